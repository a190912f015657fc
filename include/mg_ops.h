/*
 * mg_ops.h -- op-level entry points of libmg.so, exported so the test-suite can
 * check single kernels against the CPU oracle.  Not part of the decode step.
 * Same conventions as mg.h: [device] pointers owned by the caller, work enqueued
 * on `stream` (hipStream_t as void*), host-checked arguments return an error and
 * enqueue nothing.
 */
#ifndef MG_OPS_H
#define MG_OPS_H

#include <stddef.h>
#include <stdint.h>

#include "mg.h"

#ifdef __cplusplus
extern "C" {
#endif

/* dst[0..n_bytes) = src[0..n_bytes) with a plain 16-byte-per-lane copy kernel that
 * reads and writes every byte once: the reference for scaling HBM byte counters.
 * n_bytes % 16 == 0; src and dst 16-byte aligned [device]. */
mg_status mg_op_copy(int64_t n_bytes, const void* src, void* dst, void* stream);

/* Reads src[0..n_bytes) once with a grid-stride streaming kernel (eight 16-byte loads in
 * flight per thread) and stores one xor word per block into sink (mg_op_read_stream_sink_words()
 * words): the reference for the HBM read rate of the streaming kernels.  n_bytes % 16 == 0;
 * src 16-byte aligned, sink [device]. */
int mg_op_read_stream_sink_words(void);
mg_status mg_op_read_stream(int64_t n_bytes, const void* src, uint32_t* sink, void* stream);

/* out[i] = bf16 round-to-nearest-even of in[i] (NaN -> quiet NaN), the device
 * conversion used at every bf16 rounding point.  in fp32 [n], out uint16 [n]. */
mg_status mg_op_probe_bf16(int64_t n, const float* in, uint16_t* out, void* stream);
/* out[i] = the verifier's EXP(in[i]): Cody-Waite reduction with a two-part ln 2,
 * degree-7 Taylor polynomial (Horner, fma), scaling by 2^n; +inf above n = 127,
 * +0 below n = -126. */
mg_status mg_op_probe_exp(int64_t n, const float* in, float* out, void* stream);
/* q[i] = a[i] / b[i] and r[i] = sqrt(a[i]), IEEE correctly rounded fp32. */
mg_status mg_op_probe_divsqrt(int64_t n, const float* a, const float* b, float* q, float* r, void* stream);
/* One v_mfma_f32_16x16x1_4b_f32 per instance t < n_inst (one wave each), the instruction
 * the verifier's matrix-core GEMV runs its fma chains on: a, b fp32 [n_inst][64] (the
 * lane's A and B operand), c, d fp32 [n_inst][16][64] (accumulator register r of lane l
 * in and out).  Lane l = 16 k + i supplies row i of block k's A and column i of block
 * k's B; register r of lane l holds block r / 4, row 4 (l / 16) + r % 4, column l % 16.
 * The test compares d with fmaf of the matching operands. */
mg_status mg_op_probe_mfma_fma(int n_inst, const float* a, const float* b, const float* c, float* d, void* stream);
/* One v_mfma_f32_4x4x1_16b_f32 per instance t < n_inst (one wave each), the instruction the
 * matrix-core GEMV runs the fma chains of rows past the first 16-row tile on: a, b fp32
 * [n_inst][64] (the lane's A and B operand), c, d fp32 [n_inst][4][64] (accumulator register
 * r of lane l in and out).  Lane l = 4 k + i supplies row i of block k's A and column i of
 * block k's B; register r of lane l holds block l / 4, row r, column l % 4.  The test
 * compares d with fmaf of the matching operands. */
mg_status mg_op_probe_mfma4_fma(int n_inst, const float* a, const float* b, const float* c, float* d, void* stream);

/* Y[r][j] = sum_k X[r][k] * W[j][k] in fp32 (no bias, no rounding to bf16), for
 * r < n <= 256, N % 16 == 0, K % 8 == 0.  canon = 1: the verifier's canonical
 * GEMV (CDOT order, bit-reproducible) with the kernel the verifier would pick for n
 * rows; canon = 2 / 3: the same GEMV forced onto its vector-fma kernel / its
 * matrix-core kernel (the two give identical bits; tests compare both with the
 * oracle at every shape); canon = 0: the fast path's MFMA GEMM with its split-K
 * choice for this shape, which needs a workspace of
 * mg_op_linear_workspace_bytes(n, N, K) bytes (ignored when canon != 0).
 * bias must be NULL.  X bf16 [n][K], W bf16 [N][K], Y fp32 [n][N]. */
size_t mg_op_linear_workspace_bytes(int n, int N, int K);
mg_status mg_op_linear(int canon, int n, int N, int K, const uint16_t* X, const uint16_t* W, const uint16_t* bias,
                       float* Y, void* workspace, size_t workspace_bytes, void* stream);
/* The launch the fast path's MFMA GEMM makes for n rows of an N x K projection on a
 * device of n_cu compute units: *S = split-K factor, *waves = waves per block (4 or
 * 8).  Host logic only (no device call); the same limits on n, N and K as above,
 * n_cu > 0, else MG_ERR_ARG. */
mg_status mg_op_fast_gemm_config(int n, int N, int K, int n_cu, int* S, int* waves);
/* The launch the verifier's canonical GEMV makes for n host-counted rows of an N x K
 * projection (swiglu != 0: the gate/up pair of N features each, served as 8-pair groups)
 * on a device of n_cu compute units: *kernel = 2 for the vector-fma kernel (the other
 * outputs 0) or 3 for the matrix-core kernel with *tile_rows rows per block tile (16, or 32
 * as one 16-row tile plus *quads 4-row quads), *waves per feature group (8, or 16 with the
 * stage parity on the waves) and a ring *depth stages deep.  The choice never changes the
 * result bits (Sec. 3.2's verifier contract: the row result is independent of n).  Host
 * logic only (no device call); 0 < n <= 256, N > 0, K > 0, K % 8 == 0, n_cu > 0 and
 * non-NULL outputs, else MG_ERR_ARG. */
mg_status mg_op_canon_gemv_config(int n, int N, int K, int swiglu, int n_cu, int* kernel, int* tile_rows, int* quads,
                                  int* waves, int* depth);

/* y[r] = RMSNorm(x[r]) * gamma with the canonical sum of squares (one wave per
 * row, CDOT order), r < n; d % 8 == 0.  bf16 in, bf16 out. */
mg_status mg_op_rmsnorm(int n, int d, const uint16_t* x, const uint16_t* gamma, float eps, uint16_t* y, void* stream);

/* mg_decode_step (the BF16 fast path of Sec. 3.1, with its tentative K/V append of
 * Sec. 3.2) with the same launches, plus a device copy of the residual stream at every
 * layer boundary: x_taps[0] = the rows' embeddings entering layer 0, x_taps[l + 1] = the
 * output of layer l, each [B][d_model] bf16 (x_taps holds (n_layers + 1) * B * d_model
 * values [device]).  For state-forced per-layer checks of the fast path; the logits and
 * cache writes are those of mg_decode_step.  Errors as mg_decode_step, plus a NULL x_taps. */
mg_status mg_op_decode_step_taps(mg_ctx* ctx, int B, const int32_t* tokens, const int32_t* positions,
                                 const int32_t* page_table, float* logits, uint16_t* x_taps, void* stream);

#ifdef __cplusplus
}
#endif
#endif
