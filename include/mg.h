/*
 * mg.h -- C ABI of libmg.so, the MI355X (gfx950) hot path of MarginGate
 * (arXiv 2605.30218): one synchronous decode step of a batch of requests, the
 * top-1/top-2 margin gate, the deterministic verifier on the gated rows, and the
 * single-column K/V repair.
 *
 * Conventions for every call below
 *  - Pointers marked [device] are HIP device pointers owned by the caller; the
 *    library never frees them and keeps none of them beyond the call, except the
 *    weights, KV pool and workspace handed to mg_create, which must outlive the
 *    context.  Pointers marked [host] are read during the call only.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).  Every
 *    call only enqueues work on that stream and returns; results are ready when
 *    the stream is synchronised.  Kernel faults surface at that synchronisation.
 *  - Arguments the host can check (null pointers, sizes, batch above max_batch)
 *    return an error status and enqueue nothing.  Device-resident values (token
 *    ids, positions, page ids, row lists) are trusted: out-of-range values are
 *    the caller's error and are NOT checked on the device.
 *  - No call allocates device memory after mg_create.  One host thread at a time
 *    may use a given context; calls that overlap on different streams race on
 *    the context's workspace.
 *
 * Data layout
 *  - bf16 values are raw uint16 bit patterns.  Linear weights use the [out][in]
 *    row-major layout.  Logits are fp32.
 *  - Weight pointer table (mg_weight_count() entries, [device] bf16):
 *      [0] embed [V][d]
 *      layer l at 1 + 12*l: +0 attn_norm[d] +1 wq[Hq*hd][d] +2 wk[Hkv*hd][d]
 *        +3 wv[Hkv*hd][d] +4 bq[Hq*hd] +5 bk[Hkv*hd] +6 bv[Hkv*hd] (NULL when
 *        qkv_bias == 0) +7 wo[d][Hq*hd] +8 ffn_norm[d] +9 w_gate[F][d]
 *        +10 w_up[F][d] +11 w_down[d][F]
 *      [1 + 12*L] final_norm[d]   [2 + 12*L] lm_head[V][d]
 *  - KV pool: [layer][page][K|V][Hkv][page_size][hd] bf16.  K is stored after
 *    RoPE.  One head's page is page_size*hd contiguous values.
 *  - Page table: [B][max_pages_per_row] int32; position p of row b lives in page
 *    page_table[b*max_pages_per_row + p/page_size], slot p % page_size.  The
 *    caller allocates pages on the host; the page holding a row's current
 *    position must be mapped before the step.
 *  - A verifier K/V column of one row: [layer][K|V][Hkv][hd] bf16
 *    (mg_kv_col_elems() values).
 */
#ifndef MG_H
#define MG_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MG_OK = 0,
    MG_ERR_ARG = -1,       /* null pointer or value out of range */
    MG_ERR_SHAPE = -2,     /* model shape the kernels do not support */
    MG_ERR_WORKSPACE = -3, /* workspace or KV pool smaller than required */
    MG_ERR_HIP = -4,       /* a HIP runtime call failed */
    MG_ERR_STATE = -5      /* call not valid in the context's current state */
} mg_status;

typedef struct {
    int32_t n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ffn, vocab;
    int32_t qkv_bias;          /* 1: q/k/v projections carry a bias */
    float rope_theta, rms_eps;
    int32_t page_size;         /* must be 16 */
    int32_t max_batch;         /* rows per step, 1..256 */
    int32_t max_pages_per_row; /* page-table row stride; max position = this * page_size - 1 */
    int32_t n_pages;           /* pages in the KV pool */
    int32_t max_prefill;       /* items per mg_prefill call (0 = 1024) */
} mg_model_cfg;

typedef struct mg_ctx mg_ctx;

/* Entries of the weight pointer table: 3 + 12 * n_layers. */
int mg_weight_count(const mg_model_cfg* cfg);
/* Bytes of the KV pool the shape needs: n_layers*n_pages*2*Hkv*page_size*hd*2. */
size_t mg_kv_pool_bytes(const mg_model_cfg* cfg);
/* bf16 values of one row's K/V column: n_layers*2*Hkv*hd. */
size_t mg_kv_col_elems(const mg_model_cfg* cfg);
/* Bytes of device workspace mg_create needs (0 if the shape is unsupported). */
size_t mg_workspace_bytes(const mg_model_cfg* cfg);
const char* mg_status_string(int status);

/* Create a context.  Checks the shape (d_model, d_ffn, Hq*hd multiples of 64;
 * head_dim 64 or 128; Hq % Hkv == 0; page_size 16), copies the RoPE table into
 * the workspace and zeroes the workspace's counters (synchronous).  weights
 * [host array of device pointers], kv_pool and workspace [device]. */
mg_status mg_create(const mg_model_cfg* cfg, const void* const* weights, void* kv_pool, size_t kv_pool_bytes,
                    void* workspace, size_t workspace_bytes, mg_ctx** out);
mg_status mg_destroy(mg_ctx* ctx);

/* (1) The BF16 fast path: the ordinary batched decoder forward whose logits the
 * gate inspects (paper Sec. 3.1, margin trigger), which also writes the current
 * token's K/V column into the cache as a tentative entry (Sec. 3.2).  For each row b < B: consumes tokens[b] at position
 * positions[b], writes that position's K (after RoPE) and V into the paged
 * cache in every layer, attends over positions 0..positions[b], and writes
 * fp32 logits[b][V].  Its reduction plan depends on B (it may differ in the last
 * bits between batch sizes; that is the effect the method guards against).
 * tokens, positions [device int32, B]; page_table [device int32,
 * B*max_pages_per_row]; logits [device fp32, B*V]. */
mg_status mg_decode_step(mg_ctx* ctx, int B, const int32_t* tokens, const int32_t* positions,
                         const int32_t* page_table, float* logits, void* stream);

/* (2) The margin gate (Sec. 3.1): per row, top1[b] = argmax (lowest index on
 * ties), margin[b] = l_(1) - l_(2) where l_(2) is the second largest value of
 * the row (0 when the maximum is duplicated; NaN when the row holds a NaN),
 * gate[b] = protected[b] && !(margin[b] >= tau), i.e. the strict trigger
 * g < tau with NaN firing.  gated_rows receives the gated row indices in
 * increasing order and *n_gated their count (device scalar), so the verifier can
 * be launched on exactly those rows (the repair request of Sec. 3.2).
 * logits [device fp32 B*V]; protected_mask [device uint8 B] or NULL (= all rows
 * protected, Sec. 3.3's per-request policy); top1, gated_rows [device int32 B];
 * margin [device fp32 B]; gate [device uint8 B]; n_gated [device int32 1].
 * n_gated_host: NULL, or one int32 of pinned host memory (allocated with
 * hipHostMalloc) that also receives the count, stored with system scope after
 * gated_rows and *n_gated are written, so a host can poll it instead of
 * synchronising the stream (the caller sets it to a negative value first).
 * Bit-exact: comparisons only, no rounding. */
mg_status mg_margin_gate(mg_ctx* ctx, int B, const float* logits, const uint8_t* protected_mask, float tau,
                         int32_t* top1, float* margin, uint8_t* gate, int32_t* gated_rows, int32_t* n_gated,
                         int32_t* n_gated_host, void* stream);

/* The margin gate of mg_margin_gate for callers that cannot allocate device memory or hold
 * a context: code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Same outputs and the same bits as mg_margin_gate over B rows of V logits
 * (B <= 256, V >= 2, else MG_ERR_ARG), without the host-mirror count.  Its partial states
 * live in a static device array of 32 KiB per GPU, held until the process ends; the first
 * call on a device looks up that array's address (no allocation, no context).  Every call
 * on one GPU shares that array: calls that overlap on one GPU (different streams, or
 * different host threads) race and must be serialised by the caller.  All pointers
 * [device], as in mg_margin_gate; stream as everywhere. */
mg_status mg_margin_gate_noalloc(int B, int V, const float* logits, const uint8_t* protected_mask, float tau,
                                 int32_t* top1, float* margin, uint8_t* gate, int32_t* gated_rows, int32_t* n_gated,
                                 void* stream);

/* (3) The deterministic verifier (Sec. 3.2, deterministic verifier contract):
 * runs the current step again for rows rows[0..n) of the step batch with
 * the canonical reduction order (fixed per-lane groups + xor butterfly for dot
 * products, chunks of 256 positions for attention, own EXP), which depends on
 * neither n, nor the row's place in the list, nor the batch.  The row attends
 * over cache positions 0..positions[r]-1 as committed plus its OWN current
 * column, never the tentative one.  Outputs for list entry i: v_logits[i][V]
 * (fp32, may be NULL), v_tok[i] = argmax (lowest index on ties), and the K/V
 * column v_kvcol[i] (bf16, mg_kv_col_elems values).  The cache is not written.
 * n >= 0: host count.  n == -1: the count is read on the device from *n_dev
 * (graph-capturable), bounded by max_batch.  rows [device int32 n]; tokens,
 * positions, page_table as in mg_decode_step. */
mg_status mg_verify_rows(mg_ctx* ctx, int n, const int32_t* rows, const int32_t* n_dev, const int32_t* tokens,
                         const int32_t* positions, const int32_t* page_table, float* v_logits, int32_t* v_tok,
                         uint16_t* v_kvcol, void* stream);

/* A matrix-core verifier for the n listed rows (host count): the BF16 forward on
 * v_mfma_f32_16x16x32_bf16 (the fast path's kernels) with every projection's split-K
 * fixed as for 32 rows, so a row's arithmetic depends on neither n nor its place in the
 * list -- deterministic and batch-invariant by fixed tiling, which is what the
 * deterministic verifier contract of Sec. 3.2 asks for.  Its order is not the canonical
 * one of mg_verify_rows: its results match the oracle within the fast path's tolerance,
 * not bit for bit.  Outputs as mg_verify_rows: v_logits [n][vocab] fp32 (may be NULL: then
 * the LM head runs with a fused top-2 epilogue that writes no logits, and v_tok is the same
 * index), v_tok[i] = argmax (lowest index on ties), v_kvcol[i] the row's K/V column [L][2][Hkv][hd]
 * bf16; the cache is read (positions < positions[rows[i]]) and not written.  Shares the
 * context's workspace with the other calls (one call at a time per context). */
mg_status mg_verify_rows_mfma(mg_ctx* ctx, int n, const int32_t* rows, const int32_t* tokens,
                              const int32_t* positions, const int32_t* page_table, float* v_logits, int32_t* v_tok,
                              uint16_t* v_kvcol, void* stream);

/* (4) Commit and single-column repair (Sec. 3.2): for list entry i with row
 * r = rows[i]: emitted[r] = v_tok[i]; if v_tok[i] != top1[r] the verifier's
 * column v_kvcol[i] overwrites the cache at position positions[r] in every
 * layer and *n_repaired is incremented (device int32, accumulates over calls).
 * When the tokens agree the tentative column stays (verified commit).  Rows not
 * listed keep emitted[r] as the caller set it (normally top1[r]); emitted may be
 * the same buffer as top1.  n / n_dev as in mg_verify_rows. */
mg_status mg_repair_kv_column(mg_ctx* ctx, int n, const int32_t* rows, const int32_t* n_dev,
                              const int32_t* positions, const int32_t* page_table, const int32_t* top1,
                              const int32_t* v_tok, const uint16_t* v_kvcol, int32_t* emitted,
                              int32_t* n_repaired, void* stream);

/* The same commit with a choice of repair action (the variants around the rule of
 * Sec. 3.2; Sec. 4, Ablations and Robustness, describes the token-only one):
 *   MG_REPAIR_ON_MISMATCH  the method: copy the verifier column when v_tok[i] != top1[r]
 *                          (mg_repair_kv_column is this action);
 *   MG_REPAIR_TOKEN_ONLY   emit the verifier token, never copy (the tentative BF16 column
 *                          stays; *n_repaired is not incremented);
 *   MG_REPAIR_COPY_ALWAYS  copy the verifier column for every listed row, agreeing rows
 *                          included (*n_repaired counts every copy).
 * Arguments, layout and errors as mg_repair_kv_column; an action outside the three
 * returns MG_ERR_ARG and enqueues nothing. */
enum { MG_REPAIR_ON_MISMATCH = 0, MG_REPAIR_TOKEN_ONLY = 1, MG_REPAIR_COPY_ALWAYS = 2 };
mg_status mg_repair_kv_column_action(mg_ctx* ctx, int n, const int32_t* rows, const int32_t* n_dev,
                                     const int32_t* positions, const int32_t* page_table, const int32_t* top1,
                                     const int32_t* v_tok, const uint16_t* v_kvcol, int32_t* emitted,
                                     int32_t* n_repaired, int action, void* stream);

/* Prompt prefill with the verifier's canonical arithmetic, so that runs at any
 * batch size start from bit-identical prompt caches.  Item i consumes
 * tokens[i] at position positions[i] of row item_rows[i] (a row of page_table)
 * and writes that position's K/V into the cache.  Attention of an item reads
 * positions 0..positions[i] of its row, so every earlier position must be in
 * this call or an earlier one.  Items per call: at most max_prefill.  The result
 * for an item is bit-identical to a verifier recomputation at that position. */
mg_status mg_prefill(mg_ctx* ctx, int n_items, const int32_t* tokens, const int32_t* positions,
                     const int32_t* item_rows, const int32_t* page_table, void* stream);

/* Step bookkeeping: tokens[b] = emitted[b]; positions[b] += 1 for b < B. */
mg_status mg_advance(mg_ctx* ctx, int B, const int32_t* emitted, int32_t* tokens, int32_t* positions,
                     void* stream);

/* ---- measurement hooks (used by the benchmark; not part of the method) ---- */

enum {
    MG_KIND_FAST_GEMM = 0,  /* weight-streaming projections of the fast path */
    MG_KIND_FAST_ATTN = 1,  /* paged decode attention of the fast path */
    MG_KIND_CANON_GEMV = 2, /* weight-streaming projections of the verifier */
    MG_KIND_CANON_ATTN = 3, /* paged decode attention of the verifier */
    MG_KIND_GATE = 4,       /* margin gate */
    MG_KIND_COUNT = 5
};

/* Start recording a HIP event pair around every launch of kernel class `kind`
 * (on the stream it is launched on), up to max_launches launches.  Creates the
 * events (not allocation-free; call outside timed loops).  The events are
 * timing-only: recording them performs no system-scope fence. */
mg_status mg_profile_begin(mg_ctx* ctx, int kind, int max_launches);
/* Stop recording, synchronise the device and report the number of
 * launches, their summed duration in milliseconds, the summed algorithmic bytes
 * (every weight, activation, K/V and output byte the launch must move once) and
 * the summed algorithmic flops (2 per multiply-add). */
mg_status mg_profile_end(mg_ctx* ctx, int kind, int* n_launches, double* total_ms, double* algo_bytes,
                         double* algo_flops);

#ifdef __cplusplus
}
#endif
#endif
