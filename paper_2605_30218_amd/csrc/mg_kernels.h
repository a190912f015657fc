// mg_kernels.h -- launch interfaces of libmg's HIP kernels (host side).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mg {

// Which rows a kernel works on.  Row i of a launch is "item" i: its activations
// live at row i of the compact buffers; `rows` (may be NULL = identity) maps it to
// the batch row whose token / position / page-table row it uses.
struct Items {
    const int32_t* rows;     // [n] batch-row index per item, or NULL
    const int32_t* n_dev;    // device count, or NULL
    int n_host;              // host count, or the cap when n_dev is used
    const int32_t* tokens;   // [batch] token per batch row
    const int32_t* positions;// [batch] position per batch row
    const int32_t* page_table; // [batch][max_pages_per_row]
    int per_item;            // 1: tokens / positions indexed by item (prefill), else by batch row
};

__device__ __forceinline__ int items_n(const Items& it) {
    if (!it.n_dev) return it.n_host;
    const int n = *it.n_dev;
    return n < 0 ? 0 : (n > it.n_host ? it.n_host : n);
}
__device__ __forceinline__ int items_row(const Items& it, int i) { return it.rows ? it.rows[i] : i; }
__device__ __forceinline__ int items_tok(const Items& it, int i) {
    return it.per_item ? it.tokens[i] : it.tokens[items_row(it, i)];
}
__device__ __forceinline__ int items_pos(const Items& it, int i) {
    return it.per_item ? it.positions[i] : it.positions[items_row(it, i)];
}

struct ModelDims {
    int L, d, Hq, Hkv, hd, F, V;
    int page_size, max_pages_per_row, n_pages;
    float eps;
};

// ---------------------------------------------------------------- canonical GEMV
enum { EPI_BF16 = 0, EPI_RESID = 1, EPI_F32 = 2, EPI_SWIGLU = 3 };
// EPI_SWIGLU: W[0] = gate rows, W[1] = up rows (Nseg[0] = Nseg[1] = N); half of a block's
// waves take gate rows, the other half the up rows of the same outputs, and the block writes
// Y[r][j] = bf16(silu(bf16(gate)) * bf16(up)) with the verifier's EXP and IEEE division
// (bf16 [n][N])
struct GemvArgs {
    const uint16_t* X;         // [n][K] bf16 (compact rows)
    int K;
    const uint16_t* W[3];      // up to three weight matrices, concatenated along the output
    const uint16_t* bias[3];   // per segment, or NULL
    int Nseg[3];               // features per segment (0 = unused)
    int N;                     // total features
    void* Y;                   // EPI_BF16: bf16 [n][N]; EPI_F32: fp32 [n][N]; EPI_RESID: bf16 residual [n][N] (in/out)
    int n_host, cap;           // rows
    const int32_t* n_dev;
    int n_cu;                  // compute units of the device (chooses the features per wave)
};
// two kernels with bit-identical results: fma on the vector ALUs, and the same fma steps on
// the matrix cores (v_mfma_f32_16x16x1_4b_f32); launch_canon_gemv picks one by row count
hipError_t launch_canon_gemv(const GemvArgs& a, int epi, hipStream_t s);
hipError_t launch_canon_gemv_valu(const GemvArgs& a, int epi, hipStream_t s);
hipError_t launch_canon_gemv_mfma(const GemvArgs& a, int epi, hipStream_t s);
// the kernel launch_canon_gemv takes for a row count (host count, or the cap of a device count)
bool canon_gemv_on_mfma(int rows, bool device_count);
// the matrix-core kernel's launch for a row count, n_fg feature groups (16 features, or 8
// gate/up pairs) and K: rows per tile (16, or 32 with 4-row quads past 16), 4-row quads, waves
// per block (8, or 16 with the stage parity on the waves), ring depth, groups past K
struct MfmaLaunch {
    int tile_rows, quads, waves, depth;
    bool ragged;
};
MfmaLaunch choose_mfma_launch(int rows, int n_fg, int K, int n_cu);

// ---------------------------------------------------------------- fast MFMA GEMM
enum { FEPI_BF16 = 0, FEPI_PART = 1, FEPI_F32 = 2, FEPI_SWIGLU = 3, FEPI_TOP2 = 4 };
// FEPI_TOP2 (unsplit): no output tile; each block writes, per row, the top-2 state of its
// features (struct Top2, 16 bytes) to part[row * gridDim.x + block] (M x fast_gemm_blocks(...)
// states), for launch_top1_rows to merge into the row's top-1 index
// FEPI_SWIGLU (unsplit, direct-to-LDS path only): W[0] = gate rows, W[1] = up rows, N =
// outputs; half of a block's waves take gate tiles, the other half the up tiles of the same
// outputs, and Y[r][j] = bf16(silu(bf16(gate)) * bf16(up)) (bf16 [M][N], the fast path's exp)
struct FastGemmArgs {
    const uint16_t* X;         // [M][K] bf16
    int M, K;
    const uint16_t* W[3];
    const uint16_t* bias[3];   // FEPI_BF16 only
    int Nseg[3];
    int N;
    void* Y;                   // FEPI_BF16: bf16 [M][N]; FEPI_F32: fp32 [M][N]
    float* part;               // FEPI_PART: fp32 partial tiles [S][M][N]
    int S;                     // split-K factor (1 unless FEPI_PART)
    int n_cu;                  // compute units of the device (chooses the waves per block)
};
hipError_t launch_fast_gemm(const FastGemmArgs& a, int epi, hipStream_t s);
hipError_t launch_sum_partials(const float* part, int S, int64_t n, float* out, hipStream_t s);
// blocks of an unsplit fast GEMM launch of M rows over N features (the FEPI_TOP2 states per row)
int fast_gemm_blocks(int M, int N, int K, int n_cu);
// top1[r] = the lowest index of the largest non-NaN value of row r, merged from the nblk
// top-2 states per row a FEPI_TOP2 launch wrote (0 when the row has no number), r < M
hipError_t launch_top1_rows(int M, const void* states, int nblk, int32_t* top1, hipStream_t s);
int fast_gemm_splits(int M, int N, int K, int n_cu);
// the split count and the waves per block a launch of M rows uses
void fast_gemm_config(int M, int N, int K, int n_cu, int* S, int* waves);
// whether M rows of a K-long projection take the direct-to-LDS operand path
bool fast_gemm_lds_path(int M, int K);

// fast-path consumers of split partial tiles
// x[r] = bf16(x[r] + bf16(sum_s part[s][r])) (skipped when part == NULL; with embed != NULL,
// x[r] = embed[token of r] instead), then h[r] = bf16((x * rms^-1) * gamma)
hipError_t launch_resid_norm(int B, const float* part, int S, const uint16_t* embed, const int32_t* tokens, int d,
                             const uint16_t* gamma, float eps, uint16_t* x, uint16_t* h, hipStream_t s);
// act[r] = bf16(silu(bf16(sum gate partials)) * bf16(sum up partials)); part rows [gate F | up F]
hipError_t launch_swiglu_part(int B, const float* part, int S, int F, uint16_t* act, hipStream_t s);
// ---------------------------------------------------------------- small kernels
hipError_t launch_embed(const Items& it, const uint16_t* embed, int d, uint16_t* x, hipStream_t s);
hipError_t launch_rmsnorm(const uint16_t* x, const uint16_t* gamma, int n_host, const int32_t* n_dev, int cap, int d,
                          float eps, uint16_t* y, hipStream_t s);
// RoPE of q and k for each item, q' -> qrot; K', V -> destination:
//  kv_col != NULL: the verifier's own column [item][layer][K|V][Hkv][hd] (layer `layer`)
//  kv_col == NULL: the paged cache at the item's position (fast path / prefill)
hipError_t launch_rope_kv(const Items& it, const ModelDims& m, int layer, const uint16_t* qkv, const float* rope_cs,
                          uint16_t* qrot, uint16_t* kv_pool, uint16_t* kv_col, hipStream_t s);
// ---------------------------------------------------------------- attention
struct AttnArgs {
    Items it;
    ModelDims m;
    int layer;
    const uint16_t* qrot;      // [n][Hq*hd]
    const uint16_t* kv_pool;
    const uint16_t* own_col;   // verifier scratch columns [n][L][2][Hkv][hd], or NULL (read the cache)
    // qkv != NULL (with own_col): the kernel rotates the queries and the own K column itself
    // from the QKV output [n][Hq*hd + 2*Hkv*hd] with the cos/sin table cs, and writes the own
    // column (K', V) to own_col; qrot is then unused
    const uint16_t* qkv;
    const float* cs;
    float* part;               // [n][Hq][max_chunks][hd + 2]
    int chunk;                 // positions per chunk (canonical: 256)
    int max_chunks;
    uint16_t* out;             // [n][Hq*hd]
    // item table (or NULL): per item, its position then the page of every page slot of its row
    // clamped to the position's page, [n][1 + max_pages_per_row]; written once per forward by
    // launch_item_table, so a block finds its position and pages in one memory round trip
    const int32_t* itab;
    int n_cu;                  // compute units of the device (chooses the block size)
};
hipError_t launch_attention(const AttnArgs& a, int canon, hipStream_t s);  // canonical (canon = 1) only
hipError_t launch_item_table(const Items& it, const ModelDims& m, int32_t* itab, hipStream_t s);

// fast path: QKV split sum + bias + RoPE + tentative K/V append + attention, one block
// per (row, KV head); rows 0..B-1 of the step batch
struct FastAttnArgs {
    int B;
    const float* part;          // QKV split partials [S][B][Nq + 2 Nk]
    int S;
    const uint16_t *bq, *bk, *bv;  // biases or NULL
    const int32_t* positions;   // [B]
    const int32_t* page_table;  // [B][max_pages_per_row]
    ModelDims m;
    int layer;
    const float* cs;            // RoPE table [max_pos][hd] (cos, sin interleaved)
    uint16_t* kv_pool;
    uint16_t* out;              // [B][Hq * hd] bf16
    uint16_t* own_out;          // NULL: append K'/V at p to the cache; else [B][L][2][Hkv][hd] (the cache is not written)
    int nsplit;                 // position splits per (row, KV head): 1 = one block merges everything
    int split_pages;            // pages per split (split k covers pages [k, k+1) * split_pages of a row)
    float* split_part;          // nsplit > 1: partials [B][Hq][nsplit][hd + 2] (m, l, O), merged by a second launch
};
hipError_t launch_fast_attention(const FastAttnArgs& a, hipStream_t s);
// position splits of the fast attention for `rows` rows: 1 when the (row, KV head) blocks
// fill the device; else enough (row, KV head, split) blocks to fill it (at least 16 pages of
// capacity per split) and no split longer than 64 pages of capacity, so that rows of ragged
// lengths give blocks of bounded work
// (row, KV head) units: `n_kv_heads` is the KV-head count times the head groups
int fast_attn_splits(int rows, int n_kv_heads, int max_pages_per_row, int n_cu, int cap);
// blocks per (row, KV head, split): query-head groups of at most 4 (more than 4 heads per
// block do not fit two blocks per CU in registers)
int fast_attn_head_groups(int n_q_heads, int n_kv_heads);

// ---------------------------------------------------------------- gate / repair / misc
// top-1 / top-2 of B <= 256 logit rows in two launches (vocabulary slices, then a
// per-row merge and the ordered compaction); part_ws holds TOP2_WS_BYTES
constexpr size_t TOP2_WS_BYTES = 256 * 128 * 16;
// bytes of part_ws a launch of B rows over V logits uses (at most 2048 slice states of 16 bytes)
size_t top2_ws_bytes(int B, int V);
hipError_t launch_top2(int B, int V, const float* logits, const uint8_t* prot, float tau, int32_t* top1,
                       float* margin, uint8_t* gate, int32_t* gated_rows, int32_t* n_gated, int32_t* n_gated_host,
                       void* part_ws, const int32_t* n_dev, hipStream_t s);
// compact copies of the listed rows' token, position and page-table row
hipError_t launch_gather_rows(int n, const int32_t* rows, const int32_t* tokens, const int32_t* positions,
                              const int32_t* page_table, int maxp, int32_t* out_tok, int32_t* out_pos, int32_t* out_pt,
                              hipStream_t s);
hipError_t launch_repair(int n_host, const int32_t* n_dev, int cap, const int32_t* rows, const int32_t* positions,
                         const int32_t* page_table, const int32_t* top1, const int32_t* v_tok,
                         const uint16_t* v_kvcol, const ModelDims& m, uint16_t* kv_pool, int32_t* emitted,
                         int32_t* n_repaired, int action, hipStream_t s);
hipError_t launch_advance(int B, const int32_t* emitted, int32_t* tokens, int32_t* positions, hipStream_t s);

// element-wise numerics probes used by the tests
hipError_t launch_copy16(int64_t n16, const void* src, void* dst, hipStream_t s);
// streaming read of n16 16-byte words; sink receives read_stream_blocks() words
int read_stream_blocks();
hipError_t launch_read_stream(int64_t n16, const void* src, uint32_t* sink, hipStream_t s);
hipError_t launch_probe_bf16(int64_t n, const float* in, uint16_t* out, hipStream_t s);
hipError_t launch_probe_exp(int64_t n, const float* in, float* out, hipStream_t s);
hipError_t launch_probe_divsqrt(int64_t n, const float* a, const float* b, float* q, float* r, hipStream_t s);
hipError_t launch_probe_mfma_fma(int n_inst, const float* a, const float* b, const float* c, float* d, hipStream_t s);
hipError_t launch_probe_mfma4_fma(int n_inst, const float* a, const float* b, const float* c, float* d, hipStream_t s);

}  // namespace mg
