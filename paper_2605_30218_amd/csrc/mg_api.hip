// mg_api.hip -- the C ABI of libmg: context, workspace plan, and the step
// sequencer that launches the fast path, the margin gate, the verifier and the
// repair on the caller's stream.  See include/mg.h for the contract.
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <new>
#include <vector>

#include "../../include/mg.h"
#include "../../include/mg_ops.h"
#include "mg_kernels.h"

using namespace mg;

namespace {

constexpr int WPL = 12;
constexpr int CANON_CHUNK = 256;
// The matrix-core verifier splits every projection's K as a step of this many rows would,
// whatever its own row count, so a row's arithmetic never depends on the batch
constexpr int MFMA_VERIFIER_SPLIT_M = 32;
constexpr size_t ALIGN = 256;

size_t up(size_t x) { return (x + ALIGN - 1) / ALIGN * ALIGN; }

struct Plan {
    size_t rope, x, h, qkv, qrot, att, act, attn_part, itab, gemm_part, top2_ws, vlog, vrows, total;
    int rows_cap, max_pos, chunks_canon;
};

bool shape_ok(const mg_model_cfg* c) {
    if (!c) return false;
    if (c->n_layers <= 0 || c->d_model <= 0 || c->n_q_heads <= 0 || c->n_kv_heads <= 0 || c->vocab < 2) return false;
    if (c->n_q_heads % c->n_kv_heads) return false;
    if (c->n_q_heads / c->n_kv_heads > 8) return false;
    if (c->head_dim != 64 && c->head_dim != 128) return false;
    if (c->d_model % 64 || (c->n_q_heads * c->head_dim) % 64) return false;
    if (c->d_ffn % 16 || c->d_ffn <= 0 || c->vocab % 16) return false;
    if (c->page_size != 16) return false;
    if (c->max_batch < 1 || c->max_batch > 256) return false;
    if (c->max_pages_per_row <= 0 || c->n_pages <= 0) return false;
    if (c->max_prefill < 0 || c->max_prefill > 8192) return false;
    return true;
}

// Split factor chosen for each fast projection of a step with M rows.
struct ProjShape { int N, K; };
void fast_projs(const mg_model_cfg* c, ProjShape out[5]) {
    const int d = c->d_model, Nq = c->n_q_heads * c->head_dim, Nk = c->n_kv_heads * c->head_dim, F = c->d_ffn;
    out[0] = {Nq + 2 * Nk, d};
    out[1] = {d, Nq};
    out[2] = {2 * F, d};
    out[3] = {d, F};
    out[4] = {c->vocab, d};
}


Plan make_plan(const mg_model_cfg* c, int n_cu) {
    Plan p{};
    const int d = c->d_model, Hq = c->n_q_heads, hd = c->head_dim, Nq = Hq * hd, Nk = c->n_kv_heads * hd;
    const int F = c->d_ffn;
    const int pre = c->max_prefill ? c->max_prefill : 1024;
    p.rows_cap = c->max_batch > pre ? c->max_batch : pre;
    p.max_pos = c->max_pages_per_row * c->page_size;
    p.chunks_canon = (p.max_pos + CANON_CHUNK - 1) / CANON_CHUNK;
    const size_t R = p.rows_cap;
    size_t o = 0;
    p.rope = o; o += up((size_t)p.max_pos * hd * sizeof(float));
    p.x = o; o += up(R * d * 2);
    p.h = o; o += up(R * d * 2);
    p.qkv = o; o += up(R * (Nq + 2 * Nk) * 2);
    p.qrot = o; o += up(R * Nq * 2);
    p.att = o; o += up(R * Nq * 2);
    p.act = o; o += up(R * (size_t)F * 2);
    const size_t ap_canon = R * Hq * (size_t)p.chunks_canon * (hd + 2);
    p.attn_part = o; o += up(ap_canon * sizeof(float));
    p.itab = o; o += up(R * (1 + (size_t)c->max_pages_per_row) * sizeof(int32_t));
    ProjShape ps[5];
    fast_projs(c, ps);
    // split-K partial tiles of the QKV, O, gate/up and down projections: S * M * N
    // floats for every batch size the context accepts (the LM head is not split)
    size_t gp = 0;
    for (int M = 1; M <= c->max_batch; ++M)
        for (int k : {0, 1, 2, 3}) {
            // the step's own split, or the matrix-core verifier's fixed one
            const int S0 = fast_gemm_splits(M, ps[k].N, ps[k].K, n_cu);
            const int S1 = fast_gemm_splits(MFMA_VERIFIER_SPLIT_M, ps[k].N, ps[k].K, n_cu);
            const size_t need = (size_t)(S0 > S1 ? S0 : S1) * M * ps[k].N;
            if (need > gp) gp = need;
        }
    p.gemm_part = o; o += up((gp ? gp : 1) * sizeof(float));
    p.top2_ws = o; o += up(TOP2_WS_BYTES);
    p.vlog = o; o += up((size_t)c->max_batch * c->vocab * sizeof(float));
    // the matrix-core verifier's compact rows: token, position, page-table row, and the
    // top-2 pass's margin / gate / row list / count
    p.vrows = o; o += up((size_t)c->max_batch * (4 + c->max_pages_per_row) * sizeof(int32_t) + 4 * sizeof(int32_t) +
                         (size_t)c->max_batch * (sizeof(float) + 1));
    p.total = o;
    return p;
}

int device_cu_count() {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 256;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) return 256;
    return n;
}

}  // namespace

struct ProfKind {
    bool on = false;
    int max = 0;
    int used = 0;
    std::vector<hipEvent_t> ev0, ev1;
    double bytes = 0.0;
    double flops = 0.0;
};

struct mg_ctx {
    mg_model_cfg cfg;
    ModelDims m;
    std::vector<const uint16_t*> w;
    uint16_t* kv_pool;
    unsigned char* ws;
    Plan plan;
    int n_cu;
    ProfKind prof[MG_KIND_COUNT];

    const uint16_t* W(int i) const { return w[i]; }
    const uint16_t* LW(int l, int k) const { return w[1 + WPL * l + k]; }
    template <class T> T* at(size_t off) const { return reinterpret_cast<T*>(ws + off); }
};

namespace {

struct ProfScope {
    ProfKind* k;
    hipStream_t s;
    double bytes, flops;
    int idx;
    ProfScope(mg_ctx* c, int kind, hipStream_t st, double b, double f = 0.0)
        : k(&c->prof[kind]), s(st), bytes(b), flops(f), idx(-1) {
        if (k->on && k->used < k->max) {
            idx = k->used++;
            hipEventRecord(k->ev0[idx], s);
        }
    }
    ~ProfScope() {
        if (idx >= 0) {
            hipEventRecord(k->ev1[idx], s);
            k->bytes += bytes;
            k->flops += flops;
        }
    }
};

#define HIPCHK(x)                                   \
    do {                                            \
        hipError_t e_ = (x);                        \
        if (e_ != hipSuccess) return MG_ERR_HIP;    \
    } while (0)

// One fast projection.  FEPI_PART writes S split partial tiles (returned in *S_out)
// for the consuming kernel to sum; the other epilogues run unsplit.
mg_status fast_gemm(mg_ctx* c, const uint16_t* X, int M, int K, const uint16_t* const* W,
                    const uint16_t* const* bias, const int* Nseg, int nseg, void* Y, int epi, hipStream_t s,
                    int* S_out = nullptr, int split_M = 0) {
    FastGemmArgs a{};
    a.X = X;
    a.M = M;
    a.K = K;
    int N = 0;
    for (int k = 0; k < 3; ++k) {
        a.W[k] = k < nseg ? W[k] : nullptr;
        a.bias[k] = (k < nseg && bias) ? bias[k] : nullptr;
        a.Nseg[k] = k < nseg ? Nseg[k] : 0;
        N += a.Nseg[k];
    }
    // the SwiGLU epilogue writes one output per (gate, up) pair
    const int Nout = epi == FEPI_SWIGLU ? a.Nseg[0] : N;
    a.N = Nout;
    a.Y = Y;
    // the top-2 states of the fused LM-head epilogue go where the verifier's logits would
    // (M x blocks x 16 bytes, at most M x N x 4)
    a.part = epi == FEPI_TOP2 ? c->at<float>(c->plan.vlog) : c->at<float>(c->plan.gemm_part);
    a.S = epi == FEPI_PART ? fast_gemm_splits(split_M ? split_M : M, N, K, c->n_cu) : 1;
    a.n_cu = c->n_cu;
    if (S_out) *S_out = a.S;
    const double out_bytes = epi == FEPI_PART   ? 4.0 * a.S * M * N
                             : epi == FEPI_TOP2 ? 16.0 * M * fast_gemm_blocks(M, N, K, c->n_cu)
                                                : (double)M * Nout * (epi == FEPI_F32 ? 4 : 2);
    const double bytes = 2.0 * N * K + 2.0 * M * K + out_bytes;
    ProfScope ps(c, MG_KIND_FAST_GEMM, s, bytes, 2.0 * M * N * K);
    HIPCHK(launch_fast_gemm(a, epi, s));
    return MG_OK;
}

mg_status canon_gemv(mg_ctx* c, const uint16_t* X, int n, const int32_t* n_dev, int cap, int K,
                     const uint16_t* const* W, const uint16_t* const* bias, const int* Nseg, int nseg, void* Y,
                     int epi, hipStream_t s) {
    GemvArgs a{};
    a.X = X;
    a.K = K;
    int N = 0;
    for (int k = 0; k < 3; ++k) {
        a.W[k] = k < nseg ? W[k] : nullptr;
        a.bias[k] = (k < nseg && bias) ? bias[k] : nullptr;
        a.Nseg[k] = k < nseg ? Nseg[k] : 0;
        N += a.Nseg[k];
    }
    // the SwiGLU epilogue writes one output per (gate, up) pair
    const int Nout = epi == EPI_SWIGLU ? a.Nseg[0] : N;
    if (epi == EPI_SWIGLU && (nseg != 2 || a.Nseg[1] != a.Nseg[0] || bias)) return MG_ERR_ARG;
    a.N = Nout;
    a.Y = Y;
    a.n_host = n;
    a.cap = cap;
    a.n_dev = n_dev;
    a.n_cu = c->n_cu;
    const int rows = n_dev ? cap : n;
    const double bytes = 2.0 * N * K + 2.0 * rows * K + (double)rows * Nout * (epi == EPI_F32 ? 4 : 2) *
                                                        (epi == EPI_RESID ? 2 : 1);
    ProfScope ps(c, MG_KIND_CANON_GEMV, s, bytes, 2.0 * rows * N * K);
    HIPCHK(launch_canon_gemv(a, epi, s));
    return MG_OK;
}

#define MGCHK(x)                         \
    do {                                 \
        mg_status st_ = (x);             \
        if (st_ != MG_OK) return st_;    \
    } while (0)

// The verifier's canonical forward over a set of items.  own_col != NULL: the
// items' K/V columns go there and attention reads them from there (verifier);
// own_col == NULL: K/V go into the cache (prefill).  logits == NULL: no LM head.
mg_status canon_forward(mg_ctx* c, const Items& it, uint16_t* own_col, float* logits, hipStream_t s) {
    const mg_model_cfg& g = c->cfg;
    const ModelDims& m = c->m;
    const int d = g.d_model, Nq = g.n_q_heads * g.head_dim, Nk = g.n_kv_heads * g.head_dim, F = g.d_ffn;
    const int cap = it.n_host;
    const int n = it.n_host;
    const int32_t* nd = it.n_dev;
    uint16_t* x = c->at<uint16_t>(c->plan.x);
    uint16_t* h = c->at<uint16_t>(c->plan.h);
    uint16_t* qkv = c->at<uint16_t>(c->plan.qkv);
    uint16_t* qrot = c->at<uint16_t>(c->plan.qrot);
    uint16_t* att = c->at<uint16_t>(c->plan.att);
    uint16_t* act = c->at<uint16_t>(c->plan.act);
    int32_t* itab = c->at<int32_t>(c->plan.itab);
    HIPCHK(launch_item_table(it, m, itab, s));
    HIPCHK(launch_embed(it, c->W(0), d, x, s));
    for (int l = 0; l < g.n_layers; ++l) {
        HIPCHK(launch_rmsnorm(x, c->LW(l, 0), n, nd, cap, d, g.rms_eps, h, s));
        {
            const uint16_t* W[3] = {c->LW(l, 1), c->LW(l, 2), c->LW(l, 3)};
            const uint16_t* B[3] = {c->LW(l, 4), c->LW(l, 5), c->LW(l, 6)};
            const int Ns[3] = {Nq, Nk, Nk};
            MGCHK(canon_gemv(c, h, n, nd, cap, d, W, g.qkv_bias ? B : nullptr, Ns, 3, qkv, EPI_BF16, s));
        }
        // prefill: every item's K/V goes into the cache before any item attends (later
        // positions read earlier ones); the verifier's rows attend to committed columns and
        // their own, so its attention rotates the queries and the own column itself
        if (!own_col) HIPCHK(launch_rope_kv(it, m, l, qkv, c->at<float>(c->plan.rope), qrot, c->kv_pool, nullptr, s));
        {
            AttnArgs a{};
            a.it = it;
            a.m = m;
            a.layer = l;
            a.qrot = qrot;
            a.kv_pool = c->kv_pool;
            a.own_col = own_col;
            a.qkv = own_col ? qkv : nullptr;
            a.cs = c->at<float>(c->plan.rope);
            a.part = c->at<float>(c->plan.attn_part);
            a.chunk = CANON_CHUNK;
            a.max_chunks = c->plan.chunks_canon;
            a.out = att;
            a.itab = itab;
            a.n_cu = c->n_cu;
            ProfScope ps(c, MG_KIND_CANON_ATTN, s, 0.0);
            HIPCHK(launch_attention(a, 1, s));
        }
        {
            const uint16_t* W[1] = {c->LW(l, 7)};
            const int Ns[1] = {d};
            MGCHK(canon_gemv(c, att, n, nd, cap, Nq, W, nullptr, Ns, 1, x, EPI_RESID, s));
        }
        HIPCHK(launch_rmsnorm(x, c->LW(l, 8), n, nd, cap, d, g.rms_eps, h, s));
        {
            // gate/up projection with the SwiGLU in its epilogue: act = bf16(silu(bf16(gate)) * bf16(up))
            const uint16_t* W[2] = {c->LW(l, 9), c->LW(l, 10)};
            const int Ns[2] = {F, F};
            MGCHK(canon_gemv(c, h, n, nd, cap, d, W, nullptr, Ns, 2, act, EPI_SWIGLU, s));
        }
        {
            const uint16_t* W[1] = {c->LW(l, 11)};
            const int Ns[1] = {d};
            MGCHK(canon_gemv(c, act, n, nd, cap, F, W, nullptr, Ns, 1, x, EPI_RESID, s));
        }
    }
    if (logits) {
        HIPCHK(launch_rmsnorm(x, c->W(1 + WPL * g.n_layers), n, nd, cap, d, g.rms_eps, h, s));
        const uint16_t* W[1] = {c->W(2 + WPL * g.n_layers)};
        const int Ns[1] = {g.vocab};
        MGCHK(canon_gemv(c, h, n, nd, cap, d, W, nullptr, Ns, 1, logits, EPI_F32, s));
    }
    return MG_OK;
}

}  // namespace

extern "C" {

int mg_weight_count(const mg_model_cfg* cfg) { return cfg ? 3 + WPL * cfg->n_layers : 0; }

size_t mg_kv_pool_bytes(const mg_model_cfg* c) {
    if (!c) return 0;
    return (size_t)c->n_layers * c->n_pages * 2 * c->n_kv_heads * c->page_size * c->head_dim * 2;
}

size_t mg_kv_col_elems(const mg_model_cfg* c) {
    if (!c) return 0;
    return (size_t)c->n_layers * 2 * c->n_kv_heads * c->head_dim;
}

size_t mg_workspace_bytes(const mg_model_cfg* cfg) {
    if (!shape_ok(cfg)) return 0;
    return make_plan(cfg, device_cu_count()).total;
}

const char* mg_status_string(int s) {
    switch (s) {
        case MG_OK: return "ok";
        case MG_ERR_ARG: return "invalid argument";
        case MG_ERR_SHAPE: return "unsupported model shape";
        case MG_ERR_WORKSPACE: return "workspace or KV pool too small";
        case MG_ERR_HIP: return "HIP runtime error";
        case MG_ERR_STATE: return "invalid state";
        default: return "unknown status";
    }
}

mg_status mg_create(const mg_model_cfg* cfg, const void* const* weights, void* kv_pool, size_t kv_pool_bytes,
                    void* workspace, size_t workspace_bytes, mg_ctx** out) {
    if (!cfg || !weights || !kv_pool || !workspace || !out) return MG_ERR_ARG;
    if (!shape_ok(cfg)) return MG_ERR_SHAPE;
    const int nw = mg_weight_count(cfg);
    for (int i = 0; i < nw; ++i) {
        const int k = i >= 1 && i < 1 + WPL * cfg->n_layers ? (i - 1) % WPL : -1;
        const bool is_bias = k >= 4 && k <= 6;
        if (!weights[i] && !(is_bias && !cfg->qkv_bias)) return MG_ERR_ARG;
    }
    if (kv_pool_bytes < mg_kv_pool_bytes(cfg)) return MG_ERR_WORKSPACE;
    const int n_cu = device_cu_count();
    const Plan plan = make_plan(cfg, n_cu);
    if (workspace_bytes < plan.total) return MG_ERR_WORKSPACE;

    mg_ctx* c = new (std::nothrow) mg_ctx();
    if (!c) return MG_ERR_STATE;
    c->cfg = *cfg;
    if (!c->cfg.max_prefill) c->cfg.max_prefill = 1024;
    c->m = ModelDims{cfg->n_layers, cfg->d_model, cfg->n_q_heads, cfg->n_kv_heads, cfg->head_dim, cfg->d_ffn,
                     cfg->vocab, cfg->page_size, cfg->max_pages_per_row, cfg->n_pages, cfg->rms_eps};
    c->w.resize(nw);
    for (int i = 0; i < nw; ++i) c->w[i] = static_cast<const uint16_t*>(weights[i]);
    if (!cfg->qkv_bias)
        for (int l = 0; l < cfg->n_layers; ++l) c->w[1 + WPL * l + 4] = c->w[1 + WPL * l + 5] = c->w[1 + WPL * l + 6] = nullptr;
    c->kv_pool = static_cast<uint16_t*>(kv_pool);
    c->ws = static_cast<unsigned char*>(workspace);
    c->plan = plan;
    c->n_cu = n_cu;

    // RoPE table: inverse frequency and angle in float64, cos / sin rounded to fp32,
    // laid out [position][pair i][cos, sin]
    const int hd = cfg->head_dim, h2 = hd / 2;
    std::vector<float> cs((size_t)plan.max_pos * hd);
    for (int i = 0; i < h2; ++i) {
        const double inv = pow((double)cfg->rope_theta, -(2.0 * (double)i) / (double)hd);
        for (int pos = 0; pos < plan.max_pos; ++pos) {
            const double ang = (double)pos * inv;
            cs[(size_t)pos * hd + 2 * i] = (float)cos(ang);
            cs[(size_t)pos * hd + 2 * i + 1] = (float)sin(ang);
        }
    }
    if (hipMemcpy(c->at<float>(plan.rope), cs.data(), cs.size() * sizeof(float), hipMemcpyHostToDevice) != hipSuccess ||
        hipDeviceSynchronize() != hipSuccess) {
        delete c;
        return MG_ERR_HIP;
    }
    *out = c;
    return MG_OK;
}

mg_status mg_destroy(mg_ctx* c) {
    if (!c) return MG_ERR_ARG;
    for (int k = 0; k < MG_KIND_COUNT; ++k) {
        for (auto e : c->prof[k].ev0) hipEventDestroy(e);
        for (auto e : c->prof[k].ev1) hipEventDestroy(e);
    }
    delete c;
    return MG_OK;
}

// The fast forward of B rows: token / position / page-table row b at index b.  own_out
// NULL: the step -- the tentative K/V column of every row is appended to the cache.  Else
// the matrix-core verifier: the K/V columns go to own_out and the cache is only read;
// split_M fixes every projection's split-K (0: the row count's own split).  taps != NULL:
// the residual stream entering layer 0 and leaving every layer is copied to
// taps[0..L] ([L+1][B][d] bf16) as the launches run (the per-layer checks of the tests).
// top1_out != NULL (with logits NULL): the LM head runs with the fused top-2 epilogue and
// only each row's top-1 index is written (no logits).
static mg_status fast_forward(mg_ctx* c, int B, const int32_t* tokens, const int32_t* positions, const int32_t* page_table,
                       float* logits, uint16_t* own_out, int split_M, hipStream_t s, uint16_t* taps = nullptr,
                       int32_t* top1_out = nullptr) {
    const mg_model_cfg& g = c->cfg;
    const ModelDims& m = c->m;
    const int d = g.d_model, Nq = g.n_q_heads * g.head_dim, Nk = g.n_kv_heads * g.head_dim, F = g.d_ffn;
    uint16_t* x = c->at<uint16_t>(c->plan.x);
    uint16_t* h = c->at<uint16_t>(c->plan.h);
    uint16_t* att = c->at<uint16_t>(c->plan.att);
    uint16_t* act = c->at<uint16_t>(c->plan.act);
    float* part = c->at<float>(c->plan.gemm_part);
    // layer 0 input: embedding gather fused with the first RMSNorm
    HIPCHK(launch_resid_norm(B, nullptr, 0, c->W(0), tokens, d, c->LW(0, 0), g.rms_eps, x, h, s));
    const size_t tap_bytes = (size_t)B * d * sizeof(uint16_t);
    if (taps) HIPCHK(hipMemcpyAsync(taps, x, tap_bytes, hipMemcpyDeviceToDevice, s));
    for (int l = 0; l < g.n_layers; ++l) {
        int S = 1;
        {
            const uint16_t* W[3] = {c->LW(l, 1), c->LW(l, 2), c->LW(l, 3)};
            const int Ns[3] = {Nq, Nk, Nk};
            MGCHK(fast_gemm(c, h, B, d, W, nullptr, Ns, 3, nullptr, FEPI_PART, s, &S, split_M));
        }
        {
            // QKV split sum + bias + RoPE + K/V append (tentative, or own) + attention
            FastAttnArgs a{};
            a.B = B;
            a.part = part;
            a.S = S;
            if (g.qkv_bias) {
                a.bq = c->LW(l, 4);
                a.bk = c->LW(l, 5);
                a.bv = c->LW(l, 6);
            }
            a.positions = positions;
            a.page_table = page_table;
            a.m = m;
            a.layer = l;
            a.cs = c->at<float>(c->plan.rope);
            a.kv_pool = c->kv_pool;
            a.out = att;
            a.own_out = own_out;
            // split-KV when the (row, KV head) blocks cannot fill the device; the matrix-core
            // verifier fixes the split as for split_M rows, whatever its own row count
            a.nsplit = fast_attn_splits(split_M ? split_M : B, g.n_kv_heads * fast_attn_head_groups(g.n_q_heads, g.n_kv_heads),
                                        g.max_pages_per_row, c->n_cu, c->plan.chunks_canon);
            a.split_pages = (g.max_pages_per_row + a.nsplit - 1) / a.nsplit;
            a.split_part = c->at<float>(c->plan.attn_part);
            ProfScope ps(c, MG_KIND_FAST_ATTN, s, 0.0);
            HIPCHK(launch_fast_attention(a, s));
        }
        {
            const uint16_t* W[1] = {c->LW(l, 7)};
            const int Ns[1] = {d};
            MGCHK(fast_gemm(c, att, B, Nq, W, nullptr, Ns, 1, nullptr, FEPI_PART, s, &S, split_M));
        }
        HIPCHK(launch_resid_norm(B, part, S, nullptr, nullptr, d, c->LW(l, 8), g.rms_eps, x, h, s));
        {
            // gate/up: unsplit on the direct-to-LDS path, the SwiGLU runs in the GEMM's epilogue;
            // otherwise split partial tiles and a separate SwiGLU pass
            const uint16_t* W[2] = {c->LW(l, 9), c->LW(l, 10)};
            const int Ns[2] = {F, F};
            if (fast_gemm_splits(split_M ? split_M : B, 2 * F, d, c->n_cu) == 1 && fast_gemm_lds_path(B, d)) {
                MGCHK(fast_gemm(c, h, B, d, W, nullptr, Ns, 2, act, FEPI_SWIGLU, s));
            } else {
                MGCHK(fast_gemm(c, h, B, d, W, nullptr, Ns, 2, nullptr, FEPI_PART, s, &S, split_M));
                HIPCHK(launch_swiglu_part(B, part, S, F, act, s));
            }
        }
        {
            const uint16_t* W[1] = {c->LW(l, 11)};
            const int Ns[1] = {d};
            MGCHK(fast_gemm(c, act, B, F, W, nullptr, Ns, 1, nullptr, FEPI_PART, s, &S, split_M));
        }
        const uint16_t* next_gamma = l + 1 < g.n_layers ? c->LW(l + 1, 0) : c->W(1 + WPL * g.n_layers);
        HIPCHK(launch_resid_norm(B, part, S, nullptr, nullptr, d, next_gamma, g.rms_eps, x, h, s));
        if (taps)
            HIPCHK(hipMemcpyAsync(taps + (size_t)(l + 1) * B * d, x, tap_bytes, hipMemcpyDeviceToDevice, s));
    }
    const uint16_t* W[1] = {c->W(2 + WPL * g.n_layers)};
    const int Ns[1] = {g.vocab};
    if (top1_out) {
        MGCHK(fast_gemm(c, h, B, d, W, nullptr, Ns, 1, nullptr, FEPI_TOP2, s));
        HIPCHK(launch_top1_rows(B, c->at<void>(c->plan.vlog), fast_gemm_blocks(B, g.vocab, d, c->n_cu), top1_out, s));
        return MG_OK;
    }
    MGCHK(fast_gemm(c, h, B, d, W, nullptr, Ns, 1, logits, FEPI_F32, s));
    return MG_OK;
}

mg_status mg_decode_step(mg_ctx* c, int B, const int32_t* tokens, const int32_t* positions, const int32_t* page_table,
                         float* logits, void* stream) {
    if (!c || !tokens || !positions || !page_table || !logits) return MG_ERR_ARG;
    if (B < 0 || B > c->cfg.max_batch) return MG_ERR_ARG;
    if (B == 0) return MG_OK;
    return fast_forward(c, B, tokens, positions, page_table, logits, nullptr, 0, static_cast<hipStream_t>(stream));
}

mg_status mg_verify_rows_mfma(mg_ctx* c, int n, const int32_t* rows, const int32_t* tokens, const int32_t* positions,
                              const int32_t* page_table, float* v_logits, int32_t* v_tok, uint16_t* v_kvcol,
                              void* stream) {
    if (!c) return MG_ERR_ARG;
    if (n == 0) return MG_OK;
    if (n < 0 || n > c->cfg.max_batch) return MG_ERR_ARG;
    if (!rows || !tokens || !positions || !page_table || !v_tok || !v_kvcol) return MG_ERR_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int maxp = c->cfg.max_pages_per_row, B = c->cfg.max_batch;
    int32_t* vtok = c->at<int32_t>(c->plan.vrows);
    int32_t* vpos = vtok + B;
    int32_t* vrowlist = vpos + B;
    int32_t* vn = vrowlist + B;
    int32_t* vpt = vn + 4;
    float* vmargin = reinterpret_cast<float*>(vpt + (size_t)B * maxp);
    uint8_t* vgate = reinterpret_cast<uint8_t*>(vmargin + B);
    HIPCHK(launch_gather_rows(n, rows, tokens, positions, page_table, maxp, vtok, vpos, vpt, s));
    if (!v_logits) {
        // no logits wanted: the LM head's fused top-2 epilogue gives v_tok directly
        return fast_forward(c, n, vtok, vpos, vpt, nullptr, v_kvcol, MFMA_VERIFIER_SPLIT_M, s, nullptr, v_tok);
    }
    float* logits = v_logits;
    MGCHK(fast_forward(c, n, vtok, vpos, vpt, logits, v_kvcol, MFMA_VERIFIER_SPLIT_M, s));
    // v_tok = top-1 of each row (lowest index on ties); the gate outputs are scratch
    HIPCHK(launch_top2(n, c->cfg.vocab, logits, nullptr, 0.0f, v_tok, vmargin, vgate, vrowlist, vn, nullptr,
                       c->at<void>(c->plan.top2_ws), nullptr, s));
    return MG_OK;
}

mg_status mg_margin_gate(mg_ctx* c, int B, const float* logits, const uint8_t* protected_mask, float tau,
                         int32_t* top1, float* margin, uint8_t* gate, int32_t* gated_rows, int32_t* n_gated,
                         int32_t* n_gated_host, void* stream) {
    if (!c || !logits || !top1 || !margin || !gate || !gated_rows || !n_gated) return MG_ERR_ARG;
    if (B < 0 || B > c->cfg.max_batch) return MG_ERR_ARG;
    if (B == 0) return MG_OK;
    hipStream_t s = static_cast<hipStream_t>(stream);
    ProfScope ps(c, MG_KIND_GATE, s, (double)B * c->cfg.vocab * 4.0);
    HIPCHK(launch_top2(B, c->cfg.vocab, logits, protected_mask, tau, top1, margin, gate, gated_rows, n_gated,
                       n_gated_host, c->ws + c->plan.top2_ws, nullptr, s));
    return MG_OK;
}

mg_status mg_verify_rows(mg_ctx* c, int n, const int32_t* rows, const int32_t* n_dev, const int32_t* tokens,
                         const int32_t* positions, const int32_t* page_table, float* v_logits, int32_t* v_tok,
                         uint16_t* v_kvcol, void* stream) {
    if (!c) return MG_ERR_ARG;
    if (n == 0) return MG_OK;
    if (n < -1 || n > c->cfg.max_batch || (n == -1 && !n_dev)) return MG_ERR_ARG;
    if (!rows || !tokens || !positions || !page_table || !v_tok || !v_kvcol) return MG_ERR_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int cap = n == -1 ? c->cfg.max_batch : n;
    Items it{rows, n == -1 ? n_dev : nullptr, cap, tokens, positions, page_table, 0};
    float* lg = v_logits ? v_logits : c->at<float>(c->plan.vlog);
    MGCHK(canon_forward(c, it, v_kvcol, lg, s));
    HIPCHK(launch_top2(cap, c->cfg.vocab, lg, nullptr, 0.0f, v_tok, nullptr, nullptr, nullptr, nullptr, nullptr,
                       c->ws + c->plan.top2_ws, it.n_dev, s));
    return MG_OK;
}

mg_status mg_repair_kv_column(mg_ctx* c, int n, const int32_t* rows, const int32_t* n_dev, const int32_t* positions,
                              const int32_t* page_table, const int32_t* top1, const int32_t* v_tok,
                              const uint16_t* v_kvcol, int32_t* emitted, int32_t* n_repaired, void* stream) {
    return mg_repair_kv_column_action(c, n, rows, n_dev, positions, page_table, top1, v_tok, v_kvcol, emitted,
                                      n_repaired, MG_REPAIR_ON_MISMATCH, stream);
}

mg_status mg_repair_kv_column_action(mg_ctx* c, int n, const int32_t* rows, const int32_t* n_dev,
                                     const int32_t* positions, const int32_t* page_table, const int32_t* top1,
                                     const int32_t* v_tok, const uint16_t* v_kvcol, int32_t* emitted,
                                     int32_t* n_repaired, int action, void* stream) {
    if (!c) return MG_ERR_ARG;
    if (action != MG_REPAIR_ON_MISMATCH && action != MG_REPAIR_TOKEN_ONLY && action != MG_REPAIR_COPY_ALWAYS)
        return MG_ERR_ARG;
    if (n == 0) return MG_OK;
    if (n < -1 || n > c->cfg.max_batch || (n == -1 && !n_dev)) return MG_ERR_ARG;
    if (!rows || !positions || !page_table || !top1 || !v_tok || !v_kvcol || !emitted || !n_repaired)
        return MG_ERR_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    HIPCHK(launch_repair(n == -1 ? 0 : n, n == -1 ? n_dev : nullptr, c->cfg.max_batch, rows, positions, page_table,
                         top1, v_tok, v_kvcol, c->m, c->kv_pool, emitted, n_repaired, action, s));
    return MG_OK;
}

mg_status mg_prefill(mg_ctx* c, int n_items, const int32_t* tokens, const int32_t* positions, const int32_t* item_rows,
                     const int32_t* page_table, void* stream) {
    if (!c) return MG_ERR_ARG;
    if (n_items == 0) return MG_OK;
    if (n_items < 0 || n_items > c->cfg.max_prefill) return MG_ERR_ARG;
    if (!tokens || !positions || !item_rows || !page_table) return MG_ERR_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    Items it{item_rows, nullptr, n_items, tokens, positions, page_table, 1};
    return canon_forward(c, it, nullptr, nullptr, s);
}

mg_status mg_advance(mg_ctx* c, int B, const int32_t* emitted, int32_t* tokens, int32_t* positions, void* stream) {
    if (!c || !emitted || !tokens || !positions) return MG_ERR_ARG;
    if (B < 0 || B > c->cfg.max_batch) return MG_ERR_ARG;
    HIPCHK(launch_advance(B, emitted, tokens, positions, static_cast<hipStream_t>(stream)));
    return MG_OK;
}

mg_status mg_profile_begin(mg_ctx* c, int kind, int max_launches) {
    if (!c || kind < 0 || kind >= MG_KIND_COUNT || max_launches <= 0) return MG_ERR_ARG;
    ProfKind& k = c->prof[kind];
    while ((int)k.ev0.size() < max_launches) {
        hipEvent_t a, b;
        // timing-only events: no system-scope fence (cache writeback and invalidate) per record
        if (hipEventCreateWithFlags(&a, hipEventDisableSystemFence) != hipSuccess ||
            hipEventCreateWithFlags(&b, hipEventDisableSystemFence) != hipSuccess)
            return MG_ERR_HIP;
        k.ev0.push_back(a);
        k.ev1.push_back(b);
    }
    k.on = true;
    k.max = max_launches;
    k.used = 0;
    k.bytes = 0.0;
    k.flops = 0.0;
    return MG_OK;
}

mg_status mg_profile_end(mg_ctx* c, int kind, int* n_launches, double* total_ms, double* algo_bytes,
                         double* algo_flops) {
    if (!c || kind < 0 || kind >= MG_KIND_COUNT || !n_launches || !total_ms || !algo_bytes || !algo_flops)
        return MG_ERR_ARG;
    ProfKind& k = c->prof[kind];
    k.on = false;
    if (hipDeviceSynchronize() != hipSuccess) return MG_ERR_HIP;
    double tot = 0.0;
    for (int i = 0; i < k.used; ++i) {
        if (hipEventSynchronize(k.ev1[i]) != hipSuccess) return MG_ERR_HIP;
        float ms = 0.f;
        if (hipEventElapsedTime(&ms, k.ev0[i], k.ev1[i]) != hipSuccess) return MG_ERR_HIP;
        tot += ms;
    }
    *n_launches = k.used;
    *total_ms = tot;
    *algo_bytes = k.bytes;
    *algo_flops = k.flops;
    return MG_OK;
}

// ---------------------------------------------------------------- op-level entry points (tests)

mg_status mg_op_copy(int64_t n_bytes, const void* src, void* dst, void* stream) {
    if (n_bytes < 0 || n_bytes % 16 || (n_bytes && (!src || !dst))) return MG_ERR_ARG;
    return launch_copy16(n_bytes / 16, src, dst, static_cast<hipStream_t>(stream)) == hipSuccess ? MG_OK : MG_ERR_HIP;
}

int mg_op_read_stream_sink_words(void) { return read_stream_blocks(); }

mg_status mg_op_read_stream(int64_t n_bytes, const void* src, uint32_t* sink, void* stream) {
    if (n_bytes < 0 || n_bytes % 16 || (n_bytes && (!src || !sink))) return MG_ERR_ARG;
    return launch_read_stream(n_bytes / 16, src, sink, static_cast<hipStream_t>(stream)) == hipSuccess ? MG_OK
                                                                                                        : MG_ERR_HIP;
}

mg_status mg_op_probe_bf16(int64_t n, const float* in, uint16_t* out, void* stream) {
    if (n < 0 || (n && (!in || !out))) return MG_ERR_ARG;
    return launch_probe_bf16(n, in, out, static_cast<hipStream_t>(stream)) == hipSuccess ? MG_OK : MG_ERR_HIP;
}

mg_status mg_op_probe_exp(int64_t n, const float* in, float* out, void* stream) {
    if (n < 0 || (n && (!in || !out))) return MG_ERR_ARG;
    return launch_probe_exp(n, in, out, static_cast<hipStream_t>(stream)) == hipSuccess ? MG_OK : MG_ERR_HIP;
}

mg_status mg_op_probe_divsqrt(int64_t n, const float* a, const float* b, float* q, float* r, void* stream) {
    if (n < 0 || (n && (!a || !b || !q || !r))) return MG_ERR_ARG;
    return launch_probe_divsqrt(n, a, b, q, r, static_cast<hipStream_t>(stream)) == hipSuccess ? MG_OK : MG_ERR_HIP;
}

mg_status mg_op_probe_mfma_fma(int n_inst, const float* a, const float* b, const float* c, float* d, void* stream) {
    if (n_inst < 0 || (n_inst && (!a || !b || !c || !d))) return MG_ERR_ARG;
    return launch_probe_mfma_fma(n_inst, a, b, c, d, static_cast<hipStream_t>(stream)) == hipSuccess ? MG_OK
                                                                                                     : MG_ERR_HIP;
}

mg_status mg_op_probe_mfma4_fma(int n_inst, const float* a, const float* b, const float* c, float* d, void* stream) {
    if (n_inst < 0 || (n_inst && (!a || !b || !c || !d))) return MG_ERR_ARG;
    return launch_probe_mfma4_fma(n_inst, a, b, c, d, static_cast<hipStream_t>(stream)) == hipSuccess ? MG_OK
                                                                                                      : MG_ERR_HIP;
}

size_t mg_op_linear_workspace_bytes(int n, int N, int K) {
    if (n <= 0 || N <= 0 || K <= 0) return 0;
    const int S = fast_gemm_splits(n, N, K, device_cu_count());
    return up((size_t)S * n * N * sizeof(float));
}

mg_status mg_op_linear(int canon, int n, int N, int K, const uint16_t* X, const uint16_t* W, const uint16_t* bias,
                       float* Y, void* workspace, size_t workspace_bytes, void* stream) {
    if (n <= 0 || n > 256 || N <= 0 || K <= 0 || K % 8 || N % 16 || !X || !W || !Y || canon < 0 || canon > 3) return MG_ERR_ARG;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (canon) {
        GemvArgs a{};
        a.X = X;
        a.K = K;
        a.W[0] = W;
        a.Nseg[0] = N;
        a.N = N;
        a.Y = Y;
        a.n_host = n;
        a.cap = n;
        a.n_cu = device_cu_count();
        if (bias) return MG_ERR_ARG;  // fp32 output carries no bias; the model path tests the bias
        const hipError_t e = canon == 2   ? launch_canon_gemv_valu(a, EPI_F32, s)
                             : canon == 3 ? launch_canon_gemv_mfma(a, EPI_F32, s)
                                          : launch_canon_gemv(a, EPI_F32, s);
        return e == hipSuccess ? MG_OK : MG_ERR_HIP;
    }
    const size_t need = mg_op_linear_workspace_bytes(n, N, K);
    if (!workspace || workspace_bytes < need) return MG_ERR_WORKSPACE;
    if (bias) return MG_ERR_ARG;
    FastGemmArgs a{};
    a.X = X;
    a.M = n;
    a.K = K;
    a.W[0] = W;
    a.Nseg[0] = N;
    a.N = N;
    a.Y = Y;
    a.n_cu = device_cu_count();
    a.S = fast_gemm_splits(n, N, K, a.n_cu);
    a.part = static_cast<float*>(workspace);
    if (a.S == 1) return launch_fast_gemm(a, FEPI_F32, s) == hipSuccess ? MG_OK : MG_ERR_HIP;
    if (launch_fast_gemm(a, FEPI_PART, s) != hipSuccess) return MG_ERR_HIP;
    return launch_sum_partials(a.part, a.S, (int64_t)n * N, Y, s) == hipSuccess ? MG_OK : MG_ERR_HIP;
}

mg_status mg_op_fast_gemm_config(int n, int N, int K, int n_cu, int* S, int* waves) {
    if (n <= 0 || n > 256 || N <= 0 || K <= 0 || K % 8 || N % 16 || n_cu <= 0 || !S || !waves) return MG_ERR_ARG;
    fast_gemm_config(n, N, K, n_cu, S, waves);
    return MG_OK;
}

mg_status mg_op_canon_gemv_config(int n, int N, int K, int swiglu, int n_cu, int* kernel, int* tile_rows, int* quads,
                                  int* waves, int* depth) {
    if (n <= 0 || n > 256 || N <= 0 || K <= 0 || K % 8 || n_cu <= 0 || !kernel || !tile_rows || !quads || !waves ||
        !depth)
        return MG_ERR_ARG;
    if (!canon_gemv_on_mfma(n, false)) {
        *kernel = 2;
        *tile_rows = *quads = *waves = *depth = 0;
        return MG_OK;
    }
    const MfmaLaunch c = choose_mfma_launch(n, swiglu ? (N + 7) / 8 : (N + 15) / 16, K, n_cu);
    *kernel = 3;
    *tile_rows = c.tile_rows;
    *quads = c.quads;
    *waves = c.waves;
    *depth = c.depth;
    return MG_OK;
}

mg_status mg_op_decode_step_taps(mg_ctx* c, int B, const int32_t* tokens, const int32_t* positions,
                                 const int32_t* page_table, float* logits, uint16_t* x_taps, void* stream) {
    if (!c || !tokens || !positions || !page_table || !logits || !x_taps) return MG_ERR_ARG;
    if (B < 0 || B > c->cfg.max_batch) return MG_ERR_ARG;
    if (B == 0) return MG_OK;
    return fast_forward(c, B, tokens, positions, page_table, logits, nullptr, 0, static_cast<hipStream_t>(stream),
                        x_taps);
}

mg_status mg_op_rmsnorm(int n, int d, const uint16_t* x, const uint16_t* gamma, float eps, uint16_t* y, void* stream) {
    if (n <= 0 || d <= 0 || d % 8 || !x || !gamma || !y) return MG_ERR_ARG;
    return launch_rmsnorm(x, gamma, n, nullptr, n, d, eps, y, static_cast<hipStream_t>(stream)) == hipSuccess
               ? MG_OK
               : MG_ERR_HIP;
}

}  // extern "C"
