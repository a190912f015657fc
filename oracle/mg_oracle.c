/*
 * mg_oracle.c -- CPU oracle of the MarginGate gated decode step (arXiv 2605.30218).
 *
 * TEST INFRASTRUCTURE ONLY: loaded by the tests, the smoke check and the CPU
 * baseline of the benchmark, never by the product path.  Shares no code with
 * the GPU library.
 *
 * What is computed, and where the paper fixes it:
 *  - The decoder is a Llama/Qwen-style dense transformer run one row at a time
 *    (rows never interact, so this oracle is batch-invariant by construction).
 *    Storage is bf16 and every reduction accumulates in fp32; the fast path is
 *    the ordinary batched BF16 forward whose logits feed the gate (Sec. 3.1,
 *    margin trigger).
 *  - The margin is g = l_(1) - l_(2) over the fp32 logits of the current step,
 *    and the verifier fires iff g < tau, strictly (Sec. 3.1).
 *  - The verifier runs the current step again for the row and returns a token plus the
 *    K/V column of the current position (Sec. 3.2, Deterministic verifier
 *    contract).  It reads the committed cache for earlier positions and its own
 *    freshly computed column for the current one.
 *  - Commit: fast commit and verified commit keep the tentative column; when the
 *    verifier token differs, the verifier token is emitted and only the current
 *    column is overwritten, in every layer (Sec. 3.2, Single-Column Repair).
 *
 * Readings where the paper is silent (each is listed with its reason in the
 * design notes of the repository):
 *  - rounding points: every linear, norm, RoPE, attention and SwiGLU output is
 *    rounded once to bf16 (round to nearest even); logits stay fp32;
 *  - the verifier's fixed reduction order is the CANON mode below: CDOT for every
 *    dot product over the model width, chunked attention with chunks of 256
 *    positions combined in ascending order, and the EXP function below;
 *  - argmax ties go to the lowest index; a duplicated maximum gives g = 0;
 *    a NaN logit makes g NaN and fires the gate.
 *
 * Compile with -ffp-contract=off: every a*b+c below is two roundings unless it
 * is written as fmaf().
 */
#include "mg_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#define WPL 12 /* weight pointers per layer */
#define CANON_CHUNK 256

/* ------------------------------------------------------------------ scalars */

/* bf16 <- fp32, round to nearest, ties to even.  The upper 16 bits are the
 * truncation; the lower 16 bits decide whether to step up by one bf16 ulp. */
uint16_t mgo_bf16_from_f32(float f) {
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x0040u); /* quiet NaN */
    uint32_t hi = u >> 16, lo = u & 0xffffu;
    if (lo > 0x8000u || (lo == 0x8000u && (hi & 1u))) hi += 1u; /* carries into the exponent */
    return (uint16_t)hi;
}

float mgo_f32_from_bf16(uint16_t h) {
    uint32_t u = (uint32_t)h << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

void mgo_bf16_round_many(int64_t n, const float* in, uint16_t* out) {
    for (int64_t i = 0; i < n; ++i) out[i] = mgo_bf16_from_f32(in[i]);
}

/* EXP(x) = 2^n * P(r), x = n ln2 + r, |r| <= ln2/2 (Cody and Waite's additive
 * range reduction, with ln 2 split in two fp32 parts and fused multiply-adds),
 * P the degree-7 Taylor polynomial of e^r evaluated by Horner's rule with fma.
 * n > 127 overflows to +inf; n < -126 flushes to +0. */
float mgo_exp(float x) {
    if (x != x) return x;
    const double LN2 = 0.693147180559945309417232121458176568;
    const float log2e = (float)1.442695040888963407359924681001892137;
    const float ln2_hi = (float)LN2;
    const float ln2_lo = (float)(LN2 - (double)ln2_hi);
    float n = rintf(x * log2e);
    if (n > 127.0f) return INFINITY;
    if (n < -126.0f) return 0.0f;
    float r = fmaf(-n, ln2_hi, x);
    r = fmaf(-n, ln2_lo, r);
    /* Taylor coefficients 1/k!, each rounded once to fp32 */
    const float c[8] = {(float)(1.0 / 1.0),   (float)(1.0 / 1.0),   (float)(1.0 / 2.0),    (float)(1.0 / 6.0),
                        (float)(1.0 / 24.0),  (float)(1.0 / 120.0), (float)(1.0 / 720.0),  (float)(1.0 / 5040.0)};
    float p = c[7];
    for (int k = 6; k >= 0; --k) p = fmaf(p, r, c[k]);
    return ldexpf(p, (int)n);
}

void mgo_exp_many(int64_t n, const float* in, float* out) {
    for (int64_t i = 0; i < n; ++i) out[i] = mgo_exp(in[i]);
}

static inline float bf(uint16_t h) { return mgo_f32_from_bf16(h); }
static inline uint16_t rb(float f) { return mgo_bf16_from_f32(f); }

/* ------------------------------------------------------------ dot products */

/* CDOT, the verifier's dot product over a K-vector, K % 8 == 0.  Elements are
 * taken in groups of 8; group g belongs to lane g mod 64.  Each of the 64 lanes
 * starts at +0 and fma-accumulates its groups in increasing g, element order
 * within the group.  The 64 lane sums are then combined by the xor butterfly
 * with offsets 32, 16, 8, 4, 2, 1: a_l <- a_l + a_(l xor o). */
static float cdot_lanes(int K, const float* x, const uint16_t* wb, const float* wf) {
    float lane[64];
    const int G = K / 8;
    for (int l = 0; l < 64; ++l) {
        float a = 0.0f;
        for (int g = l; g < G; g += 64)
            for (int e = 0; e < 8; ++e) {
                const int k = 8 * g + e;
                const float w = wb ? bf(wb[k]) : wf[k];
                a = fmaf(x[k], w, a);
            }
        lane[l] = a;
    }
    for (int o = 32; o >= 1; o >>= 1) {
        float nxt[64];
        for (int l = 0; l < 64; ++l) nxt[l] = lane[l] + lane[l ^ o];
        memcpy(lane, nxt, sizeof lane);
    }
    return lane[0];
}

float mgo_cdot(int K, const float* x, const float* w) { return cdot_lanes(K, x, NULL, w); }

/* textbook sequential dot: a = a + x_k * w_k, left to right, from +0 */
static float seqdot(int K, const float* x, const uint16_t* wb) {
    float a = 0.0f;
    for (int k = 0; k < K; ++k) a = a + x[k] * bf(wb[k]);
    return a;
}

static float dot_mode(int mode, int K, const float* x, const uint16_t* wb) {
    return mode == MGO_CANON ? cdot_lanes(K, x, wb, NULL) : seqdot(K, x, wb);
}

/* ------------------------------------------------------------------- ops */

/* RMSNorm: ss = sum x_i^2; r = 1/sqrt(ss/d + eps); y_i = bf16((x_i * r) * gamma_i) */
void mgo_rmsnorm(int mode, int d, const uint16_t* x, const uint16_t* gamma, float eps, uint16_t* y) {
    float* xf = (float*)malloc(sizeof(float) * (size_t)d);
    for (int i = 0; i < d; ++i) xf[i] = bf(x[i]);
    float ss;
    if (mode == MGO_CANON) {
        ss = cdot_lanes(d, xf, NULL, xf);
    } else {
        ss = 0.0f;
        for (int i = 0; i < d; ++i) ss = ss + xf[i] * xf[i];
    }
    const float m = ss / (float)d;
    const float r = 1.0f / sqrtf(m + eps);
    for (int i = 0; i < d; ++i) y[i] = rb((xf[i] * r) * bf(gamma[i]));
    free(xf);
}

/* Linear: y_j = bf16(dot(x, W_j) + b_j); the bias is added in fp32 before the one rounding. */
void mgo_linear(int mode, int N, int K, const uint16_t* x, const uint16_t* W, const uint16_t* bias,
                uint16_t* y_bf16, float* y_f32) {
    float* xf = (float*)malloc(sizeof(float) * (size_t)K);
    for (int k = 0; k < K; ++k) xf[k] = bf(x[k]);
#pragma omp parallel for schedule(static)
    for (int j = 0; j < N; ++j) {
        float a = dot_mode(mode, K, xf, W + (size_t)j * K);
        if (bias) a = a + bf(bias[j]);
        if (y_f32) y_f32[j] = a;
        if (y_bf16) y_bf16[j] = rb(a);
    }
    free(xf);
}

/* RoPE, rotate-half convention: pair (i, i + hd/2) is rotated by angle
 * pos * theta^(-2i/hd).  Frequency and angle in float64, cos/sin rounded to
 * fp32; the rotation itself is four fp32 products and two sums, unfused. */
void mgo_rope(int hd, int pos, double theta, int n_heads, uint16_t* v) {
    const int h = hd / 2;
    for (int i = 0; i < h; ++i) {
        const double inv = pow(theta, -(2.0 * (double)i) / (double)hd);
        const double ang = (double)pos * inv;
        const float c = (float)cos(ang), s = (float)sin(ang);
        for (int head = 0; head < n_heads; ++head) {
            uint16_t* q = v + (size_t)head * hd;
            const float a = bf(q[i]), b = bf(q[i + h]);
            const float ac = a * c, bs = b * s, bc = b * c, as = a * s;
            q[i] = rb(ac - bs);
            q[i + h] = rb(bc + as);
        }
    }
}

/* SwiGLU: a = bf16(silu(g) * u), silu(g) = g / (1 + e^-g) */
void mgo_swiglu(int mode, int F, const uint16_t* g, const uint16_t* u, uint16_t* a) {
    for (int i = 0; i < F; ++i) {
        const float gv = bf(g[i]);
        const float t = mode == MGO_CANON ? mgo_exp(-gv) : expf(-gv);
        const float sg = gv / (1.0f + t);
        a[i] = rb(sg * bf(u[i]));
    }
}

/* Attention of one query head over keys/values given by row pointers.
 * PLAIN: s_j = (sum_d q_d k_jd) * scale, one softmax over all positions with expf.
 * CANON: s_j = SEQ-fma(q, k_j) * scale; positions are cut into chunks of 256;
 *        per chunk c: m_c = max s_j, e_j = EXP(s_j - m_c), l_c = SEQ(e_j),
 *        a_c[d] = SEQ-fma(e_j, v_jd); then over chunks in ascending order:
 *        M = max m_c, w_c = EXP(m_c - M), L = SEQ-fma(w_c, l_c), O[d] = SEQ-fma(w_c, a_c[d]).
 * out[d] = bf16(O[d] / L). */
static void attend_ptrs(int mode, int hd, int n_ctx, const float* q, const uint16_t* const* kr,
                        const uint16_t* const* vr, uint16_t* out) {
    const float scale = (float)(1.0 / sqrt((double)hd));
    float* s = (float*)malloc(sizeof(float) * (size_t)n_ctx);
    float* O = (float*)calloc((size_t)hd, sizeof(float));
    if (mode != MGO_CANON) {
        for (int j = 0; j < n_ctx; ++j) {
            float a = 0.0f;
            for (int d = 0; d < hd; ++d) a = a + q[d] * bf(kr[j][d]);
            s[j] = a * scale;
        }
        float m = s[0];
        for (int j = 1; j < n_ctx; ++j) m = s[j] > m ? s[j] : m;
        float L = 0.0f;
        for (int j = 0; j < n_ctx; ++j) {
            const float e = expf(s[j] - m);
            L = L + e;
            for (int d = 0; d < hd; ++d) O[d] = O[d] + e * bf(vr[j][d]);
        }
        for (int d = 0; d < hd; ++d) out[d] = rb(O[d] / L);
    } else {
        for (int j = 0; j < n_ctx; ++j) {
            float a = 0.0f;
            for (int d = 0; d < hd; ++d) a = fmaf(q[d], bf(kr[j][d]), a);
            s[j] = a * scale;
        }
        const int S = (n_ctx + CANON_CHUNK - 1) / CANON_CHUNK;
        float* mc = (float*)malloc(sizeof(float) * (size_t)S);
        float* lc = (float*)malloc(sizeof(float) * (size_t)S);
        float* ac = (float*)calloc((size_t)S * hd, sizeof(float));
        for (int c = 0; c < S; ++c) {
            const int j0 = c * CANON_CHUNK;
            const int j1 = j0 + CANON_CHUNK < n_ctx ? j0 + CANON_CHUNK : n_ctx;
            float m = s[j0];
            for (int j = j0 + 1; j < j1; ++j) m = s[j] > m ? s[j] : m;
            float l = 0.0f;
            for (int j = j0; j < j1; ++j) {
                const float e = mgo_exp(s[j] - m);
                l = l + e;
                for (int d = 0; d < hd; ++d) ac[(size_t)c * hd + d] = fmaf(e, bf(vr[j][d]), ac[(size_t)c * hd + d]);
            }
            mc[c] = m;
            lc[c] = l;
        }
        float M = mc[0];
        for (int c = 1; c < S; ++c) M = mc[c] > M ? mc[c] : M;
        float L = 0.0f;
        for (int c = 0; c < S; ++c) {
            const float wc = mgo_exp(mc[c] - M);
            L = fmaf(wc, lc[c], L);
            for (int d = 0; d < hd; ++d) O[d] = fmaf(wc, ac[(size_t)c * hd + d], O[d]);
        }
        for (int d = 0; d < hd; ++d) out[d] = rb(O[d] / L);
        free(mc);
        free(lc);
        free(ac);
    }
    free(s);
    free(O);
}

void mgo_attend(int mode, int hd, int n_ctx, const uint16_t* q, const uint16_t* K, const uint16_t* V,
                uint16_t* out) {
    const uint16_t** kr = (const uint16_t**)malloc(sizeof(void*) * (size_t)n_ctx);
    const uint16_t** vr = (const uint16_t**)malloc(sizeof(void*) * (size_t)n_ctx);
    float* qf = (float*)malloc(sizeof(float) * (size_t)hd);
    for (int j = 0; j < n_ctx; ++j) {
        kr[j] = K + (size_t)j * hd;
        vr[j] = V + (size_t)j * hd;
    }
    for (int d = 0; d < hd; ++d) qf[d] = bf(q[d]);
    attend_ptrs(mode, hd, n_ctx, qf, kr, vr, out);
    free(kr);
    free(vr);
    free(qf);
}

/* Top-1 / top-2 over one logit row.  Ranking: larger value first, equal values
 * by lower index; NaN ranks below every number.  l_(2) is the second largest
 * value of the multiset (a duplicated maximum gives margin 0). */
void mgo_top2(int V, const float* logits, int32_t* top1, float* margin) {
    int best = -1, has_nan = 0;
    float v1 = -INFINITY, v2 = -INFINITY;
    for (int j = 0; j < V; ++j) {
        const float v = logits[j];
        if (v != v) {
            has_nan = 1;
            continue;
        }
        if (best < 0) {
            v1 = v;
            best = j;
        } else if (v > v1) { /* strictly larger: the old maximum becomes the runner-up */
            v2 = v1;
            v1 = v;
            best = j;
        } else if (v > v2) { /* includes v == v1: a second copy of the maximum */
            v2 = v;
        }
    }
    if (best < 0) best = 0; /* every entry NaN */
    *top1 = best;
    *margin = has_nan ? NAN : v1 - v2;
}

/* --------------------------------------------------------------- the model */

typedef struct {
    const mgo_cfg* c;
    const uint16_t* const* w;
} model_t;

static const uint16_t* W(const model_t* m, int idx) { return m->w[idx]; }
static const uint16_t* LW(const model_t* m, int layer, int k) { return m->w[1 + WPL * layer + k]; }

static size_t kv_index(const mgo_cfg* c, int layer, int page, int kv, int kh, int slot) {
    return ((((size_t)layer * c->n_pages + page) * 2 + kv) * c->n_kv_heads + kh) * (size_t)c->page_size * c->head_dim +
           (size_t)slot * c->head_dim;
}

static size_t col_size(const mgo_cfg* c) { return (size_t)c->n_layers * 2 * c->n_kv_heads * c->head_dim; }

/* Scratch of one row's layer: every intermediate of the layer, sized for the shape. */
typedef struct {
    uint16_t *h, *q, *k, *v, *att, *y, *g, *u, *a;
    const uint16_t **kr, **vr;
    float* qf;
} layer_buf_t;

static int layer_buf_init(const mgo_cfg* c, int pos, layer_buf_t* b) {
    const int d = c->d_model, Hq = c->n_q_heads, Hkv = c->n_kv_heads, hd = c->head_dim, F = c->d_ffn;
    b->h = (uint16_t*)malloc(2 * (size_t)d);
    b->q = (uint16_t*)malloc(2 * (size_t)Hq * hd);
    b->k = (uint16_t*)malloc(2 * (size_t)Hkv * hd);
    b->v = (uint16_t*)malloc(2 * (size_t)Hkv * hd);
    b->att = (uint16_t*)malloc(2 * (size_t)Hq * hd);
    b->y = (uint16_t*)malloc(2 * (size_t)(d > F ? d : F));
    b->g = (uint16_t*)malloc(2 * (size_t)F);
    b->u = (uint16_t*)malloc(2 * (size_t)F);
    b->a = (uint16_t*)malloc(2 * (size_t)F);
    b->kr = (const uint16_t**)malloc(sizeof(void*) * (size_t)(pos + 1));
    b->vr = (const uint16_t**)malloc(sizeof(void*) * (size_t)(pos + 1));
    b->qf = (float*)malloc(sizeof(float) * (size_t)hd);
    return b->h && b->q && b->k && b->v && b->att && b->y && b->g && b->u && b->a && b->kr && b->vr && b->qf;
}

static void layer_buf_free(layer_buf_t* b) {
    free(b->h); free(b->q); free(b->k); free(b->v); free(b->att); free(b->y); free(b->g); free(b->u); free(b->a);
    free(b->kr); free(b->vr); free(b->qf);
}

/* Checks a row's token (token < 0: not checked), position and mapped pages 0..pos. */
static int row_ok(const mgo_cfg* c, int token, int pos, const int32_t* ptab) {
    const int ps = c->page_size;
    if ((token >= 0 && token >= c->vocab) || pos < 0 || pos >= c->max_pages_per_row * ps) return 0;
    for (int p = 0; p <= pos; ++p) {
        const int pg = ptab[p / ps];
        if (pg < 0 || pg >= c->n_pages) return 0;
    }
    return 1;
}

/* One decoder layer of one row at position pos, on the residual stream x [d] (in place):
 * pre-norm attention with the row's own K/V column (after RoPE) placed in the cache
 * (kvcol == NULL: the fast path's tentative append) or in kvcol (the verifier's scratch
 * column, cache untouched), earlier positions read from kv_read, then the pre-norm SwiGLU
 * block; both blocks add into x with one bf16 rounding each. */
static void layer_row(const model_t* m, int mode, int l, int pos, const int32_t* ptab, uint16_t* kv_pool,
                      const uint16_t* kv_read, uint16_t* kvcol, uint16_t* x, layer_buf_t* b) {
    const mgo_cfg* c = m->c;
    const int d = c->d_model, Hq = c->n_q_heads, Hkv = c->n_kv_heads, hd = c->head_dim, F = c->d_ffn;
    const int G = Hq / Hkv, ps = c->page_size;
    mgo_rmsnorm(mode, d, x, LW(m, l, 0), c->rms_eps, b->h);
    mgo_linear(mode, Hq * hd, d, b->h, LW(m, l, 1), c->qkv_bias ? LW(m, l, 4) : NULL, b->q, NULL);
    mgo_linear(mode, Hkv * hd, d, b->h, LW(m, l, 2), c->qkv_bias ? LW(m, l, 5) : NULL, b->k, NULL);
    mgo_linear(mode, Hkv * hd, d, b->h, LW(m, l, 3), c->qkv_bias ? LW(m, l, 6) : NULL, b->v, NULL);
    mgo_rope(hd, pos, (double)c->rope_theta, Hq, b->q);
    mgo_rope(hd, pos, (double)c->rope_theta, Hkv, b->k);
    /* own column */
    const uint16_t *ownk[64], *ownv[64];
    for (int kh = 0; kh < Hkv; ++kh) {
        uint16_t *dk, *dv;
        if (kvcol) {
            dk = kvcol + (((size_t)l * 2 + 0) * Hkv + kh) * hd;
            dv = kvcol + (((size_t)l * 2 + 1) * Hkv + kh) * hd;
        } else {
            const int pg = ptab[pos / ps], sl = pos % ps;
            dk = kv_pool + kv_index(c, l, pg, 0, kh, sl);
            dv = kv_pool + kv_index(c, l, pg, 1, kh, sl);
        }
        memcpy(dk, b->k + (size_t)kh * hd, 2 * (size_t)hd);
        memcpy(dv, b->v + (size_t)kh * hd, 2 * (size_t)hd);
        ownk[kh] = dk;
        ownv[kh] = dv;
    }
    for (int hh = 0; hh < Hq; ++hh) {
        const int kh = hh / G;
        for (int p = 0; p < pos; ++p) {
            const int pg = ptab[p / ps], sl = p % ps;
            b->kr[p] = kv_read + kv_index(c, l, pg, 0, kh, sl);
            b->vr[p] = kv_read + kv_index(c, l, pg, 1, kh, sl);
        }
        b->kr[pos] = ownk[kh];
        b->vr[pos] = ownv[kh];
        for (int dd = 0; dd < hd; ++dd) b->qf[dd] = bf(b->q[(size_t)hh * hd + dd]);
        attend_ptrs(mode, hd, pos + 1, b->qf, b->kr, b->vr, b->att + (size_t)hh * hd);
    }
    mgo_linear(mode, d, Hq * hd, b->att, LW(m, l, 7), NULL, b->y, NULL);
    for (int i = 0; i < d; ++i) x[i] = rb(bf(x[i]) + bf(b->y[i]));
    mgo_rmsnorm(mode, d, x, LW(m, l, 8), c->rms_eps, b->h);
    mgo_linear(mode, F, d, b->h, LW(m, l, 9), NULL, b->g, NULL);
    mgo_linear(mode, F, d, b->h, LW(m, l, 10), NULL, b->u, NULL);
    mgo_swiglu(mode, F, b->g, b->u, b->a);
    mgo_linear(mode, d, F, b->a, LW(m, l, 11), NULL, b->y, NULL);
    for (int i = 0; i < d; ++i) x[i] = rb(bf(x[i]) + bf(b->y[i]));
}

/* The head of one row: final RMSNorm, then the LM head with fp32 logits (never rounded). */
static void head_row(const model_t* m, int mode, const uint16_t* x, uint16_t* h, float* logits) {
    const mgo_cfg* c = m->c;
    mgo_rmsnorm(mode, c->d_model, x, W(m, 1 + WPL * c->n_layers), c->rms_eps, h);
    mgo_linear(mode, c->vocab, c->d_model, h, W(m, 2 + WPL * c->n_layers), NULL, NULL, logits);
}

/* One row's forward at position pos: the embedding row of the token, every layer in
 * order (layer_row), then the head when logits != NULL (prefill passes NULL). */
static int forward_row(const model_t* m, int mode, int token, int pos, const int32_t* ptab, uint16_t* kv_pool,
                       const uint16_t* kv_read, uint16_t* kvcol, float* logits) {
    const mgo_cfg* c = m->c;
    const int d = c->d_model;
    if (token < 0 || !row_ok(c, token, pos, ptab)) return -2;
    layer_buf_t b = {0};
    uint16_t* x = (uint16_t*)malloc(2 * (size_t)d);
    if (!x || !layer_buf_init(c, pos, &b)) {
        free(x);
        layer_buf_free(&b);
        return -3;
    }
    memcpy(x, W(m, 0) + (size_t)token * d, 2 * (size_t)d);
    for (int l = 0; l < c->n_layers; ++l) layer_row(m, mode, l, pos, ptab, kv_pool, kv_read, kvcol, x, &b);
    if (logits) head_row(m, mode, x, b.h, logits);
    free(x);
    layer_buf_free(&b);
    return 0;
}

static int cfg_ok(const mgo_cfg* c) {
    if (!c) return 0;
    if (c->n_layers <= 0 || c->d_model <= 0 || c->n_q_heads <= 0 || c->n_kv_heads <= 0) return 0;
    if (c->n_q_heads % c->n_kv_heads || c->n_kv_heads > 64) return 0;
    if (c->d_model % 8 || c->d_ffn % 8 || (c->n_q_heads * c->head_dim) % 8 || c->head_dim % 2) return 0;
    if (c->page_size <= 0 || c->max_pages_per_row <= 0 || c->n_pages <= 0 || c->vocab <= 0) return 0;
    return 1;
}

int mgo_decode_step(const mgo_cfg* c, const void* const* w, int mode, int B, const int32_t* tokens,
                    const int32_t* positions, const int32_t* page_table, uint16_t* kv_pool, float* logits) {
    if (!cfg_ok(c) || !w || B < 0 || !tokens || !positions || !page_table || !kv_pool || !logits) return -1;
    model_t m = {c, (const uint16_t* const*)w};
    for (int b = 0; b < B; ++b) {
        int rc = forward_row(&m, mode, tokens[b], positions[b], page_table + (size_t)b * c->max_pages_per_row,
                             kv_pool, kv_pool, NULL, logits + (size_t)b * c->vocab);
        if (rc) return rc;
    }
    return 0;
}

int mgo_margin_gate(int B, int V, const float* logits, const uint8_t* protected_mask, float tau,
                    int32_t* top1, float* margin, uint8_t* gate, int32_t* gated_rows, int32_t* n_gated) {
    if (B < 0 || V < 2 || !logits || !top1 || !margin || !gate || !gated_rows || !n_gated) return -1;
    int n = 0;
    for (int b = 0; b < B; ++b) {
        mgo_top2(V, logits + (size_t)b * V, &top1[b], &margin[b]);
        const int prot = protected_mask ? protected_mask[b] != 0 : 1;
        /* strict trigger g < tau; a NaN margin is never >= tau, so it fires */
        const int fire = prot && !(margin[b] >= tau);
        gate[b] = (uint8_t)fire;
        if (fire) gated_rows[n++] = b;
    }
    *n_gated = n;
    return 0;
}

int mgo_verify_rows(const mgo_cfg* c, const void* const* w, int mode, int n, const int32_t* rows,
                    const int32_t* tokens, const int32_t* positions, const int32_t* page_table,
                    const uint16_t* kv_pool, float* v_logits, int32_t* v_tok, uint16_t* v_kvcol) {
    if (!cfg_ok(c) || !w || n < 0 || (n && (!rows || !tokens || !positions || !page_table || !kv_pool || !v_tok ||
                                             !v_kvcol)))
        return -1;
    model_t m = {c, (const uint16_t* const*)w};
    float* lg = (float*)malloc(sizeof(float) * (size_t)c->vocab);
    for (int i = 0; i < n; ++i) {
        const int r = rows[i];
        float* out = v_logits ? v_logits + (size_t)i * c->vocab : lg;
        int rc = forward_row(&m, mode, tokens[r], positions[r], page_table + (size_t)r * c->max_pages_per_row, NULL,
                             kv_pool, v_kvcol + (size_t)i * col_size(c), out);
        if (rc) {
            free(lg);
            return rc;
        }
        float mg;
        mgo_top2(c->vocab, out, &v_tok[i], &mg);
    }
    free(lg);
    return 0;
}

/* Sec. 3.2 commit rule (action 0) and the two variants around it: token only -- the
 * verifier's token is emitted and the tentative BF16 column stays, the ablation of Sec. 4
 * (Ablations and Robustness, repair action); copy always -- the verifier's column is copied
 * on every verified row, agreeing ones included. */
int mgo_repair_kv_column_action(const mgo_cfg* c, int n, const int32_t* rows, const int32_t* positions,
                                const int32_t* page_table, const int32_t* top1, const int32_t* v_tok,
                                const uint16_t* v_kvcol, uint16_t* kv_pool, int32_t* emitted, int32_t* n_repaired,
                                int action) {
    if (!cfg_ok(c) || n < 0 || !n_repaired || action < 0 || action > 2) return -1;
    const int hd = c->head_dim, Hkv = c->n_kv_heads, ps = c->page_size;
    for (int i = 0; i < n; ++i) {
        const int r = rows[i];
        emitted[r] = v_tok[i];
        const int copy = action == 2 || (action == 0 && v_tok[i] != top1[r]);
        if (!copy) continue; /* verified commit (or token only): keep the tentative column */
        const int p = positions[r];
        const int pg = page_table[(size_t)r * c->max_pages_per_row + p / ps], sl = p % ps;
        for (int l = 0; l < c->n_layers; ++l)
            for (int kv = 0; kv < 2; ++kv)
                for (int kh = 0; kh < Hkv; ++kh)
                    memcpy(kv_pool + kv_index(c, l, pg, kv, kh, sl),
                           v_kvcol + (size_t)i * col_size(c) + (((size_t)l * 2 + kv) * Hkv + kh) * hd, 2 * (size_t)hd);
        *n_repaired += 1;
    }
    return 0;
}

int mgo_repair_kv_column(const mgo_cfg* c, int n, const int32_t* rows, const int32_t* positions,
                         const int32_t* page_table, const int32_t* top1, const int32_t* v_tok,
                         const uint16_t* v_kvcol, uint16_t* kv_pool, int32_t* emitted, int32_t* n_repaired) {
    return mgo_repair_kv_column_action(c, n, rows, positions, page_table, top1, v_tok, v_kvcol, kv_pool, emitted,
                                       n_repaired, 0);
}

int mgo_prefill(const mgo_cfg* c, const void* const* w, int mode, int n_tok, const int32_t* tokens,
                const int32_t* page_table_row, uint16_t* kv_pool) {
    if (!cfg_ok(c) || !w || n_tok < 0 || (n_tok && (!tokens || !page_table_row || !kv_pool))) return -1;
    model_t m = {c, (const uint16_t* const*)w};
    for (int t = 0; t < n_tok; ++t) {
        int rc = forward_row(&m, mode, tokens[t], t, page_table_row, kv_pool, kv_pool, NULL, NULL);
        if (rc) return rc;
    }
    return 0;
}

/* ---------------------------------------------------- layer-level entry points */

int mgo_embed(const mgo_cfg* c, const void* const* w, int B, const int32_t* tokens, uint16_t* x) {
    if (!cfg_ok(c) || !w || B < 0 || (B && (!tokens || !x))) return -1;
    const uint16_t* E = ((const uint16_t* const*)w)[0];
    for (int b = 0; b < B; ++b) {
        if (tokens[b] < 0 || tokens[b] >= c->vocab) return -2;
        memcpy(x + (size_t)b * c->d_model, E + (size_t)tokens[b] * c->d_model, 2 * (size_t)c->d_model);
    }
    return 0;
}

int mgo_layer(const mgo_cfg* c, const void* const* w, int mode, int layer, int B, const int32_t* positions,
              const int32_t* page_table, uint16_t* kv_pool, uint16_t* x) {
    if (!cfg_ok(c) || !w || B < 0 || layer < 0 || layer >= c->n_layers ||
        (B && (!positions || !page_table || !kv_pool || !x)))
        return -1;
    model_t m = {c, (const uint16_t* const*)w};
    for (int b = 0; b < B; ++b) {
        const int32_t* ptab = page_table + (size_t)b * c->max_pages_per_row;
        if (!row_ok(c, -1, positions[b], ptab)) return -2;
        layer_buf_t lb = {0};
        if (!layer_buf_init(c, positions[b], &lb)) {
            layer_buf_free(&lb);
            return -3;
        }
        layer_row(&m, mode, layer, positions[b], ptab, kv_pool, kv_pool, NULL, x + (size_t)b * c->d_model, &lb);
        layer_buf_free(&lb);
    }
    return 0;
}

int mgo_head(const mgo_cfg* c, const void* const* w, int mode, int B, const uint16_t* x, float* logits) {
    if (!cfg_ok(c) || !w || B < 0 || (B && (!x || !logits))) return -1;
    model_t m = {c, (const uint16_t* const*)w};
    uint16_t* h = (uint16_t*)malloc(2 * (size_t)c->d_model);
    if (!h) return -3;
    for (int b = 0; b < B; ++b)
        head_row(&m, mode, x + (size_t)b * c->d_model, h, logits + (size_t)b * c->vocab);
    free(h);
    return 0;
}
