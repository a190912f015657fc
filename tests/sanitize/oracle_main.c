/* Drives every entry point of the CPU oracle on a tiny model, for a build with the address
 * and undefined-behaviour sanitizers (test infrastructure).  Inputs come from a fixed linear
 * congruential sequence; the results are only checked for being finite and in range, the
 * numerics being pinned by the Python tests. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "../../oracle/mg_oracle.h"

static uint32_t state = 12345u;
static float urand(void) { /* in [-1, 1) */
    state = state * 1664525u + 1013904223u;
    return (float)((state >> 8) & 0xffffff) / 8388608.0f - 1.0f;
}

static uint16_t* tensor(size_t n, float scale) {
    uint16_t* t = (uint16_t*)malloc(2 * n);
    for (size_t i = 0; i < n; ++i) t[i] = mgo_bf16_from_f32(scale * urand());
    return t;
}

static uint16_t* ones(size_t n) {
    uint16_t* t = (uint16_t*)malloc(2 * n);
    for (size_t i = 0; i < n; ++i) t[i] = mgo_bf16_from_f32(1.0f);
    return t;
}

#define CHECK(c)                                                   \
    do {                                                           \
        if (!(c)) {                                                \
            fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
            return 1;                                              \
        }                                                          \
    } while (0)

int main(void) {
    mgo_cfg c = {2, 64, 4, 2, 16, 96, 512, 1, 10000.0f, 1e-5f, 16, 3, 4, 12};
    const int L = c.n_layers, d = c.d_model, Hq = c.n_q_heads, Hkv = c.n_kv_heads, hd = c.head_dim, F = c.d_ffn,
              V = c.vocab;
    const int nw = 3 + 12 * L;
    void** w = (void**)calloc((size_t)nw, sizeof(void*));
    w[0] = tensor((size_t)V * d, 0.5f);
    for (int l = 0; l < L; ++l) {
        void** b = w + 1 + 12 * l;
        b[0] = ones(d);
        b[1] = tensor((size_t)Hq * hd * d, 0.1f);
        b[2] = tensor((size_t)Hkv * hd * d, 0.1f);
        b[3] = tensor((size_t)Hkv * hd * d, 0.1f);
        b[4] = tensor((size_t)Hq * hd, 0.1f);
        b[5] = tensor((size_t)Hkv * hd, 0.1f);
        b[6] = tensor((size_t)Hkv * hd, 0.1f);
        b[7] = tensor((size_t)d * Hq * hd, 0.1f);
        b[8] = ones(d);
        b[9] = tensor((size_t)F * d, 0.1f);
        b[10] = tensor((size_t)F * d, 0.1f);
        b[11] = tensor((size_t)d * F, 0.1f);
    }
    w[1 + 12 * L] = ones(d);
    w[2 + 12 * L] = tensor((size_t)V * d, 0.1f);
    const size_t kv_elems = (size_t)L * c.n_pages * 2 * Hkv * c.page_size * hd;
    uint16_t* kv = (uint16_t*)calloc(kv_elems, 2);
    int32_t pt[3][4] = {{0, 3, 6, 9}, {1, 4, 7, 10}, {2, 5, 8, 11}};
    int32_t prompt[3][40];
    for (int r = 0; r < 3; ++r)
        for (int t = 0; t < 40; ++t) prompt[r][t] = (int32_t)((7 * t + 13 * r + 5) % V);
    const int plen[3] = {40, 17, 2};
    for (int mode = 0; mode < 2; ++mode) {
        memset(kv, 0, 2 * kv_elems);
        for (int r = 0; r < 3; ++r) CHECK(mgo_prefill(&c, (const void* const*)w, mode, plen[r] - 1, prompt[r], pt[r], kv) == 0);
        int32_t tok[3], pos[3];
        for (int r = 0; r < 3; ++r) {
            tok[r] = prompt[r][plen[r] - 1];
            pos[r] = plen[r] - 1;
        }
        float* logits = (float*)malloc(sizeof(float) * 3 * V);
        CHECK(mgo_decode_step(&c, (const void* const*)w, mode, 3, tok, pos, (const int32_t*)pt, kv, logits) == 0);
        for (int i = 0; i < 3 * V; ++i) CHECK(isfinite(logits[i]));
        int32_t top1[3], rows[3], ng = -1, nrep = 0, vt[3], emitted[3];
        float margin[3];
        uint8_t gate[3], prot[3] = {1, 0, 1};
        CHECK(mgo_margin_gate(3, V, logits, prot, 1e9f, top1, margin, gate, rows, &ng) == 0);
        CHECK(ng == 2 && rows[0] == 0 && rows[1] == 2);
        float* vl = (float*)malloc(sizeof(float) * 2 * V);
        uint16_t* vc = (uint16_t*)malloc(2 * 2 * (size_t)L * 2 * Hkv * hd);
        CHECK(mgo_verify_rows(&c, (const void* const*)w, mode, ng, rows, tok, pos, (const int32_t*)pt, kv, vl, vt, vc) == 0);
        for (int i = 0; i < 3; ++i) emitted[i] = top1[i];
        for (int a = 0; a < 3; ++a)
            CHECK(mgo_repair_kv_column_action(&c, ng, rows, pos, (const int32_t*)pt, top1, vt, vc, kv, emitted, &nrep, a) == 0);
        CHECK(mgo_repair_kv_column(&c, ng, rows, pos, (const int32_t*)pt, top1, vt, vc, kv, emitted, &nrep) == 0);
        uint16_t* x = (uint16_t*)malloc(2 * 3 * (size_t)d);
        CHECK(mgo_embed(&c, (const void* const*)w, 3, tok, x) == 0);
        for (int l = 0; l < L; ++l) CHECK(mgo_layer(&c, (const void* const*)w, mode, l, 3, pos, (const int32_t*)pt, kv, x) == 0);
        CHECK(mgo_head(&c, (const void* const*)w, mode, 3, x, logits) == 0);
        /* bad arguments are refused without writes */
        int32_t bad_pos[3] = {63, 64, 0};
        CHECK(mgo_decode_step(&c, (const void* const*)w, mode, 3, tok, bad_pos, (const int32_t*)pt, kv, logits) != 0);
        CHECK(mgo_layer(&c, (const void* const*)w, mode, L, 3, pos, (const int32_t*)pt, kv, x) != 0);
        free(x);
        free(vl);
        free(vc);
        free(logits);
    }
    /* op-level entry points */
    float xs[4096], ws[4096], ex[64];
    for (int i = 0; i < 4096; ++i) {
        xs[i] = urand();
        ws[i] = urand();
    }
    CHECK(isfinite(mgo_cdot(4096, xs, ws)));
    for (int i = 0; i < 64; ++i) ex[i] = 4.0f * urand() * (float)i;
    float eo[64];
    mgo_exp_many(64, ex, eo);
    uint16_t q[16], K[5 * 16], Vv[5 * 16], out[16];
    for (int i = 0; i < 16; ++i) q[i] = mgo_bf16_from_f32(urand());
    for (int i = 0; i < 80; ++i) {
        K[i] = mgo_bf16_from_f32(urand());
        Vv[i] = mgo_bf16_from_f32(urand());
    }
    for (int mode = 0; mode < 2; ++mode) mgo_attend(mode, 16, 5, q, K, Vv, out);
    uint16_t rv[2 * 16];
    for (int i = 0; i < 32; ++i) rv[i] = mgo_bf16_from_f32(urand());
    mgo_rope(16, 7, 1e4, 2, rv);
    float lg[9] = {1, 3, 3, -2, NAN, 0, 1, 2, 3};
    int32_t t1;
    float mg;
    mgo_top2(9, lg, &t1, &mg);
    CHECK(t1 == 1 && isnan(mg));
    for (int i = 0; i < nw; ++i) free(w[i]);
    free(w);
    free(kv);
    printf("oracle sanitizer run ok\n");
    return 0;
}
