/*
 * mg_oracle.h -- CPU oracle of the MarginGate gated decode step (arXiv 2605.30218).
 *
 * TEST INFRASTRUCTURE ONLY.  This library is the plain, slow reference that the
 * GPU path is checked against.  Only the test-suite, the smoke check and the
 * CPU-baseline leg of the benchmark may load it; the product path never does.
 * It shares no code, header, table or constant with the GPU library: every
 * number it produces is recomputed here from the definitions.
 *
 * Paper anchors (section / equation names of arXiv 2605.30218):
 *   Sec. 3.1 "Margin trigger"       g = l_(1) - l_(2); verify iff g < tau
 *   Sec. 3.2 "Single-Column Repair" fast commit / verified commit / repair
 *   Sec. 3.2 "Deterministic verifier contract"
 *   Sec. 3.3 "Verifier Accounting"  r_verify, r_repair
 *   Sec. 2.4 (Obs. 3) N(Delta) = |{j : l_j >= l_(1) - Delta}|
 *
 * Two arithmetic modes share one decoder:
 *   MGO_PLAIN  textbook order: sequential fp32 sums, one-pass softmax with libm expf.
 *   MGO_CANON  the verifier's fixed, documented reduction order (CDOT, chunked
 *              attention, EXP); see the definitions in mg_oracle.c.
 * Storage is bf16 (uint16_t bit patterns), compute fp32, logits fp32.
 *
 * All pointers are host pointers owned by the caller.  Functions return 0 on
 * success and a negative value on a bad argument (nothing is written then).
 */
#ifndef MG_ORACLE_H
#define MG_ORACLE_H
#include <stdint.h>
#ifdef __cplusplus
extern "C" {
#endif

enum { MGO_PLAIN = 0, MGO_CANON = 1 };

typedef struct {
    int32_t n_layers, d_model, n_q_heads, n_kv_heads, head_dim, d_ffn, vocab, qkv_bias;
    float rope_theta, rms_eps;
    int32_t page_size, max_batch, max_pages_per_row, n_pages;
} mgo_cfg;

/* Weight pointer table, 3 + 12*n_layers entries, in this order:
 *   [0] embed [V][d]
 *   per layer l at 1 + 12*l:
 *     +0 attn_norm [d]   +1 wq [Hq*hd][d]   +2 wk [Hkv*hd][d]  +3 wv [Hkv*hd][d]
 *     +4 bq [Hq*hd]      +5 bk [Hkv*hd]     +6 bv [Hkv*hd]      (NULL when qkv_bias == 0)
 *     +7 wo [d][Hq*hd]   +8 ffn_norm [d]    +9 w_gate [F][d]   +10 w_up [F][d]  +11 w_down [d][F]
 *   [1 + 12*L] final_norm [d]    [2 + 12*L] lm_head [V][d]
 * Linear weights are nn.Linear layout [out][in], row-major bf16.
 * KV pool: [layer][page][K|V][Hkv][page_size][hd] bf16; K is stored after RoPE.
 * Page table: [row][max_pages_per_row] int32 page ids; position p of a row lives in
 * page page_table[row][p / page_size], slot p % page_size.
 * A verifier K/V column for one row: [layer][K|V][Hkv][hd] bf16. */

/* scalar primitives */
uint16_t mgo_bf16_from_f32(float f);
float    mgo_f32_from_bf16(uint16_t h);
float    mgo_exp(float x);                 /* EXP: Cody-Waite + degree-7 Taylor, fma Horner */
void     mgo_bf16_round_many(int64_t n, const float* in, uint16_t* out);
void     mgo_exp_many(int64_t n, const float* in, float* out);

/* op-level entry points (one vector / one row), used by the pins and the op parity tests */
float mgo_cdot(int K, const float* x, const float* w);           /* canonical dot, fp32 inputs */
void  mgo_rmsnorm(int mode, int d, const uint16_t* x, const uint16_t* gamma, float eps, uint16_t* y);
void  mgo_linear(int mode, int N, int K, const uint16_t* x, const uint16_t* W, const uint16_t* bias,
                 uint16_t* y_bf16, float* y_f32);                  /* either output may be NULL */
void  mgo_rope(int hd, int pos, double theta, int n_heads, uint16_t* v);   /* in place, [n_heads][hd] */
void  mgo_swiglu(int mode, int F, const uint16_t* g, const uint16_t* u, uint16_t* a);
/* attention of one query head over n_ctx contiguous keys/values [n_ctx][hd] */
void  mgo_attend(int mode, int hd, int n_ctx, const uint16_t* q, const uint16_t* K, const uint16_t* V,
                 uint16_t* out);
/* top-1 index (lowest index on ties) and margin l_(1) - l_(2); NaN entries rank below -inf and
   make the margin NaN */
void  mgo_top2(int V, const float* logits, int32_t* top1, float* margin);

/* the four calls of the step, on host memory */
int mgo_decode_step(const mgo_cfg* c, const void* const* w, int mode, int B, const int32_t* tokens,
                    const int32_t* positions, const int32_t* page_table, uint16_t* kv_pool, float* logits);
int mgo_margin_gate(int B, int V, const float* logits, const uint8_t* protected_mask, float tau,
                    int32_t* top1, float* margin, uint8_t* gate, int32_t* gated_rows, int32_t* n_gated);
int mgo_verify_rows(const mgo_cfg* c, const void* const* w, int mode, int n, const int32_t* rows,
                    const int32_t* tokens, const int32_t* positions, const int32_t* page_table,
                    const uint16_t* kv_pool, float* v_logits, int32_t* v_tok, uint16_t* v_kvcol);
int mgo_repair_kv_column(const mgo_cfg* c, int n, const int32_t* rows, const int32_t* positions,
                         const int32_t* page_table, const int32_t* top1, const int32_t* v_tok,
                         const uint16_t* v_kvcol, uint16_t* kv_pool, int32_t* emitted, int32_t* n_repaired);
/* the commit rule with a repair action: 0 copy the verifier column when the tokens differ
 * (Sec. 3.2), 1 token only (the repair-action ablation of Sec. 4), 2 copy on every verified row */
int mgo_repair_kv_column_action(const mgo_cfg* c, int n, const int32_t* rows, const int32_t* positions,
                                const int32_t* page_table, const int32_t* top1, const int32_t* v_tok,
                                const uint16_t* v_kvcol, uint16_t* kv_pool, int32_t* emitted, int32_t* n_repaired,
                                int action);
/* The step cut at layer boundaries, for state-forced per-layer checks.  Composing
 * mgo_embed, mgo_layer for layers 0..L-1 and mgo_head over the same rows gives exactly
 * mgo_decode_step (logits and cache).
 * mgo_embed: x[b] = embedding row of tokens[b], x bf16 [B][d].
 * mgo_layer: one decoder layer in `mode` on the residual stream x [B][d] (in place): row b
 *   at positions[b] writes its K/V column of that layer into kv_pool (the tentative
 *   append) and attends over positions 0..positions[b] of its page-table row.
 * mgo_head: final RMSNorm and LM head, fp32 logits [B][V] from x [B][d]. */
int mgo_embed(const mgo_cfg* c, const void* const* w, int B, const int32_t* tokens, uint16_t* x);
int mgo_layer(const mgo_cfg* c, const void* const* w, int mode, int layer, int B, const int32_t* positions,
              const int32_t* page_table, uint16_t* kv_pool, uint16_t* x);
int mgo_head(const mgo_cfg* c, const void* const* w, int mode, int B, const uint16_t* x, float* logits);
/* prompt prefill of one row, positions [0, n_tok), causal, in `mode` */
int mgo_prefill(const mgo_cfg* c, const void* const* w, int mode, int n_tok, const int32_t* tokens,
                const int32_t* page_table_row, uint16_t* kv_pool);

#ifdef __cplusplus
}
#endif
#endif
