// mg_device.h -- device helpers of libmg (gfx950): bf16 conversion, the verifier's
// EXP, wave reductions.  Compiled with -ffp-contract=off: a*b+c is two roundings
// unless written as __builtin_fmaf.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#define MG_WAVE 64

namespace mg {

__device__ __forceinline__ float bf2f(uint32_t h16) { return __uint_as_float(h16 << 16); }
__device__ __forceinline__ float bf_lo(uint32_t pair) { return __uint_as_float(pair << 16); }
__device__ __forceinline__ float bf_hi(uint32_t pair) { return __uint_as_float(pair & 0xffff0000u); }

// fp32 -> bf16, round to nearest even; NaN becomes a quiet NaN with the same sign
// and upper payload bits.  Adding 0x7fff plus the kept lsb carries into the upper
// half exactly when the discarded half exceeds one half ulp, or equals it with an
// odd kept lsb.
__device__ __forceinline__ uint32_t f2bf(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return (u >> 16) | 0x40u;
    u += 0x7fffu + ((u >> 16) & 1u);
    return u >> 16;
}

__device__ __forceinline__ uint32_t pack_bf2(float lo, float hi) { return f2bf(lo) | (f2bf(hi) << 16); }

// The verifier's exponential: x = n ln2 + r with n = rint(x log2e), r reduced by
// the two-part ln2 (fp32 head + fp32 tail) with fused multiply-adds; e^r by the
// degree-7 Taylor polynomial in Horner form with fma; then r scaled by 2^n.
// n > 127 -> +inf, n < -126 -> +0.  Constants: log2e, ln2 and 1/k! each rounded to
// fp32; the tail is the fp32 rounding of (ln2 - fp32(ln2)).
__device__ __forceinline__ float canon_exp(float x) {
    if (x != x) return x;
    const float n = __builtin_rintf(x * 0x1.715476p+0f);
    if (n > 127.0f) return __builtin_inff();
    if (n < -126.0f) return 0.0f;
    float r = __builtin_fmaf(-n, 0x1.62e430p-1f, x);
    r = __builtin_fmaf(-n, -0x1.05c610p-29f, r);
    float p = 0x1.a01a02p-13f;              // 1/7!
    p = __builtin_fmaf(p, r, 0x1.6c16c2p-10f);  // 1/6!
    p = __builtin_fmaf(p, r, 0x1.111112p-7f);   // 1/5!
    p = __builtin_fmaf(p, r, 0x1.555556p-5f);   // 1/4!
    p = __builtin_fmaf(p, r, 0x1.555556p-3f);   // 1/3!
    p = __builtin_fmaf(p, r, 0x1.0p-1f);        // 1/2!
    p = __builtin_fmaf(p, r, 1.0f);             // 1/1!
    p = __builtin_fmaf(p, r, 1.0f);             // 1/0!
    return __builtin_ldexpf(p, (int)n);
}

// Correctly rounded fp32 division and square root (IEEE), as used by the
// verifier's RMSNorm, SwiGLU and attention normalisation.  The library is built
// with -fhip-fp32-correctly-rounded-divide-sqrt, so plain '/' and sqrtf are the
// IEEE operations; the GPU tests check them against the host bit for bit.
__device__ __forceinline__ float ieee_div(float a, float b) { return a / b; }
__device__ __forceinline__ float ieee_sqrt(float a) { return __builtin_sqrtf(a); }

// xor butterfly over the 64 lanes: a_l <- a_l + a_(l xor o), o = 32..1.
// IEEE addition is commutative, so every lane ends with the same bits.
__device__ __forceinline__ float butterfly_sum(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = v + __shfl_xor(v, o, MG_WAVE);
    return v;
}

// The same xor butterfly for NV = 2^k values at once.  At offset o a lane keeps the
// level sum of one value of each pair and gets its partner's copy of that value, so
// every sum is formed from exactly the operands the single-value butterfly adds at
// that lane (own value + partner at l xor o); after k levels each lane holds one
// value, and the remaining offsets run as the plain butterfly.  Value index
// v = sum_j bit(lane, 5 - j) << j ends up in every lane whose bits 5..6-k spell v.
template <int NV>
__device__ __forceinline__ float butterfly_sum_multi(float (&v)[NV], int lane) {
    static_assert(NV >= 1 && NV <= 64 && (NV & (NV - 1)) == 0, "power of two up to 64");
    int o = 32;
#pragma unroll
    for (int cnt = NV; cnt > 1; cnt >>= 1) {
        const bool hi = (lane & o) != 0;
#pragma unroll
        for (int i = 0; i < cnt / 2; ++i) {
            const float a = v[2 * i], b = v[2 * i + 1];
            const float recv = __shfl_xor(hi ? a : b, o, MG_WAVE);
            v[i] = hi ? b + recv : a + recv;
        }
        o >>= 1;
    }
    float r = v[0];
    for (; o >= 1; o >>= 1) r = r + __shfl_xor(r, o, MG_WAVE);
    return r;
}

// index of the value butterfly_sum_multi<NV> leaves in `lane`, and whether this lane
// is the lowest of the lanes holding it
template <int NV>
__device__ __forceinline__ int multi_index(int lane, bool* writer) {
    int k = 0;
    while ((1 << k) < NV) ++k;
    int v = 0;
    for (int j = 0; j < k; ++j) v |= ((lane >> (5 - j)) & 1) << j;
    *writer = (lane & ((1 << (6 - k)) - 1)) == 0;
    return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, MG_WAVE));
    return v;
}

__device__ __forceinline__ float wave_sum_fast(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, MG_WAVE);
    return v;
}

// ---- top-1 / top-2 states (the margin gate and the matrix-core verifier's fused LM-head epilogue)
// Partial state of a top-2 scan: best value/index and the runner-up value of the
// multiset seen so far.  Merging two states is associative and commutative: the
// winner is the larger value, the lower index on equal values; the runner-up is
// the larger of the winner's runner-up and the loser's best.  NaN entries are
// skipped and only flagged.
struct Top2 {
    float v1, v2;
    int i1;
    int nan;
};

__device__ __forceinline__ Top2 top2_merge(const Top2& a, const Top2& b) {
    if (a.i1 < 0) return Top2{b.v1, b.v2, b.i1, b.nan | a.nan};
    if (b.i1 < 0) return Top2{a.v1, a.v2, a.i1, a.nan | b.nan};
    const bool aw = (a.v1 > b.v1) || (a.v1 == b.v1 && a.i1 < b.i1);
    Top2 o;
    if (aw) {
        o.v1 = a.v1; o.i1 = a.i1; o.v2 = fmaxf(a.v2, b.v1);
    } else {
        o.v1 = b.v1; o.i1 = b.i1; o.v2 = fmaxf(b.v2, a.v1);
    }
    o.nan = a.nan | b.nan;
    return o;
}

__device__ __forceinline__ void top2_push(Top2& s, float v, int j) {
    if (v != v) { s.nan = 1; return; }
    if (s.i1 < 0) { s.v1 = v; s.i1 = j; return; }
    if (v > s.v1) { s.v2 = s.v1; s.v1 = v; s.i1 = j; }   // j increases within a thread: ties keep the old index
    else if (v > s.v2) s.v2 = v;
}

__device__ __forceinline__ Top2 top2_shfl(const Top2& s, int o) {
    Top2 t;
    t.v1 = __shfl_xor(s.v1, o, MG_WAVE);
    t.v2 = __shfl_xor(s.v2, o, MG_WAVE);
    t.i1 = __shfl_xor(s.i1, o, MG_WAVE);
    t.nan = __shfl_xor(s.nan, o, MG_WAVE);
    return t;
}

// Row set of a launch: `n` rows, or the count read on the device (capped).
struct RowCount {
    const int32_t* dev;
    int host;
    int cap;
    __device__ __forceinline__ int get() const {
        if (!dev) return host;
        int n = *dev;
        return n < 0 ? 0 : (n > cap ? cap : n);
    }
};

}  // namespace mg
