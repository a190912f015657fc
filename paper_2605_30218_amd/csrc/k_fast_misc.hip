// k_fast_misc.hip -- the fast path's consumers of split-K partial tiles.
//
// resid_norm: one block per row.  Sums the S fp32 partial tiles of the O or down
// projection in split order, rounds the projection to bf16, adds it to the residual
// stream (x = bf16(x + y)), and applies the next RMSNorm (h = bf16((x * r) * gamma),
// r = 1 / sqrt(mean(x^2) + eps)) from registers.  At layer 0 it takes x from the
// embedding table instead.
// swiglu_part: sums the gate/up partial tiles, rounds g and u to bf16 and writes
// a = bf16(silu(g) * u) once, for the down projection to stage.
// (The QKV partial tiles are consumed by the fused attention kernel, k_attn_fast.hip.)
#include "mg_device.h"
#include "mg_kernels.h"

namespace mg {

constexpr int RN_THREADS = 1024;
constexpr int RN_MAXQ = 2;  // float4 groups per thread: d <= 8192

// sum of the S split partials of 4 consecutive features, in split order; loads are
// issued in batches of 8 before they are added
__device__ __forceinline__ float4 sum_splits4(const float* p, size_t sstride, int S) {
    float4 y = *reinterpret_cast<const float4*>(p);
    int sp = 1;
    for (; sp + 8 <= S; sp += 8) {
        float4 t[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) t[k] = *reinterpret_cast<const float4*>(p + (size_t)(sp + k) * sstride);
#pragma unroll
        for (int k = 0; k < 8; ++k) { y.x += t[k].x; y.y += t[k].y; y.z += t[k].z; y.w += t[k].w; }
    }
    for (; sp < S; ++sp) {
        const float4 t = *reinterpret_cast<const float4*>(p + (size_t)sp * sstride);
        y.x += t.x; y.y += t.y; y.z += t.z; y.w += t.w;
    }
    return y;
}

__global__ __launch_bounds__(RN_THREADS) void resid_norm_kernel(int M, const float* __restrict__ part, int S,
                                                                const uint16_t* __restrict__ embed,
                                                                const int32_t* __restrict__ tokens, int d,
                                                                const uint16_t* __restrict__ gamma, float eps,
                                                                uint16_t* __restrict__ x, uint16_t* __restrict__ h) {
    const int r = blockIdx.x;
    const int d4 = d / 4;
    uint2* xr = reinterpret_cast<uint2*>(x + (size_t)r * d);
    const uint2* src = embed ? reinterpret_cast<const uint2*>(embed + (size_t)tokens[r] * d) : xr;
    // gamma is requested first, so the block waits for memory once
    const uint2* g2 = reinterpret_cast<const uint2*>(gamma);
    uint2 gv[RN_MAXQ];
#pragma unroll
    for (int k = 0; k < RN_MAXQ; ++k) {
        const int q = threadIdx.x + RN_THREADS * k;
        gv[k] = q < d4 ? g2[q] : make_uint2(0, 0);
    }
    float4 xv[RN_MAXQ];
    float ss = 0.0f;
#pragma unroll
    for (int k = 0; k < RN_MAXQ; ++k) {
        const int q = threadIdx.x + RN_THREADS * k;
        if (q >= d4) break;
        const uint2 v = src[q];
        float4 o = make_float4(bf_lo(v.x), bf_hi(v.x), bf_lo(v.y), bf_hi(v.y));
        if (part) {
            const float4 y = sum_splits4(part + (size_t)r * d + 4 * q, (size_t)M * d, S);
            o.x = bf2f(f2bf(o.x + bf2f(f2bf(y.x))));
            o.y = bf2f(f2bf(o.y + bf2f(f2bf(y.y))));
            o.z = bf2f(f2bf(o.z + bf2f(f2bf(y.z))));
            o.w = bf2f(f2bf(o.w + bf2f(f2bf(y.w))));
        }
        if (part || embed) xr[q] = make_uint2(pack_bf2(o.x, o.y), pack_bf2(o.z, o.w));
        xv[k] = o;
        ss += o.x * o.x + o.y * o.y + o.z * o.z + o.w * o.w;
    }
    __shared__ float red[RN_THREADS / 64];
    ss = wave_sum_fast(ss);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    float tot = 0.0f;
#pragma unroll
    for (int w = 0; w < RN_THREADS / 64; ++w) tot += red[w];
    const float rs = ieee_div(1.0f, ieee_sqrt(ieee_div(tot, (float)d) + eps));
    uint2* hr = reinterpret_cast<uint2*>(h + (size_t)r * d);
#pragma unroll
    for (int k = 0; k < RN_MAXQ; ++k) {
        const int q = threadIdx.x + RN_THREADS * k;
        if (q >= d4) break;
        const uint2 g = gv[k];
        const float4 o = xv[k];
        hr[q] = make_uint2(pack_bf2((o.x * rs) * bf_lo(g.x), (o.y * rs) * bf_hi(g.x)),
                           pack_bf2((o.z * rs) * bf_lo(g.y), (o.w * rs) * bf_hi(g.y)));
    }
}

hipError_t launch_resid_norm(int B, const float* part, int S, const uint16_t* embed, const int32_t* tokens, int d,
                             const uint16_t* gamma, float eps, uint16_t* x, uint16_t* h, hipStream_t s) {
    if (B <= 0) return hipSuccess;
    if (d % 4 || d / 4 > RN_THREADS * RN_MAXQ) return hipErrorInvalidValue;
    hipLaunchKernelGGL(resid_norm_kernel, dim3(B), dim3(RN_THREADS), 0, s, B, part, S, embed, tokens, d, gamma, eps,
                       x, h);
    return hipGetLastError();
}

// SwiGLU of the split gate/up projection: g = bf16(sum of gate partials),
// u = bf16(sum of up partials), a = bf16(silu(g) * u); part rows are [gate F | up F]
__global__ __launch_bounds__(256) void swiglu_part_kernel(int M, const float* __restrict__ part, int S, int F,
                                                          uint16_t* __restrict__ act) {
    const int r = blockIdx.y;
    const int q = blockIdx.x * 256 + threadIdx.x;  // float4 group of the gate half
    if (q >= F / 4) return;
    const size_t sstride = (size_t)M * 2 * F;
    const float4 g = sum_splits4(part + (size_t)r * 2 * F + 4 * q, sstride, S);
    const float4 u = sum_splits4(part + (size_t)r * 2 * F + F + 4 * q, sstride, S);
    const float gg[4] = {bf2f(f2bf(g.x)), bf2f(f2bf(g.y)), bf2f(f2bf(g.z)), bf2f(f2bf(g.w))};
    const float uu[4] = {bf2f(f2bf(u.x)), bf2f(f2bf(u.y)), bf2f(f2bf(u.z)), bf2f(f2bf(u.w))};
    float a[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) a[k] = (gg[k] / (1.0f + __expf(-gg[k]))) * uu[k];
    reinterpret_cast<uint2*>(act + (size_t)r * F)[q] = make_uint2(pack_bf2(a[0], a[1]), pack_bf2(a[2], a[3]));
}

hipError_t launch_swiglu_part(int B, const float* part, int S, int F, uint16_t* act, hipStream_t s) {
    if (B <= 0) return hipSuccess;
    if (F % 4) return hipErrorInvalidValue;
    hipLaunchKernelGGL(swiglu_part_kernel, dim3((F / 4 + 255) / 256, B), dim3(256), 0, s, B, part, S, F, act);
    return hipGetLastError();
}

}  // namespace mg
