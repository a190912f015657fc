// k_attn.hip -- paged GQA decode attention, fast and canonical.
//
// One block per (item, KV head, chunk of positions).  The block serves the G
// query heads that share the KV head, so each K/V page row is read from HBM
// once per item.  K and V of the chunk are staged in LDS 64 positions at a time
// (K rows padded to an odd word stride: a lane per position reads conflict-free).
//   score      s_j = (sum_d q_d k_jd, sequential fma over d) * fp32(1/sqrt(hd))
//   chunk      m = max_j s_j, e_j = exp(s_j - m), l = sum_j e_j,
//              a[d] = sum_j e_j v_jd (sequential fma over j)
//   combine    over chunks in ascending order: M = max m_c, w_c = exp(m_c - M),
//              L = sum w_c l_c, O[d] = sum w_c a_c[d] (sequential fma), out = bf16(O / L)
// Canonical (the verifier): chunks of 256 positions, so the chunk count depends
// only on the context length; the verifier's EXP; l summed sequentially in
// position order.  Fast: any chunk size, hardware exp, tree sum for l.
// The current position p comes from the item's own column when one is given
// (the verifier never reads the tentative column of the cache).
#include "mg_device.h"
#include "mg_kernels.h"

namespace mg {

constexpr int ATT_MAXG = 8;     // query heads per KV head
constexpr int ATT_MAXHD = 128;
constexpr int ATT_MAXC = 256;   // positions per chunk
constexpr int ATT_SUB = 64;     // positions staged at a time

__device__ __forceinline__ float attn_scale(int hd) { return hd == 128 ? 0x1.6a09e6p-4f : 0x1.0p-3f; }

template <bool CANON>
__global__ __launch_bounds__(256) void attn_chunk_kernel(AttnArgs a) {
    const int i = blockIdx.z;
    if (i >= items_n(a.it)) return;
    const int kh = blockIdx.y, c = blockIdx.x;
    const int r = items_row(a.it, i), p = items_pos(a.it, i);
    const int C = a.chunk;
    const int j0 = c * C;
    if (j0 > p) return;
    const int nj = min(C, p + 1 - j0);
    const ModelDims& m = a.m;
    const int hd = m.hd, G = m.Hq / m.Hkv, Nk = m.Hkv * hd;
    const int KW = hd / 2 + 1;  // 32-bit words per staged K row (odd)

    __shared__ float qs[ATT_MAXG * ATT_MAXHD];
    __shared__ uint32_t ks[ATT_SUB * (ATT_MAXHD / 2 + 1)];
    __shared__ float ps[ATT_MAXG * ATT_MAXC];
    __shared__ __attribute__((aligned(16))) uint16_t vsh[ATT_SUB * ATT_MAXHD];
    __shared__ float red[ATT_MAXG][2];

    const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
    const uint16_t* qrow = a.qrot + (size_t)i * m.Hq * hd + (size_t)kh * G * hd;
    for (int e = t; e < G * hd; e += 256) qs[e] = bf2f(qrow[e]);
    const float scale = attn_scale(hd);
    const int32_t* ptab = a.it.page_table + (size_t)r * m.max_pages_per_row;
    const uint16_t* own = a.own_col ? a.own_col + ((size_t)i * m.L + a.layer) * 2 * Nk + (size_t)kh * hd : nullptr;

    auto src_row = [&](int jpos, int kv) -> const uint16_t* {
        if (own && jpos == p) return own + (size_t)kv * Nk;
        const int page = ptab[jpos / m.page_size], slot = jpos % m.page_size;
        return a.kv_pool + ((((size_t)a.layer * m.n_pages + page) * 2 + kv) * m.Hkv + kh) * (size_t)m.page_size * hd +
               (size_t)slot * hd;
    };

    const int nsub = (nj + ATT_SUB - 1) / ATT_SUB;
    const int u4 = hd / 8;  // 16-byte pieces per row
    // ---- scores
    for (int sc = 0; sc < nsub; ++sc) {
        const int jb = j0 + sc * ATT_SUB;
        const int nn = min(ATT_SUB, j0 + nj - jb);
        __syncthreads();
        for (int e = t; e < nn * u4; e += 256) {
            const int pp = e / u4, uu = e % u4;
            const uint4 v = reinterpret_cast<const uint4*>(src_row(jb + pp, 0))[uu];
            uint32_t* dst = ks + pp * KW + uu * 4;
            dst[0] = v.x; dst[1] = v.y; dst[2] = v.z; dst[3] = v.w;
        }
        __syncthreads();
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
            const int h = wave + 4 * hh;
            if (h < G && lane < nn) {
                const uint32_t* kr = ks + lane * KW;
                const float* qh = qs + h * hd;
                float s = 0.0f;
                for (int w2 = 0; w2 < hd / 2; ++w2) {
                    const uint32_t kw = kr[w2];
                    s = __builtin_fmaf(qh[2 * w2], bf_lo(kw), s);
                    s = __builtin_fmaf(qh[2 * w2 + 1], bf_hi(kw), s);
                }
                ps[h * ATT_MAXC + sc * ATT_SUB + lane] = s * scale;
            }
        }
    }
    __syncthreads();
    // ---- chunk max, exponentials (and the fast sum)
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
        const int h = wave + 4 * hh;
        if (h < G) {
            float mx = -__builtin_inff();
            for (int j = lane; j < nj; j += 64) mx = fmaxf(mx, ps[h * ATT_MAXC + j]);
            mx = wave_max(mx);
            float ls = 0.0f;
            for (int j = lane; j < nj; j += 64) {
                const float d = ps[h * ATT_MAXC + j] - mx;
                const float e = CANON ? canon_exp(d) : __expf(d);
                ps[h * ATT_MAXC + j] = e;
                ls += e;
            }
            if (!CANON) ls = wave_sum_fast(ls);
            if (lane == 0) {
                red[h][0] = mx;
                red[h][1] = ls;
            }
        }
    }
    __syncthreads();
    if (CANON && t < G) {  // l = sum of e_j in position order
        float l = 0.0f;
        for (int j = 0; j < nj; ++j) l = l + ps[t * ATT_MAXC + j];
        red[t][1] = l;
    }
    // ---- weighted values
    float acc[4] = {0.f, 0.f, 0.f, 0.f};
    for (int sc = 0; sc < nsub; ++sc) {
        const int jb = j0 + sc * ATT_SUB;
        const int nn = min(ATT_SUB, j0 + nj - jb);
        __syncthreads();
        for (int e = t; e < nn * u4; e += 256) {
            const int pp = e / u4, uu = e % u4;
            reinterpret_cast<uint4*>(vsh + pp * hd)[uu] = reinterpret_cast<const uint4*>(src_row(jb + pp, 1))[uu];
        }
        __syncthreads();
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const int o = t + 256 * k;
            if (o < G * hd) {
                const int h = o / hd, d = o % hd;
                const float* ph = ps + h * ATT_MAXC + sc * ATT_SUB;
                float s = acc[k];
                for (int pp = 0; pp < nn; ++pp) s = __builtin_fmaf(ph[pp], bf2f(vsh[pp * hd + d]), s);
                acc[k] = s;
            }
        }
    }
    __syncthreads();
    const int stride = hd + 2;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int o = t + 256 * k;
        if (o < G * hd) {
            const int h = o / hd, d = o % hd;
            float* dst = a.part + (((size_t)i * m.Hq + kh * G + h) * a.max_chunks + c) * stride;
            if (d == 0) {
                dst[0] = red[h][0];
                dst[1] = red[h][1];
            }
            dst[2 + d] = acc[k];
        }
    }
}

template <bool CANON>
__global__ void attn_combine_kernel(AttnArgs a) {
    const int i = blockIdx.y;
    if (i >= items_n(a.it)) return;
    const int h = blockIdx.x, d = threadIdx.x;
    const int hd = a.m.hd;
    if (d >= hd) return;
    const int p = items_pos(a.it, i);
    const int S = (p + 1 + a.chunk - 1) / a.chunk;
    const int stride = hd + 2;
    const float* base = a.part + ((size_t)i * a.m.Hq + h) * a.max_chunks * stride;
    float M = base[0];
    for (int c = 1; c < S; ++c) M = fmaxf(M, base[(size_t)c * stride]);
    float L = 0.0f, O = 0.0f;
    for (int c = 0; c < S; ++c) {
        const float mc = base[(size_t)c * stride];
        const float w = CANON ? canon_exp(mc - M) : __expf(mc - M);
        L = __builtin_fmaf(w, base[(size_t)c * stride + 1], L);
        O = __builtin_fmaf(w, base[(size_t)c * stride + 2 + d], O);
    }
    a.out[(size_t)i * a.m.Hq * hd + (size_t)h * hd + d] = (uint16_t)f2bf(ieee_div(O, L));
}

hipError_t launch_attention(const AttnArgs& a, int canon, hipStream_t s) {
    const int n = a.it.n_host;
    if (n <= 0) return hipSuccess;
    dim3 g1(a.max_chunks, a.m.Hkv, n), g2(a.m.Hq, n);
    if (canon) {
        hipLaunchKernelGGL(attn_chunk_kernel<true>, g1, dim3(256), 0, s, a);
        hipLaunchKernelGGL(attn_combine_kernel<true>, g2, dim3(a.m.hd), 0, s, a);
    } else {
        hipLaunchKernelGGL(attn_chunk_kernel<false>, g1, dim3(256), 0, s, a);
        hipLaunchKernelGGL(attn_combine_kernel<false>, g2, dim3(a.m.hd), 0, s, a);
    }
    return hipGetLastError();
}

}  // namespace mg
