// k_attn.hip -- the verifier's (and the prefill's) paged GQA decode attention.
//
// A block serves the G query heads that share a KV head, so each K/V page row is
// read from HBM once per item; the context is split into chunks whose partial
// (m, l, a) a combine kernel merges:
//   score      s_j = (q . k_j) * fp32(1/sqrt(hd))
//   chunk      m = max_j s_j, e_j = exp(s_j - m), l = sum_j e_j, a[d] = sum_j e_j v_jd
//   combine    over chunks in ascending order: M = max m_c, w_c = exp(m_c - M),
//              L = sum w_c l_c, O[d] = sum w_c a_c[d], out = bf16(O / L)
// Chunks of 256 positions, so the chunk count depends only on the context length;
// every sum is sequential in a fixed order (d for the scores, position for l and a,
// chunk for L and O), with fma where the definition has a product; the verifier's EXP.
// (The fast path's attention is in k_attn_fast.hip.)
// The current position p comes from the item's own column when one is given
// (the verifier never reads the tentative column of the cache).
#include "mg_device.h"
#include "mg_kernels.h"

namespace mg {

constexpr int ATT_MAXG = 8;     // query heads per KV head
constexpr int ATT_MAXHD = 128;
constexpr int ATT_MAXC = 256;   // positions per canonical chunk

__device__ __forceinline__ float attn_scale(int hd) { return hd == 128 ? 0x1.6a09e6p-4f : 0x1.0p-3f; }

// Canonical attention: one block of 256 threads per (item, KV head, chunk of 256
// positions).  Every K and V load of the chunk is issued at once (coalesced: a wave reads
// 4 whole rows per instruction), so the block waits for memory once.  K goes through LDS,
// where the 16-byte pieces of row j sit in xor-swizzled slots (piece k at slot k ^ (j mod
// U4)) so that thread j reads its own row without bank conflicts; V then takes the same
// LDS space.  The sequential chains below read LDS in unrolled batches, so their loads are
// in flight together.
//   scores  thread j: s_j for each query head of the group, sequential fma over d, * scale
//   chunk   wave w: heads w, w + 4: m = max_j s_j, e_j = EXP(s_j - m) in place
//   values  thread t: d pair (2 dp, 2 dp + 1) of the heads hg, hg + 256 / (hd/2), ...:
//           a[d] = sequential fma over j of e_j v_jd, and in the same loop
//           l = sequential sum of e_j in position order
template <int HD, int GP>  // GP: query heads per KV head, 1..8
__global__ __launch_bounds__(256) void attn_canon_kernel(AttnArgs a) {
    constexpr int U4 = HD / 8;                // 16-byte pieces per K/V row
    constexpr int NLD = ATT_MAXC * U4 / 256;  // V pieces per thread
    constexpr int HP = HD / 2;                // d pairs (words per V row)
    constexpr int HPT = 256 / HP;             // head groups over the block's threads
    constexpr int NPG = ATT_MAXC / 16;        // pages per chunk
#ifndef MG_ATT_UB
#define MG_ATT_UB 16
#endif
    constexpr int UB = MG_ATT_UB;             // positions per batch of LDS reads
    static_assert(UB % 4 == 0 && ATT_MAXC % UB == 0, "whole float4 batches");
    static_assert(NLD * 256 == ATT_MAXC * U4, "pieces must divide evenly");

    __shared__ __attribute__((aligned(16))) uint32_t vs[ATT_MAXC * HP];
    __shared__ __attribute__((aligned(16))) float qs[8 * 256];  // the group's queries, then padding
    __shared__ __attribute__((aligned(16))) float ps[GP * ATT_MAXC];
    __shared__ float red[GP][1];

    const int i = blockIdx.z;
    if (i >= items_n(a.it)) return;
    const int kh = blockIdx.y, c = blockIdx.x;
    const int r = items_row(a.it, i), p = items_pos(a.it, i);
    const int j0 = c * ATT_MAXC;
    if (j0 > p) return;
    const int nj = min(ATT_MAXC, p + 1 - j0);
    const ModelDims& m = a.m;
    constexpr int G = GP;  // query heads per KV head (a template parameter, so the head loops have no branch)
    const int Nk = m.Hkv * HD;
    const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
    const size_t kv_stride = (size_t)m.Hkv * m.page_size * HD;  // K -> V of the same page

    // page indices of the chunk (uniform, so read through the scalar cache together with the
    // queries); entries past the current position's page are clamped to it (always mapped)
    const int32_t* ptab = a.it.page_table + (size_t)r * m.max_pages_per_row;
    int pgs[NPG];
#pragma unroll
    for (int k = 0; k < NPG; ++k) pgs[k] = ptab[min(j0 / 16 + k, p >> 4)];
    // the group's rotated queries: one 16-byte load per thread (threads past the group's
    // 8-element pieces re-read the last piece and stage it into an unused part of qs)
    static_assert(GP * HD <= 8 * 256, "one 16-byte load per thread covers the group's queries");
    // (with qkv: the piece's RoPE partner piece and the cos/sin of its 8 pairs come too)
    const bool fold = a.qkv != nullptr;
    const uint16_t* qkv_row = fold ? a.qkv + (size_t)i * (m.Hq * HD + 2 * Nk) : nullptr;
    const int tq = min(t, G * HD / 8 - 1), e0 = (tq % U4) * 8;
    const bool qlow = e0 < HD / 2;  // the piece holds first-half elements of its head
    uint4 qv, qp;
    float4 cq[4];
    if (!fold) {
        qv = *reinterpret_cast<const uint4*>(a.qrot + (size_t)i * m.Hq * HD + (size_t)kh * G * HD + 8 * tq);
    } else {
        const uint16_t* qh = qkv_row + (size_t)(kh * G + tq / U4) * HD;
        qv = *reinterpret_cast<const uint4*>(qh + e0);
        qp = *reinterpret_cast<const uint4*>(qh + (qlow ? e0 + HD / 2 : e0 - HD / 2));
        const float* csr = a.cs + (size_t)p * HD + 2 * (qlow ? e0 : e0 - HD / 2);
#pragma unroll
        for (int k = 0; k < 4; ++k) cq[k] = *reinterpret_cast<const float4*>(csr + 4 * k);
    }
    // the own column: read from own_col, or (fold) rotated here into kown by the block whose
    // chunk holds position p, which also writes it to own_col for the repair
    const uint16_t* own = (a.own_col && !fold) ? a.own_col + ((size_t)i * m.L + a.layer) * 2 * Nk + (size_t)kh * HD
                                               : nullptr;
    const bool own_here = fold && p < j0 + ATT_MAXC;
    __shared__ __attribute__((aligned(16))) uint16_t kown[HD];
    // K block of page pg for this KV head
    auto page_k = [&](int pg) -> const uint16_t* {
        return a.kv_pool + ((((size_t)a.layer * m.n_pages + pg) * 2) * m.Hkv + kh) * (size_t)m.page_size * HD;
    };
    // K and V pieces: iteration k covers positions PPI*k .. PPI*k + PPI-1 (PPI/16 pages), thread t
    // piece t mod U4 of position t / U4 of those.  Every load is unconditional, so the waits
    // below count requests exactly and the queries can be staged while K and V are in flight:
    // positions past the chunk's last live one (nj - 1) re-read that position (a cache hit;
    // those values are never used).  The verifier's own column stands in for the cache's
    // tentative column p (the fold path's rotated own K row is taken from kown below).
    // (pieces as a native vector type: a struct copy held across the scores stays in memory)
    using u32x4 = uint32_t __attribute__((ext_vector_type(4)));
    constexpr int PPI = 256 / U4, PGI = PPI / 16;
    const int sub = (t / U4) >> 4;
    u32x4 kq[NLD], vr[NLD];
    const uint16_t* vps[NLD];
#pragma unroll
    for (int k = 0; k < NLD; ++k) {
        const int e = t + 256 * k;
        const int jj = min(e / U4, nj - 1), pc = e % U4;
        int pg = pgs[PGI * k];
#pragma unroll
        for (int q2 = 1; q2 < PGI; ++q2) pg = sub == q2 ? pgs[PGI * k + q2] : pg;
        const uint16_t* kc = page_k(pg) + (size_t)(jj & 15) * HD + pc * 8;
        const bool at_p = j0 + jj == p;
        kq[k] = *reinterpret_cast<const u32x4*>((own && at_p) ? own + pc * 8 : kc);
        vps[k] = (own && at_p)    ? own + Nk + pc * 8
                 : (fold && at_p) ? qkv_row + m.Hq * HD + Nk + (size_t)kh * HD + pc * 8
                                  : kc + kv_stride;
    }
#pragma unroll
    for (int k = 0; k < NLD; ++k) vr[k] = *reinterpret_cast<const u32x4*>(vps[k]);
    if (!fold) {
        float4* qd = reinterpret_cast<float4*>(qs + 8 * t);
        qd[0] = make_float4(bf_lo(qv.x), bf_hi(qv.x), bf_lo(qv.y), bf_hi(qv.y));
        qd[1] = make_float4(bf_lo(qv.z), bf_hi(qv.z), bf_lo(qv.w), bf_hi(qv.w));
    } else {
        // rotate-half RoPE of the piece, as the RoPE kernel computes it: pair (x_i, x_(i+hd/2))
        // -> (bf16(x_i c - x_(i+hd/2) s), bf16(x_(i+hd/2) c + x_i s)), products rounded apart
        const float pv[8] = {bf_lo(qv.x), bf_hi(qv.x), bf_lo(qv.y), bf_hi(qv.y),
                             bf_lo(qv.z), bf_hi(qv.z), bf_lo(qv.w), bf_hi(qv.w)};
        const float pp[8] = {bf_lo(qp.x), bf_hi(qp.x), bf_lo(qp.y), bf_hi(qp.y),
                             bf_lo(qp.z), bf_hi(qp.z), bf_lo(qp.w), bf_hi(qp.w)};
        const float cc[16] = {cq[0].x, cq[0].y, cq[0].z, cq[0].w, cq[1].x, cq[1].y, cq[1].z, cq[1].w,
                              cq[2].x, cq[2].y, cq[2].z, cq[2].w, cq[3].x, cq[3].y, cq[3].z, cq[3].w};
        float qf[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float lo = qlow ? pv[e] : pp[e], hi = qlow ? pp[e] : pv[e];
            const float c = cc[2 * e], sn = cc[2 * e + 1];
            const float ac = lo * c, bs = hi * sn, bc = hi * c, as = lo * sn;
            qf[e] = bf2f(f2bf(qlow ? ac - bs : bc + as));
        }
        float4* qd = reinterpret_cast<float4*>(qs + 8 * t);
        qd[0] = make_float4(qf[0], qf[1], qf[2], qf[3]);
        qd[1] = make_float4(qf[4], qf[5], qf[6], qf[7]);
        if (own_here && wave == 0) {
            const uint16_t* ks = qkv_row + m.Hq * HD + (size_t)kh * HD;
            const uint16_t* vsrc = ks + Nk;
            uint16_t* ow = a.own_col ? const_cast<uint16_t*>(a.own_col) + ((size_t)i * m.L + a.layer) * 2 * Nk +
                                           (size_t)kh * HD
                                     : nullptr;
            for (int ii = lane; ii < HD / 2; ii += 64) {
                const float lo = bf2f(ks[ii]), hi = bf2f(ks[ii + HD / 2]);
                const float c = a.cs[(size_t)p * HD + 2 * ii], sn = a.cs[(size_t)p * HD + 2 * ii + 1];
                const float ac = lo * c, bs = hi * sn, bc = hi * c, as = lo * sn;
                const uint16_t o1 = (uint16_t)f2bf(ac - bs), o2 = (uint16_t)f2bf(bc + as);
                kown[ii] = o1;
                kown[ii + HD / 2] = o2;
                if (ow) {
                    ow[ii] = o1;
                    ow[ii + HD / 2] = o2;
                    ow[Nk + ii] = vsrc[ii];
                    ow[Nk + ii + HD / 2] = vsrc[ii + HD / 2];
                }
            }
        }
    }
    // K into LDS, swizzled (the V requests stay in flight: loads complete in order)
#pragma unroll
    for (int k = 0; k < NLD; ++k) {
        const int e = t + 256 * k;
        const int jj = e / U4, pc = e % U4;
        *reinterpret_cast<u32x4*>(vs + (jj * U4 + (pc ^ (jj % U4))) * 4) = kq[k];
    }
    // the queries and K rows staged by other threads are needed from here on
    __syncthreads();
    // thread t's K row (the fold path's thread of position p takes the rotated own K row)
    uint4 kr[U4];
#pragma unroll
    for (int k = 0; k < U4; ++k) kr[k] = *reinterpret_cast<const uint4*>(vs + (t * U4 + (k ^ (t % U4))) * 4);
    if (own_here && t == nj - 1) {
#pragma unroll
        for (int k = 0; k < U4; ++k) kr[k] = reinterpret_cast<const uint4*>(kown)[k];
    }

    // ---- scores: position t, all heads of the group at once (K in registers), computed
    // while the V requests are still in flight

    const float scale = attn_scale(HD);
    if (t < nj) {
        float sc[GP];
#pragma unroll
        for (int h = 0; h < GP; ++h) sc[h] = 0.0f;
#pragma unroll
        for (int k = 0; k < U4; ++k) {
            const float kf[8] = {bf_lo(kr[k].x), bf_hi(kr[k].x), bf_lo(kr[k].y), bf_hi(kr[k].y),
                                 bf_lo(kr[k].z), bf_hi(kr[k].z), bf_lo(kr[k].w), bf_hi(kr[k].w)};
#pragma unroll
            for (int h = 0; h < GP; ++h) {
                {
                    const float4 q0 = *reinterpret_cast<const float4*>(qs + h * HD + 8 * k);
                    const float4 q1 = *reinterpret_cast<const float4*>(qs + h * HD + 8 * k + 4);
                    float s = sc[h];
                    s = __builtin_fmaf(q0.x, kf[0], s);
                    s = __builtin_fmaf(q0.y, kf[1], s);
                    s = __builtin_fmaf(q0.z, kf[2], s);
                    s = __builtin_fmaf(q0.w, kf[3], s);
                    s = __builtin_fmaf(q1.x, kf[4], s);
                    s = __builtin_fmaf(q1.y, kf[5], s);
                    s = __builtin_fmaf(q1.z, kf[6], s);
                    s = __builtin_fmaf(q1.w, kf[7], s);
                    sc[h] = s;
                }
            }
        }
#pragma unroll
        for (int h = 0; h < GP; ++h) ps[h * ATT_MAXC + t] = sc[h] * scale;
    }
    // every K read is done before V takes the LDS space
    __syncthreads();
#pragma unroll
    for (int k = 0; k < NLD; ++k) {
        const int e = t + 256 * k;
        *reinterpret_cast<u32x4*>(vs + (e / U4) * HP + (e % U4) * 4) = vr[k];
    }

    // ---- chunk max and exponentials (scores only: no barrier needed after the V stores)
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
        const int h = wave + 4 * hh;
        if (h < G) {
            float mx = -__builtin_inff();
            for (int j = lane; j < nj; j += 64) mx = fmaxf(mx, ps[h * ATT_MAXC + j]);
            mx = wave_max(mx);
            for (int j = lane; j < nj; j += 64) ps[h * ATT_MAXC + j] = canon_exp(ps[h * ATT_MAXC + j] - mx);
            if (lane == 0) red[h][0] = mx;
        }
    }
    __syncthreads();

    // ---- the weighted values, with l (the sequential sum of e_j in position order) carried
    // along in the same loop: every thread of head h forms the same l, the d-pair-0 thread
    // stores it
    const int nb = nj / UB * UB;  // positions handled in whole batches
    const int dp = t % HP, hg = t / HP;
    constexpr int NH = (GP + HPT - 1) / HPT;  // heads per thread
    float acc[NH][2], lsum[NH];
#pragma unroll
    for (int u = 0; u < NH; ++u) acc[u][0] = acc[u][1] = lsum[u] = 0.0f;
    for (int j = 0; j < nb; j += UB) {
        uint32_t vw[UB];
#pragma unroll
        for (int b = 0; b < UB; ++b) vw[b] = vs[(j + b) * HP + dp];
#pragma unroll
        for (int u = 0; u < NH; ++u) {
            const int h = hg + HPT * u;
            if (h < G) {
                float e[UB];
#pragma unroll
                for (int q4 = 0; q4 < UB / 4; ++q4) {
                    const float4 t4 = *reinterpret_cast<const float4*>(ps + h * ATT_MAXC + j + 4 * q4);
                    e[4 * q4] = t4.x; e[4 * q4 + 1] = t4.y; e[4 * q4 + 2] = t4.z; e[4 * q4 + 3] = t4.w;
                }
#pragma unroll
                for (int b = 0; b < UB; ++b) {
                    lsum[u] = lsum[u] + e[b];
                    acc[u][0] = __builtin_fmaf(e[b], bf_lo(vw[b]), acc[u][0]);
                    acc[u][1] = __builtin_fmaf(e[b], bf_hi(vw[b]), acc[u][1]);
                }
            }
        }
    }
    for (int j = nb; j < nj; ++j) {
        const uint32_t vw = vs[j * HP + dp];
#pragma unroll
        for (int u = 0; u < NH; ++u) {
            const int h = hg + HPT * u;
            if (h < G) {
                const float e = ps[h * ATT_MAXC + j];
                lsum[u] = lsum[u] + e;
                acc[u][0] = __builtin_fmaf(e, bf_lo(vw), acc[u][0]);
                acc[u][1] = __builtin_fmaf(e, bf_hi(vw), acc[u][1]);
            }
        }
    }
    constexpr int stride = HD + 2;
#pragma unroll
    for (int u = 0; u < NH; ++u) {
        const int h = hg + HPT * u;
        if (h < G) {
            float* dst = a.part + (((size_t)i * m.Hq + kh * G + h) * a.max_chunks + c) * stride;
            if (dp == 0) {
                dst[0] = red[h][0];
                dst[1] = lsum[u];
            }
            dst[2 + 2 * dp] = acc[u][0];
            dst[3 + 2 * dp] = acc[u][1];
        }
    }
}

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
    // the chunk partials are read in batches of CB (all loads of a batch in flight together)
    constexpr int CB = 8;
    float M = -__builtin_inff(), L = 0.0f, O = 0.0f;
    if (S <= CB) {
        float mc[CB], lc[CB], ac[CB];
#pragma unroll
        for (int c = 0; c < CB; ++c) {
            const int cc = min(c, S - 1);
            mc[c] = base[(size_t)cc * stride];
            lc[c] = base[(size_t)cc * stride + 1];
            ac[c] = base[(size_t)cc * stride + 2 + d];
        }
        M = mc[0];
#pragma unroll
        for (int c = 1; c < CB; ++c)
            if (c < S) M = fmaxf(M, mc[c]);
#pragma unroll
        for (int c = 0; c < CB; ++c) {
            if (c < S) {
                const float w = canon_exp(mc[c] - M);
                L = __builtin_fmaf(w, lc[c], L);
                O = __builtin_fmaf(w, ac[c], O);
            }
        }
    } else {
        M = base[0];
        for (int c = 1; c < S; ++c) M = fmaxf(M, base[(size_t)c * stride]);
        for (int c = 0; c < S; ++c) {
            const float w = canon_exp(base[(size_t)c * stride] - M);
            L = __builtin_fmaf(w, base[(size_t)c * stride + 1], L);
            O = __builtin_fmaf(w, base[(size_t)c * stride + 2 + d], O);
        }
    }
    a.out[(size_t)i * a.m.Hq * hd + (size_t)h * hd + d] = (uint16_t)f2bf(ieee_div(O, L));
}

template <int HD>
static void launch_canon_g(const AttnArgs& a, int G, dim3 g1, hipStream_t s) {
    switch (G) {
        case 1: hipLaunchKernelGGL((attn_canon_kernel<HD, 1>), g1, dim3(256), 0, s, a); break;
        case 2: hipLaunchKernelGGL((attn_canon_kernel<HD, 2>), g1, dim3(256), 0, s, a); break;
        case 3: hipLaunchKernelGGL((attn_canon_kernel<HD, 3>), g1, dim3(256), 0, s, a); break;
        case 4: hipLaunchKernelGGL((attn_canon_kernel<HD, 4>), g1, dim3(256), 0, s, a); break;
        case 5: hipLaunchKernelGGL((attn_canon_kernel<HD, 5>), g1, dim3(256), 0, s, a); break;
        case 6: hipLaunchKernelGGL((attn_canon_kernel<HD, 6>), g1, dim3(256), 0, s, a); break;
        case 7: hipLaunchKernelGGL((attn_canon_kernel<HD, 7>), g1, dim3(256), 0, s, a); break;
        default: hipLaunchKernelGGL((attn_canon_kernel<HD, 8>), g1, dim3(256), 0, s, a); break;
    }
}

hipError_t launch_attention(const AttnArgs& a, int canon, hipStream_t s) {
    const int n = a.it.n_host;
    if (n <= 0) return hipSuccess;
    if (!canon || a.chunk != ATT_MAXC) return hipErrorInvalidValue;  // the fast path has its own kernel
    dim3 g1(a.max_chunks, a.m.Hkv, n), g2(a.m.Hq, n);
    const int G = a.m.Hq / a.m.Hkv;
    if (G < 1 || G > ATT_MAXG) return hipErrorInvalidValue;
    if (a.m.hd == 128)
        launch_canon_g<128>(a, G, g1, s);
    else
        launch_canon_g<64>(a, G, g1, s);
    hipLaunchKernelGGL(attn_combine_kernel, g2, dim3(a.m.hd), 0, s, a);
    return hipGetLastError();
}

}  // namespace mg
