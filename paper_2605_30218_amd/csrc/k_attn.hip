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

// Canonical attention: one block of NT threads (NT = 512 or 1024) per (item, KV head, chunk
// of 256 positions).  Every K and V load of the chunk is issued at once (coalesced: a wave
// reads whole rows), so the block waits for memory once, and the V loads stay in flight
// while the scores run.  K goes through LDS, where the 16-byte pieces of row j sit in
// xor-swizzled slots (piece k at slot k ^ (j mod U4)) so that the threads of one position
// read its row without bank conflicts; V then takes the same LDS space.  Every chain below
// is one thread's sequential loop, in the order of the definition:
//   scores  thread (j, group hg): s_j of heads hg, hg + NT/256, ...: sequential fma over d,
//           then * scale (K row and query read from LDS piece by piece)
//   chunk   m = max_j s_j (wave max, then across the waves of a head group through LDS),
//           e_j = EXP(s_j - m) by the thread that holds s_j
//   values  thread (h, d): a[d] = sequential fma over j of e_j v_jd; l = sequential sum of
//           e_j in position order by a thread of its own (or by the d = 0 thread when every
//           thread has a value chain)
template <int HD, int GP, int NT>  // GP: query heads per KV head, 1..8
__global__ __launch_bounds__(NT) void attn_canon_kernel(AttnArgs a) {
    constexpr int U4 = HD / 8;                  // 16-byte pieces per K/V row
    constexpr int NLD = ATT_MAXC * U4 / NT;     // K (and V) pieces per thread
    constexpr int HP = HD / 2;                  // d pairs (words per V row)
    constexpr int NPG = ATT_MAXC / 16;          // pages per chunk
    constexpr int HGN = NT / ATT_MAXC;          // head groups of the score phase
    constexpr int HG = (GP + HGN - 1) / HGN;    // heads per score thread
    constexpr int PPK = NT / (16 * U4);         // pages per load iteration
    constexpr bool LS_SPARE = GP * HD + GP <= NT;  // l chains on threads of their own
    constexpr int UB = 16;                      // positions per batch of LDS reads (values)
    static_assert(NLD * NT == ATT_MAXC * U4, "pieces must divide evenly");
    static_assert(GP * HD <= NT, "one value chain per thread");
    static_assert(HGN >= 1 && PPK >= 1, "block shape");

    __shared__ __attribute__((aligned(16))) uint32_t vs[ATT_MAXC * HP];
    __shared__ __attribute__((aligned(16))) float qs[GP * HD];
    __shared__ __attribute__((aligned(16))) float ps[GP * ATT_MAXC];
    __shared__ float wmx[GP][4];
    __shared__ float red[GP];
    __shared__ __attribute__((aligned(16))) uint16_t kown[HD];

    // chunk-major block order (item fastest, chunk slowest): every item's full leading chunks
    // are dispatched before the short last ones, so a launch of more blocks than CUs runs its
    // long blocks in the first wave of blocks
    const int i = blockIdx.x;
    if (i >= items_n(a.it)) return;
    const int kh = blockIdx.y, c = blockIdx.z;
    const ModelDims& m = a.m;
    const int j0 = c * ATT_MAXC;
    // position and page indices of the chunk (uniform, read through the scalar cache); entries
    // past the current position's page are clamped to it (always mapped).  From the item table
    // when there is one (one round trip), else from the item's row, position and page table.
    int p, pgs[NPG];
    if (a.itab) {
        const int32_t* tb = a.itab + (size_t)i * (1 + m.max_pages_per_row);
        p = tb[0];
#pragma unroll
        for (int k = 0; k < NPG; ++k) pgs[k] = tb[1 + min(j0 / 16 + k, m.max_pages_per_row - 1)];
    } else {
        const int r = items_row(a.it, i);
        p = items_pos(a.it, i);
        const int32_t* ptab = a.it.page_table + (size_t)r * m.max_pages_per_row;
#pragma unroll
        for (int k = 0; k < NPG; ++k) pgs[k] = ptab[min(j0 / 16 + k, p >> 4)];
    }
    if (j0 > p) return;
    const int nj = min(ATT_MAXC, p + 1 - j0);
    constexpr int G = GP;
    const int Nk = m.Hkv * HD;
    const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
    const size_t kv_stride = (size_t)m.Hkv * m.page_size * HD;  // K -> V of the same page
    // the group's queries: one 16-byte piece per thread for the first G * HD / 8 threads
    // (with qkv: the piece's RoPE partner piece and the cos/sin of its 8 pairs come too)
    const bool fold = a.qkv != nullptr;
    const uint16_t* qkv_row = fold ? a.qkv + (size_t)i * (m.Hq * HD + 2 * Nk) : nullptr;
    const bool qthr = t < G * HD / 8;
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
    auto page_k = [&](int pg) -> const uint16_t* {
        return a.kv_pool + ((((size_t)a.layer * m.n_pages + pg) * 2) * m.Hkv + kh) * (size_t)m.page_size * HD;
    };
    // K and V pieces: iteration k covers positions (NT / U4) k .. + NT / U4 - 1 (PPK pages),
    // thread t piece t mod U4 of position t / U4 of those.  Every load is unconditional:
    // positions past the chunk's last live one (nj - 1) re-read that position (a cache hit;
    // those values are never used).  The verifier's own column stands in for the cache's
    // tentative column p (the fold path's rotated own K row is taken from kown below).
    using u32x4 = uint32_t __attribute__((ext_vector_type(4)));
    const int sub = (t / U4) >> 4;
    u32x4 kq[NLD], vr[NLD];
    const uint16_t* vps[NLD];
#pragma unroll
    for (int k = 0; k < NLD; ++k) {
        const int e = t + NT * k;
        const int jj = min(e / U4, nj - 1), pc = e % U4;
        int pg = pgs[PPK * k];
#pragma unroll
        for (int q2 = 1; q2 < PPK; ++q2) pg = sub == q2 ? pgs[PPK * k + q2] : pg;
        const uint16_t* kc = page_k(pg) + (size_t)(jj & 15) * HD + pc * 8;
        const bool at_p = j0 + jj == p;
        kq[k] = *reinterpret_cast<const u32x4*>((own && at_p) ? own + pc * 8 : kc);
        vps[k] = (own && at_p)    ? own + Nk + pc * 8
                 : (fold && at_p) ? qkv_row + m.Hq * HD + Nk + (size_t)kh * HD + pc * 8
                                  : kc + kv_stride;
    }
#pragma unroll
    for (int k = 0; k < NLD; ++k) vr[k] = *reinterpret_cast<const u32x4*>(vps[k]);
    if (qthr) {
        float4* qd = reinterpret_cast<float4*>(qs + 8 * t);
        if (!fold) {
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
                const float cs_ = cc[2 * e], sn = cc[2 * e + 1];
                const float ac = lo * cs_, bs = hi * sn, bc = hi * cs_, as = lo * sn;
                qf[e] = bf2f(f2bf(qlow ? ac - bs : bc + as));
            }
            qd[0] = make_float4(qf[0], qf[1], qf[2], qf[3]);
            qd[1] = make_float4(qf[4], qf[5], qf[6], qf[7]);
        }
    }
    if (own_here && wave == 0) {
        const uint16_t* ks = qkv_row + m.Hq * HD + (size_t)kh * HD;
        const uint16_t* vsrc = ks + Nk;
        uint16_t* ow = a.own_col ? const_cast<uint16_t*>(a.own_col) + ((size_t)i * m.L + a.layer) * 2 * Nk +
                                       (size_t)kh * HD
                                 : nullptr;
        for (int ii = lane; ii < HD / 2; ii += 64) {
            const float lo = bf2f(ks[ii]), hi = bf2f(ks[ii + HD / 2]);
            const float cs_ = a.cs[(size_t)p * HD + 2 * ii], sn = a.cs[(size_t)p * HD + 2 * ii + 1];
            const float ac = lo * cs_, bs = hi * sn, bc = hi * cs_, as = lo * sn;
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
    // K into LDS, swizzled (the V requests stay in flight: loads complete in order)
#pragma unroll
    for (int k = 0; k < NLD; ++k) {
        const int e = t + NT * k;
        const int jj = e / U4, pc = e % U4;
        *reinterpret_cast<u32x4*>(vs + (jj * U4 + (pc ^ (jj % U4))) * 4) = kq[k];
    }
    // the queries and K rows staged by other threads are needed from here on
    __syncthreads();

    // ---- scores: position j, heads hg + HGN u (the fold path's thread of position p takes
    // the rotated own K row from kown), computed while the V requests are still in flight
    const float scale = attn_scale(HD);
    const int j = t % ATT_MAXC, hg = t / ATT_MAXC;
    float sc[HG];
#pragma unroll
    for (int u = 0; u < HG; ++u) sc[u] = 0.0f;
    const bool live = j < nj;
    if (live) {
        const bool from_own = own_here && j == nj - 1;
        // (unrolled by 4 pieces: fully unrolled, the compiler hoists every K and query read of
        // two heads and spills)
#pragma unroll 4
        for (int k = 0; k < U4; ++k) {
            const uint4 kp = from_own ? reinterpret_cast<const uint4*>(kown)[k]
                                      : *reinterpret_cast<const uint4*>(vs + (j * U4 + (k ^ (j % U4))) * 4);
            const float kf[8] = {bf_lo(kp.x), bf_hi(kp.x), bf_lo(kp.y), bf_hi(kp.y),
                                 bf_lo(kp.z), bf_hi(kp.z), bf_lo(kp.w), bf_hi(kp.w)};
#pragma unroll
            for (int u = 0; u < HG; ++u) {
                const int h = hg + HGN * u;
                if (h < G) {
                    const float4 q0 = *reinterpret_cast<const float4*>(qs + h * HD + 8 * k);
                    const float4 q1 = *reinterpret_cast<const float4*>(qs + h * HD + 8 * k + 4);
                    float s = sc[u];
                    s = __builtin_fmaf(q0.x, kf[0], s);
                    s = __builtin_fmaf(q0.y, kf[1], s);
                    s = __builtin_fmaf(q0.z, kf[2], s);
                    s = __builtin_fmaf(q0.w, kf[3], s);
                    s = __builtin_fmaf(q1.x, kf[4], s);
                    s = __builtin_fmaf(q1.y, kf[5], s);
                    s = __builtin_fmaf(q1.z, kf[6], s);
                    s = __builtin_fmaf(q1.w, kf[7], s);
                    sc[u] = s;
                }
            }
        }
#pragma unroll
        for (int u = 0; u < HG; ++u) sc[u] = sc[u] * scale;
    }
    // chunk max: each wave's max of its positions, per head (waves of a head group cover
    // 64 positions each)
#pragma unroll
    for (int u = 0; u < HG; ++u) {
        const int h = hg + HGN * u;
        const float mx = wave_max(live ? sc[u] : -__builtin_inff());
        if (h < G && lane == 0) wmx[h][(j >> 6)] = mx;
    }
    // every K read is done and every wave max is in before V takes the LDS space
    __syncthreads();
#pragma unroll
    for (int k = 0; k < NLD; ++k) {
        const int e = t + NT * k;
        *reinterpret_cast<u32x4*>(vs + (e / U4) * HP + (e % U4) * 4) = vr[k];
    }
#pragma unroll
    for (int u = 0; u < HG; ++u) {
        const int h = hg + HGN * u;
        if (h < G) {
            const float mx = fmaxf(fmaxf(wmx[h][0], wmx[h][1]), fmaxf(wmx[h][2], wmx[h][3]));
            if (live) ps[h * ATT_MAXC + j] = canon_exp(sc[u] - mx);
            if (j == 0) red[h] = mx;
        }
    }
    __syncthreads();

    // ---- the weighted values: thread (h, d); l on a thread of its own (or the d = 0 thread)
    const int vh = t / HD, vd = t % HD;
    const bool vthr = t < G * HD;
    const int lh = t - G * HD;  // the head whose l this spare thread forms
    const bool lthr = LS_SPARE ? (lh >= 0 && lh < G) : (vthr && vd == 0);
    const int eh = vthr ? vh : (LS_SPARE && lthr ? lh : 0);
    float acc = 0.0f, lsum = 0.0f;
    if (vthr || lthr) {
        const int nb = nj / UB * UB;  // positions handled in whole batches
        const float* eh_row = ps + eh * ATT_MAXC;
        const int vw_i = vd >> 1;
        // this thread's bf16 of a V word moved to the top half with zeros below (one v_perm)
        const uint32_t vsel = (vd & 1) ? 0x03020c0cu : 0x01000c0cu;
        for (int jb = 0; jb < nb; jb += UB) {
            float e[UB];
#pragma unroll
            for (int q4 = 0; q4 < UB / 4; ++q4) {
                const float4 t4 = *reinterpret_cast<const float4*>(eh_row + jb + 4 * q4);
                e[4 * q4] = t4.x; e[4 * q4 + 1] = t4.y; e[4 * q4 + 2] = t4.z; e[4 * q4 + 3] = t4.w;
            }
            if (vthr) {
                uint32_t vw[UB];
#pragma unroll
                for (int b = 0; b < UB; ++b) vw[b] = vs[(jb + b) * HP + vw_i];
#pragma unroll
                for (int b = 0; b < UB; ++b)
                    acc = __builtin_fmaf(e[b], __uint_as_float(__builtin_amdgcn_perm(vw[b], vw[b], vsel)), acc);
            }
            if (lthr) {
#pragma unroll
                for (int b = 0; b < UB; ++b) lsum = lsum + e[b];
            }
        }
        for (int jj = nb; jj < nj; ++jj) {
            const float e = eh_row[jj];
            if (vthr) {
                const uint32_t vw = vs[jj * HP + vw_i];
                acc = __builtin_fmaf(e, __uint_as_float(__builtin_amdgcn_perm(vw, vw, vsel)), acc);
            }
            if (lthr) lsum = lsum + e;
        }
    }
    constexpr int stride = HD + 2;
    if (vthr) {
        float* dst = a.part + (((size_t)i * m.Hq + kh * G + vh) * a.max_chunks + c) * stride;
        dst[2 + vd] = acc;
        if (!LS_SPARE && lthr) {
            dst[0] = red[vh];
            dst[1] = lsum;
        }
    }
    if (LS_SPARE && lthr) {
        float* dst = a.part + (((size_t)i * m.Hq + kh * G + lh) * a.max_chunks + c) * stride;
        dst[0] = red[lh];
        dst[1] = lsum;
    }
}

__global__ void attn_combine_kernel(AttnArgs a) {
    const int i = blockIdx.y;
    if (i >= items_n(a.it)) return;
    const int h = blockIdx.x, d = threadIdx.x;
    const int hd = a.m.hd;
    if (d >= hd) return;
    const int p = a.itab ? a.itab[(size_t)i * (1 + a.m.max_pages_per_row)] : items_pos(a.it, i);
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

// 1024 threads per block where the grid gives each CU about one block (a block's latency is
// the kernel's: measured at the Llama-8B shape, 13 rows: 25k vs 31k cycles per block with 512);
// 512 where each CU has several blocks to run and G * HD <= 512, so two blocks share a CU and
// one block's loads overlap the other's chains
template <int HD, int G>
static void launch_canon_gt(const AttnArgs& a, dim3 g1, bool many, hipStream_t s) {
    if constexpr (G * HD <= 512) {
        if (many) {
            hipLaunchKernelGGL((attn_canon_kernel<HD, G, 512>), g1, dim3(512), 0, s, a);
            return;
        }
    }
    hipLaunchKernelGGL((attn_canon_kernel<HD, G, 1024>), g1, dim3(1024), 0, s, a);
}
template <int HD>
static void launch_canon_g(const AttnArgs& a, int G, dim3 g1, bool many, hipStream_t s) {
    switch (G) {
        case 1: launch_canon_gt<HD, 1>(a, g1, many, s); break;
        case 2: launch_canon_gt<HD, 2>(a, g1, many, s); break;
        case 3: launch_canon_gt<HD, 3>(a, g1, many, s); break;
        case 4: launch_canon_gt<HD, 4>(a, g1, many, s); break;
        case 5: launch_canon_gt<HD, 5>(a, g1, many, s); break;
        case 6: launch_canon_gt<HD, 6>(a, g1, many, s); break;
        case 7: launch_canon_gt<HD, 7>(a, g1, many, s); break;
        default: launch_canon_gt<HD, 8>(a, g1, many, s); break;
    }
}

// item i: tab[i][0] = its position p, tab[i][1 + k] = its row's page of slot min(k, p / 16)
__global__ __launch_bounds__(256) void item_table_kernel(Items it, int mpr, int32_t* __restrict__ tab) {
    const int i = blockIdx.x;
    if (i >= items_n(it)) return;
    const int r = items_row(it, i), p = items_pos(it, i);
    const int32_t* ptab = it.page_table + (size_t)r * mpr;
    int32_t* tb = tab + (size_t)i * (1 + mpr);
    if (threadIdx.x == 0) tb[0] = p;
    for (int k = threadIdx.x; k < mpr; k += 256) tb[1 + k] = ptab[min(k, p >> 4)];
}

hipError_t launch_item_table(const Items& it, const ModelDims& m, int32_t* itab, hipStream_t s) {
    if (it.n_host <= 0) return hipSuccess;
    hipLaunchKernelGGL(item_table_kernel, dim3(it.n_host), dim3(256), 0, s, it, m.max_pages_per_row, itab);
    return hipGetLastError();
}

hipError_t launch_attention(const AttnArgs& a, int canon, hipStream_t s) {
    const int n = a.it.n_host;
    if (n <= 0) return hipSuccess;
    if (!canon || a.chunk != ATT_MAXC) return hipErrorInvalidValue;  // the fast path has its own kernel
    dim3 g1(n, a.m.Hkv, a.max_chunks), g2(a.m.Hq, n);
    const int G = a.m.Hq / a.m.Hkv;
    if (G < 1 || G > ATT_MAXG) return hipErrorInvalidValue;
    // blocks of the launch (an upper bound: chunks past a row's position exit at once)
    const long blocks = (long)n * a.m.Hkv * a.max_chunks;
    const bool many = blocks >= 4L * (a.n_cu > 0 ? a.n_cu : 256);
    if (a.m.hd == 128)
        launch_canon_g<128>(a, G, g1, many, s);
    else
        launch_canon_g<64>(a, G, g1, many, s);
    hipLaunchKernelGGL(attn_combine_kernel, g2, dim3(a.m.hd), 0, s, a);
    return hipGetLastError();
}

}  // namespace mg
