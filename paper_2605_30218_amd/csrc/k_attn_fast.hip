// k_attn_fast.hip -- the fast path's decode attention, fused with the split-K sum of
// the QKV projection, the bias, RoPE and the tentative K/V append.
//
// One block of 4 waves per (row, KV head, position split).  With one split (enough rows to
// fill the device) the block merges everything itself; with several (split-KV, for long
// contexts at small batch) split k takes an equal share of the pages of positions 0..p-1,
// split 0 also takes position p, and a second launch merges the splits' (m, l, O) in split
// order.
// Prologue: sums the QKV split partials of the block's features (the G query heads of
// the group, then k, then v) in split order, adds the bias and rounds to bf16 (the
// projection's rounding point); rotates q and k (rotate-half RoPE from the fp32
// cos/sin table, products and sums rounded separately, then bf16); appends K' and V
// to the paged cache at the row's position p (the tentative column) -- or, for the
// matrix-core verifier, to the row's own column buffer, leaving the cache untouched;
// keeps q' (bf16,
// the MFMA A operand) and k'_p, v_p in LDS, and copies the row's page indices for
// positions < p into LDS.
// Main loop: wave w takes the pages w, w + 4, ... of positions 0..p-1 (16 positions
// per step).  Scores on MFMA: S[h][pos] = Q[h][:] . K[pos][:] with the
// query heads as the rows of a 16-row A operand (rows >= G are zero) and 16
// positions of a page as the B operand read straight from the page (lane (j, q) reads
// 16 bytes of position j).  Softmax online in the exp2 domain; O += P V on the vector
// ALU with the wave split as hd/8 d-groups x 512/hd positions per 16-byte load.  The
// K and V of the wave's next step are requested before the current step's
// arithmetic (register ping-pong); values of positions >= p are zeroed when used.
// Epilogue: each wave's (m, l, O) goes to LDS; position p contributes its own partial
// (m = score of q' . k'_p, l = 1, O = v_p) in split 0; the partials are merged and
// out = bf16(O / L), or the split's merged partial is stored for the split merge.  Every
// split recomputes the prologue (q' is needed by all); only split 0 writes the column.
// The summation order depends on the context length and the split of positions over
// waves: this path is not the verifier's order.
#include "mg_device.h"
#include "mg_kernels.h"

namespace mg {

typedef __bf16 bf16x8_ft __attribute__((ext_vector_type(8)));
typedef float f32x4_ft __attribute__((ext_vector_type(4)));

#ifndef MG_FA_WAVES
#define MG_FA_WAVES 4
#endif
#ifndef MG_FA_MIN_WAVES
#define MG_FA_MIN_WAVES 2  // waves per SIMD the register budget must allow (up to 4 query heads per KV head: two blocks per CU without spilling; 8 would spill)
#endif
constexpr int FA_WAVES = MG_FA_WAVES;
constexpr int FA_THREADS = 64 * FA_WAVES;
constexpr int FA_PGCAP = 1024;  // page indices held in LDS (positions < 16384); more are read from memory

__device__ __forceinline__ float fa_scale(int hd) { return hd == 128 ? 0x1.6a09e6p-4f : 0x1.0p-3f; }

template <int HD, int GP>
__global__ __launch_bounds__(FA_THREADS) __attribute__((amdgpu_waves_per_eu(MG_FA_MIN_WAVES))) void attn_fast_fused_kernel(FastAttnArgs a) {
    constexpr int DG = HD / 8;    // 16-byte d-groups per row
    constexpr int PPI = 64 / DG;  // positions per V load instruction
    constexpr int VL = 16 / PPI;  // V loads per lane per page step
    constexpr int KST = HD / 32;  // MFMA k-steps over d
    constexpr int H2 = HD / 2;
    const ModelDims& m = a.m;
    const int Gall = m.Hq / m.Hkv, Nq = m.Hq * HD, Nk = m.Hkv * HD, N = Nq + 2 * Nk;
    // block -> (row, KV head, head group of up to GP query heads).  With several head groups
    // the blocks of one (row, KV head) are 8 block ids apart: blocks are dealt to the 8 XCDs
    // round-robin, so they run on the same XCD at about the same time and all but the first
    // read the pages from that XCD's L2
    const int HG = (Gall + GP - 1) / GP;
    int u = blockIdx.x, hg = 0;
    if (HG > 1) {
        const int w = blockIdx.x % (8 * HG);
        u = blockIdx.x / (8 * HG) * 8 + w % 8;
        hg = w / 8;
    }
    if (u >= a.B * m.Hkv) return;
    const int kh = u % m.Hkv, r = u / m.Hkv, split = blockIdx.z;
    const int hoff = hg * GP, G = min(GP, Gall - hoff);  // this block's query heads: hoff .. hoff + G - 1 of the group
    const int t = threadIdx.x, wave = t >> 6, lane = t & 63;
    const int jl = lane & 15, qg = lane >> 4;
    const int dg = lane % DG, po = lane / DG;
    const float sl2 = fa_scale(HD) * 1.4426950408889634f;  // scores in log2 units

    __shared__ float y[(GP + 2) * HD];
    __shared__ __attribute__((aligned(16))) uint16_t qb[GP * HD];
    __shared__ float kps[HD], vps[HD];
    __shared__ int pgs[FA_PGCAP];
    __shared__ float sp[GP];
    __shared__ float wm[FA_WAVES][GP], wl[FA_WAVES][GP];
    __shared__ float wo[FA_WAVES][GP * HD];

    const int p = a.positions[r];
    const int32_t* ptab = a.page_table + (size_t)r * m.max_pages_per_row;
    const int npg = (p + 15) / 16;  // pages holding positions 0..p-1
    // this split's pages [pg0, pg1): a fixed share of the capacity, so a block's work is
    // bounded whatever the row's length; a split past the row's pages has nothing to do (the
    // merge reads only the row's live splits)
    const int pg0 = split * a.split_pages, pg1 = min(npg, pg0 + a.split_pages);
    const bool first = split == 0;
    const bool writer = first && hg == 0;  // the block that appends the tentative column
    if (!first && pg0 >= npg) return;
    const bool pg_lds = pg1 - pg0 <= FA_PGCAP;

    // ---- prologue: split sum + bias + bf16 of this block's q, k, v features
    {
        const float* pp = a.part + (size_t)r * N;
        const size_t sstride = (size_t)a.B * N;
        const int nf = (G + 2) * HD;
        for (int q4 = t; q4 < nf / 4; q4 += FA_THREADS) {
            const int f = 4 * q4;
            int n, nb;
            const uint16_t* b;
            if (f < G * HD) { n = (kh * Gall + hoff) * HD + f; b = a.bq; nb = n; }
            else if (f < (G + 1) * HD) { nb = kh * HD + f - G * HD; n = Nq + nb; b = a.bk; }
            else { nb = kh * HD + f - (G + 1) * HD; n = Nq + Nk + nb; b = a.bv; }
            // splits summed in split order; loads issued in batches of 8
            float4 v = *reinterpret_cast<const float4*>(pp + n);
            int sp2 = 1;
            for (; sp2 + 8 <= a.S; sp2 += 8) {
                float4 u[8];
#pragma unroll
                for (int k = 0; k < 8; ++k) u[k] = *reinterpret_cast<const float4*>(pp + (size_t)(sp2 + k) * sstride + n);
#pragma unroll
                for (int k = 0; k < 8; ++k) { v.x += u[k].x; v.y += u[k].y; v.z += u[k].z; v.w += u[k].w; }
            }
            for (; sp2 < a.S; ++sp2) {
                const float4 u = *reinterpret_cast<const float4*>(pp + (size_t)sp2 * sstride + n);
                v.x += u.x; v.y += u.y; v.z += u.z; v.w += u.w;
            }
            if (b) { v.x += bf2f(b[nb]); v.y += bf2f(b[nb + 1]); v.z += bf2f(b[nb + 2]); v.w += bf2f(b[nb + 3]); }
            y[f] = bf2f(f2bf(v.x));
            y[f + 1] = bf2f(f2bf(v.y));
            y[f + 2] = bf2f(f2bf(v.z));
            y[f + 3] = bf2f(f2bf(v.w));
        }
        if (pg_lds)
            for (int j = t; j < pg1 - pg0; j += FA_THREADS) pgs[j] = ptab[pg0 + j];
        for (int e = G * HD + t; e < GP * HD; e += FA_THREADS) qb[e] = 0;
    }
    __syncthreads();
    // ---- RoPE on q and k, tentative K/V append at p, q' / k'_p / v_p into LDS
    {
        const float* csp = a.cs + (size_t)p * HD;  // [pos][i][cos, sin]
        // the tentative column in the cache, or (own_out) the row's own column buffer
        uint16_t *kdst, *vdst;
        if (a.own_out) {
            kdst = a.own_out + ((size_t)r * m.L + a.layer) * 2 * Nk + (size_t)kh * HD;
            vdst = kdst + Nk;
        } else {
            kdst = a.kv_pool + ((((size_t)a.layer * m.n_pages + ptab[p / 16]) * 2) * m.Hkv + kh) * (size_t)16 * HD +
                   (size_t)(p % 16) * HD;
            vdst = kdst + (size_t)m.Hkv * 16 * HD;
        }
        for (int t2 = t; t2 < (G + 1) * H2; t2 += FA_THREADS) {
            const int head = t2 / H2, ii = t2 % H2;  // head == G: the k head
            const float* s = y + head * HD;
            const float x1 = s[ii], x2 = s[ii + H2];
            const float c = csp[2 * ii], sn = csp[2 * ii + 1];
            const float ac = x1 * c, bs = x2 * sn, bc = x2 * c, as = x1 * sn;
            const uint32_t o1 = f2bf(ac - bs), o2 = f2bf(bc + as);
            if (head < G) {
                qb[head * HD + ii] = (uint16_t)o1;
                qb[head * HD + ii + H2] = (uint16_t)o2;
            } else {
                if (writer) {
                    kdst[ii] = (uint16_t)o1;
                    kdst[ii + H2] = (uint16_t)o2;
                }
                kps[ii] = bf2f(o1);
                kps[ii + H2] = bf2f(o2);
            }
        }
        for (int d = t; d < HD; d += FA_THREADS) {
            const float v = y[(G + 1) * HD + d];
            if (writer) vdst[d] = (uint16_t)f2bf(v);
            vps[d] = v;
        }
    }
    __syncthreads();

    // ---- position p's own score (log2 units): wave w takes heads w, w + 4
#pragma unroll
    for (int hh = 0; hh < (GP + FA_WAVES - 1) / FA_WAVES; ++hh) {
        const int h = wave + FA_WAVES * hh;
        if (h < G) {
            float s = 0.0f;
            for (int d = lane; d < HD; d += 64) s += bf2f(qb[h * HD + d]) * kps[d];
            s = wave_sum_fast(s);
            if (lane == 0) sp[h] = s * sl2;
        }
    }

    // ---- main loop over positions 0..p-1
    uint4 qa[KST];
#pragma unroll
    for (int st = 0; st < KST; ++st)
        qa[st] = jl < G ? *reinterpret_cast<const uint4*>(qb + jl * HD + st * 32 + qg * 8) : make_uint4(0, 0, 0, 0);
    float mrow[4], lrow[4];  // per head h = 4 qg + v (lanes of group qg)
#pragma unroll
    for (int v = 0; v < 4; ++v) { mrow[v] = -__builtin_inff(); lrow[v] = 0.0f; }
    float o[GP][8];
#pragma unroll
    for (int h = 0; h < GP; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) o[h][e] = 0.0f;

    const size_t kv_stride = (size_t)m.Hkv * 16 * HD;  // K -> V of the same page
    // loads of page step s (positions 16 s .. 16 s + 15): K rows straight into B-operand
    // registers, V rows for the P V product; positions >= p read the step's last valid
    // row (never used: their scores are masked and their V zeroed)
    auto fetch = [&](int s, uint4 (&kb)[KST], uint4 (&vb)[VL]) {
        int page;
        if (pg_lds)
            page = pgs[s - pg0];
        else
            page = ptab[s];
        const uint16_t* kp = a.kv_pool + ((((size_t)a.layer * m.n_pages + page) * 2) * m.Hkv + kh) * (size_t)16 * HD;
#pragma unroll
        for (int st = 0; st < KST; ++st) kb[st] = *reinterpret_cast<const uint4*>(kp + jl * HD + st * 32 + qg * 8);
#pragma unroll
        for (int tt = 0; tt < VL; ++tt) {
            const int pl = min(PPI * tt + po, p - 1 - 16 * s);
            vb[tt] = *reinterpret_cast<const uint4*>(kp + kv_stride + pl * HD + dg * 8);
        }
    };
    auto compute = [&](int s, const uint4 (&kb)[KST], const uint4 (&vb)[VL]) {
        const int base = 16 * s;
        f32x4_ft sc = f32x4_ft{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int st = 0; st < KST; ++st)
            sc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_ft, qa[st]),
                                                         __builtin_bit_cast(bf16x8_ft, kb[st]), sc, 0, 0, 0);
        float alpha[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const float x = (base + jl < p) ? sc[v] * sl2 : -__builtin_inff();
            float mx = x;
#pragma unroll
            for (int o2 = 1; o2 < 16; o2 <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o2, 64));
            const float mn = fmaxf(mrow[v], mx);
            alpha[v] = exp2f(mrow[v] - mn);
            mrow[v] = mn;
            const float pv = exp2f(x - mn);
            sc[v] = pv;
            lrow[v] = lrow[v] * alpha[v] + pv;
        }
        // rescale O and accumulate P V; head h's P of position pl sits in lane pl + 16 (h / 4)
#pragma unroll
        for (int h = 0; h < GP; ++h) {
            const float al = __shfl(alpha[h & 3], 16 * (h >> 2), 64);
#pragma unroll
            for (int e = 0; e < 8; ++e) o[h][e] *= al;
        }
#pragma unroll
        for (int tt = 0; tt < VL; ++tt) {
            const int pl = PPI * tt + po;
            const uint4 vr = base + pl < p ? vb[tt] : make_uint4(0, 0, 0, 0);
            const float v8[8] = {bf_lo(vr.x), bf_hi(vr.x), bf_lo(vr.y), bf_hi(vr.y),
                                 bf_lo(vr.z), bf_hi(vr.z), bf_lo(vr.w), bf_hi(vr.w)};
#pragma unroll
            for (int h = 0; h < GP; ++h) {
                const float ph = __shfl(sc[h & 3], pl + 16 * (h >> 2), 64);
#pragma unroll
                for (int e = 0; e < 8; ++e) o[h][e] = __builtin_fmaf(ph, v8[e], o[h][e]);
            }
        }
    };
    const int nst = pg1;  // page steps of this split: pg0 + wave, pg0 + wave + 4, ... < pg1
    int s = pg0 + wave;
    if (s < nst) {
        uint4 kA[KST], vA[VL], kB[KST], vB[VL];
        fetch(s, kA, vA);
        while (true) {
            if (s + FA_WAVES >= nst) { compute(s, kA, vA); break; }
            fetch(s + FA_WAVES, kB, vB);
            __builtin_amdgcn_sched_barrier(0);
            compute(s, kA, vA);
            s += FA_WAVES;
            if (s + FA_WAVES >= nst) { compute(s, kB, vB); break; }
            fetch(s + FA_WAVES, kA, vA);
            __builtin_amdgcn_sched_barrier(0);
            compute(s, kB, vB);
            s += FA_WAVES;
        }
    }

    // ---- wave partials: O reduced over the position groups, l over the 16 position lanes
#pragma unroll
    for (int h = 0; h < GP; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e)
            for (int off = DG; off < 64; off <<= 1) o[h][e] += __shfl_xor(o[h][e], off, 64);
#pragma unroll
    for (int v = 0; v < 4; ++v)
        for (int off = 1; off < 16; off <<= 1) lrow[v] += __shfl_xor(lrow[v], off, 64);
#pragma unroll
    for (int h = 0; h < GP; ++h) {
        const float mh = __shfl(mrow[h & 3], 16 * (h >> 2), 64);
        const float lh = __shfl(lrow[h & 3], 16 * (h >> 2), 64);
        if (lane == 0) {
            wm[wave][h] = mh;
            wl[wave][h] = lh;
        }
        if (po == 0) {
#pragma unroll
            for (int e = 0; e < 8; ++e) wo[wave][h * HD + dg * 8 + e] = o[h][e];
        }
    }
    __syncthreads();

    // ---- merge the wave partials and (split 0) position p
    for (int oi = t; oi < G * HD; oi += FA_THREADS) {
        const int h = oi / HD, d = oi % HD;
        float M = first ? sp[h] : -__builtin_inff();
#pragma unroll
        for (int w = 0; w < FA_WAVES; ++w) M = fmaxf(M, wm[w][h]);
        float L = 0.0f, O = 0.0f;
        if (first) {
            const float ws = exp2f(sp[h] - M);
            L = ws;
            O = ws * vps[d];
        }
        if (M != -__builtin_inff()) {  // (a split with no position keeps L = O = 0)
#pragma unroll
            for (int w = 0; w < FA_WAVES; ++w) {
                const float ww = exp2f(wm[w][h] - M);
                L += ww * wl[w][h];
                O += ww * wo[w][h * HD + d];
            }
        }
        if (a.nsplit == 1) {
            a.out[(size_t)r * Nq + (size_t)(kh * Gall + hoff + h) * HD + d] = (uint16_t)f2bf(O / L);
        } else {
            float* dst = a.split_part + (((size_t)r * m.Hq + kh * Gall + hoff + h) * a.nsplit + split) * (HD + 2);
            if (d == 0) {
                dst[0] = M;
                dst[1] = L;
            }
            dst[2 + d] = O;
        }
    }
}

// The split merge of split-KV: for each (row, query head), the splits' (m, l, O) combined in
// split order (exp2 domain, as the partials), out = bf16(O / L).
__global__ void attn_fast_split_merge_kernel(FastAttnArgs a) {
    const int h = blockIdx.x, r = blockIdx.y, d = threadIdx.x;
    const int hd = a.m.hd, ns = a.nsplit;
    if (d >= hd) return;
    // the row's live splits: split 0 (position p) and those holding pages of positions < p
    const int npg = (a.positions[r] + 15) / 16;
    const int live = max(1, min(ns, (npg + a.split_pages - 1) / a.split_pages));
    const float* base = a.split_part + ((size_t)r * a.m.Hq + h) * ns * (hd + 2);
    float M = -__builtin_inff();
    for (int k = 0; k < live; ++k) M = fmaxf(M, base[(size_t)k * (hd + 2)]);
    float L = 0.0f, O = 0.0f;
    for (int k = 0; k < live; ++k) {
        const float* pk = base + (size_t)k * (hd + 2);
        if (pk[0] == -__builtin_inff()) continue;  // a split with no position
        const float w = exp2f(pk[0] - M);
        L += w * pk[1];
        O += w * pk[2 + d];
    }
    a.out[(size_t)r * a.m.Hq * hd + (size_t)h * hd + d] = (uint16_t)f2bf(O / L);
}

template <int HD>
static void launch_hd(const FastAttnArgs& a, int gp, dim3 grid, hipStream_t s) {
    switch (gp) {
        case 1: hipLaunchKernelGGL((attn_fast_fused_kernel<HD, 1>), grid, dim3(FA_THREADS), 0, s, a); break;
        case 2: hipLaunchKernelGGL((attn_fast_fused_kernel<HD, 2>), grid, dim3(FA_THREADS), 0, s, a); break;
        default: hipLaunchKernelGGL((attn_fast_fused_kernel<HD, 4>), grid, dim3(FA_THREADS), 0, s, a); break;
    }
}

hipError_t launch_fast_attention(const FastAttnArgs& a, hipStream_t s) {
    if (a.B <= 0) return hipSuccess;
    const int G = a.m.Hq / a.m.Hkv;
    if (G < 1 || G > 8 || a.m.page_size != 16 || (a.m.hd != 64 && a.m.hd != 128)) return hipErrorInvalidValue;
    if (a.nsplit < 1 || a.split_pages < 1 || (long)a.nsplit * a.split_pages < a.m.max_pages_per_row ||
        (a.nsplit > 1 && !a.split_part))
        return hipErrorInvalidValue;
    const int gp = G <= 1 ? 1 : G <= 2 ? 2 : 4;
    const int HG = fast_attn_head_groups(a.m.Hq, a.m.Hkv), units = a.B * a.m.Hkv;
    const dim3 grid(HG == 1 ? units : (units + 7) / 8 * 8 * HG, 1, a.nsplit);
    if (a.m.hd == 128)
        launch_hd<128>(a, gp, grid, s);
    else
        launch_hd<64>(a, gp, grid, s);
    if (a.nsplit > 1) hipLaunchKernelGGL(attn_fast_split_merge_kernel, dim3(a.m.Hq, a.B), dim3(a.m.hd), 0, s, a);
    return hipGetLastError();
}

int fast_attn_head_groups(int n_q_heads, int n_kv_heads) {
    const int G = n_q_heads / n_kv_heads;
    return G <= 4 ? 1 : (G + 3) / 4;
}

int fast_attn_splits(int rows, int n_kv_heads, int max_pages_per_row, int n_cu, int cap) {
    const int blocks = rows * n_kv_heads;
    if (blocks <= 0 || blocks >= 2 * n_cu) return 1;  // enough blocks: one per (row, KV head)
    int ns = (2 * n_cu + blocks - 1) / blocks;
    ns = ns < max_pages_per_row / 16 ? ns : max_pages_per_row / 16;
    // small batches: also shares of at most 64 pages, so that a long row does not leave
    // its one block working after the short rows' blocks are done
    const int by_length = (max_pages_per_row + 63) / 64;
    ns = ns > by_length ? ns : by_length;
    ns = ns < cap ? ns : cap;
    return ns < 1 ? 1 : ns;
}

}  // namespace mg
