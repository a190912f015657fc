// k_gemv.hip -- the verifier's canonical GEMV.
//
// y[r][j] = CDOT(x[r], W[j]) for a set of rows r and output features j, where
// CDOT fixes the reduction order independently of how many rows are processed
// and where a row sits in the launch:
//   groups of 8 consecutive K elements; group g belongs to lane g mod 64; each
//   lane fma-accumulates its groups in increasing g (element order inside the
//   group) starting from +0; the 64 lane sums are combined by the xor butterfly
//   over offsets 32, 16, 8, 4, 2, 1 (all J*R butterflies of a wave are run
//   together with the same pairings, see butterfly_sum_multi).
// A wave owns J features (2, or 3 for wide outputs); a block of 8 waves owns 8J
// features and a tile of R rows (so the tile's activations, staged once per block,
// serve 8J features).  K is walked in chunks of 512 elements (one group per lane).
// While the fma work of chunk c runs, the weights of chunk c+1 (or c+1 and c+2 on the
// narrow, short-K launches) are in flight (registers: one 16-byte group per feature and
// lane, 1 KiB coalesced per feature, in a ping-pong pair or a ring of three) and the rows' activations of chunk c+1 are loaded into
// registers, then staged into the fp32 LDS tile: tiles up to 16 rows have two buffers
// and one barrier per chunk; larger tiles restage one buffer between two barriers,
// which keeps their LDS footprint at R * 2 KiB.  No split-K, no atomics: a row's
// arithmetic is the same whatever R, J, the tile or the count.
// Row tiles: when the host knows the row count (up to 24 rows) one tile of exactly
// ceil(n/4)*4 rows runs every row without a branch, which lets the compiler read later
// rows' activations from LDS while earlier rows compute (the dead rows compute on a copy
// of the last live row and are not written); other counts use 16-row tiles that skip
// dead rows by a uniform branch.  The tile never changes a row's arithmetic.
// Block order: the row tiles of one feature block get consecutive slots on the
// same XCD (blocks are dealt to the 8 XCDs round-robin), so they share its L2
// copy of the weights.
#include "mg_device.h"
#include "mg_kernels.h"

namespace mg {

constexpr int KCH = 512;  // K elements per chunk (64 lanes x 8)

#ifndef MG_GEMV_J_R8
#define MG_GEMV_J_R8 2
#endif
#ifndef MG_GEMV_J_R16
#define MG_GEMV_J_R16 2
#endif
#ifndef MG_GEMV_J_R12
#define MG_GEMV_J_R12 2  // features per wave of the exact 9..16-row tiles
#endif
// exact 9..16-row tiles give each wave 3 features when the output is wide (N >=
// MG_GEMV_BIG_N: the MLP up projection, the LM head: a third fewer LDS activation reads
// per fma, and still over a thousand blocks; measured at 12 rows: LM head 239 vs 261 us,
// gate/up 60 vs 61 us; 4 features drop to 3 waves per SIMD and are slower); exact
// 5..16-row tiles of a narrower output take 3 when that leaves the busiest CU fewer
// features than 2 (6144 features: 256 blocks of 24 instead of 384 of 16, measured at 8
// and 12 rows 12.8 vs 14.1 and 15.4 vs 18.1 us; 4096 features keep 256 blocks of 16)
#ifndef MG_GEMV_J_BIG
#define MG_GEMV_J_BIG 3
#endif
#ifndef MG_GEMV_BIG_N
#define MG_GEMV_BIG_N 16384
#endif
#ifndef MG_GEMV_EXACT_MAX
#define MG_GEMV_EXACT_MAX 24  // largest host row count served by one branch-free tile
#endif
#ifndef MG_GEMV_NW
#define MG_GEMV_NW 8  // waves per block (measured: 8 beats 4 and 16)
#endif
constexpr int GV_NW = MG_GEMV_NW, GV_THREADS = 64 * MG_GEMV_NW;

__host__ __device__ constexpr int pow2_at_least(int v) { return v <= 1 ? 1 : 2 * pow2_at_least((v + 1) / 2); }

#ifndef MG_GEMV_XB_MAXR
#define MG_GEMV_XB_MAXR 16  // row tiles up to this size get two LDS activation buffers
#endif

template <int R>
struct GemvShape {
    static constexpr int XLD = (R * 64 + GV_THREADS - 1) / GV_THREADS;  // staging loads (16 bytes) per thread per chunk
    static constexpr int XB = R <= MG_GEMV_XB_MAXR ? 2 : 1;               // LDS activation buffers
};

// activations of chunk kc for rows r0 .. r0+R-1: rows past nr read row nr-1 and k past
// K reads the last group (those values are never used: rows past nr are skipped and
// lanes past the last group do no arithmetic), so every load is unconditional.  A
// thread's row is its wave's (wave-uniform: a scalar row base), its group its lane's.
template <int R>
__device__ __forceinline__ void gemv_load_x(const GemvArgs& a, int r0, int nr, int kc, int wave, int lane,
                                            uint4 (&xr)[GemvShape<R>::XLD]) {
#pragma unroll
    for (int it = 0; it < GemvShape<R>::XLD; ++it) {
        const int rr = min(min(wave + GV_NW * it, R - 1), nr - 1);
        const int k = min(kc + lane * 8, a.K - 8);
        xr[it] = *reinterpret_cast<const uint4*>(a.X + (size_t)(r0 + rr) * a.K + k);
    }
}

template <int R>
__device__ __forceinline__ void gemv_store_x(float4 (*xs)[2][64], int wave, int lane, const uint4 (&xr)[GemvShape<R>::XLD]) {
#pragma unroll
    for (int it = 0; it < GemvShape<R>::XLD; ++it) {
        const int rr = wave + GV_NW * it;
        if (GV_THREADS * GemvShape<R>::XLD > R * 64 && rr >= R) continue;
        const uint4 v = xr[it];
        xs[rr][0][lane] = make_float4(bf_lo(v.x), bf_hi(v.x), bf_lo(v.y), bf_hi(v.y));
        xs[rr][1][lane] = make_float4(bf_lo(v.z), bf_hi(v.z), bf_lo(v.w), bf_hi(v.w));
    }
}

// weights of group g (clamped to the last group) of the J feature rows
template <int J>
__device__ __forceinline__ void gemv_load_w(const uint16_t* const (&wrow)[J], int g, int G, uint4 (&w)[J]) {
    const int gc = min(g, G - 1);
#pragma unroll
    for (int jj = 0; jj < J; ++jj) w[jj] = *reinterpret_cast<const uint4*>(wrow[jj] + (size_t)gc * 8);
}

// this lane's group of one chunk for every live row: sequential fma in element order
template <int J, int R, bool EXACT>
__device__ __forceinline__ void gemv_fma_chunk(const float4 (*xb)[2][64], int lane, int nr, const uint4 (&wv)[J],
                                               float (&acc)[J][R]) {
    float w[J][8];
#pragma unroll
    for (int jj = 0; jj < J; ++jj) {
        const uint4 v = wv[jj];
        w[jj][0] = bf_lo(v.x); w[jj][1] = bf_hi(v.x); w[jj][2] = bf_lo(v.y); w[jj][3] = bf_hi(v.y);
        w[jj][4] = bf_lo(v.z); w[jj][5] = bf_hi(v.z); w[jj][6] = bf_lo(v.w); w[jj][7] = bf_hi(v.w);
    }
    // EXACT tiles (sized by the host to the row count) run every row with no branch, so
    // the compiler reads later rows' activations from LDS while earlier rows compute;
    // otherwise rows past nr are skipped by a uniform branch.  The loop stays fully
    // unrolled so every accumulator index is a compile-time constant (no scratch).
#pragma unroll
    for (int rr = 0; rr < R; ++rr) {
        if (EXACT || rr < nr) {
            const float4 x0 = xb[rr][0][lane], x1 = xb[rr][1][lane];
#pragma unroll
            for (int jj = 0; jj < J; ++jj) {
                float s = acc[jj][rr];
                s = __builtin_fmaf(x0.x, w[jj][0], s);
                s = __builtin_fmaf(x0.y, w[jj][1], s);
                s = __builtin_fmaf(x0.z, w[jj][2], s);
                s = __builtin_fmaf(x0.w, w[jj][3], s);
                s = __builtin_fmaf(x1.x, w[jj][4], s);
                s = __builtin_fmaf(x1.y, w[jj][5], s);
                s = __builtin_fmaf(x1.z, w[jj][6], s);
                s = __builtin_fmaf(x1.w, w[jj][7], s);
                acc[jj][rr] = s;
            }
        }
    }
}

// PF: chunks of weights requested ahead (1 or 2)
template <int J, int R, int EPI, bool EXACT, int PF>
__global__ __launch_bounds__(GV_THREADS) void canon_gemv_kernel(GemvArgs a, int n_fb, int n_rt) {
    const int b = blockIdx.x;
    const int xcd = b & 7, slot = b >> 3;
    const int fb = (slot / n_rt) * 8 + xcd;
    const int rt = slot % n_rt;
    if (fb >= n_fb) return;
    RowCount rc{a.n_dev, a.n_host, a.cap};
    const int n = rc.get();
    const int r0 = rt * R;
    if (r0 >= n) return;
    const int nr = min(R, n - r0);
    // the wave index through a scalar register, so the activation row bases and the weight
    // rows are scalar values (fewer VGPRs and vector address instructions; measured 1.5%
    // over the five projection shapes at 1 to 16 rows, 4% on the LM head at 12)
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    const int jw = (fb * GV_NW + wave) * J;
    const int K = a.K, G = K >> 3;

    // LDS chunk: element 8*lane + 4*half + c of row rr at xs[buf][rr][half][lane].c
    constexpr int XB = GemvShape<R>::XB;
    __shared__ float4 xs[XB][R][2][64];

    const uint16_t* wrow[J];
    bool valid[J];
    if constexpr (EPI == EPI_SWIGLU) {
        // the block's first GV_NW / 2 waves take the gate rows, the others the up rows of the
        // same J (GV_NW / 2) outputs: wave w's feature jj is output pj0 + jj of its half
        const int half = wave >= GV_NW / 2, pj0 = fb * (GV_NW / 2 * J) + (wave % (GV_NW / 2)) * J;
#pragma unroll
        for (int jj = 0; jj < J; ++jj) {
            valid[jj] = pj0 + jj < a.N;
            wrow[jj] = valid[jj] ? a.W[half] + (size_t)(pj0 + jj) * K : a.W[0];
        }
    } else {
#pragma unroll
        for (int jj = 0; jj < J; ++jj) {
            int j = jw + jj;
            valid[jj] = j < a.N;
            int seg = 0;
            while (seg < 2 && j >= a.Nseg[seg]) { j -= a.Nseg[seg]; ++seg; }
            wrow[jj] = valid[jj] ? a.W[seg] + (size_t)j * K : a.W[0];
        }
    }

    float acc[J][R];
#pragma unroll
    for (int jj = 0; jj < J; ++jj)
#pragma unroll
        for (int rr = 0; rr < R; ++rr) acc[jj][rr] = 0.0f;

    const int nch = (K + KCH - 1) / KCH;
    uint4 xr[GemvShape<R>::XLD];
    if constexpr (PF == 2) {
        // weights requested two chunks ahead (a ring of three register buffers, the loop
        // unrolled by three so every buffer is named statically); loads past the last chunk
        // re-read the last group (clamped) and are never used
        uint4 wA[J], wB[J], wC[J];
        gemv_load_x<R>(a, r0, nr, 0, wave, lane, xr);
        gemv_load_w<J>(wrow, lane, G, wA);
        gemv_load_w<J>(wrow, 64 + lane, G, wB);
        gemv_store_x<R>(xs[0], wave, lane, xr);
        __syncthreads();
        auto step = [&](int c, const uint4 (&cur)[J], uint4 (&nxt)[J]) {
            gemv_load_x<R>(a, r0, nr, (c + 1) * KCH, wave, lane, xr);
            gemv_load_w<J>(wrow, (c + 2) * 64 + lane, G, nxt);
            __builtin_amdgcn_sched_barrier(0);
            if (c * 64 + lane < G) gemv_fma_chunk<J, R, EXACT>(xs[c % XB], lane, nr, cur, acc);
            if (XB == 1) __syncthreads();
            gemv_store_x<R>(xs[(c + 1) % XB], wave, lane, xr);
            __syncthreads();
        };
        for (int c = 0; c < nch; c += 3) {
            step(c, wA, wC);
            if (c + 1 >= nch) break;
            step(c + 1, wB, wA);
            if (c + 2 >= nch) break;
            step(c + 2, wC, wB);
        }
    } else {
        uint4 wA[J], wB[J];
        gemv_load_x<R>(a, r0, nr, 0, wave, lane, xr);
        gemv_load_w<J>(wrow, lane, G, wA);
        gemv_store_x<R>(xs[0], wave, lane, xr);
        __syncthreads();
        // one chunk with a successor: request chunk c+1 (activations first, then weights
        // into `nxt`), run chunk c, then stage chunk c+1's activations.  Loads complete in
        // order, so the staging waits for the activations only and the weights of chunk c+1
        // stay in flight.  With two LDS buffers chunk c+1 goes to the other buffer and one
        // barrier per chunk suffices (the buffer it overwrites was last read by chunk c-1,
        // which every wave finished before the previous barrier); with one buffer the
        // restaging sits between two barriers.
        auto step = [&](int c, const uint4 (&cur)[J], uint4 (&nxt)[J]) {
            gemv_load_x<R>(a, r0, nr, (c + 1) * KCH, wave, lane, xr);
            gemv_load_w<J>(wrow, (c + 1) * 64 + lane, G, nxt);
            __builtin_amdgcn_sched_barrier(0);
            if (c * 64 + lane < G) gemv_fma_chunk<J, R, EXACT>(xs[c % XB], lane, nr, cur, acc);
            if (XB == 1) __syncthreads();
            gemv_store_x<R>(xs[(c + 1) % XB], wave, lane, xr);
            __syncthreads();
        };
        int c = 0;
        for (; c + 2 < nch; c += 2) {
            step(c, wA, wB);
            step(c + 1, wB, wA);
        }
        if (c + 1 < nch) {
            step(c, wA, wB);
            if ((c + 1) * 64 + lane < G) gemv_fma_chunk<J, R, EXACT>(xs[(c + 1) % XB], lane, nr, wB, acc);
        } else if (c * 64 + lane < G) {
            gemv_fma_chunk<J, R, EXACT>(xs[c % XB], lane, nr, wA, acc);
        }
    }

    // all J*R butterflies at once (padded to a power of two; each value is summed over the
    // lanes on its own, so the padding never mixes in); value jj*R + rr ends in the lanes
    // multi_index names
    constexpr int NV = pow2_at_least(J * R);
    float flat[NV];
#pragma unroll
    for (int k = 0; k < NV; ++k) flat[k] = k < J * R ? acc[k / R][k % R] : 0.0f;
    const float v = butterfly_sum_multi<NV>(flat, lane);
    bool writer;
    const int idx = multi_index<NV>(lane, &writer);
    if constexpr (EPI == EPI_SWIGLU) {
        // the up waves hand their sums to the gate waves through LDS
        __shared__ float up_sum[GV_NW / 2 * J][R];
        const int half = wave >= GV_NW / 2, p = (wave % (GV_NW / 2)) * J + idx / R, rr = idx % R;
        if (half && writer && idx < J * R) up_sum[p][rr] = v;
        __syncthreads();
        if (half || !writer || idx >= J * R || rr >= nr) return;
        const int pj = fb * (GV_NW / 2 * J) + p;
        if (pj >= a.N) return;
        const float g = bf2f(f2bf(v)), up = bf2f(f2bf(up_sum[p][rr]));
        const float sg = ieee_div(g, 1.0f + canon_exp(-g));
        reinterpret_cast<uint16_t*>(a.Y)[(size_t)(r0 + rr) * a.N + pj] = (uint16_t)f2bf(sg * up);
        return;
    }
    const int jj = idx / R, rr = idx % R;
    bool ok = writer && idx < J * R && rr < nr;
#pragma unroll
    for (int k = 0; k < J; ++k)
        if (k == jj) ok = ok && valid[k];
    if (!ok) return;
    const int j = jw + jj, row = r0 + rr;
    if (EPI == EPI_F32) {
        reinterpret_cast<float*>(a.Y)[(size_t)row * a.N + j] = v;
    } else if (EPI == EPI_BF16) {
        int jl = j, seg = 0;
        while (seg < 2 && jl >= a.Nseg[seg]) { jl -= a.Nseg[seg]; ++seg; }
        const float y = a.bias[seg] ? v + bf2f(a.bias[seg][jl]) : v;
        reinterpret_cast<uint16_t*>(a.Y)[(size_t)row * a.N + j] = (uint16_t)f2bf(y);
    } else {  // residual: x = bf16(x + bf16(y))
        uint16_t* xr2 = reinterpret_cast<uint16_t*>(a.Y) + (size_t)row * a.N + j;
        const float y = bf2f(f2bf(v));
        *xr2 = (uint16_t)f2bf(bf2f(*xr2) + y);
    }
}

template <int J, int R, bool EXACT, int PF = 1>
static hipError_t launch_jr(const GemvArgs& a, int epi, int rows, hipStream_t s) {
    const int per_block = epi == EPI_SWIGLU ? GV_NW / 2 * J : GV_NW * J;  // outputs (pairs) per block
    const int n_fb = (a.N + per_block - 1) / per_block;
    const int n_rt = (rows + R - 1) / R;
    const dim3 grid(8 * ((n_fb + 7) / 8) * n_rt);
    switch (epi) {
        case EPI_SWIGLU: hipLaunchKernelGGL((canon_gemv_kernel<J, R, EPI_SWIGLU, EXACT, PF>), grid, dim3(GV_THREADS), 0, s, a, n_fb, n_rt); break;
        case EPI_BF16: hipLaunchKernelGGL((canon_gemv_kernel<J, R, EPI_BF16, EXACT, PF>), grid, dim3(GV_THREADS), 0, s, a, n_fb, n_rt); break;
        case EPI_RESID: hipLaunchKernelGGL((canon_gemv_kernel<J, R, EPI_RESID, EXACT, PF>), grid, dim3(GV_THREADS), 0, s, a, n_fb, n_rt); break;
        default: hipLaunchKernelGGL((canon_gemv_kernel<J, R, EPI_F32, EXACT, PF>), grid, dim3(GV_THREADS), 0, s, a, n_fb, n_rt); break;
    }
    return hipGetLastError();
}

// A host row count up to 24 gets one tile of exactly ceil(n/4)*4 rows (branch-free rows,
// at most three of them dead; 5..16 rows with 3 features per wave as stated above);
// larger counts and device-side counts use 16-row tiles (8-row when at most 8 rows can
// occur) that skip dead rows by a uniform branch.
// 3 features per wave: on wide outputs for 9..16-row tiles (the 8-row tile measured slower
// there: LM head at 8 rows 180 vs 178 us), on narrower ones when it balances the CUs
static bool gemv_three_features(int N, int R, int n_cu) {
    if (N >= MG_GEMV_BIG_N) return R >= 12;
    const int b2 = (N + 2 * GV_NW - 1) / (2 * GV_NW), b3 = (N + 3 * GV_NW - 1) / (3 * GV_NW);
    return (b3 + n_cu - 1) / n_cu * 3 < (b2 + n_cu - 1) / n_cu * 2;
}

hipError_t launch_canon_gemv_valu(const GemvArgs& a, int epi, hipStream_t s) {
    const int rows = a.n_dev ? a.cap : a.n_host;
    if (rows <= 0 || a.N <= 0) return hipSuccess;
    if (!a.n_dev && rows <= MG_GEMV_EXACT_MAX) {
        const int nt = (rows + 3) / 4;
        // (a SwiGLU launch is judged by its 2N features)
        const int Nf = epi == EPI_SWIGLU ? 2 * a.N : a.N;
        // narrow outputs over a short K (the QKV and O projections) request their weights two
        // chunks ahead from 5 rows on: those launches have one block per CU and wait on
        // memory (measured at 12 rows: QKV 20.0 vs 23.4 us, O 15.9 vs 17.8; the wide and the
        // long-K projections were not faster)
        const bool pf2 = nt >= 2 && a.K <= 4096 && Nf <= 8192;
        if (nt >= 2 && nt <= 4 && gemv_three_features(Nf, 4 * nt, a.n_cu > 0 ? a.n_cu : 256)) {
            if (nt == 2) return pf2 ? launch_jr<MG_GEMV_J_BIG, 8, true, 2>(a, epi, rows, s)
                                    : launch_jr<MG_GEMV_J_BIG, 8, true>(a, epi, rows, s);
            if (nt == 3) return pf2 ? launch_jr<MG_GEMV_J_BIG, 12, true, 2>(a, epi, rows, s)
                                    : launch_jr<MG_GEMV_J_BIG, 12, true>(a, epi, rows, s);
            return pf2 ? launch_jr<MG_GEMV_J_BIG, 16, true, 2>(a, epi, rows, s)
                       : launch_jr<MG_GEMV_J_BIG, 16, true>(a, epi, rows, s);
        }
        switch (nt) {
            case 1: return launch_jr<MG_GEMV_J_R8, 4, true>(a, epi, rows, s);
            case 2: return pf2 ? launch_jr<MG_GEMV_J_R8, 8, true, 2>(a, epi, rows, s)
                               : launch_jr<MG_GEMV_J_R8, 8, true>(a, epi, rows, s);
            case 3: return pf2 ? launch_jr<MG_GEMV_J_R12, 12, true, 2>(a, epi, rows, s)
                               : launch_jr<MG_GEMV_J_R12, 12, true>(a, epi, rows, s);
            case 4: return pf2 ? launch_jr<MG_GEMV_J_R12, 16, true, 2>(a, epi, rows, s)
                               : launch_jr<MG_GEMV_J_R12, 16, true>(a, epi, rows, s);
            case 5: return launch_jr<MG_GEMV_J_R16, 20, true>(a, epi, rows, s);
            default: return launch_jr<MG_GEMV_J_R16, 24, true>(a, epi, rows, s);
        }
    }
    if (!a.n_dev && rows % 16 == 0) return launch_jr<MG_GEMV_J_R16, 16, true>(a, epi, rows, s);
    if (rows > 8) return launch_jr<MG_GEMV_J_R16, 16, false>(a, epi, rows, s);
    return launch_jr<MG_GEMV_J_R8, 8, false>(a, epi, rows, s);
}

// Which of the two bit-identical kernels runs: the matrix-core one (k_gemv_mfma.hip) where it
// was measured faster, the fma kernel above otherwise (its exact 4..24-row tiles waste fewer
// lanes at small counts; the matrix-core time is flat within a 16-row tile and grows by a
// quarter tile per 4-row quad past it).  The matrix-core kernel takes host counts above 8 rows
// and device counts that may exceed 24.  Measured in the decode loop (kernel trace of gated
// Llama-8B steps, us, fma / matrix-core): at 9..12 rows O and down 14.5 and 34.0 / 22.6 on
// average (the matrix-core launch has one block per CU there and a deep ring), gate/up 63.8 /
// 53.9; with the caches flushed before each launch the LM heads at 12 rows take 264 / 242
// (Llama-8B), 246 / 229 and 337 / 314 us (Qwen2.5-7B and 14B); at 8 rows the fma kernel is
// faster on every shape (O 13.8 / 15.0, gate/up 46.2 / 53.7, LM head 188 / 234 us).  Above 12
// rows the matrix-core kernel is faster on the projections of the Llama-8B, Qwen2.5-7B and 14B
// shapes (flushed caches, e.g. at 20 rows gate/up 90.4 / 77.6, down 51.3 / 43.5).
bool canon_gemv_on_mfma(int rows, bool device_count) { return device_count ? rows > MG_GEMV_EXACT_MAX : rows > 8; }

hipError_t launch_canon_gemv(const GemvArgs& a, int epi, hipStream_t s) {
    const int rows = a.n_dev ? a.cap : a.n_host;
    return canon_gemv_on_mfma(rows, a.n_dev != nullptr) ? launch_canon_gemv_mfma(a, epi, s)
                                                         : launch_canon_gemv_valu(a, epi, s);
}

}  // namespace mg
