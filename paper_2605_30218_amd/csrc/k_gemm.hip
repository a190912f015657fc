// k_gemm.hip -- the fast path's weight-streaming projection on MFMA (gfx950).
//
// Y[M][N] = X[M][K] * W[N][K]^T with v_mfma_f32_16x16x32_bf16, M <= 256 (rows
// padded to 16-row tiles).  A block of NW waves (8, or 4 on the direct-to-LDS path;
// the host's launch rule picks the waves and the split count per launch) owns 16 NW
// output features; a wave owns 16 of them for all rows (the activation chunk staged in
// LDS serves all of the block's waves).  The block walks its K range in chunks of KC,
// requesting later chunks while the MFMAs of the current one run.  Two operand paths:
//  * K % 128 == 0 and up to 128 rows (128-element chunks): both operands go through
//    LDS by direct-to-LDS loads -- each wave's weights through its own ring of DEPTH
//    stages (two chunks ahead up to 64 rows, one above), the activations through a
//    block-wide double buffer --
//    in a swizzled layout whose loads read each row's chunk as one contiguous run and
//    whose MFMA fragment reads are free of bank conflicts (see issue_w_lds).
//  * otherwise: weights straight from HBM into MFMA B-operand registers (lane (j, q)
//    loads W[n+j][k+8q .. k+8q+7], 16 rows x 64 contiguous bytes per k step of 16
//    features) in a ping-pong register pair, the activations staged through a
//    double-buffered, padded LDS tile.  Loads complete in order, so staging the
//    activations of chunk c+1 waits only for those, and the weights of chunk c+1 stay
//    in flight across the barrier.  Every load is unconditional (rows past N read row
//    0, k past K reads the row's last group; the activations there are zero and the
//    results are discarded).
// The K range may be split over blocks (split-K): each split writes its fp32 partial
// tile and the kernel that consumes the projection (RoPE and K/V append, SwiGLU, or
// residual add + RMSNorm) sums the splits in split order, so blocks never wait for each
// other.  An unsplit gate/up projection on the direct-to-LDS path instead applies the
// SwiGLU in its epilogue (FEPI_SWIGLU).  The summation order depends on the split count
// only (split boundaries in 128-element units); the fast path's choice of split count
// depends on M, so the fast path may be batch-variant.
#include "mg_device.h"
#include "mg_kernels.h"

namespace mg {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

#ifndef MG_GEMM_KC_SMALL
#define MG_GEMM_KC_SMALL 128
#endif
// waves per block of the register operand path (measured: 8 beats 4 and 16)
constexpr int GM_NW = 8, GM_THREADS = 64 * GM_NW;
// K per chunk for a tile of MT 16-row tiles (host and device must agree)
__host__ __device__ constexpr int gemm_kc(int MT) { return MT <= 4 ? MG_GEMM_KC_SMALL : MT <= 8 ? 128 : 64; }

template <int MT>
struct GemmShape {
    static constexpr int KC = gemm_kc(MT);  // K per chunk
    static constexpr int ROWS = 16 * MT;
    static constexpr int STRIDE = KC * 2 + 16;    // LDS bytes per staged row
    static constexpr int NST = KC / 32;           // MFMA k-steps per chunk
    static constexpr int GPR = KC / 8;            // 16-byte groups per staged row
    static constexpr int XLD = (ROWS * GPR + GM_THREADS - 1) / GM_THREADS;  // staging loads per thread per chunk
    // 128-element chunks take the weights through a per-wave LDS ring of DEPTH stages and
    // the activations through a double buffer (direct-to-LDS loads; 160 KiB of LDS)
    static constexpr bool LDSW = KC == 128;  // (with K % 128 == 0, chosen at launch)
    static constexpr int DEPTH = MT <= 4 ? 3 : 2;
};

template <int EPI>
__device__ __forceinline__ void fast_epilogue(const FastGemmArgs& a, int split, int row, int n, float v) {
    if (EPI == FEPI_F32) {
        reinterpret_cast<float*>(a.Y)[(size_t)row * a.N + n] = v;
    } else if (EPI == FEPI_BF16) {
        int nl = n, seg = 0;
        while (seg < 2 && nl >= a.Nseg[seg]) { nl -= a.Nseg[seg]; ++seg; }
        const float y = a.bias[seg] ? v + bf2f(a.bias[seg][nl]) : v;
        reinterpret_cast<uint16_t*>(a.Y)[(size_t)row * a.N + n] = (uint16_t)f2bf(y);
    } else {  // FEPI_PART: fp32 partial tile of this split
        a.part[((size_t)split * a.M + row) * a.N + n] = v;
    }
}

// activations of chunk kc: rows past M read row M-1; groups past K read the row's
// last group and are zeroed when staged (so the wait for the data happens at the store)
template <int MT>
__device__ __forceinline__ void load_x(const FastGemmArgs& a, int kc, uint4 (&xr)[GemmShape<MT>::XLD]) {
    using S = GemmShape<MT>;
#pragma unroll
    for (int it = 0; it < S::XLD; ++it) {
        const int t = threadIdx.x + GM_THREADS * it;
        const int row = min(min(t / S::GPR, S::ROWS - 1), a.M - 1), k = kc + (t % S::GPR) * 8;
        xr[it] = *reinterpret_cast<const uint4*>(a.X + (size_t)row * a.K + min(k, a.K - 8));
    }
}

template <int MT>
__device__ __forceinline__ void store_x(unsigned char* buf, int kc, int K, const uint4 (&xr)[GemmShape<MT>::XLD]) {
    using S = GemmShape<MT>;
#pragma unroll
    for (int it = 0; it < S::XLD; ++it) {
        const int t = threadIdx.x + GM_THREADS * it;
        const int row = t / S::GPR, g = t % S::GPR;
        if (GM_THREADS * S::XLD > S::ROWS * S::GPR && row >= S::ROWS) continue;
        const uint32_t keep = 0u - (uint32_t)(kc + g * 8 < K);
        const uint4 v = make_uint4(xr[it].x & keep, xr[it].y & keep, xr[it].z & keep, xr[it].w & keep);
        *reinterpret_cast<uint4*>(buf + row * S::STRIDE + g * 16) = v;
    }
}

// weights of chunk kc: lane group q supplies k = kc + 32 st + 8 q .. +7 at k-step st
template <int MT, int FT>
__device__ __forceinline__ void load_w(const uint16_t* const (&wrow)[FT], int kc, int K, int q,
                                       uint4 (&wr)[GemmShape<MT>::NST][FT]) {
    using S = GemmShape<MT>;
#pragma unroll
    for (int st = 0; st < S::NST; ++st) {
        const int k = min(kc + st * 32 + q * 8, K - 8);
#pragma unroll
        for (int f = 0; f < FT; ++f) wr[st][f] = *reinterpret_cast<const uint4*>(wrow[f] + k);
    }
}

// ---- operands through LDS by direct-to-LDS loads (128-element chunks, K % 128 == 0)
// A 16-row block of a chunk (16 rows x 128 bf16 = 4 KiB, weights or activations) is 256
// 16-byte pieces; piece (row j, group G) sits at slot 64 (j >> 2) + 16 (j & 3) + (G ^ j).
// It is filled by 4 direct-to-LDS loads: load st, lane 16 r + g writes slot 64 st + 16 r + g,
// so it fetches row j = 4 st + r, group g ^ j -- each row's 256 bytes in one contiguous run
// (measured: 5.5 TB/s over the LM head against 4.4 for 16 rows x 64 bytes per load).  The
// MFMA fragment of k-step st (lane jl + 16 q: row jl, elements 32 st + 8 q ..) is the piece
// (jl, 4 st + q); the xor puts the 16 rows of one read on distinct banks.  The weights go
// through a per-wave ring of DEPTH stages (requested DEPTH - 1 chunks ahead), the
// activation chunk (MT blocks) through a double buffer shared by the block (one ahead).
// The compiler does not count direct-to-LDS loads when it places its waits, and it would
// wait for all of them before an ordinary access to LDS; so the fragment reads and the
// barrier are inline asm and every wait below is explicit (loads complete in order).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

__device__ __forceinline__ int piece_slot(int j, int G) { return 64 * (j >> 2) + 16 * (j & 3) + (G ^ j); }

// load st of a 16-row block whose row j starts at rowp(j)
__device__ __forceinline__ void issue_block_load(const uint16_t* src, uint4* block, int st, int lane) {
    __builtin_amdgcn_global_load_lds(src, block + 64 * st, 16, 0, 0);
}

__device__ __forceinline__ void issue_w_lds(const uint16_t* tile, int K, int kc, int lane, uint4* stage) {
    const int r = lane >> 4, g = lane & 15;
#pragma unroll
    for (int st = 0; st < 4; ++st) {
        const int j = 4 * st + r;
        issue_block_load(tile + (size_t)j * K + kc + 8 * (g ^ j), stage, st, lane);
    }
}

// this wave's XI of the 4 MT activation loads of chunk kc (rows past M read row M - 1; with
// fewer loads than waves, several waves issue each load, writing the same bytes)
// activation loads per wave per chunk (the 4 MT loads of a chunk shared by the NW waves)
__host__ __device__ constexpr int gemm_xi(int MT, int NW) { return 4 * MT >= NW ? 4 * MT / NW : 1; }

template <int MT, int NW>
__device__ __forceinline__ void issue_x_lds(const FastGemmArgs& a, int kc, int wave, int lane, uint4* xt) {
    constexpr int NI = 4 * MT, XI = gemm_xi(MT, NW);
    static_assert(XI * NW >= NI, "the block's waves cover every activation load");
    const int r = lane >> 4, g = lane & 15;
#pragma unroll
    for (int t = 0; t < XI; ++t) {
        const int ii = (wave * XI + t) % NI, bb = ii >> 2, st = ii & 3;
        const int j = 4 * st + r, row = min(16 * bb + j, a.M - 1);
        issue_block_load(a.X + (size_t)row * a.K + kc + 8 * (g ^ j), xt + 256 * bb, st, lane);
    }
}

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ void lds_read(u32x4_t& v, const uint4* p) {
    asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"((uint32_t)(uintptr_t)p));
}
// Waits for the LDS reads and names every fragment as read and written by the wait, so no
// use of a fragment can be scheduled before it.
template <int MT>
__device__ __forceinline__ void lds_wait_frags(u32x4_t (&wv)[2], u32x4_t (&xv)[2][MT]) {
    if constexpr (MT == 1) {
        asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(wv[0]), "+v"(wv[1]), "+v"(xv[0][0]), "+v"(xv[1][0]) : : "memory");
    } else if constexpr (MT == 2) {
        asm volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(wv[0]), "+v"(wv[1]), "+v"(xv[0][0]), "+v"(xv[0][1]), "+v"(xv[1][0]), "+v"(xv[1][1]) : : "memory");
    } else if constexpr (MT == 4) {
        asm volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(wv[0]), "+v"(wv[1]), "+v"(xv[0][0]), "+v"(xv[0][1]), "+v"(xv[0][2]), "+v"(xv[0][3]),
                       "+v"(xv[1][0]), "+v"(xv[1][1]), "+v"(xv[1][2]), "+v"(xv[1][3]) : : "memory");
    } else {
        static_assert(MT == 8, "tile count");
        asm volatile("s_waitcnt lgkmcnt(0)"
                     : "+v"(wv[0]), "+v"(wv[1]), "+v"(xv[0][0]), "+v"(xv[0][1]), "+v"(xv[0][2]), "+v"(xv[0][3]),
                       "+v"(xv[0][4]), "+v"(xv[0][5]), "+v"(xv[0][6]), "+v"(xv[0][7]), "+v"(xv[1][0]), "+v"(xv[1][1]),
                       "+v"(xv[1][2]), "+v"(xv[1][3]), "+v"(xv[1][4]), "+v"(xv[1][5]), "+v"(xv[1][6]), "+v"(xv[1][7]) : : "memory");
    }
}
__device__ __forceinline__ void lds_barrier() { asm volatile("s_barrier" ::: "memory"); }

// the MFMAs of one chunk from the LDS stage `ws` (this wave's weights) and tile `xt`,
// two k-steps at a time
template <int MT>
__device__ __forceinline__ void mfma_chunk_lds(const uint4* ws, const uint4* xt, int jl, int q, f32x4_t (&acc)[MT][1]) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        u32x4_t wv[2], xv[2][MT];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
            const int sl = piece_slot(jl, 4 * (2 * h + u) + q);
            lds_read(wv[u], ws + sl);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) lds_read(xv[u][mt], xt + 256 * mt + sl);
        }
        lds_wait_frags<MT>(wv, xv);
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                acc[mt][0] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, xv[u][mt]),
                                                                      __builtin_bit_cast(bf16x8_t, wv[u]), acc[mt][0], 0, 0, 0);
    }
}

template <int MT, int FT>
__device__ __forceinline__ void mfma_chunk(const unsigned char* buf, int jl, int q, const uint4 (&w)[GemmShape<MT>::NST][FT],
                                           f32x4_t (&acc)[MT][FT]) {
    using S = GemmShape<MT>;
#pragma unroll
    for (int st = 0; st < S::NST; ++st) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const uint4 av = *reinterpret_cast<const uint4*>(buf + (16 * mt + jl) * S::STRIDE + (st * 32 + q * 8) * 2);
            const bf16x8_t A = __builtin_bit_cast(bf16x8_t, av);
#pragma unroll
            for (int f = 0; f < FT; ++f)
                acc[mt][f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, __builtin_bit_cast(bf16x8_t, w[st][f]), acc[mt][f],
                                                                      0, 0, 0);
        }
    }
}

template <int MT, int NW, int FT, int EPI, bool LDSP>
__global__ __launch_bounds__(64 * NW) void fast_gemm_kernel(FastGemmArgs a) {
    using S = GemmShape<MT>;
    static_assert(NW == GM_NW || (LDSP && S::LDSW), "4-wave blocks only on the direct-to-LDS path");
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int jl = lane & 15, q = lane >> 4;
    const int nb = blockIdx.x, split = blockIdx.y;
    const int FB = 16 * NW * FT;  // features per block
    const int K = a.K, M = a.M;

    const uint16_t* wrow[FT];
    bool wok[FT];
    int nf[FT];
#pragma unroll
    for (int f = 0; f < FT; ++f) {
        if constexpr (EPI == FEPI_SWIGLU) {
            // waves [0, NW/2) take the gate rows, the others the up rows of the same outputs
            const int n0 = nb * (NW / 2) * 16 + (wave % (NW / 2)) * 16;
            nf[f] = n0;
            wok[f] = n0 < a.N;
            wrow[f] = wok[f] ? a.W[wave >= NW / 2] + (size_t)(n0 + jl) * K : a.W[0];
        } else {
            const int n0 = nb * FB + (wave * FT + f) * 16;
            nf[f] = n0;
            wok[f] = n0 < a.N;
            int seg = 0, nl = n0;
            while (seg < 2 && nl >= a.Nseg[seg]) { nl -= a.Nseg[seg]; ++seg; }
            wrow[f] = wok[f] ? a.W[seg] + (size_t)(nl + jl) * K : a.W[0];
        }
    }

    // split boundaries in 128-element units whatever the chunk size, so that a row's
    // summation order depends only on the split count (the matrix-core verifier fixes it)
    static_assert(128 % S::KC == 0, "chunks tile the 128-element split unit");
    const int nchunks = (K + S::KC - 1) / S::KC, nunits = (K + 127) / 128;
    const int c0 = min(nchunks, (int)((long)split * nunits / a.S) * (128 / S::KC));
    const int c1 = min(nchunks, (int)((long)(split + 1) * nunits / a.S) * (128 / S::KC));

    f32x4_t acc[MT][FT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int f = 0; f < FT; ++f) acc[mt][f] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    if constexpr (LDSP && S::LDSW) {
        static_assert(FT == 1 && S::NST == 4, "LDS operand path: one 16-feature tile, 128-element chunks");
        constexpr int D = S::DEPTH, XI = gemm_xi(MT, NW);
        __shared__ __attribute__((aligned(16))) uint4 wring[D][NW][256];
        __shared__ __attribute__((aligned(16))) uint4 xt[2][MT * 256];
        // the tile's first weight row (a tile past N reads rows 0 .. 15: results discarded)
        const uint16_t* tile = wok[0] ? wrow[0] - (size_t)jl * K : a.W[0];
        if (c0 < c1) {
            issue_x_lds<MT, NW>(a, c0 * S::KC, wave, lane, xt[c0 & 1]);
#pragma unroll
            for (int d = 0; d < D - 1; ++d)
                if (c0 + d < c1) issue_w_lds(tile, K, (c0 + d) * S::KC, lane, wring[(c0 + d) % D][wave]);
            __builtin_amdgcn_sched_barrier(0);
            if (c0 + D - 1 <= c1) wait_vmcnt<4 * (D - 1)>();  // this wave's activation loads
            else wait_vmcnt<0>();
            lds_barrier();
        }
        // steady state: chunk c + D - 1 (and so c + 1) exists.  Request this wave's share of
        // the activations of c + 1 and the weights of c + D - 1 (into the stage chunk c - 1
        // used), then wait for the weights of c: after them come at most D - 2 weight
        // chunks, the activations of c + 1 and chunk c + D - 1.  The activations of c are
        // complete: every wave waited for its share before the last barrier.
        int c = c0;
        for (; c + D - 1 < c1; ++c) {
            issue_x_lds<MT, NW>(a, (c + 1) * S::KC, wave, lane, xt[(c + 1) & 1]);
            issue_w_lds(tile, K, (c + D - 1) * S::KC, lane, wring[(c + D - 1) % D][wave]);
            __builtin_amdgcn_sched_barrier(0);
            wait_vmcnt<4 * (D - 1) + XI>();
            mfma_chunk_lds<MT>(wring[c % D][wave], xt[c & 1], jl, q, acc);
            __builtin_amdgcn_sched_barrier(0);
            wait_vmcnt<4>();  // this wave's activations of c + 1 (only chunk c + D - 1 may remain)
            lds_barrier();    // every wave's share of c + 1 is in, and every read of chunk c is done
        }
        // the last D - 1 chunks (or fewer): no more weights to request
        for (; c < c1; ++c) {
            const bool more = c + 1 < c1;
            if (more) issue_x_lds<MT, NW>(a, (c + 1) * S::KC, wave, lane, xt[(c + 1) & 1]);
            __builtin_amdgcn_sched_barrier(0);
            wait_vmcnt<0>();
            mfma_chunk_lds<MT>(wring[c % D][wave], xt[c & 1], jl, q, acc);
            __builtin_amdgcn_sched_barrier(0);
            lds_barrier();
        }
        if constexpr (EPI == FEPI_SWIGLU) {
            // every wave is past its last read of the rings (the loops end on a barrier and
            // no load is outstanding): the up waves leave their sums in the weight ring
            float* up_sum = reinterpret_cast<float*>(&wring[0][0][0]) + (wave % (NW / 2)) * MT * 256;
            static_assert((NW / 2) * MT * 256 * 4 <= (int)sizeof(wring), "up sums fit in the weight ring");
            if (wave >= NW / 2) {
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int v = 0; v < 4; ++v) up_sum[mt * 256 + (4 * q + v) * 16 + jl] = acc[mt][0][v];
            }
            __syncthreads();
            if (wave >= NW / 2 || !wok[0]) return;
            uint16_t* act = reinterpret_cast<uint16_t*>(a.Y);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int row = 16 * mt + 4 * q + v;
                    if (row >= M) continue;
                    const float g = bf2f(f2bf(acc[mt][0][v]));
                    const float u = bf2f(f2bf(up_sum[mt * 256 + (4 * q + v) * 16 + jl]));
                    act[(size_t)row * a.N + nf[0] + jl] = (uint16_t)f2bf((g / (1.0f + __expf(-g))) * u);
                }
            return;
        }
    } else {
    __shared__ __attribute__((aligned(16))) unsigned char xs[2][S::ROWS * S::STRIDE];
    uint4 wA[S::NST][FT], wB[S::NST][FT];
    uint4 xr[S::XLD];
    if (c0 < c1) {
        load_x<MT>(a, c0 * S::KC, xr);
        load_w<MT, FT>(wrow, c0 * S::KC, K, q, wA);
        store_x<MT>(xs[c0 & 1], c0 * S::KC, K, xr);
    }
    __syncthreads();
    // one chunk with a successor: request chunk c+1 (activations, then weights into
    // `nxt`), run chunk c from `cur`, stage the activations of c+1, barrier.  The
    // requests are unconditional inside the loop, so the compiler's wait for `cur`
    // leaves the requests of c+1 in flight.
    auto step = [&](int c, uint4 (&cur)[S::NST][FT], uint4 (&nxt)[S::NST][FT]) {
        load_x<MT>(a, (c + 1) * S::KC, xr);
        load_w<MT, FT>(wrow, (c + 1) * S::KC, K, q, nxt);
        // keep every request of chunk c+1 ahead of the MFMAs of chunk c
        __builtin_amdgcn_sched_barrier(0);
        mfma_chunk<MT, FT>(xs[c & 1], jl, q, cur, acc);
        store_x<MT>(xs[(c + 1) & 1], (c + 1) * S::KC, K, xr);
        __syncthreads();
    };
    int c = c0;
    for (; c + 2 < c1; c += 2) {
        step(c, wA, wB);
        step(c + 1, wB, wA);
    }
    // the last one or two chunks
    if (c + 1 < c1) {
        step(c, wA, wB);
        mfma_chunk<MT, FT>(xs[(c + 1) & 1], jl, q, wB, acc);
    } else if (c < c1) {
        mfma_chunk<MT, FT>(xs[c & 1], jl, q, wA, acc);
    }
    }

    // D[i][j] of a 16x16 tile sits in lane j + 16*(i/4), element i%4
    if constexpr (EPI == FEPI_TOP2) {
        // per row: the top-2 of the wave's 16 features (xor shuffles inside the lane group of
        // the row), then of the block's waves (LDS), stored as the block's state of the row
        static_assert(FT == 1, "one 16-feature tile per wave");
        __shared__ Top2 wst[NW][16 * MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                Top2 st{-__builtin_inff(), -__builtin_inff(), -1, 0};
                if (wok[0]) top2_push(st, acc[mt][0][v], nf[0] + jl);
#pragma unroll
                for (int o = 1; o < 16; o <<= 1) st = top2_merge(st, top2_shfl(st, o));
                if (jl == 0) wst[wave][16 * mt + 4 * q + v] = st;
            }
        __syncthreads();
        Top2* states = reinterpret_cast<Top2*>(a.part);
        for (int row = threadIdx.x; row < 16 * MT && row < M; row += 64 * NW) {
            // (states moved as 16-byte words: field-wise struct copies through memory would
            // otherwise be staged in scratch)
            auto ld = [&](int w) {
                const uint4 u = *reinterpret_cast<const uint4*>(&wst[w][row]);
                return Top2{__uint_as_float(u.x), __uint_as_float(u.y), (int)u.z, (int)u.w};
            };
            Top2 st = ld(0);
#pragma unroll
            for (int w = 1; w < NW; ++w) st = top2_merge(st, ld(w));
            reinterpret_cast<uint4*>(states)[(size_t)row * gridDim.x + nb] =
                make_uint4(__float_as_uint(st.v1), __float_as_uint(st.v2), (uint32_t)st.i1, (uint32_t)st.nan);
        }
        return;
    } else {
#pragma unroll
    for (int f = 0; f < FT; ++f) {
        if (!wok[f]) continue;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int row = 16 * mt + 4 * q + v;
                if (row < M) fast_epilogue<EPI>(a, split, row, nf[f] + jl, acc[mt][f][v]);
            }
    }
    }
}

// one block per row: merges the row's nblk block states (top2_merge is associative and
// commutative, so the grouping does not change the result) and writes the top-1 index
__global__ __launch_bounds__(256) void top1_rows_kernel(const Top2* __restrict__ states, int nblk,
                                                        int32_t* __restrict__ top1) {
    const int r = blockIdx.x, t = threadIdx.x;
    Top2 st{-__builtin_inff(), -__builtin_inff(), -1, 0};
    for (int k = t; k < nblk; k += 256) {
        const uint4 u = reinterpret_cast<const uint4*>(states)[(size_t)r * nblk + k];  // one 16-byte load
        st = top2_merge(st, Top2{__uint_as_float(u.x), __uint_as_float(u.y), (int)u.z, (int)u.w});
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) st = top2_merge(st, top2_shfl(st, o));
    __shared__ Top2 ws[4];
    if ((t & 63) == 0) ws[t >> 6] = st;
    __syncthreads();
    if (t == 0) {
        const Top2 m = top2_merge(top2_merge(ws[0], ws[1]), top2_merge(ws[2], ws[3]));
        top1[r] = m.i1 < 0 ? 0 : m.i1;
    }
}

hipError_t launch_top1_rows(int M, const void* states, int nblk, int32_t* top1, hipStream_t s) {
    if (M <= 0) return hipSuccess;
    if (nblk <= 0) return hipErrorInvalidValue;
    hipLaunchKernelGGL(top1_rows_kernel, dim3(M), dim3(256), 0, s, static_cast<const Top2*>(states), nblk, top1);
    return hipGetLastError();
}

// out[i] = sum over s of part[s][i] in split order (the op-level entry point)
__global__ void sum_partials_kernel(const float* __restrict__ part, int S, int64_t n, float* __restrict__ out) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        float s = part[i];
        for (int sp = 1; sp < S; ++sp) s += part[(size_t)sp * n + i];
        out[i] = s;
    }
}

hipError_t launch_sum_partials(const float* part, int S, int64_t n, float* out, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(sum_partials_kernel, dim3(1024), dim3(256), 0, s, part, S, n, out);
    return hipGetLastError();
}

static int mt_for(int M) {
    const int t = (M + 15) / 16;
    return t <= 1 ? 1 : t <= 2 ? 2 : t <= 4 ? 4 : t <= 8 ? 8 : 16;
}

// One 16-feature B tile per wave: blocks of 16 NW features with one tile each measured
// faster than two tiles per wave (fewer blocks, more registers per wave).
constexpr int GM_FT = 1;
constexpr int LDS_PER_CU = 160 * 1024;

// whole 128-element chunks take both operands through LDS by direct-to-LDS loads
static bool lds_path(int M, int K) { return gemm_kc(mt_for(M)) == 128 && K % 128 == 0; }

// blocks of NW waves that fit on one CU at once on the direct-to-LDS path (its LDS: the
// weight ring of DEPTH x NW stages of 4 KiB and the activation double buffer of 2 x MT x 4 KiB)
static int lds_slots(int MT, int NW) {
    const int depth = MT <= 4 ? 3 : 2;
    const int bytes = (depth * NW + 2 * MT) * 4096;
    return LDS_PER_CU / bytes > 1 ? LDS_PER_CU / bytes : 1;
}

// Launch cost of NW-wave blocks with S splits on the direct-to-LDS path.  Launches whose
// blocks are all resident at once (one round) come first, compared by the weight bytes
// of the busiest CU, then the resident waves (more requests in flight), the split count
// (partial-tile traffic), and a preference for 4-wave blocks at up to 16 rows (measured
// faster there) and for 8-wave blocks above.  Launches of several rounds already have
// blocks enough: fewest splits first, then the block size.  A block streams 16 NW
// features over its split's 128-element units (splits differ by at most one unit).
struct LaunchCost {
    int rounds;
    long cu_bytes;
    long waves;
    int S, pref;
    bool operator<(const LaunchCost& o) const {
        if ((rounds == 1) != (o.rounds == 1)) return rounds == 1;
        if (rounds != 1) {
            if (S != o.S) return S < o.S;
            if (pref != o.pref) return pref < o.pref;
            return cu_bytes < o.cu_bytes;
        }
        if (cu_bytes != o.cu_bytes) return cu_bytes < o.cu_bytes;
        if (waves != o.waves) return waves > o.waves;
        if (S != o.S) return S < o.S;
        return pref < o.pref;
    }
};

static LaunchCost lds_cost(int M, int N, int K, int S, int NW, int n_cu) {
    const int MT = mt_for(M), slots = lds_slots(MT, NW);
    const long nb = (N + 16 * NW * GM_FT - 1) / (16 * NW * GM_FT), blocks = nb * S;
    const long units = (K + 127) / 128, split_units = (units + S - 1) / S;
    const long per_cu = (blocks + n_cu - 1) / n_cu;
    LaunchCost c;
    c.rounds = (int)((per_cu + slots - 1) / slots);
    c.cu_bytes = per_cu * split_units * 128 * 16 * NW * GM_FT * 2;
    c.waves = (blocks < (long)n_cu * slots ? blocks : (long)n_cu * slots) * NW;
    c.S = S;
    // several rounds: two 4-wave blocks per CU overlap one block's start with the other's
    // stream (measured on the 128256-feature LM head); one round: as stated above
    if (c.rounds != 1) c.pref = (NW == 4) == (lds_slots(MT, 4) >= 2) ? 0 : 1;
    else c.pref = (NW == 4) == (M <= 16) ? 0 : 1;
    return c;
}

// the most splits the partial tiles allow: each split at least 4 chunks, and the partial
// tiles (S*M*N fp32, written once and read once by the consumer) at most an eighth of
// the weight bytes (measured at 64 rows: 5.54 ms per fast step against 5.69 with a quarter)
static int max_splits(int M, int K) {
    const int KC = gemm_kc(mt_for(M));
    const int nchunks = (K + KC - 1) / KC;
    const int by_chunks = nchunks / 4 > 1 ? nchunks / 4 : 1;
    const long by_traffic = (long)K / (16L * (M < 16 ? 16 : M));
    int S = by_chunks;
    if (S > by_traffic) S = (int)by_traffic;
    if (S > 32) S = 32;
    return S < 1 ? 1 : S;
}

bool fast_gemm_lds_path(int M, int K) { return lds_path(M, K); }

// waves per block for a launch with S splits
static int fast_gemm_waves(int M, int N, int K, int S, int n_cu) {
    if (!lds_path(M, K)) return GM_NW;
    return lds_cost(M, N, K, S, 4, n_cu) < lds_cost(M, N, K, S, 8, n_cu) ? 4 : 8;
}

int fast_gemm_splits(int M, int N, int K, int n_cu) {
    const int Smax = max_splits(M, K);
    if (lds_path(M, K)) {
        // the cheapest (splits, waves) pair; the launch picks the waves again for its S
        int best_S = 1;
        LaunchCost best = lds_cost(M, N, K, 1, 8, n_cu);
        for (int S = 1; S <= Smax; ++S)
            for (int NW : {8, 4}) {
                const LaunchCost c = lds_cost(M, N, K, S, NW, n_cu);
                if (c < best) { best = c; best_S = S; }
            }
        return best_S;
    }
    // register operand path: enough 8-wave blocks for about one per CU (two for small
    // batches, whose blocks carry little MFMA work per weight byte)
    const int nb = (N + 16 * GM_NW * GM_FT - 1) / (16 * GM_NW * GM_FT);
    const int target = (M <= 16 ? 2 : 1) * n_cu;
    const int S = (target + nb - 1) / nb;
    return S < Smax ? S : Smax;
}

int fast_gemm_blocks(int M, int N, int K, int n_cu) {
    const int NW = fast_gemm_waves(M, N, K, 1, n_cu);
    return (N + 16 * NW * GM_FT - 1) / (16 * NW * GM_FT);
}

void fast_gemm_config(int M, int N, int K, int n_cu, int* S, int* waves) {
    *S = fast_gemm_splits(M, N, K, n_cu);
    *waves = fast_gemm_waves(M, N, K, *S, n_cu);
}

template <int MT, int NW, int FT, int EPI>
static void launch_epi(const FastGemmArgs& a, dim3 g, hipStream_t s) {
    if constexpr (EPI == FEPI_SWIGLU) {  // direct-to-LDS path only (checked by the launcher)
        if constexpr (gemm_kc(MT) == 128)
            hipLaunchKernelGGL((fast_gemm_kernel<MT, NW, FT, EPI, true>), g, dim3(64 * NW), 0, s, a);
        return;
    }
    if constexpr (NW == GM_NW) {
        if (!(gemm_kc(MT) == 128 && a.K % 128 == 0)) {
            hipLaunchKernelGGL((fast_gemm_kernel<MT, NW, FT, EPI, false>), g, dim3(64 * NW), 0, s, a);
            return;
        }
    }
    if constexpr (gemm_kc(MT) == 128)
        hipLaunchKernelGGL((fast_gemm_kernel<MT, NW, FT, EPI, true>), g, dim3(64 * NW), 0, s, a);
}

template <int MT, int NW, int FT>
static void launch_ft(const FastGemmArgs& a, int epi, dim3 g, hipStream_t s) {
    switch (epi) {
        case FEPI_BF16: launch_epi<MT, NW, FT, FEPI_BF16>(a, g, s); break;
        case FEPI_PART: launch_epi<MT, NW, FT, FEPI_PART>(a, g, s); break;
        case FEPI_SWIGLU: launch_epi<MT, NW, FT, FEPI_SWIGLU>(a, g, s); break;
        case FEPI_TOP2: launch_epi<MT, NW, FT, FEPI_TOP2>(a, g, s); break;
        default: launch_epi<MT, NW, FT, FEPI_F32>(a, g, s); break;
    }
}

template <int MT>
static void launch_mt(const FastGemmArgs& a, int epi, int NW, hipStream_t s) {
    const int per_block = epi == FEPI_SWIGLU ? 16 * (NW / 2) : 16 * NW * GM_FT;  // outputs per block
    dim3 g((a.N + per_block - 1) / per_block, a.S);
    if constexpr (gemm_kc(MT) == 128) {
        if (NW == 4) return launch_ft<MT, 4, GM_FT>(a, epi, g, s);
    }
    launch_ft<MT, GM_NW, GM_FT>(a, epi, g, s);
}

hipError_t launch_fast_gemm(const FastGemmArgs& a, int epi, hipStream_t s) {
    if (a.M <= 0 || a.N <= 0) return hipSuccess;
    if (a.K < 8 || a.K % 8 || a.N % 16) return hipErrorInvalidValue;
    if (epi != FEPI_PART && a.S != 1) return hipErrorInvalidValue;  // only partial tiles may be split
    if (epi == FEPI_SWIGLU && (a.S != 1 || !lds_path(a.M, a.K) || a.Nseg[0] != a.N || a.Nseg[1] != a.N))
        return hipErrorInvalidValue;
    // a SwiGLU launch streams the gate and the up rows: 2N weight rows
    const int NW = fast_gemm_waves(a.M, epi == FEPI_SWIGLU ? 2 * a.N : a.N, a.K, a.S, a.n_cu > 0 ? a.n_cu : 256);
    switch (mt_for(a.M)) {
        case 1: launch_mt<1>(a, epi, NW, s); break;
        case 2: launch_mt<2>(a, epi, NW, s); break;
        case 4: launch_mt<4>(a, epi, NW, s); break;
        case 8: launch_mt<8>(a, epi, NW, s); break;
        default: launch_mt<16>(a, epi, NW, s); break;
    }
    return hipGetLastError();
}

}  // namespace mg
