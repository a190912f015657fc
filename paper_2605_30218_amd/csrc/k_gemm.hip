// k_gemm.hip -- the fast path's weight-streaming projection on MFMA (gfx950).
//
// Y[M][N] = X[M][K] * W[N][K]^T with v_mfma_f32_16x16x32_bf16, M <= 256 (rows
// padded to 16-row tiles).  A block of 4 waves owns 64*FT output features; a wave
// owns 16*FT of them for all rows.  Weights go straight from HBM into MFMA
// B-operand registers: lane (j, q) loads W[n+j][k+8q .. k+8q+7] (16 bytes), so a
// 32-wide k step of 16 features reads 16 rows x 64 contiguous bytes.  The block
// walks its K range in chunks of KC; while the MFMAs of chunk c run, the weights
// of chunks c+1 and c+2 are already in flight (three register buffers) and the activations
// of chunk c+1 are staged into the other half of a double-buffered LDS tile (rows
// padded by 16 bytes so the A-operand lanes of a k group hit distinct banks).
// One barrier per chunk.  The K range may be split over blocks (split-K): each
// split writes its fp32 partial tile and the kernel that consumes the projection
// (RoPE and K/V append, or residual add + RMSNorm) sums the splits in split order,
// so blocks never wait for each other and no cache-flushing fence is needed.  The
// summation order depends on M (tile and chunk choice) and on the split count:
// this path may be batch-variant.
#include "mg_device.h"
#include "mg_kernels.h"

namespace mg {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

#ifndef MG_GEMM_KC_SMALL
#define MG_GEMM_KC_SMALL 128
#endif
// K per chunk for a tile of MT 16-row tiles (host and device must agree)
__host__ __device__ constexpr int gemm_kc(int MT) { return MT <= 4 ? MG_GEMM_KC_SMALL : MT <= 8 ? 128 : 64; }

template <int MT>
struct GemmShape {
    static constexpr int KC = gemm_kc(MT);  // K per chunk
    static constexpr int ROWS = 16 * MT;
    static constexpr int STRIDE = KC * 2 + 16;    // LDS bytes per staged row
    static constexpr int NST = KC / 32;           // MFMA k-steps per chunk
    static constexpr int GPR = KC / 8;            // 16-byte groups per staged row
    static constexpr int XLD = ROWS * GPR / 256;  // staging loads per thread per chunk
    static_assert(XLD * 256 == ROWS * GPR, "staging must divide evenly");
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

__device__ __forceinline__ float silu_fast(float g) { return g / (1.0f + __expf(-g)); }

template <int MT, bool SWI>
__device__ __forceinline__ void load_x(const FastGemmArgs& a, int kc, uint4 (&xr)[GemmShape<MT>::XLD]) {
    using S = GemmShape<MT>;
#pragma unroll
    for (int it = 0; it < S::XLD; ++it) {
        const int t = threadIdx.x + 256 * it;
        const int row = t / S::GPR, g = t % S::GPR;
        const int k = kc + g * 8;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (row < a.M && k < a.K) {
            if (!SWI) {
                v = *reinterpret_cast<const uint4*>(a.X + (size_t)row * a.K + k);
            } else {
                const uint4 gv = *reinterpret_cast<const uint4*>(a.X + (size_t)row * 2 * a.K + k);
                const uint4 uv = *reinterpret_cast<const uint4*>(a.X + (size_t)row * 2 * a.K + a.K + k);
                v.x = pack_bf2(silu_fast(bf_lo(gv.x)) * bf_lo(uv.x), silu_fast(bf_hi(gv.x)) * bf_hi(uv.x));
                v.y = pack_bf2(silu_fast(bf_lo(gv.y)) * bf_lo(uv.y), silu_fast(bf_hi(gv.y)) * bf_hi(uv.y));
                v.z = pack_bf2(silu_fast(bf_lo(gv.z)) * bf_lo(uv.z), silu_fast(bf_hi(gv.z)) * bf_hi(uv.z));
                v.w = pack_bf2(silu_fast(bf_lo(gv.w)) * bf_lo(uv.w), silu_fast(bf_hi(gv.w)) * bf_hi(uv.w));
            }
        }
        xr[it] = v;
    }
}

template <int MT>
__device__ __forceinline__ void store_x(unsigned char* buf, const uint4 (&xr)[GemmShape<MT>::XLD]) {
    using S = GemmShape<MT>;
#pragma unroll
    for (int it = 0; it < S::XLD; ++it) {
        const int t = threadIdx.x + 256 * it;
        const int row = t / S::GPR, g = t % S::GPR;
        *reinterpret_cast<uint4*>(buf + row * S::STRIDE + g * 16) = xr[it];
    }
}

#ifndef MG_GEMM_KPERM
#define MG_GEMM_KPERM 0
#endif
// k offset, inside a chunk, of the 8 values lane group q supplies at MFMA k-step st.
// MG_GEMM_KPERM = 1 permutes the chunk so a lane's NST groups are contiguous (each
// weight row read as 4 lanes x 16*NST contiguous bytes per chunk instead of 64 bytes
// per k-step); measured slower than the natural order on MI355X, so off by default.
template <int NST>
__device__ __forceinline__ int kofs(int st, int q) { return MG_GEMM_KPERM ? q * 8 * NST + st * 8 : st * 32 + q * 8; }

template <int MT, int FT>
__device__ __forceinline__ void load_w(const uint16_t* const (&wrow)[FT], const bool (&wok)[FT], int kc, int K, int q,
                                       uint4 (&wr)[GemmShape<MT>::NST][FT]) {
    using S = GemmShape<MT>;
#pragma unroll
    for (int st = 0; st < S::NST; ++st) {
        const int k = kc + kofs<S::NST>(st, q);
#pragma unroll
        for (int f = 0; f < FT; ++f)
            wr[st][f] = (wok[f] && k < K) ? *reinterpret_cast<const uint4*>(wrow[f] + k) : make_uint4(0, 0, 0, 0);
    }
}

template <int MT, int FT, int EPI, bool SWI, int PF>
__global__ __launch_bounds__(256) void fast_gemm_kernel(FastGemmArgs a) {
    using S = GemmShape<MT>;
    __shared__ __attribute__((aligned(16))) unsigned char xs[2][S::ROWS * S::STRIDE];
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int jl = lane & 15, q = lane >> 4;
    const int nb = blockIdx.x, split = blockIdx.y;
    const int FB = 64 * FT;  // features per block
    const int K = a.K, M = a.M;

    const uint16_t* wrow[FT];
    bool wok[FT];
    int nf[FT];
#pragma unroll
    for (int f = 0; f < FT; ++f) {
        const int n0 = nb * FB + (wave * FT + f) * 16;
        nf[f] = n0;
        wok[f] = n0 < a.N;
        int seg = 0, nl = n0;
        while (seg < 2 && nl >= a.Nseg[seg]) { nl -= a.Nseg[seg]; ++seg; }
        wrow[f] = wok[f] ? a.W[seg] + (size_t)(nl + jl) * K : a.W[0];
    }

    const int nchunks = (K + S::KC - 1) / S::KC;
    const int c0 = (int)((long)split * nchunks / a.S);
    const int c1 = (int)((long)(split + 1) * nchunks / a.S);

    f32x4_t acc[MT][FT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int f = 0; f < FT; ++f) acc[mt][f] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    if constexpr (PF == 1) {
        // weights prefetched one chunk ahead (register double buffer)
        uint4 wcur[S::NST][FT], wnext[S::NST][FT];
        uint4 xr[S::XLD];
        if (c0 < c1) {
            load_w<MT, FT>(wrow, wok, c0 * S::KC, K, q, wcur);
            load_x<MT, SWI>(a, c0 * S::KC, xr);
            store_x<MT>(xs[c0 & 1], xr);
        }
        __syncthreads();
        for (int c = c0; c < c1; ++c) {
            const bool more = c + 1 < c1;
            if (more) {
                load_w<MT, FT>(wrow, wok, (c + 1) * S::KC, K, q, wnext);
                load_x<MT, SWI>(a, (c + 1) * S::KC, xr);
            }
            const unsigned char* buf = xs[c & 1];
#pragma unroll
            for (int st = 0; st < S::NST; ++st) {
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    const uint4 av = *reinterpret_cast<const uint4*>(buf + (16 * mt + jl) * S::STRIDE + kofs<S::NST>(st, q) * 2);
                    const bf16x8_t A = __builtin_bit_cast(bf16x8_t, av);
#pragma unroll
                    for (int f = 0; f < FT; ++f)
                        acc[mt][f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                            A, __builtin_bit_cast(bf16x8_t, wcur[st][f]), acc[mt][f], 0, 0, 0);
                }
            }
            if (more) store_x<MT>(xs[(c + 1) & 1], xr);
            __syncthreads();
            if (more) {
#pragma unroll
                for (int st = 0; st < S::NST; ++st)
#pragma unroll
                    for (int f = 0; f < FT; ++f) wcur[st][f] = wnext[st][f];
            }
        }
    } else {
        // weights are prefetched two chunks ahead into three rotating register buffers;
        // the chunk loop is unrolled by three so every buffer index is a constant
        uint4 wb0[S::NST][FT], wb1[S::NST][FT], wb2[S::NST][FT];
        uint4 xr[S::XLD];
        if (c0 < c1) {
            load_w<MT, FT>(wrow, wok, c0 * S::KC, K, q, wb0);
            if (c0 + 1 < c1) load_w<MT, FT>(wrow, wok, (c0 + 1) * S::KC, K, q, wb1);
            load_x<MT, SWI>(a, c0 * S::KC, xr);
            store_x<MT>(xs[c0 & 1], xr);  // chunk c always lives in buffer c & 1
        }
        __syncthreads();
        auto step = [&](int c, uint4 (&cur)[S::NST][FT], uint4 (&far)[S::NST][FT]) {
            if (c + 2 < c1) load_w<MT, FT>(wrow, wok, (c + 2) * S::KC, K, q, far);
            const bool more = c + 1 < c1;
            if (more) load_x<MT, SWI>(a, (c + 1) * S::KC, xr);
            const unsigned char* buf = xs[c & 1];
    #pragma unroll
            for (int st = 0; st < S::NST; ++st) {
    #pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    const uint4 av = *reinterpret_cast<const uint4*>(buf + (16 * mt + jl) * S::STRIDE + kofs<S::NST>(st, q) * 2);
                    const bf16x8_t A = __builtin_bit_cast(bf16x8_t, av);
    #pragma unroll
                    for (int f = 0; f < FT; ++f)
                        acc[mt][f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A, __builtin_bit_cast(bf16x8_t, cur[st][f]),
                                                                              acc[mt][f], 0, 0, 0);
                }
            }
            if (more) store_x<MT>(xs[(c + 1) & 1], xr);
            __syncthreads();
        };
        for (int c = c0; c < c1; c += 3) {
            step(c, wb0, wb2);
            if (c + 1 < c1) step(c + 1, wb1, wb0);
            if (c + 2 < c1) step(c + 2, wb2, wb1);
        }
    }

    // D[i][j] of a 16x16 tile sits in lane j + 16*(i/4), element i%4
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

// Features per wave / 16: two B tiles per wave when the output is wide enough for
// two 128-feature blocks per CU, one otherwise.
static int g_n_cu = 256;
int fast_gemm_ft(int M, int N) {
    (void)M;
#ifndef MG_GEMM_FT2_MIN_N
#define MG_GEMM_FT2_MIN_N 8192
#endif
    return N >= MG_GEMM_FT2_MIN_N ? 2 : 1;
}

int fast_gemm_splits(int M, int N, int K, int n_cu) {
    g_n_cu = n_cu;
    const int KC = gemm_kc(mt_for(M));
    const int nchunks = (K + KC - 1) / KC;
    const int FB = 64 * fast_gemm_ft(M, N);
    const int nb = (N + FB - 1) / FB;
    // enough blocks for about two per CU (four for small batches, whose blocks carry
    // little MFMA work per weight byte), each with at least 4 chunks, and the
    // partial tiles (S*M*N fp32, written once and read once by the consumer) at most
    // a quarter of the weight bytes
    const int target = (M <= 16 ? 4 : 2) * n_cu;
    int S = (target + nb - 1) / nb;
    const int by_chunks = nchunks / 4 > 1 ? nchunks / 4 : 1;
    const long by_traffic = (long)K / (8L * (M < 16 ? 16 : M));
    if (S > by_chunks) S = by_chunks;
    if (S > by_traffic) S = (int)by_traffic;
    if (S > 32) S = 32;
    return S < 1 ? 1 : S;
}

#ifndef MG_GEMM_PF
#define MG_GEMM_PF 1
#endif
template <int MT, int FT, int EPI>
static void launch_epi(const FastGemmArgs& a, dim3 g, hipStream_t s) {
    if (a.swiglu_x)
        hipLaunchKernelGGL((fast_gemm_kernel<MT, FT, EPI, true, MG_GEMM_PF>), g, dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL((fast_gemm_kernel<MT, FT, EPI, false, MG_GEMM_PF>), g, dim3(256), 0, s, a);
}

template <int MT, int FT>
static void launch_ft(const FastGemmArgs& a, int epi, dim3 g, hipStream_t s) {
    switch (epi) {
        case FEPI_BF16: launch_epi<MT, FT, FEPI_BF16>(a, g, s); break;
        case FEPI_PART: launch_epi<MT, FT, FEPI_PART>(a, g, s); break;
        default: launch_epi<MT, FT, FEPI_F32>(a, g, s); break;
    }
}

template <int MT>
static void launch_mt(const FastGemmArgs& a, int epi, int ft, hipStream_t s) {
    dim3 g((a.N + 64 * ft - 1) / (64 * ft), a.S);
    if (ft == 2)
        launch_ft<MT, 2>(a, epi, g, s);
    else
        launch_ft<MT, 1>(a, epi, g, s);
}

hipError_t launch_fast_gemm(const FastGemmArgs& a, int epi, hipStream_t s) {
    if (a.M <= 0 || a.N <= 0) return hipSuccess;
    if (epi != FEPI_PART && a.S != 1) return hipErrorInvalidValue;  // only partial tiles may be split
    const int ft = fast_gemm_ft(a.M, a.N);
    switch (mt_for(a.M)) {
        case 1: launch_mt<1>(a, epi, ft, s); break;
        case 2: launch_mt<2>(a, epi, ft, s); break;
        case 4: launch_mt<4>(a, epi, ft, s); break;
        case 8: launch_mt<8>(a, epi, ft, s); break;
        default: launch_mt<16>(a, epi, ft, s); break;
    }
    return hipGetLastError();
}

}  // namespace mg
