// k_gemm.hip -- the fast path's weight-streaming projection on MFMA (gfx950).
//
// Y[M][N] = X[M][K] * W[N][K]^T with v_mfma_f32_16x16x32_bf16.  A block of 4
// waves owns 64 output features; each wave owns 16 of them for all M rows
// (M <= 256, padded to 16-row tiles).  Weights are read straight from HBM into
// the MFMA B-operand registers: lane (j, q) loads the 16 bytes
// W[n+j][k+8q .. k+8q+7], so a 32-wide k step of 16 features is 16 rows x 64
// contiguous bytes.  Activations are staged per K chunk in LDS (rows padded by
// 16 bytes so the 16 A-operand lanes of a k group hit distinct banks).  The K
// range may be split across blocks (split-K); partial tiles go to a workspace
// and the last block of a feature tile to arrive sums them in split order, so
// the result is deterministic for a given shape.  The summation order depends on
// M (through the chunk size) and on the split count: this path is allowed to be
// batch-variant.
#include "mg_device.h"
#include "mg_kernels.h"

namespace mg {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

template <int MT>
struct GemmShape {
    static constexpr int KC = MT <= 4 ? 256 : 128;  // K per chunk
    static constexpr int ROWS = 16 * MT;
    static constexpr int STRIDE = KC * 2 + 16;      // LDS bytes per staged row
    static constexpr int NST = KC / 32;             // MFMA k-steps per chunk
};

template <int EPI>
__device__ __forceinline__ void fast_epilogue(const FastGemmArgs& a, int row, int n, float v) {
    if (EPI == FEPI_F32) {
        reinterpret_cast<float*>(a.Y)[(size_t)row * a.N + n] = v;
    } else if (EPI == FEPI_BF16) {
        int nl = n, seg = 0;
        while (seg < 2 && nl >= a.Nseg[seg]) { nl -= a.Nseg[seg]; ++seg; }
        const float y = a.bias[seg] ? v + bf2f(a.bias[seg][nl]) : v;
        reinterpret_cast<uint16_t*>(a.Y)[(size_t)row * a.N + n] = (uint16_t)f2bf(y);
    } else {
        uint16_t* xr = reinterpret_cast<uint16_t*>(a.Y) + (size_t)row * a.N + n;
        *xr = (uint16_t)f2bf(bf2f(*xr) + bf2f(f2bf(v)));
    }
}

__device__ __forceinline__ float silu_fast(float g) { return g / (1.0f + __expf(-g)); }

template <int MT, int EPI, bool SWI>
__global__ __launch_bounds__(256) void fast_gemm_kernel(FastGemmArgs a) {
    using S = GemmShape<MT>;
    __shared__ __attribute__((aligned(16))) unsigned char xs[S::ROWS * S::STRIDE];
    __shared__ int s_last;
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int jl = lane & 15, q = lane >> 4;
    const int nb = blockIdx.x, split = blockIdx.y;
    const int n_w = nb * 64 + wave * 16;
    const bool wvalid = n_w < a.N;
    const int K = a.K, M = a.M;

    int seg = 0, nloc = n_w;
    while (seg < 2 && nloc >= a.Nseg[seg]) { nloc -= a.Nseg[seg]; ++seg; }
    const uint16_t* wrow = wvalid ? a.W[seg] + (size_t)(nloc + jl) * K : a.W[0];

    const int nchunks = (K + S::KC - 1) / S::KC;
    const int c0 = (int)((long)split * nchunks / a.S);
    const int c1 = (int)((long)(split + 1) * nchunks / a.S);

    f32x4_t acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    for (int c = c0; c < c1; ++c) {
        const int kc = c * S::KC;
        uint4 wr[S::NST];
#pragma unroll
        for (int st = 0; st < S::NST; ++st) {
            const int k = kc + st * 32 + q * 8;
            wr[st] = (wvalid && k < K) ? *reinterpret_cast<const uint4*>(wrow + k) : make_uint4(0, 0, 0, 0);
        }
        __syncthreads();
        constexpr int GPR = S::KC / 8;  // 16-byte groups per staged row
        for (int t = threadIdx.x; t < S::ROWS * GPR; t += 256) {
            const int row = t / GPR, g = t % GPR;
            const int k = kc + g * 8;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (row < M && k < K) {
                if (!SWI) {
                    v = *reinterpret_cast<const uint4*>(a.X + (size_t)row * K + k);
                } else {
                    const uint4 gv = *reinterpret_cast<const uint4*>(a.X + (size_t)row * 2 * K + k);
                    const uint4 uv = *reinterpret_cast<const uint4*>(a.X + (size_t)row * 2 * K + K + k);
                    v.x = pack_bf2(silu_fast(bf_lo(gv.x)) * bf_lo(uv.x), silu_fast(bf_hi(gv.x)) * bf_hi(uv.x));
                    v.y = pack_bf2(silu_fast(bf_lo(gv.y)) * bf_lo(uv.y), silu_fast(bf_hi(gv.y)) * bf_hi(uv.y));
                    v.z = pack_bf2(silu_fast(bf_lo(gv.z)) * bf_lo(uv.z), silu_fast(bf_hi(gv.z)) * bf_hi(uv.z));
                    v.w = pack_bf2(silu_fast(bf_lo(gv.w)) * bf_lo(uv.w), silu_fast(bf_hi(gv.w)) * bf_hi(uv.w));
                }
            }
            *reinterpret_cast<uint4*>(xs + row * S::STRIDE + g * 16) = v;
        }
        __syncthreads();
#pragma unroll
        for (int st = 0; st < S::NST; ++st) {
            const bf16x8_t bv = __builtin_bit_cast(bf16x8_t, wr[st]);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const uint4 av = *reinterpret_cast<const uint4*>(xs + (16 * mt + jl) * S::STRIDE + (st * 32 + q * 8) * 2);
                acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, av), bv, acc[mt], 0, 0, 0);
            }
        }
    }

    // D[i][j] of a 16x16 tile sits in lane j + 16*(i/4), element i%4
    if (a.S == 1) {
        if (!wvalid) return;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int row = 16 * mt + 4 * q + v;
                if (row < M) fast_epilogue<EPI>(a, row, n_w + jl, acc[mt][v]);
            }
        return;
    }
    if (wvalid) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int row = 16 * mt + 4 * q + v;
                if (row < M) a.part[((size_t)split * M + row) * a.N + n_w + jl] = acc[mt][v];
            }
    }
    __threadfence();
    __syncthreads();
    if (threadIdx.x == 0) s_last = (atomicAdd(a.tickets + nb, 1) == a.S - 1);
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    for (int t = threadIdx.x; t < M * 64; t += 256) {
        const int row = t >> 6, n = nb * 64 + (t & 63);
        if (n >= a.N) continue;
        float sum = 0.0f;
        for (int sp = 0; sp < a.S; ++sp)
            sum += __hip_atomic_load(a.part + ((size_t)sp * M + row) * a.N + n, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        fast_epilogue<EPI>(a, row, n, sum);
    }
    if (threadIdx.x == 0) __hip_atomic_store(a.tickets + nb, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

static int mt_for(int M) {
    const int t = (M + 15) / 16;
    return t <= 1 ? 1 : t <= 2 ? 2 : t <= 4 ? 4 : t <= 8 ? 8 : 16;
}

int fast_gemm_splits(int M, int N, int K, int n_cu) {
    const int KC = mt_for(M) <= 4 ? 256 : 128;
    const int nchunks = (K + KC - 1) / KC;
    const int nb = (N + 63) / 64;
    int want = (4 * n_cu + nb - 1) / nb;
    int maxs = nchunks / 2 > 1 ? nchunks / 2 : 1;
    if (want > maxs) want = maxs;
    if (want > 32) want = 32;
    return want < 1 ? 1 : want;
}

template <int MT, int EPI>
static void launch_mt_epi(const FastGemmArgs& a, dim3 g, hipStream_t s) {
    if (a.swiglu_x)
        hipLaunchKernelGGL((fast_gemm_kernel<MT, EPI, true>), g, dim3(256), 0, s, a);
    else
        hipLaunchKernelGGL((fast_gemm_kernel<MT, EPI, false>), g, dim3(256), 0, s, a);
}

template <int MT>
static void launch_mt(const FastGemmArgs& a, int epi, dim3 g, hipStream_t s) {
    switch (epi) {
        case FEPI_BF16: launch_mt_epi<MT, FEPI_BF16>(a, g, s); break;
        case FEPI_RESID: launch_mt_epi<MT, FEPI_RESID>(a, g, s); break;
        default: launch_mt_epi<MT, FEPI_F32>(a, g, s); break;
    }
}

hipError_t launch_fast_gemm(const FastGemmArgs& a, int epi, hipStream_t s) {
    if (a.M <= 0 || a.N <= 0) return hipSuccess;
    dim3 g((a.N + 63) / 64, a.S);
    switch (mt_for(a.M)) {
        case 1: launch_mt<1>(a, epi, g, s); break;
        case 2: launch_mt<2>(a, epi, g, s); break;
        case 4: launch_mt<4>(a, epi, g, s); break;
        case 8: launch_mt<8>(a, epi, g, s); break;
        default: launch_mt<16>(a, epi, g, s); break;
    }
    return hipGetLastError();
}

}  // namespace mg
