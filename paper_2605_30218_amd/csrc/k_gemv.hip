// k_gemv.hip -- the verifier's canonical GEMV.
//
// y[r][j] = CDOT(x[r], W[j]) for a set of rows r and output features j, where
// CDOT fixes the reduction order independently of how many rows are processed
// and where a row sits in the launch:
//   groups of 8 consecutive K elements; group g belongs to lane g mod 64; each
//   lane fma-accumulates its groups in increasing g (element order inside the
//   group) starting from +0; the 64 lane sums are combined by the xor butterfly
//   over offsets 32, 16, 8, 4, 2, 1.
// A wave owns J features; a block of 4 waves owns 4J features and a tile of R
// rows.  The K dimension is walked in chunks of 512 elements (one group per
// lane): the block stages the chunk of its R rows in LDS as fp32, every wave
// streams one 16-byte weight group per feature and lane (1 KiB coalesced per
// feature) and applies it to all R rows.  No split-K, no atomics: a row's
// arithmetic is the same whatever R, J, the tile or the row count.
#include "mg_device.h"
#include "mg_kernels.h"

namespace mg {

constexpr int KCH = 512;  // K elements per chunk (64 lanes x 8)

template <int J, int R, int EPI>
__global__ __launch_bounds__(256) void canon_gemv_kernel(GemvArgs a) {
    RowCount rc{a.n_dev, a.n_host, a.cap};
    const int n = rc.get();
    const int r0 = blockIdx.x * R;
    if (r0 >= n) return;
    const int nr = min(R, n - r0);
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int jw = (blockIdx.y * 4 + wave) * J;
    const int K = a.K, G = K >> 3;

    // LDS chunk: element 8*lane + 4*half + c of row rr at xs[rr][half][lane].c
    __shared__ float4 xs[R][2][64];

    const uint16_t* wrow[J];
    bool valid[J];
#pragma unroll
    for (int jj = 0; jj < J; ++jj) {
        int j = jw + jj;
        valid[jj] = j < a.N;
        int seg = 0;
        while (seg < 2 && j >= a.Nseg[seg]) { j -= a.Nseg[seg]; ++seg; }
        wrow[jj] = valid[jj] ? a.W[seg] + (size_t)j * K : a.W[0];
    }

    float acc[J][R];
#pragma unroll
    for (int jj = 0; jj < J; ++jj)
#pragma unroll
        for (int rr = 0; rr < R; ++rr) acc[jj][rr] = 0.0f;

    for (int kc = 0; kc < K; kc += KCH) {
        __syncthreads();
        for (int t = threadIdx.x; t < R * 64; t += 256) {
            const int rr = t >> 6, gl = t & 63;
            const int k = kc + gl * 8;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (rr < nr && k < K) v = *reinterpret_cast<const uint4*>(a.X + (size_t)(r0 + rr) * K + k);
            xs[rr][0][gl] = make_float4(bf_lo(v.x), bf_hi(v.x), bf_lo(v.y), bf_hi(v.y));
            xs[rr][1][gl] = make_float4(bf_lo(v.z), bf_hi(v.z), bf_lo(v.w), bf_hi(v.w));
        }
        __syncthreads();
        const int g = (kc >> 3) + lane;
        if (g < G) {
            float w[J][8];
#pragma unroll
            for (int jj = 0; jj < J; ++jj) {
                uint4 v = make_uint4(0, 0, 0, 0);
                if (valid[jj]) v = *reinterpret_cast<const uint4*>(wrow[jj] + (size_t)g * 8);
                w[jj][0] = bf_lo(v.x); w[jj][1] = bf_hi(v.x); w[jj][2] = bf_lo(v.y); w[jj][3] = bf_hi(v.y);
                w[jj][4] = bf_lo(v.z); w[jj][5] = bf_hi(v.z); w[jj][6] = bf_lo(v.w); w[jj][7] = bf_hi(v.w);
            }
#pragma unroll
            for (int rr = 0; rr < R; ++rr) {
                if (rr >= nr) break;
                const float4 x0 = xs[rr][0][lane], x1 = xs[rr][1][lane];
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

    // butterfly, then lane (jj*R + rr) % 64 writes result (jj, rr); every lane holds it
#pragma unroll
    for (int jj = 0; jj < J; ++jj) {
#pragma unroll
        for (int rr = 0; rr < R; ++rr) {
            const float v = butterfly_sum(acc[jj][rr]);
            if (lane != ((jj * R + rr) & 63) || rr >= nr || !valid[jj]) continue;
            const int j = jw + jj, row = r0 + rr;
            if (EPI == EPI_F32) {
                reinterpret_cast<float*>(a.Y)[(size_t)row * a.N + j] = v;
            } else if (EPI == EPI_BF16) {
                int jl = j, seg = 0;
                while (seg < 2 && jl >= a.Nseg[seg]) { jl -= a.Nseg[seg]; ++seg; }
                const float y = a.bias[seg] ? v + bf2f(a.bias[seg][jl]) : v;
                reinterpret_cast<uint16_t*>(a.Y)[(size_t)row * a.N + j] = (uint16_t)f2bf(y);
            } else {  // residual: x = bf16(x + bf16(y))
                uint16_t* xr = reinterpret_cast<uint16_t*>(a.Y) + (size_t)row * a.N + j;
                const float y = bf2f(f2bf(v));
                *xr = (uint16_t)f2bf(bf2f(*xr) + y);
            }
        }
    }
}

template <int J, int R>
static hipError_t launch_jr(const GemvArgs& a, int epi, int rows, hipStream_t s) {
    dim3 grid((rows + R - 1) / R, (a.N + 4 * J - 1) / (4 * J));
    switch (epi) {
        case EPI_BF16: hipLaunchKernelGGL((canon_gemv_kernel<J, R, EPI_BF16>), grid, dim3(256), 0, s, a); break;
        case EPI_RESID: hipLaunchKernelGGL((canon_gemv_kernel<J, R, EPI_RESID>), grid, dim3(256), 0, s, a); break;
        default: hipLaunchKernelGGL((canon_gemv_kernel<J, R, EPI_F32>), grid, dim3(256), 0, s, a); break;
    }
    return hipGetLastError();
}

hipError_t launch_canon_gemv(const GemvArgs& a, int epi, hipStream_t s) {
    const int rows = a.n_dev ? a.cap : a.n_host;
    if (rows <= 0 || a.N <= 0) return hipSuccess;
    if (rows <= 8) return launch_jr<4, 8>(a, epi, rows, s);
    return launch_jr<4, 16>(a, epi, rows, s);
}

}  // namespace mg
