// k_misc.hip -- embedding gather, RMSNorm, RoPE + K/V placement, SwiGLU, the
// top-1/top-2 margin gate, the K/V column repair, step bookkeeping, numerics probes.
#include "mg_device.h"
#include "mg_kernels.h"
#include "../../include/mg.h"

namespace mg {

// ------------------------------------------------------------------ embedding
// x[i][:] = embed[token of item i][:]
__global__ __launch_bounds__(256) void embed_kernel(Items it, const uint16_t* __restrict__ E, int d,
                                                    uint16_t* __restrict__ x) {
    const int i = blockIdx.x;
    if (i >= items_n(it)) return;
    const int tok = items_tok(it, i);
    const uint4* src = reinterpret_cast<const uint4*>(E + (size_t)tok * d);
    uint4* dst = reinterpret_cast<uint4*>(x + (size_t)i * d);
    for (int t = threadIdx.x; t < d / 8; t += blockDim.x) dst[t] = src[t];
}

hipError_t launch_embed(const Items& it, const uint16_t* embed, int d, uint16_t* x, hipStream_t s) {
    if (it.n_host <= 0) return hipSuccess;
    hipLaunchKernelGGL(embed_kernel, dim3(it.n_host), dim3(256), 0, s, it, embed, d, x);
    return hipGetLastError();
}

// ------------------------------------------------------------------ RMSNorm
// One wave per row.  ss = CDOT(x, x) (lane l owns groups l, l+64, ...; fma in
// element order; xor butterfly), m = ss / d, r = 1 / sqrt(m + eps),
// y_i = bf16((x_i * r) * gamma_i).  Used by both paths (it is batch-invariant).
constexpr int RMS_MAXG = 16;  // groups of 8 per lane: d <= 8192

__global__ __launch_bounds__(256) void rmsnorm_kernel(const uint16_t* __restrict__ x, const uint16_t* __restrict__ g,
                                                      RowCount rc, int d, float eps, uint16_t* __restrict__ y) {
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int row = blockIdx.x * 4 + wave;
    if (row >= rc.get()) return;
    const uint4* xr = reinterpret_cast<const uint4*>(x + (size_t)row * d);
    const int G = d >> 3;
    // the lane's groups lane, lane+64, ... are loaded together and kept in registers
    // gamma is requested with x, so the block waits for memory once
    const uint4* gr = reinterpret_cast<const uint4*>(g);
    uint4 xv[RMS_MAXG], gv[RMS_MAXG];
#pragma unroll
    for (int k = 0; k < RMS_MAXG; ++k) {
        const int gi = lane + 64 * k;
        xv[k] = gi < G ? xr[gi] : make_uint4(0, 0, 0, 0);
        gv[k] = gi < G ? gr[gi] : make_uint4(0, 0, 0, 0);
    }
    float a = 0.0f;
#pragma unroll
    for (int k = 0; k < RMS_MAXG; ++k) {
        if (lane + 64 * k < G) {
            const uint4 v = xv[k];
            const float e[8] = {bf_lo(v.x), bf_hi(v.x), bf_lo(v.y), bf_hi(v.y),
                                bf_lo(v.z), bf_hi(v.z), bf_lo(v.w), bf_hi(v.w)};
#pragma unroll
            for (int i = 0; i < 8; ++i) a = __builtin_fmaf(e[i], e[i], a);
        }
    }
    const float ss = butterfly_sum(a);
    const float m = ieee_div(ss, (float)d);
    const float r = ieee_div(1.0f, ieee_sqrt(m + eps));
    uint4* yr = reinterpret_cast<uint4*>(y + (size_t)row * d);
#pragma unroll
    for (int k = 0; k < RMS_MAXG; ++k) {
        const int gi = lane + 64 * k;
        if (gi < G) {
            const uint4 v = xv[k], w = gv[k];
            uint4 o;
            o.x = pack_bf2((bf_lo(v.x) * r) * bf_lo(w.x), (bf_hi(v.x) * r) * bf_hi(w.x));
            o.y = pack_bf2((bf_lo(v.y) * r) * bf_lo(w.y), (bf_hi(v.y) * r) * bf_hi(w.y));
            o.z = pack_bf2((bf_lo(v.z) * r) * bf_lo(w.z), (bf_hi(v.z) * r) * bf_hi(w.z));
            o.w = pack_bf2((bf_lo(v.w) * r) * bf_lo(w.w), (bf_hi(v.w) * r) * bf_hi(w.w));
            yr[gi] = o;
        }
    }
}

hipError_t launch_rmsnorm(const uint16_t* x, const uint16_t* gamma, int n_host, const int32_t* n_dev, int cap, int d,
                          float eps, uint16_t* y, hipStream_t s) {
    const int rows = n_dev ? cap : n_host;
    if (rows <= 0) return hipSuccess;
    if (d % 8 || d / 8 > 64 * RMS_MAXG) return hipErrorInvalidValue;
    RowCount rc{n_dev, n_host, cap};
    hipLaunchKernelGGL(rmsnorm_kernel, dim3((rows + 3) / 4), dim3(256), 0, s, x, gamma, rc, d, eps, y);
    return hipGetLastError();
}

// ------------------------------------------------------------------ RoPE + K/V placement
// Rotate-half RoPE: pair (i, i + hd/2) of every q and k head is rotated by the
// angle pos * theta^(-2i/hd), using the fp32 cos/sin table built on the host in
// float64.  q'_i = bf16(q_i c - q_(i+h) s), q'_(i+h) = bf16(q_(i+h) c + q_i s),
// products and sums separately rounded.  K' and V go to the verifier's own column
// (kv_col != NULL) or into the paged cache at the item's position.
__global__ __launch_bounds__(256) void rope_kv_kernel(Items it, ModelDims m, int layer, const uint16_t* __restrict__ qkv,
                                                      const float* __restrict__ cs, uint16_t* __restrict__ qrot,
                                                      uint16_t* __restrict__ kv_pool, uint16_t* __restrict__ kv_col) {
    const int i = blockIdx.x;
    if (i >= items_n(it)) return;
    const int r = items_row(it, i);
    const int pos = items_pos(it, i);
    const int hd = m.hd, h2 = hd / 2, Nq = m.Hq * hd, Nk = m.Hkv * hd;
    const uint16_t* src = qkv + (size_t)i * (Nq + 2 * Nk);
    const float* csp = cs + (size_t)pos * hd;  // [pos][i][cos, sin]
    uint16_t *kdst, *vdst;
    if (kv_col) {
        kdst = kv_col + ((size_t)i * m.L + layer) * 2 * Nk;
        vdst = kdst + Nk;
    } else {
        const int page = it.page_table[(size_t)r * m.max_pages_per_row + pos / m.page_size];
        const int slot = pos % m.page_size;
        // [layer][page][K|V][Hkv][page_size][hd]: head kh's row is at +kh*page_size*hd
        kdst = kv_pool + (((size_t)layer * m.n_pages + page) * 2) * (size_t)Nk * m.page_size + (size_t)slot * hd;
        vdst = kdst + (size_t)Nk * m.page_size;
    }
    const int kv_head_stride = kv_col ? hd : hd * m.page_size;
    // task = 8 consecutive pairs (i, i + hd/2) of one q or k head, or 8 values of v;
    // each thread's tasks are loaded together before any arithmetic
    const int gph = h2 / 8;                       // pair groups per head
    const int n_rot = (m.Hq + m.Hkv) * gph, n_v = Nk / 8;
    constexpr int TPT = 4;                        // tasks per thread per round
    for (int t0 = 0; t0 < n_rot + n_v; t0 += 256 * TPT) {
        uint4 lo[TPT], hi[TPT];
        float4 c4[TPT][4];
#pragma unroll
        for (int u = 0; u < TPT; ++u) {
            const int t = t0 + threadIdx.x + 256 * u;
            if (t < n_rot) {
                const int head = t / gph, ii = (t % gph) * 8;
                const uint16_t* sh = head < m.Hq ? src + head * hd : src + Nq + (head - m.Hq) * hd;
                lo[u] = *reinterpret_cast<const uint4*>(sh + ii);
                hi[u] = *reinterpret_cast<const uint4*>(sh + ii + h2);
#pragma unroll
                for (int q = 0; q < 4; ++q) c4[u][q] = *reinterpret_cast<const float4*>(csp + 2 * ii + 4 * q);
            } else if (t < n_rot + n_v) {
                lo[u] = *reinterpret_cast<const uint4*>(src + Nq + Nk + (t - n_rot) * 8);
            }
        }
#pragma unroll
        for (int u = 0; u < TPT; ++u) {
            const int t = t0 + threadIdx.x + 256 * u;
            if (t < n_rot) {
                const int head = t / gph, ii = (t % gph) * 8;
                const float a[8] = {bf_lo(lo[u].x), bf_hi(lo[u].x), bf_lo(lo[u].y), bf_hi(lo[u].y),
                                    bf_lo(lo[u].z), bf_hi(lo[u].z), bf_lo(lo[u].w), bf_hi(lo[u].w)};
                const float b[8] = {bf_lo(hi[u].x), bf_hi(hi[u].x), bf_lo(hi[u].y), bf_hi(hi[u].y),
                                    bf_lo(hi[u].z), bf_hi(hi[u].z), bf_lo(hi[u].w), bf_hi(hi[u].w)};
                const float cc[16] = {c4[u][0].x, c4[u][0].y, c4[u][0].z, c4[u][0].w, c4[u][1].x, c4[u][1].y,
                                      c4[u][1].z, c4[u][1].w, c4[u][2].x, c4[u][2].y, c4[u][2].z, c4[u][2].w,
                                      c4[u][3].x, c4[u][3].y, c4[u][3].z, c4[u][3].w};
                uint32_t o1[8], o2[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float c = cc[2 * e], sn = cc[2 * e + 1];
                    const float ac = a[e] * c, bs = b[e] * sn, bc = b[e] * c, as = a[e] * sn;
                    o1[e] = f2bf(ac - bs);
                    o2[e] = f2bf(bc + as);
                }
                const uint4 w1 = make_uint4(o1[0] | (o1[1] << 16), o1[2] | (o1[3] << 16), o1[4] | (o1[5] << 16),
                                            o1[6] | (o1[7] << 16));
                const uint4 w2 = make_uint4(o2[0] | (o2[1] << 16), o2[2] | (o2[3] << 16), o2[4] | (o2[5] << 16),
                                            o2[6] | (o2[7] << 16));
                uint16_t* dst = head < m.Hq ? qrot + (size_t)i * Nq + head * hd
                                            : kdst + (size_t)(head - m.Hq) * kv_head_stride;
                *reinterpret_cast<uint4*>(dst + ii) = w1;
                *reinterpret_cast<uint4*>(dst + ii + h2) = w2;
            } else if (t < n_rot + n_v) {
                const int e = (t - n_rot) * 8, head = e / hd, dd = e % hd;
                *reinterpret_cast<uint4*>(vdst + (size_t)head * kv_head_stride + dd) = lo[u];
            }
        }
    }
}

hipError_t launch_rope_kv(const Items& it, const ModelDims& m, int layer, const uint16_t* qkv, const float* rope_cs,
                          uint16_t* qrot, uint16_t* kv_pool, uint16_t* kv_col, hipStream_t s) {
    if (it.n_host <= 0) return hipSuccess;
    hipLaunchKernelGGL(rope_kv_kernel, dim3(it.n_host), dim3(256), 0, s, it, m, layer, qkv, rope_cs, qrot, kv_pool,
                       kv_col);
    return hipGetLastError();
}

// ------------------------------------------------------------------ top-1 / top-2
constexpr int TOP2_MAX_SLICES = 128;

// Stage 1: block (s, b) scans slice s of row b (16-byte loads), merges its lanes by
// wave shuffles and its waves through LDS, and stores the slice's state.
__global__ __launch_bounds__(256) void top2_slice_kernel(int B, int V, int slice, const float* __restrict__ logits,
                                                         Top2* __restrict__ part, int nsl, const int32_t* n_dev) {
    const int s = blockIdx.x, b = blockIdx.y;
    const int nrows = n_dev ? min(max(*n_dev, 0), B) : B;
    if (b >= nrows) return;
    const float* row = logits + (size_t)b * V;
    const int j0 = s * slice, j1 = min(j0 + slice, V);
    Top2 st{-__builtin_inff(), -__builtin_inff(), -1, 0};
    const int t = threadIdx.x;
    if ((V & 3) == 0) {  // slice is a multiple of 4, so are j0 and j1
        const float4* r4 = reinterpret_cast<const float4*>(row);
        for (int q = j0 / 4 + t; q < j1 / 4; q += 256) {
            const float4 v = r4[q];
            top2_push(st, v.x, 4 * q);
            top2_push(st, v.y, 4 * q + 1);
            top2_push(st, v.z, 4 * q + 2);
            top2_push(st, v.w, 4 * q + 3);
        }
    } else {
        for (int q = j0 + t; q < j1; q += 256) top2_push(st, row[q], q);
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) st = top2_merge(st, top2_shfl(st, o));
    __shared__ Top2 ws[4];
    if ((t & 63) == 0) ws[t >> 6] = st;
    __syncthreads();
    if (t == 0) part[(size_t)b * nsl + s] = top2_merge(top2_merge(ws[0], ws[1]), top2_merge(ws[2], ws[3]));
}

// Stage 2: one block of 1024 threads.  Row b's nsl slice states sit in nsl/2
// consecutive threads (2 states each, nsl a power of two, B * nsl <= 2048), merged
// by xor shuffles inside that lane group; then top1 / margin / gate, and the gated
// rows compacted in increasing order with per-wave ballots.
__global__ __launch_bounds__(1024) void top2_final_kernel(int B, const Top2* __restrict__ part, int nsl,
                                                          const uint8_t* __restrict__ prot, float tau, int32_t* top1,
                                                          float* margin, uint8_t* gate, int32_t* gated_rows,
                                                          int32_t* n_gated, int32_t* n_gated_host,
                                                          const int32_t* n_dev) {
    const int nrows = n_dev ? min(max(*n_dev, 0), B) : B;
    const int t = threadIdx.x;
    const int tpr = nsl / 2;            // threads per row (power of two, <= 64)
    const int b = t / tpr;
    const bool live = b < nrows;
    Top2 st{-__builtin_inff(), -__builtin_inff(), -1, 0};
    if (live) st = top2_merge(part[(size_t)b * nsl + 2 * (t % tpr)], part[(size_t)b * nsl + 2 * (t % tpr) + 1]);
    for (int o = 1; o < tpr; o <<= 1) st = top2_merge(st, top2_shfl(st, o));
    __shared__ uint8_t fire_s[256];
    __shared__ int wave_cnt[4];
    if (t % tpr == 0 && b < B) {
        int fire = 0;
        if (live) {
            const int i1 = st.i1 < 0 ? 0 : st.i1;
            const float g = st.nan ? __builtin_nanf("") : st.v1 - st.v2;
            top1[b] = i1;
            if (margin) margin[b] = g;
            if (gate) {
                const int p = prot ? (prot[b] != 0) : 1;
                fire = p && !(g >= tau);
                gate[b] = (uint8_t)fire;
            }
        }
        fire_s[b] = (uint8_t)fire;
    }
    if (!gated_rows) return;
    __syncthreads();  // fire_s complete
    // rows 0..255 -> waves 0..3 of 64 rows: ballot, then prefix over the waves
    const int w = t >> 6, l = t & 63;
    const int f = (t < nrows) ? fire_s[t] : 0;  // t < 256 whenever t < nrows
    const unsigned long long bal = __ballot(f);
    if (w < 4 && l == 0) wave_cnt[w] = __popcll(bal);
    __syncthreads();
    if (w < 4) {
        int base = 0;
        for (int k = 0; k < w; ++k) base += wave_cnt[k];
        if (f) gated_rows[base + __popcll(bal & ((1ull << l) - 1ull))] = t;
        if (t == 0) {
            const int cnt = wave_cnt[0] + wave_cnt[1] + wave_cnt[2] + wave_cnt[3];
            *n_gated = cnt;
            // mirror for a host that polls pinned memory (a system-scope release store; the
            // device-side consumers of the rows are ordered by the stream)
            if (n_gated_host) __hip_atomic_store(n_gated_host, cnt, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
        }
    }
}

int top2_slices(int B, int V) {
    int nsl = 2;
    while (nsl * 2 <= TOP2_MAX_SLICES && (nsl * 2) * (B > 0 ? B : 1) <= 2048 && (V + nsl * 2 - 1) / (nsl * 2) >= 1024)
        nsl *= 2;
    return nsl;
}

size_t top2_ws_bytes(int B, int V) {
    return B <= 0 ? 0 : (size_t)top2_slices(B, V) * B * sizeof(Top2);
}

hipError_t launch_top2(int B, int V, const float* logits, const uint8_t* prot, float tau, int32_t* top1, float* margin,
                       uint8_t* gate, int32_t* gated_rows, int32_t* n_gated, int32_t* n_gated_host, void* part_ws,
                       const int32_t* n_dev, hipStream_t s) {
    if (B <= 0) return hipSuccess;
    if (B > 256) return hipErrorInvalidValue;
    const int nsl = top2_slices(B, V);
    int slice = (V + nsl - 1) / nsl;
    slice = (slice + 3) & ~3;
    Top2* part = static_cast<Top2*>(part_ws);
    hipLaunchKernelGGL(top2_slice_kernel, dim3(nsl, B), dim3(256), 0, s, B, V, slice, logits, part, nsl, n_dev);
    hipLaunchKernelGGL(top2_final_kernel, dim3(1), dim3(1024), 0, s, B, part, nsl, prot, tau, top1, margin, gate,
                       gated_rows, n_gated, n_gated_host, n_dev);
    return hipGetLastError();
}

// ------------------------------------------------------------------ single-column repair
// One block per listed row.  The decision is taken once (v_tok vs top1, read
// before anything is written, so emitted may alias top1); on a mismatch the
// verifier column [L][K|V][Hkv][hd] is copied to the row's current position in
// every layer, then emitted and the repair counter are updated.
__global__ void gather_rows_kernel(int n, const int32_t* __restrict__ rows, const int32_t* __restrict__ tokens,
                                   const int32_t* __restrict__ positions, const int32_t* __restrict__ page_table,
                                   int maxp, int32_t* __restrict__ out_tok, int32_t* __restrict__ out_pos,
                                   int32_t* __restrict__ out_pt) {
    const int i = blockIdx.x;
    if (i >= n) return;
    const int r = rows[i];
    if (threadIdx.x == 0) {
        out_tok[i] = tokens[r];
        out_pos[i] = positions[r];
    }
    for (int k = threadIdx.x; k < maxp; k += blockDim.x) out_pt[(size_t)i * maxp + k] = page_table[(size_t)r * maxp + k];
}

hipError_t launch_gather_rows(int n, const int32_t* rows, const int32_t* tokens, const int32_t* positions,
                              const int32_t* page_table, int maxp, int32_t* out_tok, int32_t* out_pos, int32_t* out_pt,
                              hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(gather_rows_kernel, dim3(n), dim3(256), 0, s, n, rows, tokens, positions, page_table, maxp,
                       out_tok, out_pos, out_pt);
    return hipGetLastError();
}

__global__ __launch_bounds__(256) void repair_kernel(RowCount rc, const int32_t* __restrict__ rows,
                                                     const int32_t* __restrict__ positions,
                                                     const int32_t* __restrict__ page_table, const int32_t* top1,
                                                     const int32_t* __restrict__ v_tok,
                                                     const uint16_t* __restrict__ v_kvcol, ModelDims m,
                                                     uint16_t* __restrict__ kv_pool, int32_t* emitted,
                                                     int32_t* n_repaired, int action) {
    const int i = blockIdx.x;
    if (i >= rc.get()) return;
    __shared__ int decide[2];
    const int r = rows[i];
    if (threadIdx.x == 0) {
        decide[0] = v_tok[i];
        // the method copies on a disagreement; the variants never copy (token only) or
        // always copy
        decide[1] = action == MG_REPAIR_COPY_ALWAYS ? 1 : action == MG_REPAIR_TOKEN_ONLY ? 0 : (v_tok[i] != top1[r]);
    }
    __syncthreads();
    const int vt = decide[0];
    if (decide[1]) {
        const int pos = positions[r];
        const int page = page_table[(size_t)r * m.max_pages_per_row + pos / m.page_size];
        const int slot = pos % m.page_size;
        const int hd = m.hd, per_head = hd / 8;  // uint4 per head row
        const int segs = m.L * 2 * m.Hkv;
        const uint4* src = reinterpret_cast<const uint4*>(v_kvcol + (size_t)i * segs * hd);
        for (int t = threadIdx.x; t < segs * per_head; t += blockDim.x) {
            const int seg = t / per_head, u = t % per_head;
            const int layer = seg / (2 * m.Hkv), kv = (seg / m.Hkv) % 2, kh = seg % m.Hkv;
            uint16_t* dst = kv_pool + ((((size_t)layer * m.n_pages + page) * 2 + kv) * m.Hkv + kh) * (size_t)m.page_size * hd +
                            (size_t)slot * hd;
            reinterpret_cast<uint4*>(dst)[u] = src[t];
        }
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        emitted[r] = vt;
        if (decide[1]) atomicAdd(n_repaired, 1);
    }
}

hipError_t launch_repair(int n_host, const int32_t* n_dev, int cap, const int32_t* rows, const int32_t* positions,
                         const int32_t* page_table, const int32_t* top1, const int32_t* v_tok, const uint16_t* v_kvcol,
                         const ModelDims& m, uint16_t* kv_pool, int32_t* emitted, int32_t* n_repaired, int action, hipStream_t s) {
    const int grid = n_dev ? cap : n_host;
    if (grid <= 0) return hipSuccess;
    RowCount rc{n_dev, n_host, cap};
    hipLaunchKernelGGL(repair_kernel, dim3(grid), dim3(256), 0, s, rc, rows, positions, page_table, top1, v_tok,
                       v_kvcol, m, kv_pool, emitted, n_repaired, action);
    return hipGetLastError();
}

// ------------------------------------------------------------------ bookkeeping
__global__ void advance_kernel(int B, const int32_t* __restrict__ emitted, int32_t* tokens, int32_t* positions) {
    const int b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b < B) {
        tokens[b] = emitted[b];
        positions[b] += 1;
    }
}

hipError_t launch_advance(int B, const int32_t* emitted, int32_t* tokens, int32_t* positions, hipStream_t s) {
    if (B <= 0) return hipSuccess;
    hipLaunchKernelGGL(advance_kernel, dim3((B + 255) / 256), dim3(256), 0, s, B, emitted, tokens, positions);
    return hipGetLastError();
}

// ------------------------------------------------------------------ numerics probes
__global__ void probe_bf16_kernel(int64_t n, const float* in, uint16_t* out) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        out[i] = (uint16_t)f2bf(in[i]);
}
__global__ void probe_exp_kernel(int64_t n, const float* in, float* out) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
        out[i] = canon_exp(in[i]);
}
__global__ void probe_divsqrt_kernel(int64_t n, const float* a, const float* b, float* q, float* r) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
        q[i] = ieee_div(a[i], b[i]);
        r[i] = ieee_sqrt(a[i]);
    }
}

// plain 16-byte copy: reads and writes n16 * 16 bytes once (counter calibration)
__global__ __launch_bounds__(256) void copy16_kernel(int64_t n16, const uint4* __restrict__ src, uint4* __restrict__ dst) {
    // four independent 16-byte loads in flight per thread before the stores
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    for (; i + 3 * stride < n16; i += 4 * stride) {
        const uint4 a = src[i], b = src[i + stride], c = src[i + 2 * stride], d = src[i + 3 * stride];
        dst[i] = a;
        dst[i + stride] = b;
        dst[i + 2 * stride] = c;
        dst[i + 3 * stride] = d;
    }
    for (; i < n16; i += stride) dst[i] = src[i];
}

hipError_t launch_copy16(int64_t n16, const void* src, void* dst, hipStream_t s) {
    if (n16 <= 0) return hipSuccess;
    hipLaunchKernelGGL(copy16_kernel, dim3(2048), dim3(256), 0, s, n16, static_cast<const uint4*>(src),
                       static_cast<uint4*>(dst));
    return hipGetLastError();
}

// Streaming read of n16 16-byte words (eight loads in flight per thread, grid-stride): the
// reference for the HBM read rate the weight- and K/V-streaming kernels could reach.  Each
// block stores the xor of its words to sink[block], which keeps every load.
constexpr int READ_STREAM_BLOCKS = 16384;
__global__ __launch_bounds__(256) void read_stream_kernel(int64_t n16, const uint4* __restrict__ src,
                                                          uint32_t* __restrict__ sink) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    uint32_t acc = 0;
    for (; i + 7 * stride < n16; i += 8 * stride) {
        uint4 v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) v[u] = src[i + u * stride];
#pragma unroll
        for (int u = 0; u < 8; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    for (; i < n16; i += stride) {
        const uint4 v = src[i];
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    __shared__ uint32_t red[4];
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) acc ^= __shfl_xor(acc, o, MG_WAVE);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (threadIdx.x == 0) sink[blockIdx.x] = red[0] ^ red[1] ^ red[2] ^ red[3];
}

int read_stream_blocks() { return READ_STREAM_BLOCKS; }

hipError_t launch_read_stream(int64_t n16, const void* src, uint32_t* sink, hipStream_t s) {
    if (n16 <= 0) return hipSuccess;
    hipLaunchKernelGGL(read_stream_kernel, dim3(READ_STREAM_BLOCKS), dim3(256), 0, s, n16,
                       static_cast<const uint4*>(src), sink);
    return hipGetLastError();
}

static int probe_grid(int64_t n) { return (int)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096); }

hipError_t launch_probe_bf16(int64_t n, const float* in, uint16_t* out, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(probe_bf16_kernel, dim3(probe_grid(n)), dim3(256), 0, s, n, in, out);
    return hipGetLastError();
}
hipError_t launch_probe_exp(int64_t n, const float* in, float* out, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(probe_exp_kernel, dim3(probe_grid(n)), dim3(256), 0, s, n, in, out);
    return hipGetLastError();
}
hipError_t launch_probe_divsqrt(int64_t n, const float* a, const float* b, float* q, float* r, hipStream_t s) {
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(probe_divsqrt_kernel, dim3(probe_grid(n)), dim3(256), 0, s, n, a, b, q, r);
    return hipGetLastError();
}

typedef float probe_v16f __attribute__((ext_vector_type(16)));

// The instruction the matrix-core canonical GEMV (k_gemv_mfma.hip) relies on, bare: per instance t (one wave),
// D = v_mfma_f32_16x16x1_4b_f32(a[t][lane], b[t][lane], C) with C and D [t][register][lane]
__global__ __launch_bounds__(64) void probe_mfma_fma_kernel(const float* __restrict__ a, const float* __restrict__ b,
                                                            const float* __restrict__ c, float* __restrict__ d) {
    const size_t t = blockIdx.x;
    const int lane = threadIdx.x;
    probe_v16f acc;
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = c[(t * 16 + r) * 64 + lane];
    acc = __builtin_amdgcn_mfma_f32_16x16x1f32(a[t * 64 + lane], b[t * 64 + lane], acc, 0, 0, 0);
#pragma unroll
    for (int r = 0; r < 16; ++r) d[(t * 16 + r) * 64 + lane] = acc[r];
}

hipError_t launch_probe_mfma_fma(int n_inst, const float* a, const float* b, const float* c, float* d, hipStream_t s) {
    if (n_inst <= 0) return hipSuccess;
    hipLaunchKernelGGL(probe_mfma_fma_kernel, dim3(n_inst), dim3(64), 0, s, a, b, c, d);
    return hipGetLastError();
}

// one v_mfma_f32_4x4x1_16b_f32 per wave: a, b [n][64], c, d [n][4][64]
typedef float probe_v4f __attribute__((ext_vector_type(4)));
__global__ __launch_bounds__(64) void probe_mfma4_fma_kernel(const float* __restrict__ a, const float* __restrict__ b,
                                                             const float* __restrict__ c, float* __restrict__ d) {
    const size_t t = blockIdx.x;
    const int lane = threadIdx.x;
    probe_v4f acc;
#pragma unroll
    for (int r = 0; r < 4; ++r) acc[r] = c[(t * 4 + r) * 64 + lane];
    acc = __builtin_amdgcn_mfma_f32_4x4x1f32(a[t * 64 + lane], b[t * 64 + lane], acc, 0, 0, 0);
#pragma unroll
    for (int r = 0; r < 4; ++r) d[(t * 4 + r) * 64 + lane] = acc[r];
}

hipError_t launch_probe_mfma4_fma(int n_inst, const float* a, const float* b, const float* c, float* d, hipStream_t s) {
    if (n_inst <= 0) return hipSuccess;
    hipLaunchKernelGGL(probe_mfma4_fma_kernel, dim3(n_inst), dim3(64), 0, s, a, b, c, d);
    return hipGetLastError();
}

}  // namespace mg
