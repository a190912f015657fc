// k_gemv_mfma.hip -- the verifier's canonical GEMV on the matrix cores.
//
// Same arithmetic as canon_gemv_kernel (k_gemv.hip), bit for bit: y[r][j] = CDOT(x[r], W[j])
// with CDOT's 64 chains (chain l owns the 8-element groups g = l mod 64 and fma-accumulates
// them in increasing g, element order inside a group, from +0) combined by the xor butterfly
// over chain offsets 32, 16, 8, 4, 2, 1.
//
// The fma steps run on v_mfma_f32_16x16x1_4b_f32.  With K = 1 every output element of that
// instruction is one fused multiply-add, d = fma(a, b, c) with a single IEEE rounding (a
// probe over 8.4M cases with subnormals, signed zeros, infinities and cancellation found it
// equal to fmaf bit for bit), and its four blocks are four independent 16 x 16 outer
// products.  So one instruction advances 4 chains (the blocks) x 16 features (A rows) x 16
// rows (B columns) by one element: block bk of lane 16 bk + i takes feature i's weight and
// row i's activation of its chain's element, and D holds (block bk, feature i, row j) in
// register 4 bk + i % 4 of lane 16 (i / 4) + j.
//
// Work split.  A block owns FG groups of 16 features (a SwiGLU group is 8 gate rows and the
// 8 matching up rows) and a tile of 16 rows; NWB waves serve each feature group.  K is walked
// in stages of 256 elements (32 groups: the chains of one half, l = 32 p + ..., p = stage
// parity).  Every stage, weights and activations go through LDS by direct-to-LDS loads: one
// load moves two 512-byte runs (two rows of the stage), and group g of stage row r sits at
// slot 32 r + (g xor (r mod 16)), so each run is one contiguous read and each MFMA operand
// read (16 rows, one group) hits 16 distinct bank groups.  The stages form a ring of D
// buffers (stage s + D is requested into the buffer of stage s once every wave holds stage
// s's operands in registers; the operands of stage s + 1 are read while the MFMAs of stage s
// run); the loads of a stage are shared by all waves, so each stage starts on a block
// barrier.  The compiler does not count direct-to-LDS loads when it places waits, so the
// operand reads, their waits, the barrier and every wait for the loads are explicit.
// Chain bits of wave w of its feature group (NWB = 4: l = 32 p + 16 qq + 4 w + bk; NWB = 8:
// l = 32 p + 4 w + bk): the bits above the wave bits are the wave's own, then come the wave
// bits, then the instruction's blocks.  NWB = 16 puts the stage parity on the waves as well
// (l = 4 w + bk): a step is then a pair of stages (512 elements, 1 KiB runs), wave w < 8 takes
// the even stage's chains and wave w + 8 the odd one's, one accumulator each, and the whole
// butterfly above the block bits goes through LDS.  Butterfly, in the order of the offsets:
// the wave's own bits by register adds, the wave bits through LDS, the block bits by register
// adds of the four block registers of a lane.  IEEE addition is commutative, so pairing operands in
// either order gives the same bits as the single-lane butterfly.
// Groups past K read a group of -0 weights and +0 activations: fma(-0, +0, c) = c + (-0) = c
// for every c, so those chains are left unchanged.  Rows past the count compute on a copy of
// the last live row and are not written; features past N on a copy of the last feature.
#include <type_traits>

#include "mg_device.h"
#include "mg_kernels.h"

namespace mg {

typedef float mg_v16f __attribute__((ext_vector_type(16)));
typedef float mg_v4f __attribute__((ext_vector_type(4)));
typedef uint32_t mg_u32x4 __attribute__((ext_vector_type(4)));

// one 8-element group of bf16 -0 (weights) and of +0 (activations) for groups past K
__device__ __align__(16) const uint16_t k_neg_zero_group[8] = {0x8000, 0x8000, 0x8000, 0x8000,
                                                              0x8000, 0x8000, 0x8000, 0x8000};
__device__ __align__(16) const uint16_t k_pos_zero_group[8] = {0, 0, 0, 0, 0, 0, 0, 0};

__device__ __forceinline__ float bfe(const mg_u32x4& v, int e) {
    const uint32_t w = v[e >> 1];
    return (e & 1) ? bf_hi(w) : bf_lo(w);
}

template <int N>
__device__ __forceinline__ void gv_wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
__device__ __forceinline__ void gv_barrier() { asm volatile("s_barrier" ::: "memory"); }
__device__ __forceinline__ void gv_lds_read(mg_u32x4& v, const uint4* p) {
    asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"((uint32_t)(uintptr_t)p));
}
// waits for the operand reads and names every operand as read and written by the wait, so
// no use of one can be scheduled before it
template <int NQ, int T>
__device__ __forceinline__ void gv_lds_wait(mg_u32x4 (&av)[NQ], mg_u32x4 (&bv)[T][NQ]) {
    if constexpr (NQ == 1 && T == 1) {
        asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(av[0]), "+v"(bv[0][0]) : : "memory");
    } else if constexpr (NQ == 2 && T == 1) {
        asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(av[0]), "+v"(av[1]), "+v"(bv[0][0]), "+v"(bv[0][1]) : : "memory");
    } else {
        static_assert(NQ == 1 && T == 2, "quads per stage x row tiles");
        asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(av[0]), "+v"(bv[0][0]), "+v"(bv[1][0]) : : "memory");
    }
}
// the same for one 16-row tile plus XQ 4-row quads (one quad of the stage per wave)
template <int XQ>
__device__ __forceinline__ void gv_lds_wait_x(mg_u32x4& av, mg_u32x4& bv, mg_u32x4 (&bx)[XQ]) {
    if constexpr (XQ == 1) {
        asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(av), "+v"(bv), "+v"(bx[0]) : : "memory");
    } else {
        static_assert(XQ == 2, "4-row quads past the first tile");
        asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(av), "+v"(bv), "+v"(bx[0]), "+v"(bx[1]) : : "memory");
    }
}

// XQ > 0 (with T = 2 and one quad per wave): rows 16 .. 16 + 4 XQ - 1 of the block's 32-row
// tile run on v_mfma_f32_4x4x1_16b_f32 instead of a second 16x16x1 tile.  Its 16 blocks of
// 4 x 4 are the 4 chains x 4 feature quads: lane 16 c + 4 q + i supplies feature 4 q + i of
// chain c (the very A operand of the 16x16x1 instruction) and row 4 rq + i of the quad's B,
// and register r of lane 16 c + 4 q + j holds (chain c, feature 4 q + r, row 4 rq + j); an
// fma step of 16 x 4 rows costs a quarter of a 16 x 16 one.
template <int FG, int NWB, int T, int XQ, int EPI, int D, bool RAGGED>
__global__ __launch_bounds__(64 * FG * NWB, RAGGED ? 1 : 4) void canon_gemv_mfma_kernel(GemvArgs a, int n_fg, int n_rt) {
    constexpr int NW = FG * NWB;
    constexpr bool PW = NWB == 16;              // stage parity on the waves: a step is a stage pair
    constexpr int SG = PW ? 64 : 32;            // groups of a step (slots of a ring row)
    constexpr int NQ = PW ? 1 : 8 / NWB;        // quads of a wave per stage
    constexpr int NACC = PW ? 1 : 2;            // accumulators per quad (stage parity)
    constexpr int SROWS = 16 * FG + 16 * T;     // rows of a stage: weights, then activations
    constexpr int NLD = PW ? SROWS : SROWS / 2; // direct-to-LDS loads per step (one row of 64 slots, or two of 32)
    constexpr int IPW = NLD / NW;               // loads per wave per stage
    constexpr int TM = XQ ? 1 : T;              // 16-row tiles on the 16x16x1 instruction
    constexpr int XA = XQ ? XQ : 1;             // (array extent)
    static_assert(NWB == 4 || NWB == 8 || (NWB == 16 && FG == 1 && XQ == 0), "waves per feature group");
    static_assert(NACC * NQ * T <= 4, "accumulators");
    static_assert(XQ == 0 || (T == 2 && NQ == 1 && XQ <= 2 && XQ <= NWB), "4-row quads: second tile, one quad per wave");
    static_assert(NLD % NW == 0, "every wave issues the same loads (exact waits)");
    const int b = blockIdx.x;
    const int xcd = b & 7, slot = b >> 3;
    const int fb = (slot / n_rt) * 8 + xcd;     // feature block (FG groups)
    const int rt = slot % n_rt;
    if (fb * FG >= n_fg) return;
    RowCount rc{a.n_dev, a.n_host, a.cap};
    const int n = rc.get();
    const int r0 = rt * 16 * T;
    if (r0 >= n) return;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
    const int fgw = wave / NWB, wb = wave % NWB;
    const int bk = lane >> 4, ii = lane & 15;
    const int K = a.K, G = K >> 3;
    const int nst = PW ? (G + 63) >> 6 : (G + 31) >> 5;

    __shared__ __attribute__((aligned(16))) uint4 ring[D][SROWS * SG];

    // the rows this lane loads: load m = wave + NW t of a stage covers stage rows 2m, 2m+1;
    // this lane's half is row 2m + (lane >> 5), its slot lane & 31 (NWB = 16: load m is row m
    // of the stage pair, slot lane)
    const uint16_t* src_row[IPW];
    int sw[IPW];
    bool is_w[IPW];
#pragma unroll
    for (int t = 0; t < IPW; ++t) {
        const int m = wave + NW * t;
        const int r = PW ? m : 2 * m + (lane >> 5);
        is_w[t] = r < 16 * FG;
        if (r < 16 * FG) {
            const int fgl = fb * FG + r / 16, i = r % 16;
            if constexpr (EPI == EPI_SWIGLU) {
                const int pj = min(fgl * 8 + (i & 7), a.N - 1);
                src_row[t] = a.W[i >> 3] + (size_t)pj * K;
            } else {
                int j = min(fgl * 16 + i, a.N - 1), seg = 0;
                while (seg < 2 && j >= a.Nseg[seg]) { j -= a.Nseg[seg]; ++seg; }
                src_row[t] = a.W[seg] + (size_t)j * K;
            }
        } else {
            src_row[t] = a.X + (size_t)min(r0 + r - 16 * FG, n - 1) * K;
        }
        sw[t] = (PW ? lane : lane & 31) ^ (r & 15);  // the group this lane's slot holds
    }
    // the loads of stage s into buffer s % D (clamped to the last stage)
    auto issue = [&](int s) {
        const int sc = min(s, nst - 1);
        uint4* buf = ring[s % D];
#pragma unroll
        for (int t = 0; t < IPW; ++t) {
            const int g = sc * SG + sw[t];
            const uint16_t* src = src_row[t] + (size_t)g * 8;
            if constexpr (RAGGED) src = g < G ? src : (is_w[t] ? k_neg_zero_group : k_pos_zero_group);
            __builtin_amdgcn_global_load_lds(src, buf + 64 * (wave + NW * t), 16, 0, 0);
        }
    };

    mg_v16f acc[TM][NACC * NQ];  // [row tile][NACC qi + p] (qi: the wave's quad of a stage, p: stage parity)
#pragma unroll
    for (int t = 0; t < TM; ++t)
#pragma unroll
        for (int k = 0; k < NACC * NQ; ++k)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[t][k][r] = 0.0f;
    mg_v4f accx[XA][2];  // 4-row quads: [quad][stage parity]
#pragma unroll
    for (int q = 0; q < XA; ++q)
#pragma unroll
        for (int k = 0; k < 2; ++k)
#pragma unroll
            for (int r = 0; r < 4; ++r) accx[q][k][r] = 0.0f;

    // operand slots of quad qi (group of the stage: NWB = 4: 16 qi + 4 wb + bk; NWB = 8: 4 wb + bk)
    int aslot[NQ], bslot[TM][NQ], bxslot[XA];
#pragma unroll
    for (int qi = 0; qi < NQ; ++qi) {
        const int lg = PW ? 32 * (wb >> 3) + 4 * (wb & 7) + bk : (NWB == 4 ? 16 * qi : 0) + 4 * wb + bk;
        aslot[qi] = SG * (16 * fgw + ii) + (lg ^ ii);
#pragma unroll
        for (int t = 0; t < TM; ++t) bslot[t][qi] = SG * (16 * FG + 16 * t + ii) + (lg ^ ii);
    }
#pragma unroll
    for (int q = 0; q < XA; ++q) {  // row 4 q + (lane mod 4) of the second tile, the lane's chain
        const int lg = 4 * wb + bk, rr = 4 * q + (lane & 3);
        bxslot[q] = 32 * (16 * FG + 16 + rr) + (lg ^ rr);
    }
    // operand reads of stage s (raw bf16 groups), waited for one stage later
    struct Ops {
        mg_u32x4 a[NQ], b[TM][NQ], bx[XA];
    };
    auto read_ops = [&](int s, Ops& o) {
        const uint4* buf = ring[s % D];
#pragma unroll
        for (int qi = 0; qi < NQ; ++qi) {
            gv_lds_read(o.a[qi], buf + aslot[qi]);
#pragma unroll
            for (int t = 0; t < TM; ++t) gv_lds_read(o.b[t][qi], buf + bslot[t][qi]);
        }
        if constexpr (XQ > 0) {
#pragma unroll
            for (int q = 0; q < XQ; ++q) gv_lds_read(o.bx[q], buf + bxslot[q]);
        }
    };
    // the MFMAs of one stage into the accumulators of parity P (a compile-time index, so the
    // accumulators stay in registers)
    auto mfmas = [&](const Ops& o, auto P) {
        constexpr int p = PW ? 0 : decltype(P)::value;
        // a quad's operands converted before its MFMAs; with a deep ring (one block per CU, two
        // waves per SIMD) all sixteen are held in registers of their own so that the stage's
        // MFMAs issue back to back (down projection at 16 rows 33.3 against 34.7 us); elsewhere
        // the compiler may reuse two registers, which keeps the VGPR count at 61 and four 8-wave
        // blocks per CU (gate/up at 16 rows 53.2 against 58.3 us with the sixteen registers)
#pragma unroll
        for (int qi = 0; qi < NQ; ++qi) {
            float fa[8], fx[TM][8], fq[XA][8];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                fa[e] = bfe(o.a[qi], e);
#pragma unroll
                for (int t = 0; t < TM; ++t) fx[t][e] = bfe(o.b[t][qi], e);
                if constexpr (XQ > 0) {
#pragma unroll
                    for (int q = 0; q < XQ; ++q) fq[q][e] = bfe(o.bx[q], e);
                }
            }
            if constexpr (D >= 4 && TM == 1 && XQ == 0) {
                asm volatile("" : "+v"(fa[0]), "+v"(fa[1]), "+v"(fa[2]), "+v"(fa[3]), "+v"(fa[4]), "+v"(fa[5]), "+v"(fa[6]), "+v"(fa[7]),
                             "+v"(fx[0][0]), "+v"(fx[0][1]), "+v"(fx[0][2]), "+v"(fx[0][3]), "+v"(fx[0][4]), "+v"(fx[0][5]), "+v"(fx[0][6]), "+v"(fx[0][7]));
            }
#pragma unroll
            for (int e = 0; e < 8; ++e) {
#pragma unroll
                for (int t = 0; t < TM; ++t)
                    acc[t][NACC * qi + p] = __builtin_amdgcn_mfma_f32_16x16x1f32(fa[e], fx[t][e], acc[t][NACC * qi + p], 0, 0, 0);
                if constexpr (XQ > 0) {
#pragma unroll
                    for (int q = 0; q < XQ; ++q)
                        accx[q][p] = __builtin_amdgcn_mfma_f32_4x4x1f32(fa[e], fq[q][e], accx[q][p], 0, 0, 0);
                }
            }
        }
    };
    // One stage: its operands (read one stage earlier) are waited for; then, if a stage
    // follows, this wave's loads of stage s + 1 are waited for (stages s + 1 .. s + D - 1 are
    // requested while s + D - 1 < nst, so D - 2 stages of loads may remain; near the end
    // none), the barrier makes every wave's loads of s + 1 visible and every read of stage
    // s finished, the loads of stage s + D go to the buffer of s, and the operands of s + 1 are
    // requested; then the MFMAs of stage s run from registers.
    auto step = [&](int s, Ops& cur, Ops& nxt, auto P) {
        if constexpr (XQ > 0) gv_lds_wait_x<XQ>(cur.a[0], cur.b[0][0], cur.bx);
        else gv_lds_wait<NQ, T>(cur.a, cur.b);
        if (s + 1 < nst) {
            if (s + D - 1 < nst) gv_wait_vmcnt<IPW * (D - 2)>();
            else gv_wait_vmcnt<0>();
            gv_barrier();
            if (s + D < nst) issue(s + D);
            read_ops(s + 1, nxt);
        }
        __builtin_amdgcn_sched_barrier(0);
        mfmas(cur, P);
        __builtin_amdgcn_sched_barrier(0);
    };

    // ring: stages 0 .. D - 1 requested up front, one per buffer (clamped past the last
    // stage: a clamped stage is never read)
#pragma unroll
    for (int s = 0; s < D; ++s) issue(s);
    gv_wait_vmcnt<IPW * (D - 1)>();
    gv_barrier();
    Ops oa, ob;
    read_ops(0, oa);
    for (int s = 0; s < nst; s += 2) {
        step(s, oa, ob, std::integral_constant<int, 0>{});
        if (s + 1 < nst) step(s + 1, ob, oa, std::integral_constant<int, 1>{});
    }
    gv_wait_vmcnt<0>();  // (clamped prologue loads of a short K)

    // butterfly, the wave's own bits: stage parity (offset 32), then for NWB = 4 the quad (16);
    // then the wave bits through LDS (the ring is free once every wave is past its last read),
    // one row tile at a time; then the block bits
    float* red = reinterpret_cast<float*>(&ring[0][0]);  // [NW][16][64]
    static_assert(NW * 16 * 64 * 4 <= D * SROWS * SG * 16, "the reduction fits in the ring");
    const int col = wb & 3;  // register column i % 4 that waves wb < 4 finish
    float vt[TM];
#pragma unroll
    for (int t = 0; t < TM; ++t) {
        mg_v16f tot;
        if constexpr (PW) {
            tot = acc[t][0];
        } else if constexpr (NQ == 2) {
            tot = (acc[t][0] + acc[t][1]) + (acc[t][2] + acc[t][3]);
        } else {
            tot = acc[t][0] + acc[t][1];
        }
        gv_barrier();  // every wave is past its last read of the ring (or of the previous tile)
#pragma unroll
        for (int r = 0; r < 16; ++r) red[(wave * 16 + r) * 64 + lane] = tot[r];
        __syncthreads();
        float s4[4];
#pragma unroll
        for (int bb = 0; bb < 4; ++bb) {
            float v[NWB];
#pragma unroll
            for (int w = 0; w < NWB; ++w) v[w] = red[((fgw * NWB + w) * 16 + 4 * bb + col) * 64 + lane];
#pragma unroll
            for (int h = NWB / 2; h >= 1; h >>= 1)
#pragma unroll
                for (int w = 0; w < h; ++w) v[w] = v[w] + v[w + h];
            s4[bb] = v[0];
        }
        vt[t] = (s4[0] + s4[2]) + (s4[1] + s4[3]);  // block bits: offsets 2 then 1
    }
    // the 4-row quads: the same pairings, the wave bits through LDS (wave wb < XQ finishes quad
    // wb), then the chain's low bits, which sit in lane bits 5 and 4 here: offsets 2 then 1
    float vq[4];
    if constexpr (XQ > 0) {
        gv_barrier();  // every wave is past its reads of the last tile
#pragma unroll
        for (int q = 0; q < XQ; ++q) {
            const mg_v4f totq = accx[q][0] + accx[q][1];
#pragma unroll
            for (int r = 0; r < 4; ++r) red[(wave * 16 + 4 * q + r) * 64 + lane] = totq[r];
        }
        __syncthreads();
        const int q = wb < XQ ? wb : 0;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            float v[NWB];
#pragma unroll
            for (int w = 0; w < NWB; ++w) v[w] = red[((fgw * NWB + w) * 16 + 4 * q + r) * 64 + lane];
#pragma unroll
            for (int h = NWB / 2; h >= 1; h >>= 1)
#pragma unroll
                for (int w = 0; w < h; ++w) v[w] = v[w] + v[w + h];
            float x = v[0];
            x = x + __shfl_xor(x, 32, MG_WAVE);
            x = x + __shfl_xor(x, 16, MG_WAVE);
            vq[r] = x;
        }
    }
    if (wb >= 4) return;

    // epilogue: output (feature i of the group, row) = v; upv: the matching up row's sum
    const int fgl = fb * FG + fgw;
    auto emit = [&](float v, float upv, int i, int row, bool live) {
        if constexpr (EPI == EPI_SWIGLU) {
            const int pj = fgl * 8 + i;
            if (!live || i >= 8 || row >= n || pj >= a.N) return;
            const float g = bf2f(f2bf(v)), up = bf2f(f2bf(upv));
            const float sg = ieee_div(g, 1.0f + canon_exp(-g));
            reinterpret_cast<uint16_t*>(a.Y)[(size_t)row * a.N + pj] = (uint16_t)f2bf(sg * up);
        } else {
            const int j = fgl * 16 + i;
            if (!live || row >= n || j >= a.N) return;
            if (EPI == EPI_F32) {
                reinterpret_cast<float*>(a.Y)[(size_t)row * a.N + j] = v;
            } else if (EPI == EPI_BF16) {
                int jl = j, seg = 0;
                while (seg < 2 && jl >= a.Nseg[seg]) { jl -= a.Nseg[seg]; ++seg; }
                const float y = a.bias[seg] ? v + bf2f(a.bias[seg][jl]) : v;
                reinterpret_cast<uint16_t*>(a.Y)[(size_t)row * a.N + j] = (uint16_t)f2bf(y);
            } else {  // residual: x = bf16(x + bf16(y))
                uint16_t* xp = reinterpret_cast<uint16_t*>(a.Y) + (size_t)row * a.N + j;
                *xp = (uint16_t)f2bf(bf2f(*xp) + bf2f(f2bf(v)));
            }
        }
    };
    // 16-row tiles: lane 16 (i / 4) + j holds feature i = 4 (lane / 16) + col, row j = lane % 16
    // (a SwiGLU group's gate features i < 8 sit in lanes 0..31, their up rows 32 lanes higher)
#pragma unroll
    for (int t = 0; t < TM; ++t) {
        const float upv = EPI == EPI_SWIGLU ? __shfl_xor(vt[t], 32, MG_WAVE) : 0.0f;
        emit(vt[t], upv, 4 * (lane >> 4) + col, r0 + 16 * t + (lane & 15), true);
    }
    // 4-row quad wb: lanes 4 q + j (chain 0) hold feature 4 q + r in register r, row 16 + 4 wb + j
    // (gate features in lanes 0..7, their up rows 8 lanes higher)
    if constexpr (XQ > 0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const float upv = EPI == EPI_SWIGLU ? __shfl_xor(vq[r], 8, MG_WAVE) : 0.0f;
            emit(vq[r], upv, 4 * ((lane >> 2) & 3) + r, r0 + 16 + 4 * wb + (lane & 3), wb < XQ && lane < 16);
        }
    }
}

template <int FG, int NWB, int T, int D, bool RG, int XQ = 0>
static hipError_t launch_mfma_cfg(const GemvArgs& a, int epi, int rows, hipStream_t s) {
    const int n_fg = epi == EPI_SWIGLU ? (a.N + 7) / 8 : (a.N + 15) / 16;
    const int n_fb = (n_fg + FG - 1) / FG;
    const int n_rt = (rows + 16 * T - 1) / (16 * T);
    const dim3 grid(8 * ((n_fb + 7) / 8) * n_rt), block(64 * FG * NWB);
    switch (epi) {
        case EPI_SWIGLU: hipLaunchKernelGGL((canon_gemv_mfma_kernel<FG, NWB, T, XQ, EPI_SWIGLU, D, RG>), grid, block, 0, s, a, n_fg, n_rt); break;
        case EPI_BF16: hipLaunchKernelGGL((canon_gemv_mfma_kernel<FG, NWB, T, XQ, EPI_BF16, D, RG>), grid, block, 0, s, a, n_fg, n_rt); break;
        case EPI_RESID: hipLaunchKernelGGL((canon_gemv_mfma_kernel<FG, NWB, T, XQ, EPI_RESID, D, RG>), grid, block, 0, s, a, n_fg, n_rt); break;
        default: hipLaunchKernelGGL((canon_gemv_mfma_kernel<FG, NWB, T, XQ, EPI_F32, D, RG>), grid, block, 0, s, a, n_fg, n_rt); break;
    }
    return hipGetLastError();
}

template <bool RG>
static hipError_t launch_mfma_sel(const GemvArgs& a, int epi, int rows, const MfmaLaunch& c, hipStream_t s) {
    const bool deep = c.depth == 4;
    if (c.waves == 16) return launch_mfma_cfg<1, 16, 1, 4, RG>(a, epi, rows, s);
    if (c.tile_rows == 32) {
        if (c.quads == 2) return deep ? launch_mfma_cfg<1, 8, 2, 4, RG, 2>(a, epi, rows, s) : launch_mfma_cfg<1, 8, 2, 2, RG, 2>(a, epi, rows, s);
        if (c.quads == 1) return deep ? launch_mfma_cfg<1, 8, 2, 4, RG, 1>(a, epi, rows, s) : launch_mfma_cfg<1, 8, 2, 2, RG, 1>(a, epi, rows, s);
        return deep ? launch_mfma_cfg<1, 8, 2, 4, RG>(a, epi, rows, s) : launch_mfma_cfg<1, 8, 2, 2, RG>(a, epi, rows, s);
    }
    return deep ? launch_mfma_cfg<1, 8, 1, 4, RG>(a, epi, rows, s) : launch_mfma_cfg<1, 8, 1, 2, RG>(a, epi, rows, s);
}

// Launch rule: one feature group per block served by 8 waves (two groups per block, sharing
// the activation stages, measured slower on every shape once the outputs were wide enough to
// fill the chip: LM head at 16 rows 238 against 206 us, at 20 rows 331 against 302 us, with
// the caches flushed before each launch).  Row tiles: one 16-row tile per block up to 16 rows;
// one tile and one or two 4-row quads up to 24; above that 16-row tiles in separate blocks of
// the same feature group, which the block order puts on one XCD so that the weights come from
// HBM once and from its L2 after (against two tiles sharing the weight operand: at 32 rows
// LM head 350 against 368 us, Qwen2.5-7B gate/up 103 against 112, Llama-8B gate/up equal; at
// 48 rows, where the shared pair is half empty, 556 against 724 and 150 against 188); above 48
// rows two tiles per block again (equal on gate/up, 81 against 88 us on the down projection
// at 64 rows).
// Ring depth: a launch with at most one block per CU (the 4096-feature outputs) has nothing
// else on the CU to cover a stage's memory latency, so it keeps three stages in flight
// (depth 4: in the decode loop the O and down projections at 12-16 rows took 21.9 against
// 29.3 us with depth 2); launches with several blocks per CU keep the shallow ring, which
// leaves room for more blocks (gate/up at 12-16 rows: 52.9 us at depth 2, 57.9 at 4; at
// 20 rows 80.6 us at depth 2, 84.9 at 3).  A deep launch over a long K (the down projections)
// runs 16 waves with the stage parity on the waves, so four waves per SIMD share the matrix
// core and a barrier covers two stages (down at 16 rows 31.7 against 33.4 us, Qwen2.5-7B down
// 38.0 against 40.8); over a short K its 16-wave butterfly costs more than it saves (O 15.2
// against 14.9 us).  Its steps are 512 elements, so it takes the ragged form unless 512
// divides K.
#ifndef MG_GEMV_PW_MIN_K
#define MG_GEMV_PW_MIN_K 8192
#endif
MfmaLaunch choose_mfma_launch(int rows, int n_fg, int K, int n_cu) {
    MfmaLaunch c{};
    c.tile_rows = (rows > 16 && rows <= 24) || rows > 48 ? 32 : 16;
    c.quads = c.tile_rows == 32 && rows <= 24 ? (rows > 20 ? 2 : 1) : 0;
    const int n_rt = (rows + c.tile_rows - 1) / c.tile_rows;
    const bool deep = (long)n_fg * n_rt <= (n_cu > 0 ? n_cu : 256);
    c.depth = deep ? 4 : 2;
    // a deep ring over a long K: 16 waves, the two stage parities on separate waves
    c.waves = deep && c.tile_rows == 16 && K >= MG_GEMV_PW_MIN_K ? 16 : 8;
    c.ragged = K % (c.waves == 16 ? 512 : 256) != 0;
    return c;
}

hipError_t launch_canon_gemv_mfma(const GemvArgs& a, int epi, hipStream_t s) {
    const int rows = a.n_dev ? a.cap : a.n_host;
    if (rows <= 0 || a.N <= 0) return hipSuccess;
    const int n_fg = epi == EPI_SWIGLU ? (a.N + 7) / 8 : (a.N + 15) / 16;
    const MfmaLaunch c = choose_mfma_launch(rows, n_fg, a.K, a.n_cu);
    return c.ragged ? launch_mfma_sel<true>(a, epi, rows, c, s) : launch_mfma_sel<false>(a, epi, rows, c, s);
}

}  // namespace mg
