"""Op-level parity of the HIP kernels against the CPU oracle (GPU).

Bit-exact: the device bf16 rounding, the verifier's EXP, IEEE fp32 division and square
root, the canonical GEMV (CDOT order) and the canonical RMSNorm.  Tolerance: the fast
MFMA GEMM, whose summation order is free; with small-integer inputs every order is exact,
so it must then match bit for bit as well."""
import numpy as np
import pytest
import torch

from oracle import mgo
from paper_2605_30218_amd import mg, synth

pytestmark = pytest.mark.gpu
DEV = "cuda"


def to_dev_bf16(a_u16):
    return torch.from_numpy(np.ascontiguousarray(a_u16).view(np.int16)).to(DEV)


def test_bf16_rounding_bitexact():
    upper = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0, 1, 0x7FFF, 0x8000, 0x8001, 0xFFFF], np.uint32)
    u = np.concatenate([(upper[:, None] | lows[None, :]).ravel(),
                        np.random.default_rng(1).integers(0, 1 << 32, 2_000_000, dtype=np.uint64).astype(np.uint32)])
    x = u.view(np.float32)
    got = mg.op_probe_bf16(torch.from_numpy(x.copy()).to(DEV)).cpu().numpy().view(np.uint16)
    np.testing.assert_array_equal(got, mgo.bf16_from_f32(x))


def test_exp_bitexact_against_oracle():
    x = np.concatenate([np.linspace(-104.0, 90.0, 4_000_001).astype(np.float32),
                        np.float32([0.0, -0.0, np.inf, -np.inf, np.nan, 88.72, -87.33, -86.9, 1e-30, -1e-30]),
                        (np.random.default_rng(2).standard_normal(1_000_000) * 10).astype(np.float32)])
    got = mg.op_probe_exp(torch.from_numpy(x).to(DEV)).cpu().numpy()
    ref = mgo.exp(x)
    np.testing.assert_array_equal(got.view(np.uint32), ref.view(np.uint32))


def test_division_and_sqrt_are_ieee():
    rng = np.random.default_rng(3)
    a = (rng.standard_normal(2_000_000) * np.exp2(rng.integers(-140, 120, 2_000_000))).astype(np.float32)
    b = (rng.standard_normal(2_000_000) * np.exp2(rng.integers(-120, 120, 2_000_000))).astype(np.float32)
    a = np.abs(a)
    q, r = mg.op_probe_divsqrt(torch.from_numpy(a).to(DEV), torch.from_numpy(b).to(DEV))
    with np.errstate(all="ignore"):
        np.testing.assert_array_equal(q.cpu().numpy().view(np.uint32), (a / b).view(np.uint32))
        np.testing.assert_array_equal(r.cpu().numpy().view(np.uint32), np.sqrt(a).view(np.uint32))


# row counts cover every tile the vector-fma kernel picks: one branch-free tile of 4, 8, 12,
# 16, 20 or 24 rows (9..16 rows of a wide output, N >= 16384, with 3 features per wave and a
# ragged last feature block; 5..16 rows of 4608 or 6144 features with 3 features per wave,
# which balances the CUs), several 16-row tiles (a multiple of 16, and a ragged count with a
# partial last tile); and every launch of the matrix-core kernel: one 16-row tile per block
# up to 16 rows and from 25 to 48 (several blocks of row tiles on one feature group), two
# 16-row tiles per block from 49 rows, 17..24 rows as one 16-row tile plus one or two 4-row
# quads, each with the deep ring (at most one block per CU: up to 256 feature groups) and the
# shallow one (6144, 8208, 16384 and 32768 features), K a multiple of 256 or not (groups
# past K); the deep ring over K >= 8192 with the stage parity on 16 waves, K a multiple of 512,
# of 256 only, or of neither, at one and two 16-row tiles.  K covers several
# 512-element chunks and a partial last chunk.  kernel: 1 = the verifier's choice for n rows,
# 2 = the vector-fma kernel, 3 = the matrix-core kernel.
GEMV_CASES = [(1, 16, 8), (3, 48, 688), (8, 64, 4096), (13, 80, 1032), (16, 32, 14336),
              (24, 16, 512), (5, 4096, 256), (10, 32, 1032), (12, 48, 4096), (19, 32, 688),
              (21, 16, 1544), (25, 32, 1032), (32, 16, 2056), (47, 16, 520),
              (9, 16384, 264), (12, 16400, 1032), (16, 16432, 4096), (7, 6144, 520),
              (12, 4608, 1032), (16, 6144, 264), (20, 6144, 520), (14, 32784, 264), (15, 32768, 512),
              (40, 32784, 520), (29, 32768, 256), (18, 32768, 256), (23, 32784, 520), (64, 96, 4096), (100, 48, 264),
              (64, 8208, 264), (56, 4112, 512), (12, 64, 8200), (16, 48, 8448), (30, 64, 8704)]


@pytest.mark.parametrize("kernel", [1, 2, 3])
@pytest.mark.parametrize("n,N,K", GEMV_CASES)
def test_canonical_gemv_bitexact(n, N, K, kernel):
    X = synth.random_bf16((n, K), seed=n * 7 + 1)
    W = synth.random_bf16((N, K), seed=N + K, std=0.05)
    Y = mg.op_linear(kernel, to_dev_bf16(X), to_dev_bf16(W)).cpu().numpy()
    for r in range(n):
        ref = mgo.linear(mgo.CANON, X[r], W, fp32=True)
        np.testing.assert_array_equal(Y[r].view(np.uint32), ref.view(np.uint32), err_msg=f"row {r}")


def test_canonical_gemv_row_result_independent_of_row_count_and_place():
    K, N = 1032, 48
    X = synth.random_bf16((40, K), seed=11)
    W = synth.random_bf16((N, K), seed=12, std=0.05)
    full = mg.op_linear(True, to_dev_bf16(X), to_dev_bf16(W)).cpu().numpy()
    for rows in ([7], [39, 7], list(range(7, 20)), list(range(40))[::-1]):
        part = mg.op_linear(True, to_dev_bf16(X[rows]), to_dev_bf16(W)).cpu().numpy()
        np.testing.assert_array_equal(part.view(np.uint32), full[rows].view(np.uint32))


@pytest.mark.parametrize("n,N,K", [(1, 64, 4096), (5, 48, 688), (16, 128, 4096), (33, 64, 14336), (64, 6144, 4096),
                                   (100, 80, 1032), (256, 64, 512), (64, 28672, 4096), (64, 4096, 14336),
                                   (64, 128256, 4096), (1, 4096, 4096), (128, 6144, 5120)])
def test_fast_gemm_within_tolerance(n, N, K):
    X = synth.random_bf16((n, K), seed=n + 3)
    W = synth.random_bf16((N, K), seed=N + 5, std=0.02)
    Y = mg.op_linear(False, to_dev_bf16(X), to_dev_bf16(W)).cpu().numpy().astype(np.float64)
    ref = mgo.f32_from_bf16(X).astype(np.float64) @ mgo.f32_from_bf16(W).astype(np.float64).T
    bound = K * 2.0 ** -23 * (np.abs(mgo.f32_from_bf16(X)).astype(np.float64) @
                              np.abs(mgo.f32_from_bf16(W)).astype(np.float64).T) + 1e-30
    assert np.all(np.abs(Y - ref) <= bound)


# (64, 256, 4096), (20, 128, 1024), (128, 96, 2048), (9, 64, 512): the direct-to-LDS
# operand path with 4-wave blocks at 4-, 2-, 8- and 1-tile row counts; (20|64|128, 16512,
# 512) the same path with 8-wave blocks; the others the register path
@pytest.mark.parametrize("n,N,K", [(3, 48, 688), (64, 256, 4096), (130, 64, 1032), (20, 128, 1024), (128, 96, 2048),
                                   (9, 64, 512), (20, 16512, 512), (64, 16512, 512), (128, 16512, 512)])
def test_fast_gemm_small_integers_exact(n, N, K):
    X = synth.small_int_bf16((n, K), seed=21)
    W = synth.small_int_bf16((N, K), seed=22)
    Y = mg.op_linear(False, to_dev_bf16(X), to_dev_bf16(W)).cpu().numpy()
    # integer products summed in float64: exact (every |sum| < 2^53)
    ref = mgo.f32_from_bf16(X).astype(np.float64) @ mgo.f32_from_bf16(W).astype(np.float64).T
    np.testing.assert_array_equal(Y, ref.astype(np.float32))
    for kernel in (1, 2, 3):
        Yc = mg.op_linear(kernel, to_dev_bf16(X), to_dev_bf16(W)).cpu().numpy()
        np.testing.assert_array_equal(Yc, ref.astype(np.float32))


@pytest.mark.parametrize("d,eps", [(256, 1e-5), (4096, 1e-5), (3584, 1e-6), (5120, 1e-6), (688, 1e-5)])
def test_rmsnorm_bitexact(d, eps):
    x = synth.random_bf16((9, d), seed=d)
    g = synth.random_bf16((d,), seed=d + 1)
    y = mg.op_rmsnorm(to_dev_bf16(x), to_dev_bf16(g), eps).cpu().numpy().view(np.uint16)
    for r in range(9):
        np.testing.assert_array_equal(y[r], mgo.rmsnorm(mgo.CANON, x[r], g, eps))


@pytest.mark.parametrize("n_words", [0, 4, 1 << 20, (1 << 22) + 12])
def test_bandwidth_references_touch_every_word(n_words):
    """The copy and streaming-read kernels behind the bandwidth calibrations: the copy is
    exact, and the read's per-block xor words fold to the xor of the whole buffer (every
    word read once), including a tail shorter than one grid-wide batch of loads."""
    src_np = np.random.default_rng(n_words).integers(-(1 << 31), 1 << 31, n_words, dtype=np.int64).astype(np.int32)
    src = torch.from_numpy(src_np).to(DEV)
    dst = torch.zeros_like(src)
    mg.op_copy(src, dst)
    np.testing.assert_array_equal(dst.cpu().numpy(), src_np)
    sink = torch.zeros(mg.read_stream_sink_words(), dtype=torch.int32, device=DEV)
    mg.op_read_stream(src, sink)
    folded = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    expect = np.bitwise_xor.reduce(src_np.view(np.uint32)) if n_words else np.uint32(0)
    assert folded == expect


def test_fp32_mfma_k1_is_a_fused_multiply_add():
    """v_mfma_f32_16x16x1_4b_f32, on which the matrix-core canonical GEMV runs CDOT's fma
    chains: every output element equals fmaf(a, b, c) of its operands (one rounding), for
    random values over a wide exponent range, subnormals, signed zeros, infinities and
    cancellation against the product, in the lane and register layout mg_ops.h states."""
    import ctypes
    import ctypes.util
    rng = np.random.default_rng(16)
    n = 48

    def mixed(shape):
        x = (rng.standard_normal(shape) * np.exp2(rng.integers(-40, 40, shape))).astype(np.float32)
        u, m = x.view(np.uint32), rng.random(shape)
        u[m < 0.04] = rng.integers(1, 0x800000, int((m < 0.04).sum()), dtype=np.uint32)
        u[(m >= 0.04) & (m < 0.06)] = 0x80000000
        u[(m >= 0.06) & (m < 0.08)] = 0
        x[(m >= 0.08) & (m < 0.09)] = np.inf
        x[(m >= 0.09) & (m < 0.10)] = -np.inf
        return x

    a, b, c = mixed((n, 64)), mixed((n, 64)), mixed((n, 16, 64))
    r = np.arange(16)[:, None]
    l = np.arange(64)[None, :]
    ia, ib = 16 * (r // 4) + 4 * (l // 16) + r % 4, 16 * (r // 4) + l % 16
    ae, be = a[:, ia], b[:, ib]
    # a third of the accumulators cancel the product to within a few ulps
    sel = rng.random((n, 16, 64)) < 0.3
    prod = (ae.astype(np.float64) * be.astype(np.float64)).astype(np.float32)
    with np.errstate(all="ignore"):
        c[sel] = -prod[sel] * np.float32(1 + 2 ** -20)
    d = mg.op_probe_mfma_fma(*(torch.from_numpy(np.ascontiguousarray(x)).to(DEV) for x in (a, b, c))).cpu().numpy()
    libm = ctypes.CDLL(ctypes.util.find_library("m"))
    libm.fmaf.restype = ctypes.c_float
    libm.fmaf.argtypes = [ctypes.c_float] * 3
    ref = np.array([libm.fmaf(float(x), float(y), float(z)) for x, y, z in zip(ae.ravel(), be.ravel(), c.ravel())],
                   np.float32).reshape(d.shape)
    both_nan = np.isnan(d) & np.isnan(ref)
    assert np.array_equal(np.isnan(d), np.isnan(ref))
    assert np.array_equal(d.view(np.uint32)[~both_nan], ref.view(np.uint32)[~both_nan])


def test_fp32_mfma_4x4x1_is_a_fused_multiply_add():
    """v_mfma_f32_4x4x1_16b_f32, which carries the fma chains of the rows past the first 16-row
    tile: every output element equals fmaf(a, b, c) of its operands (one rounding), over the same
    operand mix as the 16x16x1 test, in the lane and register layout mg_ops.h states."""
    import ctypes
    import ctypes.util
    rng = np.random.default_rng(17)
    n = 48

    def mixed(shape):
        x = (rng.standard_normal(shape) * np.exp2(rng.integers(-40, 40, shape))).astype(np.float32)
        u, m = x.view(np.uint32), rng.random(shape)
        u[m < 0.04] = rng.integers(1, 0x800000, int((m < 0.04).sum()), dtype=np.uint32)
        u[(m >= 0.04) & (m < 0.06)] = 0x80000000
        u[(m >= 0.06) & (m < 0.08)] = 0
        x[(m >= 0.08) & (m < 0.09)] = np.inf
        x[(m >= 0.09) & (m < 0.10)] = -np.inf
        return x

    a, b, c = mixed((n, 64)), mixed((n, 64)), mixed((n, 4, 64))
    r = np.arange(4)[:, None]
    l = np.arange(64)[None, :]
    ia, ib = 4 * (l // 4) + r, l + 0 * r
    ae, be = a[:, ia], b[:, ib]
    # a third of the accumulators cancel the product to within a few ulps
    sel = rng.random((n, 4, 64)) < 0.3
    prod = (ae.astype(np.float64) * be.astype(np.float64)).astype(np.float32)
    with np.errstate(all="ignore"):
        c[sel] = -prod[sel] * np.float32(1 + 2 ** -20)
    d = mg.op_probe_mfma4_fma(*(torch.from_numpy(np.ascontiguousarray(x)).to(DEV) for x in (a, b, c))).cpu().numpy()
    libm = ctypes.CDLL(ctypes.util.find_library("m"))
    libm.fmaf.restype = ctypes.c_float
    libm.fmaf.argtypes = [ctypes.c_float] * 3
    ref = np.array([libm.fmaf(float(x), float(y), float(z)) for x, y, z in zip(ae.ravel(), be.ravel(), c.ravel())],
                   np.float32).reshape(d.shape)
    both_nan = np.isnan(d) & np.isnan(ref)
    assert np.array_equal(np.isnan(d), np.isnan(ref))
    assert np.array_equal(d.view(np.uint32)[~both_nan], ref.view(np.uint32)[~both_nan])
