"""Pins of the CPU oracle against what the mathematics and the paper fix (no GPU).

Each test checks one oracle function against something other than itself: closed forms,
exact small-integer arithmetic, brute force, library routines in float64, hand-derived
fixtures (tests/golden/), invariants of the definitions.  Paper anchors: arXiv 2605.30218
Sec. 3.1 (margin g = l_(1) - l_(2), trigger g < tau), Sec. 2.4 / Obs. 3 (N(Delta) > 1 iff
g < Delta), Sec. 3.2 (fast commit, verified commit, single-column repair), Sec. 3.3
(r_verify, r_repair).
"""
import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import mgo
from paper_2605_30218_amd import synth

GOLD = os.path.join(os.path.dirname(__file__), "golden")
f32 = np.float32


# ----------------------------------------------------------------------------- bf16 rounding

def _bf16_ref(u32: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even of fp32 bit patterns to bf16, derived in float64 from the two
    neighbouring bf16 values (distance comparison), independent of the oracle's bit trick."""
    with np.errstate(invalid="ignore"):
        x = u32.view(np.float32).astype(np.float64)
    lo = (u32 >> 16).astype(np.uint32)                      # truncation toward zero
    hi = lo + 1                                              # next bf16 away from zero
    def val(b):
        b = b.astype(np.uint32)
        e = (b >> 7) & 0xFF
        m = b & 0x7F
        s = np.where(b & 0x8000, -1.0, 1.0)
        mag = np.where(e == 0, m * 2.0 ** -133, (1 + m / 128.0) * np.exp2(e.astype(np.float64) - 127))
        mag = np.where(e == 255, 2.0 ** 128, mag)             # successor of the largest finite value
        return s * mag
    dlo = np.abs(x - val(lo))
    dhi = np.abs(val(hi) - x)
    pick_hi = (dhi < dlo) | ((dhi == dlo) & ((lo & 1) == 1))
    out = np.where(pick_hi, hi, lo).astype(np.uint32)
    exp_all_ones = ((u32 >> 23) & 0xFF) == 0xFF
    is_nan = exp_all_ones & ((u32 & 0x7FFFFF) != 0)
    is_inf = exp_all_ones & ((u32 & 0x7FFFFF) == 0)
    out = np.where(is_inf, u32 >> 16, out)
    out = np.where(is_nan, (u32 >> 16) | 0x40, out)
    return out.astype(np.uint16)


def test_bf16_rne_all_upper_halves():
    """Every bf16 upper half x the lower halves at and around each rounding decision."""
    upper = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0, 1, 0x3FFF, 0x7FFE, 0x7FFF, 0x8000, 0x8001, 0xBFFF, 0xFFFE, 0xFFFF], np.uint32)
    u = (upper[:, None] | lows[None, :]).ravel()
    got = mgo.bf16_from_f32(u.view(np.float32))
    np.testing.assert_array_equal(got, _bf16_ref(u))


def test_bf16_rne_random_sample():
    u = np.random.default_rng(7).integers(0, 1 << 32, size=4_000_000, dtype=np.uint64).astype(np.uint32)
    np.testing.assert_array_equal(mgo.bf16_from_f32(u.view(np.float32)), _bf16_ref(u))


def test_bf16_matches_torch_rounding():
    """torch's fp32 -> bfloat16 cast is round-to-nearest-even on finite values."""
    x = torch.randn(1_000_000, generator=torch.Generator().manual_seed(3)) * 37.0
    ref = x.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(mgo.bf16_from_f32(x.numpy()), ref)


# ----------------------------------------------------------------------------- EXP

def _ulp_err(got: np.ndarray, x: np.ndarray) -> np.ndarray:
    ref = np.exp(x.astype(np.float64))
    spacing = np.spacing(np.abs(ref).astype(np.float32)).astype(np.float64)
    return np.abs(got.astype(np.float64) - ref) / spacing


def test_exp_within_2ulp_dense_sweep():
    x = np.linspace(-87.0, 88.0, 3_000_001, dtype=np.float64).astype(np.float32)
    got = mgo.exp(x)
    err = _ulp_err(got, x)
    assert err.max() <= 2.0, (float(err.max()), float(x[err.argmax()]))
    # around 0 every fp32 in [-1, 1] stepping 2^-12
    y = (np.arange(-4096, 4097, dtype=np.float32) / 4096).astype(np.float32)
    assert _ulp_err(mgo.exp(y), y).max() <= 2.0


def test_exp_special_values_and_monotone():
    assert mgo.exp(np.float32([0.0]))[0] == 1.0
    assert mgo.exp(np.float32([-0.0]))[0] == 1.0
    assert math.isinf(mgo.exp(np.float32([89.0]))[0])
    assert mgo.exp(np.float32([-1000.0]))[0] == 0.0
    assert mgo.exp(np.float32([-np.inf]))[0] == 0.0
    assert np.isnan(mgo.exp(np.float32([np.nan]))[0])
    x = np.sort(np.random.default_rng(0).uniform(-80, 80, 200_000).astype(np.float32))
    y = mgo.exp(x)
    assert np.all(np.diff(y) >= 0)


# ----------------------------------------------------------------------------- CDOT

def test_cdot_golden_order_cases():
    d = json.load(open(os.path.join(GOLD, "cdot_order.json")))
    for case in d["cases"]:
        x = np.zeros(case["K"], f32)
        w = np.zeros(case["K"], f32)
        for g, e, xv, wv in case["terms"]:
            x[8 * g + e] = xv
            w[8 * g + e] = wv
        assert mgo.cdot(x, w) == f32(case["expect"]), case["name"]
        seq = f32(0)
        for xi, wi in zip(x, w):
            seq = f32(seq + f32(xi * wi))
        assert seq == f32(case["sequential"]), case["name"]


@pytest.mark.parametrize("K", [8, 64, 256, 504, 688, 4096, 14336])
def test_cdot_small_integers_exact(K):
    rng = np.random.default_rng(K)
    x = rng.integers(-3, 4, K).astype(f32)
    w = rng.integers(-3, 4, K).astype(f32)
    assert mgo.cdot(x, w) == float(np.dot(x.astype(np.int64), w.astype(np.int64)))


@pytest.mark.parametrize("K", [512, 4096])
def test_cdot_error_bound(K):
    rng = np.random.default_rng(11)
    x = rng.standard_normal(K).astype(f32)
    w = rng.standard_normal(K).astype(f32)
    exact = float(np.dot(x.astype(np.float64), w.astype(np.float64)))
    bound = K * 2.0 ** -24 * float(np.abs(x.astype(np.float64) * w).sum()) * 1.01
    assert abs(mgo.cdot(x, w) - exact) <= bound


# ----------------------------------------------------------------------------- RMSNorm

@pytest.mark.parametrize("mode", [mgo.PLAIN, mgo.CANON])
def test_rmsnorm_closed_forms(mode):
    one = mgo.bf16_from_f32(np.ones(8, f32))
    x = mgo.bf16_from_f32(np.array([3, 4, 0, 0, 0, 0, 0, 0], f32))
    eps = 1e-5
    y = mgo.f32_from_bf16(mgo.rmsnorm(mode, x, one, eps))
    r = 1.0 / math.sqrt(25.0 / 8.0 + eps)
    np.testing.assert_allclose(y[:2], [3 * r, 4 * r], rtol=2 ** -8)
    assert np.all(y[2:] == 0)
    # constant vector c -> c / sqrt(c^2 + eps), i.e. +-1 to bf16 rounding
    for c in (0.5, -2.0, 7.0):
        v = mgo.bf16_from_f32(np.full(64, c, f32))
        yy = mgo.f32_from_bf16(mgo.rmsnorm(mode, v, mgo.bf16_from_f32(np.ones(64, f32)), eps))
        np.testing.assert_allclose(yy, c / math.sqrt(c * c + eps), rtol=2 ** -8)


@pytest.mark.parametrize("mode", [mgo.PLAIN, mgo.CANON])
def test_rmsnorm_scale_invariance_and_gain(mode):
    """eps = 0: scaling x by 2 is exact in every step, so the output is bit-identical;
    a gain of 2 doubles the output exactly."""
    x = synth.random_bf16(4096, seed=4)
    x2 = mgo.bf16_from_f32(mgo.f32_from_bf16(x) * 2)
    one = mgo.bf16_from_f32(np.ones(4096, f32))
    two = mgo.bf16_from_f32(np.full(4096, 2, f32))
    y = mgo.rmsnorm(mode, x, one, 0.0)
    np.testing.assert_array_equal(mgo.rmsnorm(mode, x2, one, 0.0), y)
    np.testing.assert_array_equal(mgo.f32_from_bf16(mgo.rmsnorm(mode, x, two, 0.0)), 2 * mgo.f32_from_bf16(y))


# ----------------------------------------------------------------------------- Linear

@pytest.mark.parametrize("mode", [mgo.PLAIN, mgo.CANON])
def test_linear_one_hot_returns_column(mode):
    W = synth.random_bf16((24, 512), seed=5)
    for k in (0, 7, 8, 300, 511):
        x = np.zeros(512, np.uint16)
        x[k] = 0x3F80  # 1.0
        np.testing.assert_array_equal(mgo.linear(mode, x, W), W[:, k])


@pytest.mark.parametrize("mode", [mgo.PLAIN, mgo.CANON])
def test_linear_small_integers_exact_with_bias(mode):
    W = synth.small_int_bf16((40, 688), seed=6)
    x = synth.small_int_bf16((688,), seed=7)
    b = synth.small_int_bf16((40,), seed=8)
    Wi = mgo.f32_from_bf16(W).astype(np.int64)
    xi = mgo.f32_from_bf16(x).astype(np.int64)
    bi = mgo.f32_from_bf16(b).astype(np.int64)
    y = mgo.linear(mode, x, W, b, fp32=True)
    np.testing.assert_array_equal(y, (Wi @ xi + bi).astype(f32))


# ----------------------------------------------------------------------------- RoPE

def test_rope_position_zero_is_identity():
    v = synth.random_bf16((3, 128), seed=9)
    np.testing.assert_array_equal(mgo.rope(128, 0, 5e5, v), v)


@pytest.mark.parametrize("hd,theta", [(64, 1e4), (128, 5e5), (128, 1e6)])
def test_rope_matches_complex_rotation(hd, theta):
    """Rotate-half RoPE equals multiplying z_i = v_i + i v_(i+hd/2) by exp(i pos theta^(-2i/hd))."""
    v = synth.random_bf16((2, hd), seed=10)
    h = hd // 2
    for pos in (1, 17, 511, 16383):
        got = mgo.f32_from_bf16(mgo.rope(hd, pos, theta, v)).reshape(2, hd)
        vf = mgo.f32_from_bf16(v).reshape(2, hd).astype(np.float64)
        z = vf[:, :h] + 1j * vf[:, h:]
        ang = pos * theta ** (-2.0 * np.arange(h) / hd)
        r = z * np.exp(1j * ang)
        ref = np.concatenate([r.real, r.imag], axis=1)
        np.testing.assert_allclose(got, ref, rtol=2 ** -7, atol=2 ** -7 * np.abs(vf).max())
        # each pair keeps its norm up to bf16 rounding
        n0 = np.abs(z)
        n1 = np.hypot(got[:, :h], got[:, h:])
        np.testing.assert_allclose(n1, n0, rtol=2 ** -7, atol=1e-6)


# ----------------------------------------------------------------------------- SwiGLU

@pytest.mark.parametrize("mode", [mgo.PLAIN, mgo.CANON])
def test_swiglu_closed_forms(mode):
    g = mgo.bf16_from_f32(np.array([0, 0, 20, -20, 1, -1, 2, 3], f32))
    u = mgo.bf16_from_f32(np.array([5, -3, 2, 2, 1, 1, 0.5, -1], f32))
    a = mgo.f32_from_bf16(mgo.swiglu(mode, g, u))
    gf = mgo.f32_from_bf16(g).astype(np.float64)
    uf = mgo.f32_from_bf16(u).astype(np.float64)
    ref = gf / (1 + np.exp(-gf)) * uf
    np.testing.assert_allclose(a, ref, rtol=2 ** -8, atol=1e-7)
    assert a[0] == 0 and a[1] == 0
    assert a[2] == 40.0  # silu(20) = 20 to fp32 precision, times 2


# ----------------------------------------------------------------------------- attention

@pytest.mark.parametrize("mode", [mgo.PLAIN, mgo.CANON])
def test_attention_hand_computed_two_tokens(mode):
    hd = 64
    q = mgo.bf16_from_f32(np.r_[np.ones(4), np.zeros(hd - 4)].astype(f32))
    k = mgo.bf16_from_f32(np.zeros((2, hd), f32))
    v = mgo.bf16_from_f32(np.array([[2.0] * hd, [4.0] * hd], f32) * np.arange(1, hd + 1, dtype=f32) / 8)
    # equal scores -> mean of the two values
    out = mgo.f32_from_bf16(mgo.attend(mode, q, k, v))
    vf = mgo.f32_from_bf16(v)
    np.testing.assert_array_equal(out, mgo.f32_from_bf16(mgo.bf16_from_f32(((vf[0] + vf[1]) / 2).astype(f32))))
    # single position -> that value, exactly
    np.testing.assert_array_equal(mgo.attend(mode, q, k[:1], v[:1]), v[0])
    # score gap ln 3 -> weights 1/4, 3/4
    kk = np.zeros((2, hd), f32)
    kk[1, 0] = math.log(3.0) * math.sqrt(hd)  # q.k1 * (1/sqrt(hd)) = ln 3 (to bf16 precision)
    kb = mgo.bf16_from_f32(kk)
    gap = mgo.f32_from_bf16(kb)[1, 0] / math.sqrt(hd)
    w1 = math.exp(gap) / (1 + math.exp(gap))
    out = mgo.f32_from_bf16(mgo.attend(mode, q, kb, v))
    np.testing.assert_allclose(out, (1 - w1) * vf[0] + w1 * vf[1], rtol=2 ** -7)
    assert abs(w1 - 0.75) < 2e-3


@pytest.mark.parametrize("n", [1, 255, 256, 257, 600, 1100])
def test_attention_long_contexts_vs_float64_softmax(n):
    """Both modes, across the 256-position chunk boundaries of the canonical order."""
    hd = 128
    q = synth.random_bf16((hd,), seed=20)
    K = synth.random_bf16((n, hd), seed=21)
    V = synth.random_bf16((n, hd), seed=22)
    qf, Kf, Vf = (mgo.f32_from_bf16(a).astype(np.float64) for a in (q, K, V))
    s = Kf @ qf / math.sqrt(hd)
    p = np.exp(s - s.max())
    ref = (p / p.sum()) @ Vf
    for mode in (mgo.PLAIN, mgo.CANON):
        out = mgo.f32_from_bf16(mgo.attend(mode, q, K, V))
        np.testing.assert_allclose(out, ref, rtol=2 ** -7, atol=2 ** -8 * np.abs(ref).max())


def test_attention_equal_keys_average_all_positions():
    hd, n = 64, 700
    q = synth.random_bf16((hd,), seed=23)
    K = np.tile(synth.random_bf16((1, hd), seed=24), (n, 1))
    V = synth.small_int_bf16((n, hd), seed=25, lo=-4, hi=4)
    ref = mgo.f32_from_bf16(V).astype(np.float64).mean(0)
    for mode in (mgo.PLAIN, mgo.CANON):
        out = mgo.f32_from_bf16(mgo.attend(mode, q, K, V))
        np.testing.assert_allclose(out, ref, rtol=2 ** -7, atol=1e-2)


# ----------------------------------------------------------------------------- top-2 / gate

def _top2_bruteforce(row):
    """Stable sort of (value desc, index asc) with NaN ranked last."""
    idx = sorted(range(len(row)), key=lambda j: (0 if not np.isnan(row[j]) else 1,
                                                  -row[j] if not np.isnan(row[j]) else 0, j))
    if np.isnan(row).any():
        return idx[0], float("nan")
    return idx[0], float(f32(row[idx[0]]) - f32(row[idx[1]]))


def _adversarial_rows(V, rng):
    rows = [np.zeros(V, f32), rng.standard_normal(V).astype(f32)]
    r = rng.standard_normal(V).astype(f32); r[V - 1] = 50; rows.append(r)
    r = rng.standard_normal(V).astype(f32); r[0] = 50; rows.append(r)
    r = rng.standard_normal(V).astype(f32); r[[5, V // 2]] = 9.0; rows.append(r)          # duplicated max
    r = np.full(V, -1.0, f32); r[3] = -0.0; r[7] = 0.0; rows.append(r)                   # -0 == +0 tie
    r = rng.standard_normal(V).astype(f32); r[11] = np.nan; rows.append(r)
    r = np.round(rng.standard_normal(V) * 4).astype(f32); rows.append(r)                # many ties
    r = rng.standard_normal(V).astype(f32); r[V - 2] = 8.0; r[V - 1] = np.nextafter(f32(8.0), f32(9)); rows.append(r)
    return rows


@pytest.mark.parametrize("V", [7, 4096, 128256, 152064])
def test_top2_against_bruteforce(V):
    rng = np.random.default_rng(V)
    rows = _adversarial_rows(V, rng) if V > 20 else [rng.standard_normal(V).astype(f32) for _ in range(50)]
    for row in rows:
        t, m = mgo.top2(row)
        if V <= 4096:
            bt, bm = _top2_bruteforce(row)
        else:  # same definition through numpy's stable argsort
            if np.isnan(row).any():
                bt = int(np.argmax(np.where(np.isnan(row), -np.inf, row)))
                bm = float("nan")
            else:
                order = np.argsort(-row.astype(np.float64), kind="stable")
                bt, bm = int(order[0]), float(row[order[0]] - row[order[1]])
        assert t == bt
        assert (math.isnan(m) and math.isnan(bm)) or m == bm


def test_near_tie_count_identity():
    """Obs. 3: N(Delta) = |{j : l_j >= l_(1) - Delta}| > 1 exactly when g < Delta... for Delta at
    which l_(1) - Delta is exact; with the sign convention of the paper's Table 4."""
    rng = np.random.default_rng(5)
    for _ in range(200):
        row = (rng.standard_normal(4096) * 0.5).astype(np.float64)
        row = np.round(row * 64) / 64  # dyadic: every difference below is exact
        row = row.astype(f32)
        _, g = mgo.top2(row)
        l1 = row.max()
        for delta in (0.0, 1 / 64, 0.25, 0.5, 1.0, 2.0):
            N = int(np.sum(row.astype(np.float64) >= float(l1) - delta))
            # N counts values within Delta of the top (inclusive); g <= Delta iff a second one is there
            assert (N > 1) == (g <= delta)


def test_margin_gate_strict_threshold_mask_and_nan():
    V = 64
    base = np.linspace(-1, -0.1, V).astype(f32)
    rows = []
    for m in (0.5, np.nextafter(f32(0.5), f32(0)), np.nextafter(f32(0.5), f32(1)), 0.0, 3.0):
        r = base.copy(); r[10] = f32(m); r[20] = 0.0; rows.append(r)   # g = m - 0 exactly
    r = base.copy(); r[3] = np.nan; rows.append(r)
    L = np.stack(rows)
    tau = 0.5
    top1, margin, gate, grows = mgo.OracleModel.margin_gate(L, None, tau)
    assert list(top1[:5]) == [10, 10, 10, 10, 10]  # m = 0: tie at 0, lower index 10 wins
    assert margin[0] == f32(0.5)
    assert list(gate) == [0, 1, 0, 1, 0, 1]   # g == tau does not trigger; NaN always does
    assert list(grows) == [1, 3, 5]
    prot = np.array([1, 0, 1, 1, 1, 0], np.uint8)
    _, _, gate2, grows2 = mgo.OracleModel.margin_gate(L, prot, tau)
    assert list(gate2) == [0, 0, 0, 1, 0, 0]
    assert list(grows2) == [3]


# ----------------------------------------------------------------------------- whole decoder

def _tiny_model(max_batch=4, ctx=64, seed=0, shape=synth.TINY):
    w = synth.weights_to_numpy(synth.make_weights(shape, seed=seed))
    pt, n_pages = synth.make_page_table([ctx] * max_batch, shape.page_size, -(-ctx // shape.page_size), seed=5)
    return mgo.OracleModel(shape, w, max_batch, pt.shape[1], n_pages), w, pt


def _torch_reference_logits(shape, w, tokens):
    """A textbook causal decoder in float64 with torch library routines (rms_norm,
    scaled_dot_product_attention with GQA, silu, complex-number RoPE), rounding to bf16
    at the same points.  Returns the logits of the last position."""
    def bf(t):
        return t.to(torch.bfloat16).to(torch.float64)
    def T(a):
        return None if a is None else torch.from_numpy(a.view(np.int16).copy()).view(torch.bfloat16).to(torch.float64)
    W = [T(a) for a in w]
    d, Hq, Hkv, hd = shape.d_model, shape.n_q_heads, shape.n_kv_heads, shape.head_dim
    n = len(tokens)
    pos = torch.arange(n, dtype=torch.float64)
    ang = pos[:, None] * shape.rope_theta ** (-2.0 * torch.arange(hd // 2, dtype=torch.float64) / hd)
    rot = torch.polar(torch.ones_like(ang), ang)

    def rope(t):  # t [n, H, hd]
        z = torch.complex(t[..., : hd // 2], t[..., hd // 2:]) * rot[:, None, :]
        return bf(torch.cat([z.real, z.imag], -1))

    x = W[0][torch.as_tensor(tokens, dtype=torch.long)]
    for l in range(shape.n_layers):
        b = 1 + 12 * l
        h = bf(F.rms_norm(x, (d,), W[b + 0], shape.rms_eps))
        q = bf(h @ W[b + 1].T + (W[b + 4] if W[b + 4] is not None else 0)).view(n, Hq, hd)
        k = bf(h @ W[b + 2].T + (W[b + 5] if W[b + 5] is not None else 0)).view(n, Hkv, hd)
        v = bf(h @ W[b + 3].T + (W[b + 6] if W[b + 6] is not None else 0)).view(n, Hkv, hd)
        q, k = rope(q), rope(k)
        a = F.scaled_dot_product_attention(q.transpose(0, 1), k.transpose(0, 1), v.transpose(0, 1),
                                           is_causal=True, enable_gqa=True)
        a = bf(a.transpose(0, 1).reshape(n, Hq * hd))
        x = bf(x + bf(a @ W[b + 7].T))
        h = bf(F.rms_norm(x, (d,), W[b + 8], shape.rms_eps))
        g = bf(h @ W[b + 9].T)
        u = bf(h @ W[b + 10].T)
        x = bf(x + bf(bf(F.silu(g) * u) @ W[b + 11].T))
    h = bf(F.rms_norm(x, (d,), W[1 + 12 * shape.n_layers], shape.rms_eps))
    return (h[-1] @ W[2 + 12 * shape.n_layers].T).numpy()


def _normwise(a, ref):
    return float(np.abs(a.astype(np.float64) - ref).max() / np.abs(ref).max())


@pytest.mark.parametrize("mode", [mgo.PLAIN, mgo.CANON])
def test_decoder_matches_float64_library_reference(mode):
    shape = synth.TINY
    om, w, pt = _tiny_model(max_batch=1, ctx=48)
    toks = synth.make_prompts(1, [40], shape.vocab, seed=1)[0]
    om.prefill(mode, toks[:-1], pt[0])
    logits = om.decode_step(mode, toks[-1:], np.array([39], np.int32), pt[:1])[0]
    ref = _torch_reference_logits(shape, w, toks)
    assert _normwise(logits, ref) < 5e-3


def test_decoder_with_qkv_bias_matches_reference():
    shape = synth.ModelShape("tiny-bias", 2, 256, 8, 2, 32, 344, 1024, True, 1e6, 1e-6)
    om, w, pt = _tiny_model(max_batch=1, ctx=32, shape=shape)
    toks = synth.make_prompts(1, [20], shape.vocab, seed=3)[0]
    om.prefill(mgo.CANON, toks[:-1], pt[0])
    logits = om.decode_step(mgo.CANON, toks[-1:], np.array([19], np.int32), pt[:1])[0]
    assert _normwise(logits, _torch_reference_logits(shape, w, toks)) < 5e-3


def test_causality_future_cache_is_ignored():
    om, w, pt = _tiny_model(max_batch=1, ctx=48)
    toks = synth.make_prompts(1, [30], synth.TINY.vocab, seed=1)[0]
    om.prefill(mgo.CANON, toks[:-1], pt[0])
    snap = om.kv_pool.copy()
    a = om.decode_step(mgo.CANON, toks[-1:], np.array([29], np.int32), pt[:1])
    om.kv_pool[:] = snap
    kv = om.kv_view()
    # scribble over positions 30..47 (pages 1 slot 14.. and page 2) of row 0 in every layer
    for p in range(30, 48):
        kv[:, pt[0, p // 16], :, :, p % 16, :] = 0x4040
    b = om.decode_step(mgo.CANON, toks[-1:], np.array([29], np.int32), pt[:1])
    np.testing.assert_array_equal(a, b)


def test_batch_invariance_row_alone_vs_any_placement():
    om, w, pt = _tiny_model(max_batch=4, ctx=48)
    prompts = synth.make_prompts(4, [12, 20, 7, 30], synth.TINY.vocab, seed=1)
    for r in range(4):
        om.prefill(mgo.PLAIN, prompts[r][:-1], pt[r])
    snap = om.kv_pool.copy()
    toks = np.array([p[-1] for p in prompts], np.int32)
    pos = np.array([len(p) - 1 for p in prompts], np.int32)
    full = om.decode_step(mgo.PLAIN, toks, pos, pt)
    for perm in ([3, 1, 0, 2], [2], [0, 3]):
        om.kv_pool[:] = snap
        part = om.decode_step(mgo.PLAIN, toks[perm], pos[perm], pt[perm])
        np.testing.assert_array_equal(part, full[perm])


def test_verifier_scratch_column_equals_cache_path():
    """verify_rows (own column in scratch, cache untouched) equals a canonical decode step
    of the same row (own column appended to the cache), bit for bit."""
    om, w, pt = _tiny_model(max_batch=2, ctx=48)
    prompts = synth.make_prompts(2, [25, 33], synth.TINY.vocab, seed=1)
    for r in range(2):
        om.prefill(mgo.CANON, prompts[r][:-1], pt[r])
    toks = np.array([p[-1] for p in prompts], np.int32)
    pos = np.array([24, 32], np.int32)
    before = om.kv_pool.copy()
    vl, vt, col = om.verify_rows(np.array([1, 0], np.int32), toks, pos, pt)
    np.testing.assert_array_equal(om.kv_pool, before)  # verifier never writes the cache
    lg = om.decode_step(mgo.CANON, toks, pos, pt)
    np.testing.assert_array_equal(vl, lg[[1, 0]])
    assert list(vt) == [int(np.argmax(lg[1])), int(np.argmax(lg[0]))]
    kv = om.kv_view()
    c1 = col[0].reshape(synth.TINY.n_layers, 2, synth.TINY.n_kv_heads, synth.TINY.head_dim)
    np.testing.assert_array_equal(c1, kv[:, pt[1, 32 // 16], :, :, 32 % 16, :])


def test_repair_overwrites_only_the_current_column():
    """Sec. 3.2: a verified commit keeps the tentative column; a repair copies the verifier's
    column at the current position in every layer and nothing else."""
    om, w, pt = _tiny_model(max_batch=3, ctx=48)
    rng = np.random.default_rng(0)
    om.kv_pool[:] = rng.integers(0, 1 << 16, om.kv_pool.size, dtype=np.uint16)
    before = om.kv_pool.copy()
    rows = np.array([0, 2], np.int32)
    pos = np.array([5, 40, 17], np.int32)
    top1 = np.array([10, 11, 12], np.int32)
    v_tok = np.array([10, 99], np.int32)      # row 0 agrees (verified commit), row 2 differs (repair)
    col = rng.integers(0, 1 << 16, (2, om.col_elems()), dtype=np.uint16)
    emitted, nrep = om.repair(rows, pos, pt, top1, v_tok, col, top1)
    assert list(emitted) == [10, 11, 99] and nrep == 1
    kv, kb = om.kv_view(), before.reshape(om.kv_view().shape)
    s = synth.TINY
    np.testing.assert_array_equal(kv[:, pt[2, 1], :, :, 1, :], col[1].reshape(s.n_layers, 2, s.n_kv_heads, s.head_dim))
    mask = np.ones(kv.shape, bool)
    mask[:, pt[2, 1], :, :, 1, :] = False
    np.testing.assert_array_equal(kv[mask], kb[mask])


@pytest.mark.parametrize("action", [mgo.REPAIR_TOKEN_ONLY, mgo.REPAIR_COPY_ALWAYS])
def test_repair_action_variants(action):
    """The two repair actions around the commit rule (Sec. 3.2): token only -- the
    repair-action ablation of Sec. 4, the verifier's token is emitted and the cache keeps
    the tentative column (no byte changes, no repair counted); copy always -- every verified
    row's column is overwritten, agreeing rows included, and nothing else."""
    om, w, pt = _tiny_model(max_batch=3, ctx=48)
    rng = np.random.default_rng(1)
    om.kv_pool[:] = rng.integers(0, 1 << 16, om.kv_pool.size, dtype=np.uint16)
    before = om.kv_pool.copy()
    rows = np.array([0, 2], np.int32)
    pos = np.array([5, 40, 17], np.int32)
    top1 = np.array([10, 11, 12], np.int32)
    v_tok = np.array([10, 99], np.int32)      # row 0 agrees, row 2 differs
    col = rng.integers(0, 1 << 16, (2, om.col_elems()), dtype=np.uint16)
    emitted, nrep = om.repair(rows, pos, pt, top1, v_tok, col, top1, action)
    assert list(emitted) == [10, 11, 99]
    kv, kb = om.kv_view(), before.reshape(om.kv_view().shape)
    s = synth.TINY
    if action == mgo.REPAIR_TOKEN_ONLY:
        assert nrep == 0
        np.testing.assert_array_equal(om.kv_pool, before)
        return
    assert nrep == 2
    mask = np.ones(kv.shape, bool)
    for i, r in enumerate(rows):
        page, slot = pt[r, pos[r] // 16], pos[r] % 16
        np.testing.assert_array_equal(kv[:, page, :, :, slot, :], col[i].reshape(s.n_layers, 2, s.n_kv_heads, s.head_dim))
        mask[:, page, :, :, slot, :] = False
    np.testing.assert_array_equal(kv[mask], kb[mask])


def test_plain_and_canonical_agree_within_tolerance():
    om, w, pt = _tiny_model(max_batch=1, ctx=48)
    toks = synth.make_prompts(1, [33], synth.TINY.vocab, seed=9)[0]
    om.prefill(mgo.CANON, toks[:-1], pt[0])
    snap = om.kv_pool.copy()
    a = om.decode_step(mgo.CANON, toks[-1:], np.array([32], np.int32), pt[:1])[0]
    om.kv_pool[:] = snap
    b = om.decode_step(mgo.PLAIN, toks[-1:], np.array([32], np.int32), pt[:1])[0]
    assert _normwise(b, a.astype(np.float64)) < 1e-2


def test_gated_loop_canonical_fast_path_never_repairs():
    """When the fast path and the verifier share the canonical order, every verified step
    agrees (r_repair = 0) and the emitted token is the fast argmax."""
    om, w, pt = _tiny_model(max_batch=4, ctx=64)
    prompts = synth.make_prompts(4, [32] * 4, synth.TINY.vocab, seed=1)
    for r in range(4):
        om.prefill(mgo.CANON, prompts[r][:-1], pt[r])
    toks = np.array([p[-1] for p in prompts], np.int32)
    pos = np.full(4, 31, np.int32)
    for _ in range(4):
        emitted, rec = om.gated_step(mgo.CANON, toks, pos, pt, None, 0.5)
        assert rec["n_repaired"] == 0
        np.testing.assert_array_equal(emitted, rec["top1"])
        toks, pos = emitted, pos + 1



@pytest.mark.parametrize("mode", [mgo.PLAIN, mgo.CANON])
@pytest.mark.parametrize("bias", [False, True])
def test_step_cut_at_layers_composes_to_decode_step(mode, bias):
    """mgo_embed, mgo_layer over every layer and mgo_head, called one after another on rows
    with different positions, give the decode step's logits and cache bit for bit (the
    entry points the per-layer state-forced GPU checks feed with the GPU's own layer
    inputs)."""
    shape = synth.ModelShape("tiny-bias", 2, 256, 8, 2, 32, 344, 1024, True, 1e6, 1e-6) if bias else synth.TINY
    om, w, pt = _tiny_model(max_batch=3, ctx=48, shape=shape)
    prompts = synth.make_prompts(3, [12, 31, 5], shape.vocab, seed=2)
    for r in range(3):
        om.prefill(mode, prompts[r][:-1], pt[r])
    snap = om.kv_pool.copy()
    toks = np.array([p[-1] for p in prompts], np.int32)
    pos = np.array([len(p) - 1 for p in prompts], np.int32)
    ref = om.decode_step(mode, toks, pos, pt)
    ref_kv = om.kv_pool.copy()
    om.kv_pool[:] = snap
    x = om.embed(toks)
    np.testing.assert_array_equal(x, w[0][toks])
    for l in range(shape.n_layers):
        y = om.layer(mode, l, x, pos, pt)
        assert not np.array_equal(y, x)
        x = y
    np.testing.assert_array_equal(om.head(mode, x).view(np.uint32), ref.view(np.uint32))
    np.testing.assert_array_equal(om.kv_pool, ref_kv)
    # a layer writes only its own layer's column at each row's position
    om.kv_pool[:] = snap
    om.layer(mode, 1, om.embed(toks), pos, pt)
    changed = np.argwhere(om.kv_view() != snap.reshape(om.kv_view().shape))
    assert changed.size and set(changed[:, 0].tolist()) == {1}
    for r in range(3):
        p = int(pos[r])
        assert ((changed[:, 1] == pt[r, p // 16]) & (changed[:, 4] == p % 16)).any()
    assert set(zip(changed[:, 1].tolist(), changed[:, 4].tolist())) <= \
        {(int(pt[r, int(pos[r]) // 16]), int(pos[r]) % 16) for r in range(3)}
