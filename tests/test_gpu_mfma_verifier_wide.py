"""The matrix-core verifier (mg_verify_rows_mfma) at the Llama-3.1-8B widths, where its
fixed split-K is not 1 (GPU).

A 2-layer decoder at full width (d 4096, 32/8 heads, hd 128, FFN 14336, vocab 128256) with
256 rows of ragged context (seeded synthetic bf16 caches of 32..300 positions).  With the
split-K fixed as for 32 rows the QKV projection is split 5 ways and the O and down
projections 8 ways; the split a list of n rows would choose on its own differs for n in
{33, 64, 128, 129, 256}.  Checked (deterministic verifier contract, Sec. 3.2):
  batch invariance   a row's logits, token and K/V column are bit-identical for list sizes
                     1, 2, 31, 32, 33, 64, 128, 129, 256, at the first, the last and a
                     middle place, for three different rows
  oracle parity      logits within normwise 1e-2 of the oracle's canonical verifier on the
                     same cache, each layer's K/V column within normwise 1e-2, and the token
                     the oracle's argmax except at an oracle near-tie below twice the
                     measured l_inf gap
  cache              only read"""
import numpy as np
import pytest
import torch

from paper_2605_30218_amd import mg, synth

from _gpu_common import dev_i32, normwise, oracle_for_rows, u16

pytestmark = pytest.mark.gpu
SHAPE = synth.ModelShape("llama3.1-8b-width-2l", 2, 4096, 32, 8, 128, 14336, 128256, False, 5e5, 1e-5)
NB = 256
SIZES = (1, 2, 31, 32, 33, 64, 128, 129, 256)
TARGETS = (0, 129, 255)
SPLIT_M = 32  # the row count whose split-K the matrix-core verifier fixes


@pytest.fixture(scope="module")
def wide2():
    lens = synth.make_lengths(NB, 32, 300, seed=8)
    ctx = int(lens.max()) + 16
    maxp = -(-ctx // SHAPE.page_size)
    pt, n_pages = synth.make_page_table([ctx] * NB, SHAPE.page_size, maxp, seed=7)
    w = synth.make_weights(SHAPE, seed=3, device="cuda")
    eng = mg.Engine(SHAPE, w, NB, maxp, n_pages)
    cached = np.concatenate([pt[r, :-(-(int(lens[r]) - 1) // SHAPE.page_size)] for r in range(NB)])
    synth.fill_synthetic_kv(eng.kv_view(), cached, seed=9)
    tok = synth.make_prompts(1, [NB], SHAPE.vocab, seed=10)[0]
    pos = (lens - 1).astype(np.int32)
    yield dict(eng=eng, pt=pt, tok=tok, pos=pos, wn=synth.weights_to_numpy(w))
    eng.close()


def run(f, rows):
    eng = f["eng"]
    n = len(rows)
    vl = torch.empty((n, SHAPE.vocab), dtype=torch.float32, device="cuda")
    vt = torch.empty(n, dtype=torch.int32, device="cuda")
    vc = torch.empty((n, eng.col_elems), dtype=torch.int16, device="cuda")
    eng.verify_rows_mfma(n, dev_i32(rows), dev_i32(f["tok"]), dev_i32(f["pos"]), dev_i32(f["pt"]), vl, vt, vc)
    torch.cuda.synchronize()
    return vl.cpu().numpy(), vt.cpu().numpy(), u16(vc)


def test_fixed_split_is_not_one_and_differs_from_the_lists_own():
    d, F, Nq, Nk = SHAPE.d_model, SHAPE.d_ffn, SHAPE.n_q_heads * SHAPE.head_dim, SHAPE.n_kv_heads * SHAPE.head_dim
    projs = [(Nq + 2 * Nk, d), (d, Nq), (2 * F, d), (d, F)]
    fixed = [mg.fast_gemm_config(SPLIT_M, N, K)[0] for N, K in projs]
    print("split-K fixed for the matrix-core verifier (QKV, O, gate/up, down):", fixed)
    assert sum(S > 1 for S in fixed) >= 2
    moved = {n for n in SIZES for (N, K), S in zip(projs, fixed) if mg.fast_gemm_config(n, N, K)[0] != S}
    print("list sizes whose own split would differ:", sorted(moved))
    assert {64, 128, 256} <= moved


def test_mfma_verifier_invariant_where_split_k_is_fixed(wide2):
    f = wide2
    rng = np.random.default_rng(23)
    before = u16(f["eng"].kv_pool).copy()
    for target in TARGETS:
        l0, t0, c0 = run(f, [target])
        for n in SIZES[1:]:
            others = rng.choice(np.setdiff1d(np.arange(NB), [target]), n - 1, replace=False)
            for place in sorted({0, n - 1, n // 2}):
                rows = [int(r) for r in others[:place]] + [target] + [int(r) for r in others[place:]]
                l, t, c = run(f, rows)
                assert np.array_equal(l[place].view(np.uint32), l0[0].view(np.uint32)), (target, n, place)
                assert t[place] == t0[0], (target, n, place)
                assert np.array_equal(c[place], c0[0]), (target, n, place)
    np.testing.assert_array_equal(u16(f["eng"].kv_pool), before)


def test_mfma_verifier_within_tolerance_of_the_oracle_at_full_width(wide2):
    f = wide2
    rows = list(TARGETS)
    gl, gt, gc = run(f, rows)
    om, ptl = oracle_for_rows(SHAPE, f["wn"], f["eng"], f["pt"], rows)
    rl, rt, rc = om.verify_rows(np.arange(len(rows), dtype=np.int32), f["tok"][rows], f["pos"][rows], ptl)
    L, Hkv, hd = SHAPE.n_layers, SHAPE.n_kv_heads, SHAPE.head_dim
    f32 = lambda u: (u.astype(np.uint32) << 16).view(np.float32)  # noqa: E731
    for i in range(len(rows)):
        err = normwise(gl[i], rl[i])
        gcol = f32(gc[i]).reshape(L, 2, Hkv * hd)
        rcol = f32(rc[i]).reshape(L, 2, Hkv * hd)
        cerr = max(normwise(gcol[l, j], rcol[l, j]) for l in range(L) for j in range(2))
        print(f"row {rows[i]}: logits {err:.2e}, K/V column {cerr:.2e}, token {gt[i]} vs {rt[i]}")
        assert err <= 1e-2, (rows[i], err)
        assert cerr <= 1e-2, (rows[i], cerr)
        if gt[i] != rt[i]:
            srt = np.sort(rl[i])[::-1]
            assert srt[0] - srt[1] <= 2 * np.abs(gl[i] - rl[i]).max(), rows[i]


def test_mfma_verifier_fused_top2_epilogue(wide2):
    """Without a logits buffer the matrix-core verifier's LM head runs with the fused top-2
    epilogue (per-block states merged per row): the same tokens and K/V columns as with the
    logits written, and batch-invariant the same way."""
    f = wide2
    eng = f["eng"]

    def run_nologits(rows):
        n = len(rows)
        vt = torch.empty(n, dtype=torch.int32, device="cuda")
        vc = torch.empty((n, eng.col_elems), dtype=torch.int16, device="cuda")
        eng.verify_rows_mfma(n, dev_i32(rows), dev_i32(f["tok"]), dev_i32(f["pos"]), dev_i32(f["pt"]), None, vt, vc)
        torch.cuda.synchronize()
        return vt.cpu().numpy(), u16(vc)

    rng = np.random.default_rng(31)
    for n in (1, 12, 33, 129, 256):
        rows = [int(r) for r in rng.choice(NB, n, replace=False)]
        _, t_ref, c_ref = run(f, rows)
        t, c = run_nologits(rows)
        np.testing.assert_array_equal(t, t_ref)
        np.testing.assert_array_equal(c, c_ref)
