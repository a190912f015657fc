"""Full-size parity on the Llama-3.1-8B-shaped decoder in the benchmark's launch configuration
(batch 64, 512-token prompts), on sampled rows the oracle recomputes one by one (GPU).

  fast step logits, full width, 2 and 32 layers
                                           within max(1e-2, twice the spread between two valid fp32 orders)
                                           (the verifier's canonical order vs the oracle's plain
                                           order) measured on the same rows and state: at this
                                           depth the random-init model amplifies any change of
                                           summation order to a few percent of the logit scale
  margin gate over 64 x 128256 logits      bit-exact
  verifier (sampled rows)                  bit-exact logits, token and K/V column
  verifier batch invariance                a row alone == inside 12 and 64 rows, any place
  single-column repair                     repaired columns == the oracle verifier's columns
The prompt cache comes from the canonical prefill, then one fast step appends the tentative
column; the oracle is state-forced from the GPU cache of the sampled rows."""
import numpy as np
import pytest
import torch

from oracle import mgo
from paper_2605_30218_amd import mg, synth
from paper_2605_30218_amd.runtime import GatedDecoder, prefill_rows

from _gpu_common import dev_i32, normwise, u16

pytestmark = pytest.mark.gpu
S = synth.LLAMA8B
B, P = 64, 512
SAMPLE = [0, 1, 37, 63]


@pytest.fixture(scope="module")
def full():
    ctx = P + 8
    maxp = -(-ctx // 16)
    pt, n_pages = synth.make_page_table([ctx] * B, 16, maxp, seed=5)
    w = synth.make_weights(S, seed=0, device="cuda")
    eng = mg.Engine(S, w, B, maxp, n_pages, max_prefill=1024)
    prompts = synth.make_prompts(B, [P] * B, S.vocab, seed=1)
    last, pos0 = prefill_rows(eng, prompts, pt)
    wn = synth.weights_to_numpy(w)
    yield dict(eng=eng, pt=pt, last=last, pos0=pos0, wn=wn, maxp=maxp)
    eng.close()


def oracle_for_rows(f, rows):
    """An oracle holding only the given rows' pages, copied from the GPU cache."""
    maxp = f["maxp"]
    om = mgo.OracleModel(S, f["wn"], len(rows), maxp, len(rows) * maxp)
    src = torch.as_tensor(f["pt"][rows].reshape(-1).astype(np.int64)).cuda()
    torch.cuda.synchronize()
    om.kv_view()[:] = u16(f["eng"].kv_view()[:, src])
    return om, np.arange(len(rows) * maxp, dtype=np.int32).reshape(len(rows), maxp)


def test_full_verifier_bitexact_and_invariant(full):
    eng, pt = full["eng"], full["pt"]
    last, pos0 = full["last"], full["pos0"]
    dpt, dtok, dpos = dev_i32(pt), dev_i32(last), dev_i32(pos0)

    def run(rows):
        n = len(rows)
        vl = torch.empty((n, S.vocab), dtype=torch.float32, device="cuda")
        vt = torch.empty(n, dtype=torch.int32, device="cuda")
        vc = torch.empty((n, eng.col_elems), dtype=torch.int16, device="cuda")
        eng.verify_rows(n, dev_i32(rows), None, dtok, dpos, dpt, vl, vt, vc)
        torch.cuda.synchronize()
        return vl.cpu().numpy(), vt.cpu().numpy(), u16(vc)

    rows = [63, 0, 37]
    vl, vt, vc = run(rows)
    om, ptl = oracle_for_rows(full, rows)
    rl, rt, rc = om.verify_rows(np.arange(3, dtype=np.int32), last[rows], pos0[rows], ptl)
    np.testing.assert_array_equal(vl.view(np.uint32), rl.view(np.uint32))
    np.testing.assert_array_equal(vt, rt)
    np.testing.assert_array_equal(vc, rc)
    # the same row inside 12 and 64 rows, at several places
    rng = np.random.default_rng(0)
    for n, place in ((12, 0), (12, 11), (12, 5), (64, 63), (64, 30)):
        others = rng.choice(np.setdiff1d(np.arange(B), [37]), n - 1, replace=False)
        rr = list(others[:place]) + [37] + list(others[place:])
        l2, t2, c2 = run(rr)
        assert np.array_equal(l2[place].view(np.uint32), vl[2].view(np.uint32))
        assert t2[place] == vt[2]
        assert np.array_equal(c2[place], vc[2])


def test_full_fast_step_gate_and_repair(full):
    eng, pt = full["eng"], full["pt"]
    last, pos0 = full["last"], full["pos0"]
    snap = eng.kv_pool.clone()
    # fast-step logits vs the oracle (plain) on sampled rows, from the same pre-step cache
    om, ptl = oracle_for_rows(full, SAMPLE)
    ref = om.decode_step(mgo.PLAIN, last[SAMPLE], pos0[SAMPLE], ptl)
    dec = GatedDecoder(eng, pt, None, tau=0.06)
    dec.set_state(last, pos0)
    keep = {}
    dec.step("gated", keep=keep)
    torch.cuda.synchronize()
    post = u16(eng.kv_view())
    emitted = dec.tokens.cpu().numpy()
    # the spread between two valid orders on the same rows: the verifier (canonical order,
    # bit-exact with the oracle's canonical mode) against the oracle's plain order
    vl = torch.empty((len(SAMPLE), S.vocab), dtype=torch.float32, device="cuda")
    vt = torch.empty(len(SAMPLE), dtype=torch.int32, device="cuda")
    vc = torch.empty((len(SAMPLE), eng.col_elems), dtype=torch.int16, device="cuda")
    eng.kv_pool.copy_(snap)
    eng.verify_rows(len(SAMPLE), dev_i32(SAMPLE), None, dev_i32(last), dev_i32(pos0), dev_i32(pt), vl, vt, vc)
    torch.cuda.synchronize()
    canon = vl.cpu().numpy()
    spread = max(normwise(canon[k], ref[k]) for k in range(len(SAMPLE)))
    errs = [normwise(keep["logits"][r], ref[k]) for k, r in enumerate(SAMPLE)]
    print(f"32-layer fast-vs-plain {max(errs):.4f}, canonical-vs-plain spread {spread:.4f}")
    assert max(errs) <= max(1e-2, 2 * spread), (errs, spread)
    # the gate over the whole batch is bit-exact
    rt, rm, rg, rr = mgo.OracleModel.margin_gate(keep["logits"], None, dec.tau)
    np.testing.assert_array_equal(keep["top1"], rt)
    np.testing.assert_array_equal(keep["gate"], rg)
    np.testing.assert_array_equal(keep["rows"], rr)
    # every gated sampled row: verifier token and, on a mismatch, the repaired column
    eng.kv_pool.copy_(snap)
    gs = [r for r in SAMPLE if r in set(rr.tolist())]
    if gs:
        om2, ptl2 = oracle_for_rows(full, gs)
        _, vt, vc = om2.verify_rows(np.arange(len(gs), dtype=np.int32), last[gs], pos0[gs], ptl2,
                                    want_logits=False)
        for k, r in enumerate(gs):
            assert emitted[r] == vt[k]
            if vt[k] != rt[r]:
                p = pos0[r]
                col = post[:, pt[r, p // 16], :, :, p % 16, :]
                np.testing.assert_array_equal(col, vc[k].reshape(col.shape))
    for r in SAMPLE:
        if r not in set(rr.tolist()):
            assert emitted[r] == rt[r] and keep["margin"][r] >= dec.tau


def test_full_width_shallow_fast_step():
    """Every fast kernel at the benchmark's widths and launch configuration (d 4096, FFN
    14336, vocab 128256, 32/8 heads, hd 128, batch 64, context 512), two layers deep."""
    shape = synth.ModelShape("llama3.1-8b-width-2l", 2, 4096, 32, 8, 128, 14336, 128256, False, 5e5, 1e-5)
    ctx = P + 8
    maxp = -(-ctx // 16)
    pt, n_pages = synth.make_page_table([ctx] * B, 16, maxp, seed=5)
    w = synth.make_weights(shape, seed=3, device="cuda")
    eng = mg.Engine(shape, w, B, maxp, n_pages, max_prefill=1024)
    prompts = synth.make_prompts(B, [P] * B, shape.vocab, seed=4)
    last, pos0 = prefill_rows(eng, prompts, pt)
    rows = [0, 21, 63]
    maxpg = maxp
    om = mgo.OracleModel(shape, synth.weights_to_numpy(w), len(rows), maxpg, len(rows) * maxpg)
    src = torch.as_tensor(pt[rows].reshape(-1).astype(np.int64)).cuda()
    om.kv_view()[:] = u16(eng.kv_view()[:, src])
    logits = torch.empty((B, shape.vocab), dtype=torch.float32, device="cuda")
    eng.decode_step(B, dev_i32(last), dev_i32(pos0), dev_i32(pt), logits)
    torch.cuda.synchronize()
    ptl = np.arange(len(rows) * maxpg, dtype=np.int32).reshape(len(rows), maxpg)
    ref = om.decode_step(mgo.PLAIN, last[rows], pos0[rows], ptl)
    got = logits.cpu().numpy()
    errs = [normwise(got[r], ref[k]) for k, r in enumerate(rows)]
    # the verifier's canonical order on the same state gives the spread of valid orders
    om.kv_view()[:] = u16(eng.kv_view()[:, src])
    vl, _, _ = om.verify_rows(np.arange(len(rows), dtype=np.int32), last[rows], pos0[rows], ptl)
    spread = max(normwise(vl[k], ref[k]) for k in range(len(rows)))
    eng.close()
    print(f"2-layer full-width fast-vs-plain {max(errs):.4f}, canonical-vs-plain spread {spread:.4f}")
    assert max(errs) <= max(1e-2, 2 * spread), (errs, spread)
