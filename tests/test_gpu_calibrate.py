"""The tau calibration recipe (Sec. 3.1 threshold setting, Appendix A) on the tiny decoder (GPU).

  reference decode   the deterministic reference (verifier on every row, its column always
                     kept) equals the oracle's canonical greedy decode token for token, with a
                     bit-identical cache, and a row decoded alone equals the same row in the batch
  recipe             eps statistics, a frontier point per tau, tau_100 the smallest fully
                     deterministic tau of the grid
  repair actions     the three commits (copy on disagreement, token only, copy always); with
                     every step verified, copy always is the reference decode itself"""
import numpy as np
import pytest
import torch

from paper_2605_30218_amd import calibrate, diagnostics, mg, synth
from paper_2605_30218_amd.runtime import GatedDecoder

from _gpu_common import Pair, u16

pytestmark = pytest.mark.gpu
S = synth.TINY
STEPS = 24


@pytest.fixture(scope="module")
def pair():
    return Pair(S, max_batch=8, ctx_cap=96)


@pytest.fixture(scope="module")
def prompts():
    return synth.make_prompts(4, [32, 20, 32, 9], S.vocab, seed=1)


def fresh(pair, prompts):
    pair.eng.kv_pool.zero_()
    pair.om.kv_pool[:] = 0
    return pair.prefill(prompts)


def test_reference_decode_is_the_oracle_canonical_greedy_decode(pair, prompts):
    last, pos0 = fresh(pair, prompts)
    dec = GatedDecoder(pair.eng, pair.pt[:4], None, tau=0.0)
    dec.set_state(last, pos0)
    got = calibrate.reference_decode(dec, STEPS)
    torch.cuda.synchronize()
    rows = np.arange(4, dtype=np.int32)
    tok, pos = last.copy(), pos0.copy()
    never = np.full(4, -1, np.int32)
    for s in range(STEPS):
        _, vt, vc = pair.om.verify_rows(rows, tok, pos, pair.pt[:4], want_logits=False)
        emitted, _ = pair.om.repair(rows, pos, pair.pt[:4], never, vt, vc, never)
        np.testing.assert_array_equal(got[:, s], emitted, err_msg=f"step {s}")
        tok, pos = emitted, pos + 1
    np.testing.assert_array_equal(u16(pair.eng.kv_pool), pair.om.kv_pool)


def test_reference_decode_is_batch_invariant(pair, prompts):
    last, pos0 = fresh(pair, prompts)
    dec = GatedDecoder(pair.eng, pair.pt[:4], None, tau=0.0)
    dec.set_state(last, pos0)
    batch = calibrate.reference_decode(dec, STEPS)
    last, pos0 = fresh(pair, prompts)
    one = GatedDecoder(pair.eng, pair.pt[2:3], None, tau=0.0)
    one.set_state(last[2:3], pos0[2:3])
    alone = calibrate.reference_decode(one, STEPS)
    np.testing.assert_array_equal(alone[0], batch[2])


def test_calibration_recipe(pair, prompts):
    last, pos0 = fresh(pair, prompts)
    snap = pair.eng.kv_pool.clone()
    dec = GatedDecoder(pair.eng, pair.pt[:4], None, tau=0.0)
    res = calibrate.calibrate(dec, (last, pos0), snap, STEPS)
    print(res)
    assert 0.0 <= res["eps_median"] <= res["eps_max"] and res["pert_tau"] == pytest.approx(2 * res["eps_max"])
    assert len(res["frontier"]) == 6
    for f in res["frontier"]:
        assert 0.0 <= f["r_verify"] <= 1.0 and 0.0 <= f["seq_det"] <= 1.0
    det = [f["tau"] for f in res["frontier"] if f["seq_det"] == 1.0]
    assert res["tau_100"] == (min(det) if det else None)


def test_repair_actions(pair, prompts):
    """MarginGate under each repair action from one state, against the reference decode.
    Token only never copies (r_repair 0); copy always copies every verified row (r_repair =
    r_verify); at a tau above every margin (all rows verified every step) copy always is the
    reference decode token for token."""
    last, pos0 = fresh(pair, prompts)
    snap = pair.eng.kv_pool.clone()
    dec = GatedDecoder(pair.eng, pair.pt[:4], None, tau=0.0)
    res = calibrate.repair_actions(dec, (last, pos0), snap, STEPS, 0.05)
    print(res)
    a = res["actions"]
    assert set(a) == {"on_mismatch", "token_only", "copy_always"}
    assert a["token_only"]["r_repair"] == 0.0
    assert a["copy_always"]["r_repair"] == pytest.approx(a["copy_always"]["r_verify"])
    for v in a.values():
        assert a["on_mismatch"]["r_verify"] == pytest.approx(v["r_verify"], abs=0.5) and 0 <= v["seq_det"] <= 1
    assert dec.repair_action == mg.REPAIR_ON_MISMATCH and dec.tau == 0.0
    top = calibrate.repair_actions(dec, (last, pos0), snap, STEPS, float("inf"))
    assert top["actions"]["copy_always"]["r_verify"] == 1.0
    assert top["actions"]["copy_always"]["seq_det"] == 1.0


def test_divergence_diagnostics(pair, prompts):
    """Obs. 1-3 and the oracle-position repair on the tiny decoder: the statistics are well
    formed; until its first divergence a row of the oracle-position run is its ungated run, so
    every ungated divergence event costs at least one verification there."""
    last, pos0 = fresh(pair, synth.make_prompts(4, [32] * 4, S.vocab, seed=3))
    snap = pair.eng.kv_pool.clone()
    dec = GatedDecoder(pair.eng, pair.pt[:4], None, tau=0.0)
    st, ref = diagnostics.flip_study(dec, (last, pos0), snap, STEPS, tau=0.05)
    print(st)
    assert st["rows"] == 4 and ref.shape == (4, STEPS)
    assert 0.0 <= st["flips"]["rate"] <= 1.0 and st["flips"]["synchronous_samples"] >= 4
    assert st["near_tie"]["events"] == st["flips"]["events"]
    orc = diagnostics.oracle_position_repair(dec, (last, pos0), snap, STEPS, ref)
    print(orc)
    assert orc["verified_row_steps"] >= st["flips"]["events"] and 0.0 <= orc["seq_det"] <= 1.0


def test_diagnostics_extraction_matches_the_oracle(pair, prompts):
    """What the divergence diagnostics read from the GPU, against the oracle on the same state:
    the final layer's K/V columns after the reference decode (final_layer_kv) equal the oracle's
    canonical greedy decode cache at those positions bit for bit; on a fast step, the fast
    margins equal the oracle's top-2 over the same logits, the reference token's rank
    (_rank_of) equals a brute-force rank under the gate's order, and the near-tie counts
    N(Delta) equal a brute-force count and satisfy N(Delta) > 1 iff margin <= Delta."""
    from oracle import mgo
    last, pos0 = fresh(pair, synth.make_prompts(4, [32] * 4, S.vocab, seed=3))
    dec = GatedDecoder(pair.eng, pair.pt[:4], None, tau=0.0)
    dec.set_state(last, pos0)
    steps = 12
    ref = calibrate.reference_decode(dec, steps)
    kv_gpu = diagnostics.final_layer_kv(dec, int(pos0[0]), steps).cpu().numpy()
    # the oracle's own canonical greedy decode from the same prompts
    rows = np.arange(4, dtype=np.int32)
    tok, pos = last.copy(), pos0.copy()
    never = np.full(4, -1, np.int32)
    for s in range(steps):
        _, vt, vc = pair.om.verify_rows(rows, tok, pos, pair.pt[:4], want_logits=False)
        emitted, _ = pair.om.repair(rows, pos, pair.pt[:4], never, vt, vc, never)
        assert np.array_equal(emitted, ref[:, s])
        tok, pos = emitted, pos + 1
    kv = pair.om.kv_view()
    L = S.n_layers
    for b in range(4):
        for s in range(steps):
            p = int(pos0[b]) + s
            col = kv[L - 1, pair.pt[b, p // 16], :, :, p % 16, :]
            want = (col.astype(np.uint32) << 16).view(np.float32)
            assert np.array_equal(kv_gpu[b, s], want), (b, s)
    # a fast step from the post-reference state: margins, ranks and near-tie counts
    dec.step("off")
    torch.cuda.synchronize()
    lg = dec.logits.cpu().numpy()
    margin = dec.margin.cpu().numpy()
    probe = torch.as_tensor(ref[:, -1].astype(np.int32), device="cuda")
    rank = diagnostics._rank_of(dec.logits, probe).cpu().numpy()
    nt = diagnostics.near_tie_count(dec.logits).cpu().numpy()
    for b in range(4):
        t1, g = mgo.top2(lg[b])
        assert np.float32(g).view(np.uint32) == margin[b].view(np.uint32)
        v, t = lg[b, ref[b, -1]], int(ref[b, -1])
        assert rank[b] == int(np.sum((lg[b] > v) | ((lg[b] == v) & (np.arange(lg.shape[1]) < t))))
        for k, dlt in enumerate(diagnostics.NEAR_TIE_DELTAS):
            thr = np.float32(lg[b].max()) - np.float32(dlt)   # the threshold in fp32, as the count forms it
            assert nt[b, k] == int(np.sum(lg[b] >= thr))
            assert (nt[b, k] > 1) == (margin[b] <= dlt)
