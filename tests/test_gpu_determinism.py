"""Run-to-run determinism of the fast path on fixed inputs and a fixed batch (GPU).

The fast path may change its reduction plan with the batch (that is what the gate guards
against), but on the same inputs and the same batch every run must give the same bits: a
difference would mean a race (an LDS buffer read before every wave wrote it, a partial tile
summed before it was complete).  Each case runs the fast step five times from the same cache
and compares the logits and the tentative K/V columns bit for bit, at the full Llama-8B widths
(2 layers): batch 64 at 512 positions (the benchmark's launch shapes, split-K GEMMs), batch 4 at
1.5k-3k positions (split-KV attention), batch 1; and the matrix-core verifier likewise."""
import numpy as np
import pytest
import torch

from paper_2605_30218_amd import mg, synth

from _gpu_common import dev_i32, u16

pytestmark = pytest.mark.gpu
SHAPE = synth.ModelShape("llama3.1-8b-width-2l", 2, 4096, 32, 8, 128, 14336, 128256, False, 5e5, 1e-5)
RUNS = 5


@pytest.fixture(scope="module")
def model():
    return synth.make_weights(SHAPE, seed=3, device="cuda")


@pytest.mark.parametrize("lens", [[512] * 64, [3000, 1500, 2200, 17], [700]], ids=["b64", "b4-splitkv", "b1"])
def test_fast_step_repeats_bit_for_bit(model, lens):
    lens = np.asarray(lens, np.int32)
    B = lens.size
    ctx = int(lens.max()) + 16
    maxp = -(-ctx // 16)
    pt, n_pages = synth.make_page_table([ctx] * B, 16, maxp, seed=5)
    eng = mg.Engine(SHAPE, model, B, maxp, n_pages)
    cached = np.concatenate([pt[r, :-(-(int(lens[r]) - 1) // 16)] for r in range(B)])
    synth.fill_synthetic_kv(eng.kv_view(), cached, seed=21)
    tok = synth.make_prompts(1, [B], SHAPE.vocab, seed=22)[0]
    pos = (lens - 1).astype(np.int32)
    snap = eng.kv_pool.clone()
    cols = [(int(pt[r, int(pos[r]) // 16]), int(pos[r]) % 16) for r in range(B)]
    kv = eng.kv_view()
    ref_l = ref_c = None
    for run in range(RUNS):
        eng.kv_pool.copy_(snap)
        logits = torch.empty((B, SHAPE.vocab), dtype=torch.float32, device="cuda")
        eng.decode_step(B, dev_i32(tok), dev_i32(pos), dev_i32(pt), logits)
        torch.cuda.synchronize()
        lg = logits.cpu().numpy().view(np.uint32)
        cc = np.stack([u16(kv[:, pg, :, :, sl, :]) for pg, sl in cols])
        if run == 0:
            ref_l, ref_c = lg, cc
        else:
            assert np.array_equal(lg, ref_l), f"logits differ on run {run}"
            assert np.array_equal(cc, ref_c), f"K/V columns differ on run {run}"
    # the matrix-core verifier on every row, repeated
    ref = None
    for run in range(RUNS):
        vl = torch.empty((B, SHAPE.vocab), dtype=torch.float32, device="cuda")
        vt = torch.empty(B, dtype=torch.int32, device="cuda")
        vc = torch.empty((B, eng.col_elems), dtype=torch.int16, device="cuda")
        eng.verify_rows_mfma(B, dev_i32(np.arange(B)), dev_i32(tok), dev_i32(pos), dev_i32(pt), vl, vt, vc)
        torch.cuda.synchronize()
        got = (vl.cpu().numpy().view(np.uint32), vt.cpu().numpy(), u16(vc))
        if ref is None:
            ref = got
        else:
            for a, b in zip(got, ref):
                assert np.array_equal(a, b), f"matrix-core verifier differs on run {run}"
    eng.close()
