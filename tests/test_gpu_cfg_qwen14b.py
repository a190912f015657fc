"""The Qwen2.5-14B-shaped workload at full size (GPU).

48 layers, d 5120, 40 query / 8 KV heads, head_dim 128, SwiGLU FFN 13824, vocab 152064,
QKV bias, RoPE theta 1e6; random-init N(0, 0.02) bf16 weights.  Batch 128 with prompt
lengths drawn uniformly from 128 to 2048 (ragged page tables).  The prompt caches are seeded
synthetic bf16 values (a canonical prefill of ~140k tokens at this size takes minutes, and
every check below is state-forced from the GPU cache, so the cache need not come from a
forward pass).  tau is the 15% quantile of the fast-path margins of a 16-step calibration
run; then 256 gated greedy decode steps, every row protected.  At the first and a late
step:
  fast step, per layer      each of the 48 layers' output and tentative K/V column, and the
                            head's logits, within normwise 1e-2 of the oracle run on the
                            GPU's own input to that layer, on three rows (the shortest and the
                            longest context among them)
  gated step, state-forced  on rows picked from the step's gated list (repaired rows first; a
                            step with no repair is run and the next one checked): gate
                            bit-exact over the batch, verifier logits / token / K-V column
                            bit-exact, commit and single-column repair byte for byte."""
import numpy as np
import pytest
import torch

from paper_2605_30218_amd import mg, synth
from paper_2605_30218_amd.runtime import GatedDecoder

from _gpu_common import assert_forced, assert_layerwise, forced_steps, layerwise_check

pytestmark = pytest.mark.gpu
S = synth.QWEN14B
B, STEPS, CALIB, RATE = 128, 256, 16, 0.15
CHECK_STEPS = (0, STEPS - 16)


@pytest.fixture(scope="module")
def run():
    lens = synth.make_lengths(B, 128, 2048, seed=2)
    ctx = lens + CALIB + STEPS + 32
    maxp = -(-int(ctx.max()) // S.page_size)
    pt, n_pages = synth.make_page_table(ctx, S.page_size, maxp, seed=5)
    w = synth.make_weights(S, seed=0, device="cuda")
    eng = mg.Engine(S, w, B, maxp, n_pages)
    # synthetic cache of the prompt positions 0..len-2 of every row
    cached = np.concatenate([pt[r, :-(-(int(lens[r]) - 1) // S.page_size)] for r in range(B)])
    synth.fill_synthetic_kv(eng.kv_view(), cached, seed=6)
    prompts = synth.make_prompts(B, lens, S.vocab, seed=1)
    last = np.array([p[-1] for p in prompts], np.int32)
    pos0 = (lens - 1).astype(np.int32)
    wn = synth.weights_to_numpy(w)
    dec = GatedDecoder(eng, pt, None, tau=0.0)
    dec.set_state(last, pos0)
    margins = []
    for _ in range(CALIB):
        dec.step("off")
        margins.append(dec.margin.cpu().numpy().copy())
    tau = float(np.quantile(np.concatenate(margins), RATE))
    dec.tau = tau
    dec.protected_row_steps = dec.verified_row_steps = 0
    pos_now = dec.positions.cpu().numpy()
    sample = [int(np.argmin(pos_now)), 64, int(np.argmax(pos_now))]
    checks, layers = [], []
    step = 0
    while step < STEPS:
        if step in CHECK_STEPS:
            tok, pos = dec.tokens.cpu().numpy(), dec.positions.cpu().numpy()
            res = layerwise_check(S, wn, eng, pt, tok, pos, sample)
            print(f"step {step} layerwise: worst x {max(res['x']):.2e} k {max(res['k']):.2e} "
                  f"v {max(res['v']):.2e} head {res['head']:.2e} e2e {res['e2e']:.4f}", flush=True)
            layers.append(res)
            c, ran = forced_steps(S, wn, eng, dec, pt, 1, tau, want_repair=True)
            checks += c
            step += ran
        else:
            dec.step("gated")
            step += 1
    torch.cuda.synchronize()
    yield dict(checks=checks, layers=layers, tau=tau, r_verify=dec.r_verify, sample=sample,
               ctx=[int(pos_now[r]) for r in sample])
    eng.close()


def test_qwen14b_layerwise_fast_step(run):
    print(f"tau {run['tau']:.4f}, layer-checked rows {run['sample']} at contexts {run['ctx']}")
    for res in run["layers"]:
        assert_layerwise(res)


def test_qwen14b_gated_steps_state_forced(run):
    assert_forced(run["checks"])


def test_qwen14b_trigger_rate_near_calibration(run):
    print(f"r_verify {run['r_verify']:.3f} at the 15% calibration quantile")
    assert 0.05 <= run["r_verify"] <= 0.35, run["r_verify"]
