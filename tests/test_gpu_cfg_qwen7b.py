"""The Qwen2.5-7B-shaped workload in the high-trigger regime, at full size (GPU).

28 layers, d 3584, 28 query / 4 KV heads, head_dim 128, SwiGLU FFN 18944, vocab 152064,
QKV bias, RoPE theta 1e6; random-init N(0, 0.02) bf16 weights with the seeded tie-pair
low-rank perturbation of the LM head (about half of the steps get a top-1/top-2 margin
below tau = 0.5).  Batch 32 with seeded uniform 1024-token prompts (canonical prefill), then
512 gated greedy decode steps, every row protected.  At sampled steps the oracle is
state-forced from the GPU cache of sampled rows:
  gate over the batch                bit-exact (top-1, margin bits, gate, ordered rows)
  fast step, per layer               each of the 28 layers' output and tentative K/V column,
                                     and the head's logits, within normwise 1e-2 of the oracle
                                     run on the GPU's own input to that layer
  verifier logits, token, K/V column bit-exact, on rows picked from the step's gated list
                                     (repaired rows first; a step with no repair is run and
                                     the next one checked)
  commit / single-column repair      the verifier's token and column on gated rows; top-1
                                     with margin >= tau elsewhere
and the measured trigger rate lies near the perturbation's design point of 1/2."""
import numpy as np
import pytest
import torch

from oracle import mgo  # noqa: F401  (the oracle library is loaded through _gpu_common)
from paper_2605_30218_amd import mg, synth
from paper_2605_30218_amd.runtime import GatedDecoder, prefill_rows

from _gpu_common import assert_forced, assert_layerwise, forced_steps, layerwise_check

pytestmark = pytest.mark.gpu
S = synth.QWEN7B
B, P, STEPS, TAU = 32, 1024, 512, 0.5
CHECK_STEPS = (0, 255, 511)
SAMPLE = [0, 13, 31]


@pytest.fixture(scope="module")
def run():
    ctx = P + STEPS + 32
    maxp = -(-ctx // S.page_size)
    pt, n_pages = synth.make_page_table([ctx] * B, S.page_size, maxp, seed=5)
    w = synth.perturb_lm_head_tie_pairs(synth.make_weights(S, seed=0, device="cuda"), S, seed=4, tau=TAU)
    eng = mg.Engine(S, w, B, maxp, n_pages, max_prefill=1024)
    prompts = synth.make_prompts(B, [P] * B, S.vocab, seed=1)
    last, pos0 = prefill_rows(eng, prompts, pt)
    wn = synth.weights_to_numpy(w)
    dec = GatedDecoder(eng, pt, None, tau=TAU)
    dec.set_state(last, pos0)
    checks, layers = [], []
    step = 0
    while step < STEPS:
        if step in CHECK_STEPS:
            tok, pos = dec.tokens.cpu().numpy(), dec.positions.cpu().numpy()
            res = layerwise_check(S, wn, eng, pt, tok, pos, SAMPLE)
            print(f"step {step} layerwise: worst x {max(res['x']):.2e} k {max(res['k']):.2e} "
                  f"v {max(res['v']):.2e} head {res['head']:.2e} e2e {res['e2e']:.4f}", flush=True)
            layers.append(res)
            c, ran = forced_steps(S, wn, eng, dec, pt, 1, TAU, want_repair=True)
            checks += c
            step += ran
        else:
            dec.step("gated")
            step += 1
    torch.cuda.synchronize()
    yield dict(checks=checks, layers=layers, r_verify=dec.r_verify, r_repair=dec.r_repair())
    eng.close()


def test_qwen7b_layerwise_fast_step(run):
    for res in run["layers"]:
        assert_layerwise(res)


def test_qwen7b_gated_steps_state_forced(run):
    assert_forced(run["checks"])


def test_qwen7b_trigger_rate_near_design_point(run):
    print(f"r_verify {run['r_verify']:.3f}, r_repair {run['r_repair']:.4f}")
    assert 0.3 <= run["r_verify"] <= 0.7, run["r_verify"]
