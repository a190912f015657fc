"""The Qwen2.5-7B-shaped workload in the high-trigger regime, at full size (GPU).

28 layers, d 3584, 28 query / 4 KV heads, head_dim 128, SwiGLU FFN 18944, vocab 152064,
QKV bias, RoPE theta 1e6; random-init N(0, 0.02) bf16 weights with the seeded tie-pair
low-rank perturbation of the LM head (about half of the steps get a top-1/top-2 margin
below tau = 0.5).  Batch 32 with seeded uniform 1024-token prompts (canonical prefill), then
512 gated greedy decode steps, every row protected.  At sampled steps the oracle is
state-forced from the GPU cache of sampled rows:
  gate over the batch                bit-exact (top-1, margin bits, gate, ordered rows)
  fast logits                        within max(1e-2, twice the oracle's own spread between
                                     the plain and the canonical order on the same state)
  verifier logits, token, K/V column bit-exact
  commit / single-column repair      the verifier's token and column on gated rows; top-1
                                     with margin >= tau elsewhere
and the measured trigger rate lies near the perturbation's design point of 1/2."""
import numpy as np
import pytest
import torch

from oracle import mgo  # noqa: F401  (the oracle library is loaded through _gpu_common)
from paper_2605_30218_amd import mg, synth
from paper_2605_30218_amd.runtime import GatedDecoder, prefill_rows

from _gpu_common import forced_step_check, oracle_for_rows

pytestmark = pytest.mark.gpu
S = synth.QWEN7B
B, P, STEPS, TAU = 32, 1024, 512, 0.5
CHECK_STEPS = (0, 255, 511)
SAMPLE = [0, 13, 31]


@pytest.fixture(scope="module")
def run():
    ctx = P + STEPS + 16
    maxp = -(-ctx // S.page_size)
    pt, n_pages = synth.make_page_table([ctx] * B, S.page_size, maxp, seed=5)
    w = synth.perturb_lm_head_tie_pairs(synth.make_weights(S, seed=0, device="cuda"), S, seed=4, tau=TAU)
    eng = mg.Engine(S, w, B, maxp, n_pages, max_prefill=1024)
    prompts = synth.make_prompts(B, [P] * B, S.vocab, seed=1)
    last, pos0 = prefill_rows(eng, prompts, pt)
    wn = synth.weights_to_numpy(w)
    dec = GatedDecoder(eng, pt, None, tau=TAU)
    dec.set_state(last, pos0)
    checks = []
    for step in range(STEPS):
        if step in CHECK_STEPS:
            pre_tok, pre_pos = dec.tokens.cpu().numpy(), dec.positions.cpu().numpy()
            om, ptl = oracle_for_rows(S, wn, eng, pt, SAMPLE)
            keep = {}
            dec.step("gated", keep=keep)
            emitted = dec.top1.cpu().numpy()
            c = forced_step_check(S, eng, pt, pre_tok, pre_pos, SAMPLE, om, ptl, keep, emitted, TAU)
            print(f"step {step}: {c}", flush=True)
            checks.append(c)
        else:
            dec.step("gated")
    torch.cuda.synchronize()
    yield dict(checks=checks, r_verify=dec.r_verify, r_repair=dec.r_repair())
    eng.close()


def test_qwen7b_gated_steps_state_forced(run):
    for c in run["checks"]:
        assert c["gate"], c
        assert c["verifier"], c
        assert c["commit"], c
        assert c["err"] <= max(1e-2, 2 * c["spread"]), c
    assert sum(c["gated_in_sample"] for c in run["checks"]) > 0, "no sampled row was gated at the checked steps"


def test_qwen7b_trigger_rate_near_design_point(run):
    print(f"r_verify {run['r_verify']:.3f}, r_repair {run['r_repair']:.4f}")
    assert 0.3 <= run["r_verify"] <= 0.7, run["r_verify"]
