"""Shape matrix on shallow decoders (GPU): head_dim 128 and 64, GQA groups 1..8, QKV bias,
contexts that cross several fast (128) and canonical (256) attention chunks, ragged
FFN widths.  The fast path must agree with the oracle's plain mode within normwise 1e-2
(most rows agree to ~1e-7; a single bf16 rounding flip on a large hidden element moves a
row by a few 1e-3, and the oracle's own canonical and plain modes show the same jumps),
and the verifier must be bit-exact with the oracle's canonical mode."""
import numpy as np
import pytest
import torch

from oracle import mgo
from paper_2605_30218_amd import synth

from _gpu_common import Pair, dev_i32, normwise, u16

pytestmark = pytest.mark.gpu

SHAPES = [
    synth.ModelShape("l8-like", 1, 512, 8, 2, 128, 1024, 2048, False, 5e5, 1e-5),
    synth.ModelShape("q7-like", 2, 448, 7, 1, 128, 592, 1536, True, 1e6, 1e-6),
    synth.ModelShape("q14-like", 1, 640, 10, 2, 128, 432, 1024, True, 1e6, 1e-6),
    synth.ModelShape("g8-hd64", 2, 512, 8, 1, 64, 688, 4096, False, 1e4, 1e-5),
    synth.ModelShape("mha-hd64", 1, 256, 4, 4, 64, 256, 512, False, 1e4, 1e-5),
]
LENS = [600, 130, 257, 1, 300, 129]


@pytest.fixture(scope="module", params=SHAPES, ids=[s.name for s in SHAPES])
def setup(request):
    s = request.param
    pair = Pair(s, max_batch=len(LENS), ctx_cap=640, seed=11)
    prompts = synth.make_prompts(len(LENS), [L + 1 for L in LENS], s.vocab, seed=12)
    last, pos0 = pair.prefill(prompts)
    torch.cuda.synchronize()
    return pair, last, pos0


def test_prefill_bitexact(setup):
    pair, _, _ = setup
    np.testing.assert_array_equal(u16(pair.eng.kv_pool), pair.om.kv_pool)


def test_verifier_bitexact(setup):
    pair, last, pos0 = setup
    e, s = pair.eng, pair.shape
    n = len(LENS)
    rows = np.arange(n, dtype=np.int32)[::-1].copy()
    vl = torch.empty((n, s.vocab), dtype=torch.float32, device="cuda")
    vt = torch.empty(n, dtype=torch.int32, device="cuda")
    vc = torch.empty((n, e.col_elems), dtype=torch.int16, device="cuda")
    e.verify_rows(n, dev_i32(rows), None, dev_i32(last), dev_i32(pos0), dev_i32(pair.pt[:n]), vl, vt, vc)
    torch.cuda.synchronize()
    rl, rt, rc = pair.om.verify_rows(rows, last, pos0, pair.pt[:n])
    np.testing.assert_array_equal(vl.cpu().numpy().view(np.uint32), rl.view(np.uint32))
    np.testing.assert_array_equal(vt.cpu().numpy(), rt)
    np.testing.assert_array_equal(u16(vc), rc)


def test_fast_step_close_to_oracle(setup):
    pair, last, pos0 = setup
    e, s = pair.eng, pair.shape
    n = len(LENS)
    snap = e.kv_pool.clone()
    om_snap = pair.om.kv_pool.copy()
    logits = torch.empty((n, s.vocab), dtype=torch.float32, device="cuda")
    e.decode_step(n, dev_i32(last), dev_i32(pos0), dev_i32(pair.pt[:n]), logits)
    torch.cuda.synchronize()
    ref = pair.om.decode_step(mgo.PLAIN, last, pos0, pair.pt[:n])
    got = logits.cpu().numpy()
    errs = [normwise(got[b], ref[b]) for b in range(n)]
    e.kv_pool.copy_(snap)
    pair.om.kv_pool[:] = om_snap
    assert max(errs) <= 1e-2, errs
