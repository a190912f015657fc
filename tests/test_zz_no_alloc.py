"""mg_margin_gate_noalloc, the allocation-free margin gate (GPU): its outputs equal
mg_margin_gate's bit for bit (top-1, margin bits, gate, ordered gated rows, count) on two
calls in a row through the C ABI, the second with fewer rows and a narrower vocabulary, so
the shared static scratch array is reused with stale contents from the first call."""
import numpy as np
import pytest
import torch

from paper_2605_30218_amd import mg, synth

pytestmark = pytest.mark.gpu


def _gate_engine(V):
    # a one-layer model whose only role is to give mg_margin_gate a context with vocab V
    shape = synth.ModelShape(f"gate-v{V}", 1, 64, 1, 1, 64, 64, V, False, 1e4, 1e-5)
    w = synth.make_weights(shape, seed=0, device="cuda")
    return mg.Engine(shape, w, 256, 1, 1)


def _logits(B, V, seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    lg = torch.randn((B, V), generator=g, device="cuda") * 0.9
    # adversarial rows: duplicated maximum, a NaN, a margin exactly at tau
    lg[1, 7] = lg[1].max()
    lg[1, 3] = lg[1, 7]
    lg[2, V // 2] = float("nan")
    top = lg[3].max()
    lg[3, 0] = top + 0.25
    return lg.contiguous()


def _outputs(B):
    i32 = dict(dtype=torch.int32, device="cuda")
    return (torch.full((B,), -7, **i32), torch.full((B,), -7.0, device="cuda"),
            torch.full((B,), 9, dtype=torch.uint8, device="cuda"), torch.full((B,), -7, **i32), torch.full((1,), -7, **i32))


def _host(outs):
    t, m, g, r, n = (x.cpu().numpy() for x in outs)
    k = int(n[0])
    return t, m.view(np.uint32), g, r[:k], k


@pytest.mark.parametrize("calls", [((64, 128256, 0.25), (5, 4096, 0.3))])
def test_noalloc_gate_equals_context_gate_twice(calls):
    for i, (B, V, tau) in enumerate(calls):
        eng = _gate_engine(V)
        lg = _logits(B, V, seed=40 + i)
        prot = torch.ones(B, dtype=torch.uint8, device="cuda")
        prot[B - 1] = 0
        ref = _outputs(B)
        eng.margin_gate(B, lg, prot, tau, *ref)
        got = _outputs(B)
        mg.margin_gate_noalloc(B, V, lg, prot, tau, *got)
        torch.cuda.synchronize()
        a, b = _host(ref), _host(got)
        np.testing.assert_array_equal(a[0], b[0])
        np.testing.assert_array_equal(a[1], b[1])
        np.testing.assert_array_equal(a[2], b[2])
        np.testing.assert_array_equal(a[3], b[3])
        assert a[4] == b[4] and 0 < a[4] < B
        eng.close()


def test_noalloc_gate_rejects_sizes_beyond_its_limit():
    lg = torch.zeros((1, 16), device="cuda")
    outs = _outputs(1)
    with pytest.raises(mg.MgError):
        mg.margin_gate_noalloc(257, 16, lg, None, 0.1, *outs)
    with pytest.raises(mg.MgError):
        mg.margin_gate_noalloc(1, 1, lg, None, 0.1, *outs)
