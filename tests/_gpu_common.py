"""Shared set-up of the GPU parity tests: one synthetic model fed to both the HIP engine and
the CPU oracle (same weight bytes, same page table), and state copies between them."""
import numpy as np
import torch

from oracle import mgo
from paper_2605_30218_amd import mg, synth
from paper_2605_30218_amd.runtime import GatedDecoder, prefill_rows


def u16(t: torch.Tensor) -> np.ndarray:
    return t.cpu().numpy().view(np.uint16)


class Pair:
    """A HIP engine and an oracle model over the same weights and page table."""

    def __init__(self, shape, max_batch, ctx_cap, seed=0, weights=None, max_prefill=0):
        self.shape = shape
        ws = weights if weights is not None else synth.make_weights(shape, seed=seed)
        self.pt, self.n_pages = synth.make_page_table([ctx_cap] * max_batch, shape.page_size,
                                                      -(-ctx_cap // shape.page_size), seed=seed + 5)
        self.maxp = self.pt.shape[1]
        self.eng = mg.Engine(shape, ws, max_batch, self.maxp, self.n_pages, max_prefill=max_prefill)
        self.om = mgo.OracleModel(shape, synth.weights_to_numpy(ws), max_batch, self.maxp, self.n_pages)
        self.max_batch = max_batch

    def sync_oracle_cache(self):
        """State-forcing: copy the GPU's KV pool into the oracle."""
        torch.cuda.synchronize()
        self.om.kv_pool[:] = u16(self.eng.kv_pool)

    def prefill(self, prompts):
        last, pos0 = prefill_rows(self.eng, prompts, self.pt[: len(prompts)])
        for r, p in enumerate(prompts):
            self.om.prefill(mgo.CANON, p[:-1], self.pt[r])
        return last, pos0

    def decoder(self, B, protected=None, tau=0.5):
        return GatedDecoder(self.eng, self.pt[:B], protected, tau)


def dev_i32(a):
    return torch.as_tensor(np.ascontiguousarray(np.asarray(a, np.int32))).to("cuda")


def normwise(a, ref):
    a = np.asarray(a, np.float64)
    ref = np.asarray(ref, np.float64)
    return float(np.abs(a - ref).max() / np.abs(ref).max())
