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


def oracle_for_rows(shape, wn, eng, page_table, rows):
    """State-forcing for full-size runs: an oracle that holds only the given batch rows, with
    their KV pages copied from the GPU pool.  Returns (oracle, its page table [n][maxp]);
    unmapped (-1) entries of the batch page table stay unmapped."""
    sub = np.asarray(page_table, np.int32)[list(rows)]
    valid = sub >= 0
    n_pages = int(valid.sum())
    ptl = np.full(sub.shape, -1, np.int32)
    ptl[valid] = np.arange(n_pages, dtype=np.int32)
    om = mgo.OracleModel(shape, wn, len(rows), sub.shape[1], max(n_pages, 1))
    src = torch.as_tensor(sub[valid].astype(np.int64)).to(eng.kv_pool.device)
    torch.cuda.synchronize()
    om.kv_view()[:, :n_pages] = u16(eng.kv_view()[:, src])
    return om, ptl



def forced_step_check(shape, eng, page_table, pre_tok, pre_pos, sample, om, ptl, keep, emitted, tau,
                      protected=None):
    """State-forced parity of one gated step of a full-size run, on sampled batch rows.

    `om`/`ptl` come from oracle_for_rows() on the PRE-step cache of `sample`; `pre_tok` /
    `pre_pos` are the step's input tokens and positions, `keep` the step's kept outputs and
    `emitted` the committed tokens.  The verifier attends to positions 0..p-1 plus its own
    column, and a step writes only column p, so the GPU verifier can be re-run after the step on
    the pre-step inputs.  Returns a dict of findings (the tests assert on it):
      gate      the gate over the whole batch equals the oracle's (top1, margin bits, gate, rows)
      err       worst normwise fast-vs-oracle(plain) logit error over `sample`
      spread    worst normwise canonical-vs-plain spread of the oracle on the same rows
      verifier  GPU verifier logits / tokens / K-V columns of `sample` bit-equal to the oracle's
      commit    gated sampled rows emit the verifier token and, on a repair, hold its column;
                the others emit top-1 with margin >= tau"""
    sample = list(sample)
    n = len(sample)
    ref = om.decode_step(mgo.PLAIN, pre_tok[sample], pre_pos[sample], ptl)
    vl, vt, vc = om.verify_rows(np.arange(n, dtype=np.int32), pre_tok[sample], pre_pos[sample], ptl)
    rt, rm, rg, rr = mgo.OracleModel.margin_gate(keep["logits"], protected, tau)
    gate = (np.array_equal(keep["top1"], rt) and np.array_equal(keep["margin"].view(np.uint32), rm.view(np.uint32))
            and np.array_equal(keep["gate"], rg) and np.array_equal(keep["rows"], rr))
    spread = max(normwise(vl[k], ref[k]) for k in range(n))
    err = max(normwise(keep["logits"][r], ref[k]) for k, r in enumerate(sample))
    gl = torch.empty((n, shape.vocab), dtype=torch.float32, device="cuda")
    gt = torch.empty(n, dtype=torch.int32, device="cuda")
    gc = torch.empty((n, eng.col_elems), dtype=torch.int16, device="cuda")
    eng.verify_rows(n, dev_i32(sample), None, dev_i32(pre_tok), dev_i32(pre_pos), dev_i32(page_table), gl, gt, gc)
    torch.cuda.synchronize()
    verifier = (np.array_equal(gl.cpu().numpy().view(np.uint32), vl.view(np.uint32))
                and np.array_equal(gt.cpu().numpy(), vt) and np.array_equal(u16(gc), vc))
    gated = {int(r): i for i, r in enumerate(keep["rows"])}
    kv = eng.kv_view()
    commit, repaired = True, 0
    for k, r in enumerate(sample):
        if r in gated:
            commit &= int(keep["v_tok"][gated[r]]) == int(vt[k]) and int(emitted[r]) == int(vt[k])
            if vt[k] != rt[r]:
                p = int(pre_pos[r])
                col = u16(kv[:, int(page_table[r][p // shape.page_size]), :, :, p % shape.page_size, :])
                commit &= np.array_equal(col.reshape(-1), vc[k].reshape(-1))
                repaired += 1
        else:
            commit &= int(emitted[r]) == int(rt[r]) and float(keep["margin"][r]) >= tau
    return dict(gate=gate, err=err, spread=spread, verifier=verifier, commit=commit,
                gated_in_sample=sum(r in gated for r in sample), repaired=repaired, n_gated=len(keep["rows"]))
