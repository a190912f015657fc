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


def layerwise_check(shape, wn, eng, page_table, tok, pos, sample, B=None):
    """State-forced per-layer parity of one fast step on sampled batch rows, at full width and
    depth.  The GPU runs the step (mg_op_decode_step_taps) and hands out the residual stream
    at every layer boundary; the oracle (plain order) then runs layer l alone from the GPU's
    own input to layer l and the pre-step cache of the sampled rows, and its output, and the
    K/V column it appends, are compared with the GPU's layer l output and tentative column.
    The head is checked the same way from the GPU's final residual stream.  So no layer's
    input carries the differences of earlier layers: each comparison is one layer of
    arithmetic on identical inputs.

    Returns dict(embed=bool bit-exact, x=[per-layer normwise error], k=[...], v=[...],
    head=normwise logit error, e2e=normwise error of the whole plain-order step from the
    same pre-step state (depth-amplified; reported, not a bar))."""
    sample = list(sample)
    B = len(tok) if B is None else B
    om, ptl = oracle_for_rows(shape, wn, eng, page_table, sample)
    L, d = shape.n_layers, shape.d_model
    taps = torch.empty((L + 1, B, d), dtype=torch.int16, device="cuda")
    logits = torch.empty((B, shape.vocab), dtype=torch.float32, device="cuda")
    eng.decode_step_taps(B, dev_i32(tok), dev_i32(pos), dev_i32(page_table), logits, taps)
    torch.cuda.synchronize()
    xt = u16(taps)[:, sample]
    glog = logits.cpu().numpy()[sample]
    kv = eng.kv_view()
    spos = np.asarray(pos, np.int32)[sample]
    stok = np.asarray(tok, np.int32)[sample]
    ps = shape.page_size
    # the GPU's tentative columns, [row][layer][K|V][Hkv][hd]
    gcol = np.stack([u16(kv[:, int(page_table[r][int(pos[r]) // ps]), :, :, int(pos[r]) % ps, :]) for r in sample])
    out = dict(embed=bool(np.array_equal(xt[0], np.asarray(wn[0])[stok])), x=[], k=[], v=[])
    ov = om.kv_view()
    for l in range(L):
        y = om.layer(mgo.PLAIN, l, xt[l], spos, ptl)
        out["x"].append(max(normwise(mgo.f32_from_bf16(xt[l + 1][k]), mgo.f32_from_bf16(y[k]))
                            for k in range(len(sample))))
        for j, name in ((0, "k"), (1, "v")):
            e = 0.0
            for k in range(len(sample)):
                p = int(spos[k])
                ref = ov[l, int(ptl[k][p // ps]), j, :, p % ps, :]
                e = max(e, normwise(mgo.f32_from_bf16(gcol[k, l, j]), mgo.f32_from_bf16(ref)))
            out[name].append(e)
    ref = om.head(mgo.PLAIN, xt[L])
    out["head"] = max(normwise(glog[k], ref[k]) for k in range(len(sample)))
    e2e = om.decode_step(mgo.PLAIN, stok, spos, ptl)
    out["e2e"] = max(normwise(glog[k], e2e[k]) for k in range(len(sample)))
    return out


def assert_layerwise(res, bar=1e-2):
    """Every layer's output and tentative K/V column and the head within `bar` (normwise)."""
    worst = {n: (int(np.argmax(res[n])), float(np.max(res[n]))) for n in ("x", "k", "v")}
    print(f"per-layer worst (layer, err): {worst}; head {res['head']:.2e}; end-to-end {res['e2e']:.4f}", flush=True)
    assert res["embed"], "layer-0 input differs from the embedding rows"
    for n in ("x", "k", "v"):
        assert max(res[n]) <= bar, (n, worst[n], res[n])
    assert res["head"] <= bar, res["head"]


def pick_forced_sample(keep, n_gated=3, n_fast=1):
    """Rows for a state-forced check of a step that has run: gated rows whose verifier token
    differed from the fast top-1 (repaired) first, then other gated rows, then rows the gate
    let through (fast commits).  So a check verifies repairs whenever the step made one."""
    rows = [int(r) for r in keep["rows"]]
    rep = [r for i, r in enumerate(rows) if int(keep["v_tok"][i]) != int(keep["top1"][r])]
    ver = [r for r in rows if r not in rep]
    fast = [r for r in range(len(keep["top1"])) if r not in set(rows)]
    pick = (rep + ver)[:n_gated] + fast[:n_fast]
    return sorted(pick), len([r for r in pick if r in rep])


def forced_steps(shape, wn, eng, dec, page_table, n_steps, tau, n_gated=3, n_fast=1, max_extra=8,
                 want_repair=False):
    """Run gated steps and state-force the oracle on each of `n_steps` checked steps, on rows
    chosen after the step from its gated list (pick_forced_sample).  The oracle is built from
    the post-step cache: a step writes only column p of each row, and both the oracle's
    plain step and its verifier overwrite or bypass column p, so positions 0..p-1 are the
    pre-step state.  A step with no gated row (want_repair: no repaired row) is run but not
    checked, at most max_extra times in all.  Returns (checks, steps run)."""
    checks, extra, ran = [], 0, 0
    while len(checks) < n_steps:
        pre_tok, pre_pos = dec.tokens.cpu().numpy(), dec.positions.cpu().numpy()
        keep = {}
        dec.step("gated", keep=keep)
        ran += 1
        sample, n_rep = pick_forced_sample(keep, n_gated, n_fast)
        if (len(keep["rows"]) == 0 or (want_repair and n_rep == 0)) and extra < max_extra:
            extra += 1
            continue
        emitted = dec.top1.cpu().numpy()
        om, ptl = oracle_for_rows(shape, wn, eng, page_table, sample)
        c = forced_step_check(shape, eng, page_table, pre_tok, pre_pos, sample, om, ptl, keep, emitted, tau)
        c["sample"] = sample
        c["ctx"] = [int(pre_pos[r]) for r in sample]
        del om
        print(f"forced step {len(checks)}: {c}", flush=True)
        checks.append(c)
    return checks, ran


def assert_forced(checks, need_repair=True):
    """Every checked step bit-exact (gate, verifier, commit); gated rows were checked, and
    (need_repair) at least one repaired column was compared byte for byte."""
    for c in checks:
        assert c["gate"] and c["verifier"] and c["commit"], c
    assert sum(c["gated_in_sample"] for c in checks) > 0, "no gated row was checked"
    if need_repair:
        assert sum(c["repaired"] for c in checks) > 0, "no repaired column was checked"
    print("fast-vs-plain end-to-end logit error per checked step (reported, not a bar): "
          + ", ".join(f"{c['err']:.4f}" for c in checks), flush=True)
