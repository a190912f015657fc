"""tau calibration by the paper's recipe (Sec. 3.1, threshold setting; Appendix A; the
Pareto frontier of Sec. 4.3), on the synthetic workloads.

  reference   the deterministic reference decode: every step is the verifier's canonical
              transition for every row, and its K/V column always replaces the tentative
              one, so the whole cache and token stream are canonical.  It is batch-invariant
              by construction (the verifier is) and equals the oracle's canonical greedy
              decode token for token.
  eps_pert    per row and step of the reference trajectory, the l-infinity gap between the
              fast batched logits and the reference logits over the reference's top-50
              entries; 2 max(eps) only sets the sweep range
  sweep       MarginGate end to end from the same prefilled state for each tau of a grid:
              trigger rate, sequence-level determinism (the fraction of protected rows whose
              whole emitted sequence equals the reference), overhead over the fast path, and
              (for frontiers that never reach full determinism) the mean step at which a row
              first leaves the reference and the per-token agreement
  tau_100     the smallest tau of the grid at which every protected row is deterministic
  actions     MarginGate at one tau under each repair action of the commit: the method's
              (copy the verifier column when the tokens differ, Sec. 3.2), token only (the
              repair-action ablation of Sec. 4) and copy on every verified row

Host-side orchestration of the library's entry points; all arithmetic runs in libmg."""
from __future__ import annotations

import time

import numpy as np
import torch

from . import mg
from .runtime import GatedDecoder


def reference_decode(dec: GatedDecoder, steps: int, keep_logits=None):
    """Canonical greedy decode of every row of `dec` from its current state: the verifier on
    all rows, then the commit with the copy-always repair action, so every row emits the
    verifier token and takes the verifier column.  keep_logits(step, fast_logits, ref_logits):
    optional callback receiving host copies of both logit sets per step (the fast step runs
    first on the same state; its tentative columns are then overwritten).  Returns the
    emitted tokens [rows][steps]."""
    e, B = dec.e, dec.B
    rows = dec.always_rows
    n = int(rows.numel())
    if n != B:  # an unprotected row would be handed the placeholder token -1
        raise ValueError("the reference decode needs every row protected")
    v_logits = torch.empty((n, e.shape.vocab), dtype=torch.float32, device=dec.tokens.device) if keep_logits else None
    emitted = torch.empty(B, dtype=torch.int32, device=dec.tokens.device)
    out = np.zeros((n, steps), np.int32)
    for s in range(steps):
        if keep_logits:
            e.decode_step(B, dec.tokens, dec.positions, dec.page_table, dec.logits)
        e.verify_rows(n, rows, None, dec.tokens, dec.positions, dec.page_table, v_logits, dec.v_tok, dec.v_kvcol)
        # every row emits the verifier token and takes the verifier column
        e.repair_kv_column_action(n, rows, None, dec.positions, dec.page_table, dec.v_tok, dec.v_tok, dec.v_kvcol,
                                  emitted, dec.n_repaired, mg.REPAIR_COPY_ALWAYS)
        if keep_logits:
            keep_logits(s, dec.logits[rows.long()].cpu().numpy(), v_logits.cpu().numpy())
        e.advance(B, emitted, dec.tokens, dec.positions)
        out[:, s] = emitted[rows.long()].cpu().numpy()
    return out


def eps_pert(fast: np.ndarray, ref: np.ndarray, topk: int = 50) -> np.ndarray:
    """Per row: max over the reference's top-k entries of |fast - ref| (Appendix A)."""
    idx = np.argpartition(-ref, topk - 1, axis=1)[:, :topk]
    return np.abs(np.take_along_axis(fast, idx, 1) - np.take_along_axis(ref, idx, 1)).max(1)


def gated_run(dec: GatedDecoder, steps: int, mode: str = "gated"):
    """Emitted tokens [rows][steps] of a MarginGate (or off / always) run and its wall time."""
    rows = dec.always_rows.long()
    out = np.zeros((int(rows.numel()), steps), np.int32)
    dec.protected_row_steps = dec.verified_row_steps = 0
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    toks = []
    for _ in range(steps):
        dec.step(mode)
        toks.append(dec.tokens[rows].clone())  # advance() stored the emitted tokens as the next input
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    for s, t in enumerate(toks):
        out[:, s] = t.cpu().numpy()
    return out, wall


def calibrate(dec: GatedDecoder, state, kv_snap, steps: int, taus=None, grid_factors=(0.125, 0.25, 0.5, 1.0, 2.0, 4.0)):
    """The whole recipe from one prefilled state (`state` = (tokens, positions) host arrays,
    `kv_snap` the prefilled KV pool).  Returns a dict with the eps statistics, the per-tau
    frontier and tau_100 (None when no tested tau reaches full determinism)."""
    eng = dec.e
    eps = []

    def keep(_s, fast, ref):
        eps.append(eps_pert(fast, ref))

    eng.kv_pool.copy_(kv_snap)
    dec.set_state(*state)
    ref = reference_decode(dec, steps, keep)
    eps = np.concatenate(eps)
    pert_tau = 2.0 * float(eps.max())
    if taus is None:
        taus = [pert_tau * f for f in grid_factors]
    eng.kv_pool.copy_(kv_snap)
    dec.set_state(*state)
    _, t_off = gated_run(dec, steps, "off")
    frontier = []
    for tau in taus:
        eng.kv_pool.copy_(kv_snap)
        dec.set_state(*state)
        dec.tau = float(tau)
        toks, wall = gated_run(dec, steps, "gated")
        frontier.append(dict(tau=float(tau), r_verify=dec.r_verify, overhead=wall / t_off - 1.0,
                             **compare_to_reference(toks, ref)))
    tau100 = next((f["tau"] for f in frontier if f["seq_det"] == 1.0), None)
    return dict(eps_median=float(np.median(eps)), eps_max=float(eps.max()), pert_tau=pert_tau, steps=steps,
                rows=int(dec.always_rows.numel()), frontier=frontier, tau_100=tau100, reference=ref, t_off=t_off)


def compare_to_reference(toks: np.ndarray, ref: np.ndarray) -> dict:
    """Sequence determinism against the reference decode (Sec. 4): the fraction of rows whose
    whole sequence matches, the mean step of each row's first divergence (the step count if
    it never diverges), and the fraction of matching tokens."""
    steps = ref.shape[1]
    same = toks == ref
    first = np.where(same.all(1), steps, np.argmin(same, axis=1))
    return dict(seq_det=float(np.mean(np.all(same, axis=1))), first_divergence_mean=float(first.mean()),
                token_agreement=float(same.mean()))


ACTIONS = (("on_mismatch", mg.REPAIR_ON_MISMATCH), ("token_only", mg.REPAIR_TOKEN_ONLY),
           ("copy_always", mg.REPAIR_COPY_ALWAYS))


def repair_actions(dec: GatedDecoder, state, kv_snap, steps: int, tau: float, reference=None, t_off=None):
    """MarginGate at `tau` from the same prefilled state under each repair action -- the
    method's (copy the verifier column when the tokens differ, Sec. 3.2), token only (the
    repair-action ablation of Sec. 4) and copy on every verified row -- against the
    canonical reference decode: trigger and repair rates, sequence determinism, first
    divergence, token agreement, overhead over the fast path."""
    eng = dec.e
    if reference is None:
        eng.kv_pool.copy_(kv_snap)
        dec.set_state(*state)
        reference = reference_decode(dec, steps)
    if t_off is None:
        eng.kv_pool.copy_(kv_snap)
        dec.set_state(*state)
        _, t_off = gated_run(dec, steps, "off")
    out = {}
    tau0, act0 = dec.tau, dec.repair_action
    try:
        for name, action in ACTIONS:
            eng.kv_pool.copy_(kv_snap)
            dec.set_state(*state)
            dec.tau, dec.repair_action = float(tau), action
            dec.n_repaired.zero_()
            toks, wall = gated_run(dec, steps, "gated")
            out[name] = dict(r_verify=dec.r_verify, r_repair=dec.r_repair(), overhead=wall / t_off - 1.0,
                             **compare_to_reference(toks, reference))
    finally:
        dec.tau, dec.repair_action = tau0, act0
    return dict(tau=float(tau), steps=steps, actions=out)
