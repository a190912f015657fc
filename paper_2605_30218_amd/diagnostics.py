"""Divergence diagnostics of Sec. 2 on the synthetic workloads: the premises of the method
(Obs. 1-3) measured on this fast path against the canonical reference decode.

  flips     Obs. 1: the ungated fast path (every row, batch B) decodes freely from the
            prefilled state beside the reference; a token-divergence event is a row's first
            step whose token differs, and the rate is events over synchronous samples (the
            steps up to and including each row's first divergence).
  kv        Obs. 2: per row, the final layer's K and V at each decoded position, fast vs
            reference (l2 over KV heads and head dim), aligned at the row's first divergent
            position (the first position whose input token differs, Delta = 0): the median
            pre-divergence mean over Delta < 0 ("pre"), the Delta = 0 value over it ("spike"),
            and the median per-row slope of a linear fit over the pre-divergence window.
  near_tie  Obs. 3: at each divergence event, the rank of the reference token in the fast
            logits (top-2 / top-3 / top-8 shares) and the fast top-1/top-2 margin, against the
            margins of the stable synchronous steps; the share of events the gate at tau fires
            on (its recall); and the near-tie count N(Delta) = |{j : l_j >= l_(1) - Delta}| of
            Sec. 2.4 (its Table 4) at the paper's four scales, as a mean over the token-stable
            synchronous steps and over the divergent steps, with their ratio.
  oracle    the synthetic analogue of the oracle selective repair (Sec. 2, Table 5): the
            verifier and the repair run exactly at the steps where the fast token differs from
            the reference token; repairs per sequence (all, and those made while the row was
            still on the reference), sequence determinism, first unrepaired divergence.

Host-side orchestration and statistics over libmg's outputs; the decode arithmetic runs in
libmg."""
from __future__ import annotations

import numpy as np
import torch

from . import calibrate, mg
from .runtime import GatedDecoder


def final_layer_kv(dec: GatedDecoder, p0: int, steps: int) -> torch.Tensor:
    """The final layer's K and V at positions p0 .. p0+steps-1 of every row, as fp32
    [rows][steps][2][Hkv][hd] (on the device)."""
    e = dec.e
    s = e.shape
    n_pages = e.kv_pool.numel() // (s.n_layers * 2 * s.n_kv_heads * s.page_size * s.head_dim)
    kv = e.kv_pool.view(s.n_layers, n_pages, 2, s.n_kv_heads, s.page_size, s.head_dim)[s.n_layers - 1]
    pos = torch.arange(p0, p0 + steps, device=kv.device)
    pages = dec.page_table.long()[:, pos // s.page_size]                   # [B][steps]
    slots = (pos % s.page_size).expand_as(pages)
    col = kv[pages, :, :, slots, :]                                         # [B][steps][2][Hkv][hd]
    return (col.to(torch.int32) << 16).view(torch.float32)                 # bf16 bits -> fp32


def _rank_of(logits: torch.Tensor, tok: torch.Tensor) -> torch.Tensor:
    """Rank of tok in each row of logits under the gate's order (larger value first, lower
    index first among equals); 0 = top-1."""
    v = logits.gather(1, tok.long()[:, None])
    idx = torch.arange(logits.shape[1], device=logits.device)[None, :]
    return ((logits > v) | ((logits == v) & (idx < tok.long()[:, None]))).sum(1)


NEAR_TIE_DELTAS = (0.25, 0.5, 1.0, 2.0)  # the scales of Sec. 2.4, Table 4 (logit units)


def near_tie_count(logits: torch.Tensor, deltas=NEAR_TIE_DELTAS) -> torch.Tensor:
    """N(Delta) = |{j : l_j >= l_(1) - Delta}| for each row and Delta, [rows][len(deltas)]
    (int64).  With the inclusive comparison, N(Delta) > 1 exactly when the top-1/top-2 margin
    is at most Delta (a duplicated maximum, margin 0, counts every copy)."""
    top = logits.max(1, keepdim=True).values
    return torch.stack([(logits >= top - float(d)).sum(1) for d in deltas], 1)


def flip_study(dec: GatedDecoder, state, kv_snap, steps: int, tau: float, window: int = 16):
    """Obs. 1-3 from one prefilled state (`state` = (tokens, positions) host arrays with all
    rows at one position, `kv_snap` the prefilled pool).  Returns (statistics, the reference
    tokens [rows][steps])."""
    e = dec.e
    pos = np.asarray(state[1])
    if not (pos == pos[0]).all():
        raise ValueError("the aligned K/V study needs every row at one position")
    p0 = int(pos[0])
    e.kv_pool.copy_(kv_snap)
    dec.set_state(*state)
    reference = calibrate.reference_decode(dec, steps)
    kv_ref = final_layer_kv(dec, p0, steps)
    ref_dev = torch.as_tensor(reference, device=dec.tokens.device)
    # the free-running fast path, keeping each step's margin and the reference token's rank
    e.kv_pool.copy_(kv_snap)
    dec.set_state(*state)
    rows = dec.always_rows.long()
    n = int(rows.numel())
    margins = torch.empty((n, steps), dtype=torch.float32, device=dec.tokens.device)
    ranks = torch.empty((n, steps), dtype=torch.int64, device=dec.tokens.device)
    toks = torch.empty((n, steps), dtype=torch.int32, device=dec.tokens.device)
    ncount = torch.empty((n, steps, len(NEAR_TIE_DELTAS)), dtype=torch.int64, device=dec.tokens.device)
    for s in range(steps):
        dec.step("off")
        margins[:, s] = dec.margin[rows]
        ranks[:, s] = _rank_of(dec.logits[rows], ref_dev[:, s])
        ncount[:, s] = near_tie_count(dec.logits[rows])
        toks[:, s] = dec.tokens[rows]
    kv_fast = final_layer_kv(dec, p0, steps)
    ek = torch.linalg.vector_norm((kv_fast[:, :, 0] - kv_ref[:, :, 0]).flatten(2), dim=2).cpu().numpy()
    evv = torch.linalg.vector_norm((kv_fast[:, :, 1] - kv_ref[:, :, 1]).flatten(2), dim=2).cpu().numpy()
    stats = divergence_stats(toks.cpu().numpy(), reference, margins.cpu().numpy(), ranks.cpu().numpy(), ek, evv,
                             tau, window, ncount.cpu().numpy())
    return stats, reference


def divergence_stats(toks, reference, margins, ranks, ek, ev_, tau: float, window: int = 16, ncount=None) -> dict:
    """The statistics of flip_study from its per-row, per-step arrays: emitted tokens and the
    reference's [rows][steps], the fast margins and the reference token's rank in the fast
    logits at each step, the final-layer K and V l2 deviations at each cache step, and
    (optional) the near-tie counts N(Delta) [rows][steps][len(NEAR_TIE_DELTAS)]."""
    n, steps = reference.shape
    same = toks == reference
    diverged = ~same.all(1)
    first = np.where(diverged, np.argmin(same, axis=1), steps)
    # Obs. 1: events over synchronous samples (each row's steps up to its first divergence)
    events = int(diverged.sum())
    samples = int(np.minimum(first + 1, steps).sum())
    # Obs. 3: the event step s = first[b]; the stable synchronous steps s < first[b]
    evr = np.nonzero(diverged)[0]
    ev_rank = ranks[evr, first[evr]]
    ev_margin = margins[evr, first[evr]]
    stable = np.concatenate([margins[b, :first[b]] for b in range(n)] + [np.zeros(0, np.float32)])
    # Obs. 2: the token emitted at step s is the input at position p0 + s + 1, whose column
    # is written at step s + 1 -- so Delta = 0 is cache step first + 1; rows with fewer than
    # 3 pre-divergence columns are left out
    pre_k, pre_v, spike_k, spike_v, slope_k = [], [], [], [], []
    for b in evr:
        d0 = first[b] + 1
        if d0 >= steps or d0 < 3:
            continue
        lo = max(0, d0 - window)
        pk, pv = ek[b, lo:d0], ev_[b, lo:d0]
        pre_k.append(pk.mean())
        pre_v.append(pv.mean())
        spike_k.append(ek[b, d0] / max(pk.mean(), 1e-30))
        spike_v.append(ev_[b, d0] / max(pv.mean(), 1e-30))
        slope_k.append(np.polyfit(np.arange(lo - d0, 0), pk, 1)[0])

    def med(a):
        return float(np.median(a)) if len(a) else None

    def share(mask):
        return float(np.mean(mask)) if mask.size else None

    # Table 4: mean N(Delta) over the token-stable synchronous steps (s < first) and over the
    # divergent steps (s = first)
    cluster = None
    if ncount is not None:
        stable_mask = np.arange(steps)[None, :] < first[:, None]
        cluster = {}
        for k, dlt in enumerate(NEAR_TIE_DELTAS):
            ns = ncount[:, :, k][stable_mask]
            nd = ncount[evr, first[evr], k]
            ms = float(ns.mean()) if ns.size else None
            md = float(nd.mean()) if nd.size else None
            cluster[str(dlt)] = dict(stable=ms, divergent=md,
                                     ratio=(md / ms) if (ms and md is not None) else None)

    return dict(
        steps=steps, rows=n, tau=float(tau),
        flips=dict(events=events, synchronous_samples=samples, rate=events / max(samples, 1),
                   first_divergence_mean=float(first.mean())),
        kv=dict(trials=len(pre_k), window=window, k_pre=med(pre_k), k_spike=med(spike_k), v_pre=med(pre_v),
                v_spike=med(spike_v), k_slope_median=med(slope_k), k_slope_abs_median=med(np.abs(slope_k))),
        near_tie=dict(events=int(evr.size), top2=share(ev_rank <= 1), top3=share(ev_rank <= 2),
                      top8=share(ev_rank <= 7), event_margin_median=med(ev_margin), stable_margin_median=med(stable),
                      gate_recall=share(ev_margin < tau), stable_trigger=share(stable < tau)),
        near_tie_count=cluster)


def oracle_position_repair(dec: GatedDecoder, state, kv_snap, steps: int, reference):
    """The verifier and the repair (the method's action) exactly at the steps where a row's
    fast token differs from the reference token (known in advance, as the oracle of Sec. 2
    knows the true divergence positions).  Returns repairs per sequence, the share of rows
    whose whole sequence equals the reference, and the verified row-steps."""
    e = dec.e
    e.kv_pool.copy_(kv_snap)
    dec.set_state(*state)
    B = dec.B
    rows_all = dec.always_rows
    n_all = int(rows_all.numel())
    if n_all != B:
        raise ValueError("the oracle-position run needs every row protected")
    ref_dev = torch.as_tensor(reference, device=dec.tokens.device)
    dec.n_repaired.zero_()
    verified = 0
    out = np.zeros((n_all, steps), np.int32)
    vmask = np.zeros((n_all, steps), bool)
    for s in range(steps):
        e.decode_step(B, dec.tokens, dec.positions, dec.page_table, dec.logits)
        e.margin_gate(B, dec.logits, dec.protected, 0.0, dec.top1, dec.margin, dec.gate, dec.gated_rows, dec.n_gated,
                      None)
        rows = torch.nonzero(dec.top1 != ref_dev[:, s]).flatten().to(torch.int32)
        n = int(rows.numel())
        if n:
            vmask[rows.cpu().numpy(), s] = True
            e.verify_rows(n, rows, None, dec.tokens, dec.positions, dec.page_table, None, dec.v_tok, dec.v_kvcol)
            e.repair_kv_column(n, rows, None, dec.positions, dec.page_table, dec.top1, dec.v_tok, dec.v_kvcol,
                               dec.top1, dec.n_repaired)
        verified += n
        e.advance(B, dec.top1, dec.tokens, dec.positions)
        out[:, s] = dec.tokens.cpu().numpy()
    cmp = calibrate.compare_to_reference(out, reference)
    # repairs while a row is still on the reference (steps up to its first unrepaired
    # divergence): the count the oracle experiment of Sec. 2 reports
    same = out == reference
    first = np.where(same.all(1), steps, np.argmin(same, axis=1))
    sync = np.arange(steps)[None, :] <= first[:, None]
    return dict(steps=steps, rows=n_all, verified_row_steps=verified,
                repairs_per_sequence=int(dec.n_repaired.item()) / n_all,
                synchronous_repairs_per_sequence=float((vmask & sync).sum()) / n_all, **cmp)
