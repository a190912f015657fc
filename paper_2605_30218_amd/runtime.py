"""Host-side sequencing of the MarginGate decode loop over libmg (arXiv 2605.30218, Sec. 3).

Per step: the fast batched forward (tentative K/V append), the margin gate (which
also stores the gated-row count into pinned host memory, polled here instead of a
stream synchronisation), the verifier on exactly those rows, and the commit /
single-column repair.  Modes: "off" (fast path only, r_verify = 0),
"gated" (MarginGate), "always" (the verifier on every protected row, r_verify = 1:
the always-on baseline of Sec. 3.3).  All arithmetic runs in libmg; this module only
orders calls and keeps counters.
"""
from __future__ import annotations

import time

import numpy as np
import torch

from . import mg
from .mg import Engine


def check_positions(page_table, positions, page_size: int, n_pages: int):
    """Host guard of the device-trusted inputs of a step: every row's position must lie inside its
    page-table row and on a mapped page of the pool (the kernels write the tentative K/V column
    through that entry and read the RoPE table at that position, unchecked).  Raises ValueError."""
    pt = np.asarray(page_table)
    pos = np.asarray(positions).astype(np.int64)
    if pt.ndim != 2 or pos.shape != (pt.shape[0],):
        raise ValueError(f"page table {pt.shape} and positions {pos.shape} do not match")
    cap = pt.shape[1] * page_size
    bad = np.nonzero((pos < 0) | (pos >= cap))[0]
    if bad.size:
        r = int(bad[0])
        raise ValueError(f"row {r}: position {int(pos[r])} outside its page-table row (capacity {cap})")
    pages = pt[np.arange(pos.size), pos // page_size]
    bad = np.nonzero((pages < 0) | (pages >= n_pages))[0]
    if bad.size:
        r = int(bad[0])
        raise ValueError(f"row {r}: position {int(pos[r])} maps to page {int(pages[r])}, not a page of the pool "
                         f"(0..{n_pages - 1})")


class GatedDecoder:
    def __init__(self, engine: Engine, page_table, protected=None, tau: float = 0.5):
        self.e = engine
        dev = engine.device
        # host mirrors of the page table and the positions, for the capacity guard
        self._pt_host = np.ascontiguousarray(np.asarray(page_table, np.int32))
        self._pos_host = None
        self.page_table = torch.as_tensor(page_table, dtype=torch.int32).to(dev).contiguous()
        self.B = self.page_table.shape[0]
        B, V = self.B, engine.shape.vocab
        self.tau = float(tau)
        self.protected = None if protected is None else torch.as_tensor(protected, dtype=torch.uint8).to(dev)
        prot = np.ones(B, bool) if protected is None else np.asarray(protected, bool)
        self.always_rows = torch.as_tensor(np.nonzero(prot)[0].astype(np.int32)).to(dev)
        i32 = dict(dtype=torch.int32, device=dev)
        self.tokens = torch.zeros(B, **i32)
        self.positions = torch.zeros(B, **i32)
        self.logits = torch.empty((B, V), dtype=torch.float32, device=dev)
        self.top1 = torch.empty(B, **i32)          # also the emitted tokens (repair rewrites gated rows)
        self.margin = torch.empty(B, dtype=torch.float32, device=dev)
        self.gate = torch.empty(B, dtype=torch.uint8, device=dev)
        self.gated_rows = torch.empty(B, **i32)
        self.n_gated = torch.zeros(1, **i32)
        self.v_tok = torch.empty(B, **i32)
        self.v_kvcol = torch.empty((B, engine.col_elems), dtype=torch.int16, device=dev)
        self.n_repaired = torch.zeros(1, **i32)
        # the commit's repair action: the method's (copy the verifier column when the tokens
        # differ), or a variant for the repair-action measurements (mg.REPAIR_TOKEN_ONLY,
        # mg.REPAIR_COPY_ALWAYS)
        self.repair_action = mg.REPAIR_ON_MISMATCH
        # the verifier: "canonical" (mg_verify_rows, the oracle's order bit for bit) or "mfma"
        # (mg_verify_rows_mfma: fixed-tile matrix-core forward, batch-invariant, tolerance
        # parity)
        self.verifier = "canonical"
        # the gate mirrors its count into pinned host memory; the host polls it instead of
        # synchronising the stream
        self._count_dev, self._count = mg.host_count_slot()
        self.steps = 0
        self.protected_row_steps = 0
        self.verified_row_steps = 0
        self.hist = []

    def set_state(self, tokens, positions):
        pos = np.array(positions, np.int32, copy=True)
        check_positions(self._pt_host, pos, self.e.shape.page_size, self.e.cfg.n_pages)
        self.tokens.copy_(torch.as_tensor(np.asarray(tokens, np.int32)))
        self.positions.copy_(torch.as_tensor(pos))
        self._pos_host = pos

    def step(self, mode: str = "gated", keep=None):
        """One decode step.  keep: optional dict that receives host copies of the step's
        logits / top1 / margin / gate / rows / v_tok (tests)."""
        e, B = self.e, self.B
        if self._pos_host is None:
            raise RuntimeError("GatedDecoder.step before set_state")
        check_positions(self._pt_host, self._pos_host, e.shape.page_size, e.cfg.n_pages)
        e.decode_step(B, self.tokens, self.positions, self.page_table, self.logits)
        gated = mode not in ("off", "always")
        if gated:
            self._count[0] = -1
        e.margin_gate(B, self.logits, self.protected, self.tau, self.top1, self.margin, self.gate, self.gated_rows,
                      self.n_gated, self._count_dev if gated else None)
        if mode == "off":
            n, rows = 0, self.gated_rows
        elif mode == "always":
            rows = self.always_rows
            n = int(rows.numel())
        else:
            n, rows = self._wait_count(), self.gated_rows
        if keep is not None:
            keep.update(logits=self.logits.cpu().numpy(), top1=self.top1.cpu().numpy(),
                        margin=self.margin.cpu().numpy(), gate=self.gate.cpu().numpy(),
                        positions=self.positions.cpu().numpy(), tokens=self.tokens.cpu().numpy())
        if n:
            if self.verifier == "mfma":
                e.verify_rows_mfma(n, rows, self.tokens, self.positions, self.page_table, None, self.v_tok,
                                   self.v_kvcol)
            else:
                e.verify_rows(n, rows, None, self.tokens, self.positions, self.page_table, None, self.v_tok,
                              self.v_kvcol)
            if self.repair_action == mg.REPAIR_ON_MISMATCH:
                e.repair_kv_column(n, rows, None, self.positions, self.page_table, self.top1, self.v_tok, self.v_kvcol,
                                   self.top1, self.n_repaired)
            else:
                e.repair_kv_column_action(n, rows, None, self.positions, self.page_table, self.top1, self.v_tok,
                                          self.v_kvcol, self.top1, self.n_repaired, self.repair_action)
            if keep is not None:
                keep.update(rows=rows[:n].cpu().numpy(), v_tok=self.v_tok[:n].cpu().numpy())
        elif keep is not None:
            keep.update(rows=np.zeros(0, np.int32), v_tok=np.zeros(0, np.int32))
        e.advance(B, self.top1, self.tokens, self.positions)
        self._pos_host += 1
        self.steps += 1
        self.protected_row_steps += int(self.always_rows.numel())
        self.verified_row_steps += n
        self.hist.append(n)
        return n

    def _wait_count(self, limit_s: float = 60.0) -> int:
        """Poll the pinned count slot until the gate kernel has stored the count."""
        spins, t0 = 0, None
        while True:
            v = int(self._count[0])
            if v >= 0:
                return v
            spins += 1
            if spins % 4096 == 0:
                now = time.perf_counter()
                t0 = now if t0 is None else t0
                if now - t0 > limit_s:
                    torch.cuda.synchronize()  # surfaces a kernel error, if any
                    v = int(self._count[0])
                    if v < 0:
                        raise RuntimeError("the margin gate's count never reached host memory")
                    return v

    @property
    def r_verify(self):
        return self.verified_row_steps / max(self.protected_row_steps, 1)

    def r_repair(self):
        return int(self.n_repaired.item()) / max(self.protected_row_steps, 1)


def prefill_rows(engine: Engine, prompts, page_table, max_items: int = 1024):
    """Canonical prefill of positions 0..len-2 of every prompt (the last prompt token is
    consumed by the first decode step).  Items are issued in increasing position order, so
    every earlier position of a row is in the cache before a later one attends to it."""
    dev = engine.device
    pts = np.asarray(page_table, np.int32)
    for r, pr in enumerate(prompts):  # the last prefilled position of each row, and every earlier page
        if len(pr) > 1:
            check_positions(pts[r:r + 1], [len(pr) - 2], engine.shape.page_size, engine.cfg.n_pages)
            n_pg = (len(pr) - 2) // engine.shape.page_size + 1
            if (pts[r, :n_pg] < 0).any():
                raise ValueError(f"row {r}: a prompt page is unmapped")
    items = [(t, p, r) for r, pr in enumerate(prompts) for p, t in enumerate(pr[:-1])]
    items.sort(key=lambda x: (x[1], x[2]))
    pt = torch.as_tensor(np.asarray(page_table, np.int32)).to(dev).contiguous()
    arr = np.asarray(items, np.int32).reshape(-1, 3)
    for o in range(0, len(arr), max_items):
        chunk = arr[o:o + max_items]
        tok = torch.as_tensor(np.ascontiguousarray(chunk[:, 0])).to(dev)
        pos = torch.as_tensor(np.ascontiguousarray(chunk[:, 1])).to(dev)
        row = torch.as_tensor(np.ascontiguousarray(chunk[:, 2])).to(dev)
        engine.prefill(len(chunk), tok, pos, row, pt)
    torch.cuda.synchronize()
    last = np.array([pr[-1] for pr in prompts], np.int32)
    pos0 = np.array([len(pr) - 1 for pr in prompts], np.int32)
    return last, pos0


def prefill_fast(engine: Engine, prompts, page_table):
    """Prompt prefill through the fast path: teacher-forced decode steps over positions
    0..len-2, all rows still in their prompt advancing together.  Cheaper than the canonical
    prefill; its cache depends on the batch shape like every fast-path column."""
    dev = engine.device
    pt = np.asarray(page_table, np.int32)
    lens = np.array([len(p) for p in prompts])
    for r in range(len(prompts)):
        if lens[r] > 1:
            n_pg = (int(lens[r]) - 2) // engine.shape.page_size + 1
            check_positions(pt[r:r + 1], [int(lens[r]) - 2], engine.shape.page_size, engine.cfg.n_pages)
            if (pt[r, :n_pg] < 0).any():
                raise ValueError(f"row {r}: a prompt page is unmapped")
    logits = torch.empty((len(prompts), engine.shape.vocab), dtype=torch.float32, device=dev)
    for t in range(int(lens.max()) - 1):
        act = np.nonzero(lens - 1 > t)[0]
        tok = torch.as_tensor(np.array([prompts[r][t] for r in act], np.int32)).to(dev)
        pos = torch.full((act.size,), t, dtype=torch.int32, device=dev)
        ptr = torch.as_tensor(np.ascontiguousarray(pt[act])).to(dev)
        engine.decode_step(int(act.size), tok, pos, ptr, logits)
    torch.cuda.synchronize()
    last = np.array([pr[-1] for pr in prompts], np.int32)
    return last, (lens - 1).astype(np.int32)
