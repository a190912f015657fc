"""Benchmark of the MarginGate decode step on one MI355X.

Workloads (--config; random-init N(0, 0.02) bf16 weights of the named shape, seeded synthetic
inputs, greedy decode, every row protected):
  llama8b  (default) Llama-3.1-8B shape (32 layers, d 4096, 32/8 heads, hd 128, FFN 14336,
           vocab 128256, RoPE theta 5e5), batch 64, uniform random 512-token prompts
           (canonical prefill, not timed); tau set for the paper's Llama-3.1-8B trigger rate
           (18.56%, the quantile of the fast-path margins of an untimed run as long as the
           timed one)
  qwen7b   Qwen2.5-7B shape with QKV bias, batch 32, 1024-token prompts (canonical prefill),
           the LM head's seeded tie-pair perturbation, tau = 0.5 (about half of the steps
           trigger)
  qwen14b  Qwen2.5-14B shape with QKV bias, batch 128, prompt lengths uniform in [128, 2048]
           (seeded synthetic caches), tau = the 15% quantile of a 16-step calibration run
  longctx  Llama-3.1-8B shape, 32 slots with contexts uniform in [4096, 16384] (seeded
           synthetic caches); phases of 16 steps between which a seeded subset of rows leaves
           and new rows join (batch 8..32); the llama8b tau
Modes, each from the same prefilled state:
  off     the BF16 fast path only (r_verify = 0)
  gated   MarginGate: verify rows whose top-1/top-2 margin is below tau
  always  the verifier on every row and step (the always-on baseline, r_verify = 1)
  gated_mfma, always_mfma  (llama8b) the same with the matrix-core verifier (fixed tiling,
          batch-invariant, tolerance parity) instead of the canonical one
The timed modes record no kernel events; a separate gated pass brackets the launches of the
four main kernel kinds with HIP events for the per-kernel figures and the roofline.

One JSON line on stdout: value = gated decode tokens/s (rows * steps / time of the timed
steps, inputs resident in HBM), plus the other modes, the verifier overhead
(inc_mode = T_mode / T_off - 1, cut = inc_always / inc_gated), the roofline of the dominant
kernel, the HBM roofline fraction of each mode and of the fast forward and the verifier
alone (algorithmic bytes: every streamed weight once per forward, the live K/V of the rows
involved, the fp32 logits), and the CPU oracle baseline on a bounded sample.  llama8b also
reports the paper's tau calibration recipe, the repair actions, the divergence diagnostics,
the protected row decoded alone (bs = 1) against the same row inside the batch, and the fast
step's HBM fraction at batch 1, 8, 16 and 32.
"""
import argparse
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2605_30218_amd import calibrate, diagnostics, mg, profsum, synth  # noqa: E402
from paper_2605_30218_amd.runtime import GatedDecoder, prefill_fast, prefill_rows  # noqa: E402

METRIC = "decode tok/s + gated-vs-always-on verifier overhead, Llama-3.1-8B-shape bs=64"
HBM_PEAK = 8.0e12            # B/s, MI355X
FP32_VECTOR_PEAK = 157.3e12  # flop/s: 256 CU x 2.4 GHz x 256 fp32 flop/clk (the published vector peak;
                             # plain v_fma_f32 measures above half of it, so half is no ceiling)
PAPER_TRIGGER = 0.1856       # Llama-3.1-8B trigger rate at tau_100 (paper Sec. 4.3)
LLAMA8B_TAU = 0.059          # the llama8b workload's calibrated tau (18.56% trigger), reused by longctx
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "{kernel}_traffic_{config}.txt")
KIND_NAMES = {mg.KIND_FAST_GEMM: "fast_gemm", mg.KIND_CANON_GEMV: "canon_gemv", mg.KIND_FAST_ATTN: "fast_attention",
              mg.KIND_CANON_ATTN: "canon_attention"}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kv_bytes_per_pos(shape):
    """K and V bytes of one position in one layer."""
    return shape.n_kv_heads * shape.head_dim * 2 * 2


def attn_bytes(shape, ctxs):
    """Algorithmic HBM bytes of one layer's decode attention over rows attending `ctxs`
    positions each: their K and V, the rotated queries in and the attention outputs out."""
    ctxs = np.asarray(ctxs, np.float64)
    return float(ctxs.sum()) * kv_bytes_per_pos(shape) + ctxs.size * 2 * shape.n_q_heads * shape.head_dim * 2


def streamed_weight_bytes(shape):
    """bf16 bytes of every weight a forward streams (the embedding is gathered, not streamed)."""
    return 2 * (shape.n_params() - shape.vocab * shape.d_model)


def forward_bytes(shape, ctxs):
    """Algorithmic HBM bytes of one forward over rows attending `ctxs` positions each: every
    streamed weight once, each layer's attention bytes, the fp32 logits written."""
    n = len(ctxs)
    if n == 0:
        return 0.0
    return streamed_weight_bytes(shape) + shape.n_layers * attn_bytes(shape, ctxs) + n * shape.vocab * 4


# ---------------------------------------------------------------- workloads

class Workload:
    """A prefilled engine and the state every mode starts from.  Fixed-batch workloads have one
    phase; longctx has several (rows join and leave between phases)."""

    def __init__(self, name, shape, weights, eng, desc, global_batch, seq_len):
        self.name, self.shape, self.weights, self.eng = name, shape, weights, eng
        self.desc, self.global_batch, self.seq_len = desc, global_batch, seq_len
        self.phases = []        # list of dict(pt, tokens, positions, join): join = [(slot, ctx, seed)]
        self.kv_snap = None
        self.prefill_s = 0.0
        self.tau = None

    def start(self):
        """Restore the prefilled cache."""
        self.eng.kv_pool.copy_(self.kv_snap)


def make_llama8b(args, shape=synth.LLAMA8B):
    B, P = args.batch or 64, args.prompt or 512
    ctx_cap = P + args.warmup + args.steps + 16
    maxp = -(-ctx_cap // shape.page_size)
    pt, n_pages = synth.make_page_table([ctx_cap] * B, shape.page_size, maxp, seed=5)
    log(f"[bench] weights {shape.name} on GPU (seed 0)")
    w = synth.make_weights(shape, seed=0, device="cuda")
    eng = mg.Engine(shape, w, B, maxp, n_pages, max_prefill=1024)
    wl = Workload("llama8b", shape, w, eng,
                  f"Llama-3.1-8B-shaped random-init decoder, batch {B}, uniform random {P}-token prompts, gated "
                  f"greedy decode (all rows protected, tau for an 18.56% trigger)", B, P)
    prompts = synth.make_prompts(B, [P] * B, shape.vocab, seed=1)
    log(f"[bench] {args.prefill} prefill {B} x {P - 1} tokens")
    t0 = time.perf_counter()
    last, pos0 = (prefill_rows if args.prefill == "canonical" else prefill_fast)(eng, prompts, pt)
    wl.prefill_s = time.perf_counter() - t0
    wl.phases = [dict(pt=pt, tokens=last, positions=pos0, join=[])]
    wl.kv_snap = eng.kv_pool.clone()
    return wl


def make_qwen7b(args):
    shape, B, P, tau = synth.QWEN7B, args.batch or 32, args.prompt or 1024, 0.5
    ctx_cap = P + args.warmup + args.steps + 16
    maxp = -(-ctx_cap // shape.page_size)
    pt, n_pages = synth.make_page_table([ctx_cap] * B, shape.page_size, maxp, seed=5)
    log(f"[bench] weights {shape.name} on GPU (seed 0, tie-pair LM-head perturbation seed 4)")
    w = synth.perturb_lm_head_tie_pairs(synth.make_weights(shape, seed=0, device="cuda"), shape, seed=4, tau=tau)
    eng = mg.Engine(shape, w, B, maxp, n_pages, max_prefill=1024)
    wl = Workload("qwen7b", shape, w, eng,
                  f"Qwen2.5-7B-shaped random-init decoder with QKV bias, batch {B}, uniform random {P}-token "
                  f"prompts, LM head with the seeded tie-pair low-rank perturbation (high-trigger regime), gated "
                  f"greedy decode at tau {tau} (all rows protected)", B, P)
    prompts = synth.make_prompts(B, [P] * B, shape.vocab, seed=1)
    log(f"[bench] canonical prefill {B} x {P - 1} tokens")
    t0 = time.perf_counter()
    last, pos0 = prefill_rows(eng, prompts, pt)
    wl.prefill_s = time.perf_counter() - t0
    wl.phases = [dict(pt=pt, tokens=last, positions=pos0, join=[])]
    wl.kv_snap = eng.kv_pool.clone()
    wl.tau = tau
    return wl


def make_qwen14b(args):
    shape, B = synth.QWEN14B, args.batch or 128
    lens = synth.make_lengths(B, 128, 2048, seed=2)
    ctx = lens + args.warmup + max(args.steps, 16) + 16
    maxp = -(-int(ctx.max()) // shape.page_size)
    pt, n_pages = synth.make_page_table(ctx, shape.page_size, maxp, seed=5)
    log(f"[bench] weights {shape.name} on GPU (seed 0)")
    w = synth.make_weights(shape, seed=0, device="cuda")
    eng = mg.Engine(shape, w, B, maxp, n_pages)
    wl = Workload("qwen14b", shape, w, eng,
                  f"Qwen2.5-14B-shaped random-init decoder with QKV bias, batch {B}, prompt lengths uniform in "
                  f"[128, 2048] (seeded synthetic caches), gated greedy decode at the 15% margin quantile (all rows "
                  f"protected)", B, int(lens.mean()))
    t0 = time.perf_counter()
    cached = np.concatenate([pt[r, :-(-(int(lens[r]) - 1) // shape.page_size)] for r in range(B)])
    synth.fill_synthetic_kv(eng.kv_view(), cached, seed=6)
    torch.cuda.synchronize()
    wl.prefill_s = time.perf_counter() - t0
    prompts = synth.make_prompts(B, lens, shape.vocab, seed=1)
    last = np.array([p[-1] for p in prompts], np.int32)
    wl.phases = [dict(pt=pt, tokens=last, positions=(lens - 1).astype(np.int32), join=[])]
    wl.kv_snap = eng.kv_pool.clone()
    return wl


def make_longctx(args):
    shape, slots, phase_steps = synth.LLAMA8B, 32, 16
    n_phases = max(1, -(-args.steps // phase_steps))
    ctx_lo, ctx_hi = 4096, 16384
    maxp = -(-(ctx_hi + args.warmup + n_phases * phase_steps + 16) // shape.page_size)
    pt_slots, n_pages = synth.make_page_table([maxp * shape.page_size] * slots, shape.page_size, maxp, seed=5)
    log(f"[bench] weights {shape.name} on GPU (seed 0), {slots} slots x {maxp} pages")
    w = synth.make_weights(shape, seed=0, device="cuda")
    eng = mg.Engine(shape, w, slots, maxp, n_pages)
    wl = Workload("longctx", shape, w, eng,
                  f"Llama-3.1-8B-shaped random-init decoder with long-context paged KV: {slots} slots, contexts "
                  f"uniform in [{ctx_lo}, {ctx_hi}] (seeded synthetic caches), phases of {phase_steps} steps between "
                  f"which rows leave and join (batch 8..{slots}), gated greedy decode at the llama8b tau", slots,
                  (ctx_lo + ctx_hi) // 2)
    wl.pt_slots = pt_slots
    wl.phase_steps = phase_steps
    rng = np.random.default_rng(3)
    # the schedule: which slots are active in each phase and the rows that join at its start
    active = [int(s) for s in rng.permutation(slots)]
    joins = [[(s, int(rng.integers(ctx_lo, ctx_hi + 1)), 100 + i, int(rng.integers(0, shape.vocab)))
              for i, s in enumerate(active)]]
    sched = [active]
    nj = len(active)
    for _ in range(1, n_phases):
        b_next = int(rng.integers(8, slots + 1))
        keep_n = min(len(active) - 1, b_next)
        kept = [int(s) for s in rng.choice(active, keep_n, replace=False)]
        free = [s for s in range(slots) if s not in kept]
        new = [int(s) for s in rng.choice(free, b_next - keep_n, replace=False)]
        j = []
        for s in new:
            j.append((s, int(rng.integers(ctx_lo, ctx_hi + 1)), 100 + nj, int(rng.integers(0, shape.vocab))))
            nj += 1
        active = [int(s) for s in rng.permutation(kept + new)]
        sched.append(active)
        joins.append(j)
    wl.phases = [dict(slots=a, join=j) for a, j in zip(sched, joins)]
    wl.tau = LLAMA8B_TAU
    wl.kv_snap = None  # every run re-creates its caches from the seeded schedule
    return wl


WORKLOADS = {"llama8b": make_llama8b, "qwen7b": make_qwen7b, "qwen14b": make_qwen14b, "longctx": make_longctx}


# ---------------------------------------------------------------- runs

def join_rows(wl, join, tok, pos):
    """Seeded synthetic caches (and the first token) of rows that join (not timed)."""
    for slot, ctx, seed, t in join:
        npg = -(-(ctx - 1) // wl.shape.page_size)
        synth.fill_synthetic_kv(wl.eng.kv_view(), wl.pt_slots[slot, :npg], seed=seed)
        tok[slot] = t
        pos[slot] = ctx - 1


def run_mode(wl, mode, warmup, steps, tau, profile_kinds=(), profile_steps=32, record_row=None):
    """One mode over the workload from its start state.  Returns the timing and rate record
    (and, when profile_kinds is given, the per-kind HIP event figures in 'prof')."""
    name, _, ver = mode.partition("_")
    eng, shape = wl.eng, wl.shape
    L = shape.n_layers
    per_step = {mg.KIND_FAST_GEMM: 4 * L + 1, mg.KIND_CANON_GEMV: 4 * L + 1, mg.KIND_FAST_ATTN: L,
                mg.KIND_CANON_ATTN: L}
    prof_steps = min(steps, profile_steps)
    for k in profile_kinds:
        eng.profile_begin(k, prof_steps * per_step[k])
    wall, per, hist, fast_b, ver_b = 0.0, [], [], 0.0, 0.0
    prot = ver_rows = 0
    n_rep = 0
    fast_ctx_steps, ver_ctx_steps = [], []   # per-step context lists (for the attention bytes)
    row_tokens = []
    if wl.name == "longctx":
        slots = len(wl.pt_slots)
        tok = np.zeros(slots, np.int32)
        pos = np.zeros(slots, np.int32)
        phases = wl.phases
    else:
        wl.start()
        phases = wl.phases
    for ph_i, ph in enumerate(phases):
        if wl.name == "longctx":
            join_rows(wl, ph["join"], tok, pos)
            active = ph["slots"]
            pt, ptok, ppos = wl.pt_slots[active], tok[active], pos[active]
            ph_steps = min(wl.phase_steps, steps - ph_i * wl.phase_steps)
            ph_warm = warmup if ph_i == 0 else 0
        else:
            pt, ptok, ppos = ph["pt"], ph["tokens"], ph["positions"]
            ph_steps, ph_warm = steps, warmup
        if ph_steps <= 0:
            break
        dec = GatedDecoder(eng, pt, None, tau=tau)
        dec.verifier = "mfma" if ver == "mfma" else "canonical"
        dec.set_state(ptok, ppos)
        for _ in range(ph_warm):
            dec.step(name)
        torch.cuda.synchronize()
        dec.protected_row_steps = dec.verified_row_steps = 0
        dec.hist = []
        dec.n_repaired.zero_()
        ctx0 = dec._pos_host.copy() + 1    # positions attended at the first timed step
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(ph_steps + 1)]
        rec = []
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ev[0].record()
        for s in range(ph_steps):
            dec.step(name)
            ev[s + 1].record()
            if record_row is not None:
                rec.append(dec.tokens[record_row].clone())
        torch.cuda.synchronize()
        wall += time.perf_counter() - t0
        per += [ev[s].elapsed_time(ev[s + 1]) for s in range(ph_steps)]
        row_tokens += [int(t.item()) for t in rec]
        prot += dec.protected_row_steps
        ver_rows += dec.verified_row_steps
        n_rep += int(dec.n_repaired.item())
        hist += dec.hist
        mean_ctx = float(ctx0.mean())
        for s in range(ph_steps):
            fast_ctx_steps.append(ctx0 + s)
            ver_ctx_steps.append(np.full(dec.hist[s], mean_ctx + s))
        if wl.name == "longctx":
            tok[active] = dec.tokens.cpu().numpy()
            pos[active] = dec.positions.cpu().numpy()
    prof = {k: eng.profile_end(k) for k in profile_kinds}
    n_steps = len(per)
    # attention bytes of the recorded launches: the library does not know the positions (they
    # live on the device), the benchmark does; a kind records the launches of the first steps
    # that ran it (the verifier runs only on steps with gated rows).  Verified rows are taken
    # at the batch's mean context of their step.
    for k, ctxs in ((mg.KIND_FAST_ATTN, fast_ctx_steps), (mg.KIND_CANON_ATTN, ver_ctx_steps)):
        if k in prof:
            n, ms, b, f = prof[k]
            ran = [c for c in ctxs if len(c)][:n // L]
            prof[k] = (n, ms, float(sum(L * attn_bytes(shape, c) for c in ran)), f)
    fast_b = sum(forward_bytes(shape, c) for c in fast_ctx_steps)
    ver_b = sum(forward_bytes(shape, c) for c in ver_ctx_steps)
    rows_total = sum(len(c) for c in fast_ctx_steps)
    per = np.asarray(per)
    out = dict(ms_per_step=wall * 1e3 / n_steps, tok_s=rows_total / wall, p50_ms=float(np.median(per)),
               p99_ms=float(np.percentile(per, 99)), r_verify=ver_rows / max(prot, 1), r_repair=n_rep / max(prot, 1),
               verified_rows_per_step=float(np.mean(hist)),
               verified_rows_hist=np.bincount(np.asarray(hist, dtype=np.int64), minlength=1).tolist(),
               fast_bytes_per_step=fast_b / n_steps, verifier_bytes_per_step=ver_b / n_steps,
               hbm_frac=(fast_b + ver_b) / wall / HBM_PEAK, prof=prof)
    if record_row is not None:
        out["row_tokens"] = row_tokens
    return out


def calibrate_tau(wl, steps, rate):
    """The `rate` quantile of the fast-path margins of every row over an untimed run."""
    wl.start()
    ph = wl.phases[0]
    dec = GatedDecoder(wl.eng, ph["pt"], None, tau=0.0)
    dec.set_state(ph["tokens"], ph["positions"])
    ms = []
    for _ in range(steps):
        dec.step("off")
        ms.append(dec.margin.cpu().numpy().copy())
    return float(np.quantile(np.concatenate(ms), rate))


def kernel_table(prof):
    kernels = {}
    for k, (n, ms, b, f) in prof.items():
        kernels[KIND_NAMES[k]] = dict(launches=n, total_ms=ms, avg_us=1e3 * ms / max(n, 1), algo_bytes=b,
                                      algo_flops=f, gbps=b / (ms * 1e-3) / 1e9 if ms > 0 else 0.0,
                                      tflops=f / (ms * 1e-3) / 1e12 if ms > 0 else 0.0)
    return kernels


def roofline_of(kernels, config):
    """Roofline entry of the kernel kind with the most time."""
    if not kernels:
        return None
    dom = max(kernels, key=lambda k: kernels[k]["total_ms"])
    kd = kernels[dom]
    sec = kd["total_ms"] * 1e-3
    hbm = kd["algo_bytes"] / sec
    alu = kd["algo_flops"] / sec
    # HBM bytes per launch from the committed FETCH_SIZE / WRITE_SIZE summary of this workload,
    # if it was taken on the kernel's current source
    traffic = None
    if dom in profsum.SOURCES:
        t = profsum.read_traffic(TRAFFIC_SUMMARY.format(kernel=dom, config=config))
        if t and t[1] == profsum.source_sha(dom):
            traffic = t[0]
    common = dict(kernel=dom, traffic=traffic, traffic_unit="bytes/launch", launches=kd["launches"],
                  algo_bytes_per_launch=kd["algo_bytes"] / max(kd["launches"], 1), avg_us=kd["avg_us"])
    # the bound follows the arithmetic intensity of the launches against the ridge point
    if dom == "canon_gemv" and kd["algo_flops"] / kd["algo_bytes"] > FP32_VECTOR_PEAK / HBM_PEAK:
        return dict(bound="alu", achieved=alu / 1e12, peak=FP32_VECTOR_PEAK / 1e12, unit="TFLOP/s",
                    frac=alu / FP32_VECTOR_PEAK, **common)
    return dict(bound="hbm", achieved=hbm / 1e9, peak=HBM_PEAK / 1e9, unit="GB/s", frac=hbm / HBM_PEAK, **common)


def bs1_leg(wl, warmup, steps, tau):
    """Sequence determinism of the protected row (Sec. 4.1): row 0 decoded alone (bs = 1) under
    the gate at tau, from the same prefilled state, against its tokens inside the batch (an
    untimed gated run of the whole batch that records row 0's emitted tokens)."""
    batch = run_mode(wl, "gated", warmup, steps, tau, record_row=0)
    ph = wl.phases[0]
    one = Workload(wl.name, wl.shape, wl.weights, wl.eng, wl.desc, 1, wl.seq_len)
    one.kv_snap = wl.kv_snap
    one.phases = [dict(pt=ph["pt"][:1], tokens=ph["tokens"][:1], positions=ph["positions"][:1], join=[])]
    r = run_mode(one, "gated", warmup, steps, tau, record_row=0)
    alone = np.asarray(r.pop("row_tokens"))
    inb = np.asarray(batch["row_tokens"])
    n = min(alone.size, inb.size)
    same = alone[:n] == inb[:n]
    first = int(np.argmin(same)) if not same.all() else None
    r.pop("prof", None)
    return dict(steps=int(n), identical=bool(same.all()), token_agreement=float(same.mean()),
                first_divergence=first, bs1=r)


def small_batches(wl, sizes, warmup, steps):
    """The fast step alone (mode off) on the first B rows of the batch."""
    out = {}
    ph = wl.phases[0]
    for B in sizes:
        sub = Workload(wl.name, wl.shape, wl.weights, wl.eng, wl.desc, B, wl.seq_len)
        sub.kv_snap = wl.kv_snap
        sub.phases = [dict(pt=ph["pt"][:B], tokens=ph["tokens"][:B], positions=ph["positions"][:B], join=[])]
        r = run_mode(sub, "off", warmup, steps, 0.0)
        out[str(B)] = dict(ms_per_step=r["ms_per_step"], tok_s=r["tok_s"], hbm_frac=r["hbm_frac"])
    return out


def cpu_baseline(wl, rows, steps):
    """The oracle (plain mode, as it stands) on host cores: `rows` rows x `steps` steps of the
    same workload, started from the GPU's cache of those rows at the start state."""
    from oracle import mgo
    shape, eng = wl.shape, wl.eng
    if wl.name == "longctx":
        tok = np.zeros(len(wl.pt_slots), np.int32)
        pos = np.zeros(len(wl.pt_slots), np.int32)
        join_rows(wl, wl.phases[0]["join"], tok, pos)
        act = wl.phases[0]["slots"]
        pt, last, p0 = wl.pt_slots[act], tok[act], pos[act]
    else:
        wl.start()
        ph = wl.phases[0]
        pt, last, p0 = ph["pt"], ph["tokens"], ph["positions"]
    rows = list(rows)
    sub = pt[rows]
    valid = sub >= 0
    n_pages = int(valid.sum())
    ptl = np.full(sub.shape, -1, np.int32)
    ptl[valid] = np.arange(n_pages, dtype=np.int32)
    om = mgo.OracleModel(shape, synth.weights_to_numpy(wl.weights), len(rows), sub.shape[1], n_pages)
    src = torch.as_tensor(sub[valid].astype(np.int64)).cuda()
    om.kv_view()[:] = eng.kv_view()[:, src].cpu().numpy().view(np.uint16)
    toks, poss = last[rows].copy(), p0[rows].copy()
    t0 = time.perf_counter()
    for _ in range(steps):
        lg = om.decode_step(mgo.PLAIN, toks, poss, ptl)
        toks, poss = lg.argmax(1).astype(np.int32), poss + 1
    dt = time.perf_counter() - t0
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return dict(value=len(rows) * steps / dt, unit="tok/s", cores=threads, kind="oracle",
                sample=f"{len(rows)} rows x {steps} decode step(s) of the same workload (plain mode, contexts "
                       f"{int(p0[rows].min())}..{int(p0[rows].max())}), {dt:.1f} s")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--config", choices=sorted(WORKLOADS), default="llama8b")
    ap.add_argument("--steps", type=int, default=256)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--batch", type=int, default=0, help="rows (0 = the workload's)")
    ap.add_argument("--prompt", type=int, default=0, help="prompt tokens (0 = the workload's)")
    ap.add_argument("--modes", default=None, help="default: off,gated,always (+ gated_mfma,always_mfma on llama8b)")
    ap.add_argument("--always-steps", type=int, default=0, help="timed steps of the always modes (0 = --steps)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=4)
    ap.add_argument("--cpu-steps", type=int, default=2)
    ap.add_argument("--tau", type=float, default=None)
    ap.add_argument("--pareto-steps", type=int, default=None,
                    help="steps of the tau calibration recipe (reference decode, eps_pert, sweep; default --steps, "
                         "0 = skip; llama8b only)")
    ap.add_argument("--profile-steps", type=int, default=32,
                    help="steps of the separate gated pass whose kernel launches are bracketed by HIP events "
                         "(0 = no pass)")
    ap.add_argument("--no-extras", action="store_true", help="skip the bs=1 leg and the small-batch sweep")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run the plain copy kernel on MIB MiB five times (HBM counter scaling) and exit")
    ap.add_argument("--read-calibration", type=int, default=0, metavar="MIB",
                    help="only run the streaming-read kernel over MIB MiB five times (the HBM read rate) and exit")
    ap.add_argument("--prefill", choices=("canonical", "fast"), default="canonical",
                    help="prompt prefill before the timed steps (llama8b; not timed)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported (rows are independent, so "
              "the path scales by data parallelism over requests with no exchange)", file=sys.stderr)
        sys.exit(2)
    torch.cuda.set_device(0)
    mg.load()
    if args.copy_calibration:
        nb = args.copy_calibration << 20
        src = torch.ones(nb // 4, dtype=torch.int32, device="cuda")
        dst = torch.empty_like(src)
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
        ev[0].record()
        for i in range(5):
            mg.op_copy(src, dst)
            ev[i + 1].record()
        torch.cuda.synchronize()
        ms = [ev[i].elapsed_time(ev[i + 1]) for i in range(5)]
        print(json.dumps(dict(copy_bytes=nb, launches=5, ms=ms, gbps_read_plus_write=2 * nb / (min(ms) * 1e-3) / 1e9)))
        return
    if args.read_calibration:
        nb = args.read_calibration << 20
        src = torch.ones(nb // 4, dtype=torch.int32, device="cuda")
        sink = torch.zeros(mg.read_stream_sink_words(), dtype=torch.int32, device="cuda")
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
        ev[0].record()
        for i in range(5):
            mg.op_read_stream(src, sink)
            ev[i + 1].record()
        torch.cuda.synchronize()
        ms = [ev[i].elapsed_time(ev[i + 1]) for i in range(5)]
        print(json.dumps(dict(read_bytes=nb, launches=5, ms=ms, gbps_read=nb / (min(ms) * 1e-3) / 1e9)))
        return
    cfg = args.config
    wl = WORKLOADS[cfg](args)
    modes_list = (args.modes or ("off,gated,always,gated_mfma,always_mfma" if cfg == "llama8b" else
                                 "off,gated,always")).split(",")
    always_steps = args.always_steps or args.steps
    # tau
    if args.tau is not None:
        tau = args.tau
    elif cfg == "llama8b":
        tau = calibrate_tau(wl, args.warmup + args.steps, PAPER_TRIGGER)
    elif cfg == "qwen14b":
        tau = calibrate_tau(wl, 16, 0.15)
    else:
        tau = wl.tau
    log(f"[bench] {cfg}: tau = {tau:.5f}")
    calib = None
    pareto_steps = (args.steps if args.pareto_steps is None else args.pareto_steps) if cfg == "llama8b" else 0
    if pareto_steps > 0:
        # the paper's threshold recipe (Sec. 3.1, Appendix A): eps_pert against the deterministic
        # reference, a sweep over 2 max(eps) x {1/8 .. 4}, tau_100
        ph = wl.phases[0]
        dec = GatedDecoder(wl.eng, ph["pt"], None, tau=tau)
        state = (ph["tokens"], ph["positions"])
        log(f"[bench] tau calibration recipe over {pareto_steps} steps")
        calib = calibrate.calibrate(dec, state, wl.kv_snap, pareto_steps)
        dec.tau = tau
        log(f"[bench] eps median {calib['eps_median']:.4f} max {calib['eps_max']:.4f}, tau_100 {calib['tau_100']}")
        # the repair actions of the commit at the benchmark's tau, against the same reference
        calib["repair_actions"] = calibrate.repair_actions(dec, state, wl.kv_snap, pareto_steps, tau,
                                                           reference=calib.pop("reference"), t_off=calib.pop("t_off"))
        log("[bench] repair actions: " + ", ".join(f"{k} seq_det {v['seq_det']:.3f} first div "
                                                     f"{v['first_divergence_mean']:.1f}"
                                                     for k, v in calib["repair_actions"]["actions"].items()))
        # the divergence diagnostics of Sec. 2 (Obs. 1-3) and the oracle-position repair
        div, ref = diagnostics.flip_study(dec, state, wl.kv_snap, pareto_steps, tau)
        div["oracle_repair"] = diagnostics.oracle_position_repair(dec, state, wl.kv_snap, pareto_steps, ref)
        calib["divergence"] = div
        log(f"[bench] flips: rate {div['flips']['rate']:.4f} ({div['flips']['events']} events), oracle-position "
            f"repairs/seq {div['oracle_repair']['repairs_per_sequence']:.2f}")
    modes = {}
    for mode in modes_list:
        steps = always_steps if mode.startswith("always") else args.steps
        log(f"[bench] mode {mode}: {args.warmup} warmup + {steps} timed steps")
        modes[mode] = run_mode(wl, mode, args.warmup, steps, tau)
        modes[mode].pop("prof", None)
        log(f"[bench] mode {mode}: {modes[mode]['ms_per_step']:.3f} ms/step, {modes[mode]['tok_s']:.0f} tok/s, "
            f"r_verify {modes[mode]['r_verify']:.4f}")
    # per-kernel HIP-event figures from a separate gated pass (the timed modes record none)
    kernels, roofline = {}, None
    if args.profile_steps > 0:
        kinds = (mg.KIND_FAST_GEMM, mg.KIND_CANON_GEMV, mg.KIND_FAST_ATTN, mg.KIND_CANON_ATTN)
        log(f"[bench] profiled gated pass: {args.profile_steps} steps with kernel events")
        pr = run_mode(wl, "gated", args.warmup, min(args.profile_steps, args.steps), tau, kinds, args.profile_steps)
        kernels = kernel_table(pr["prof"])
        roofline = roofline_of(kernels, f"{cfg}_b{wl.global_batch}" if cfg != "llama8b" else "llama8b_bs64")
    g = modes.get("gated") or next(iter(modes.values()))
    out = dict(metric=METRIC if cfg == "llama8b" else f"{METRIC} (workload {cfg})", value=g["tok_s"], unit="tok/s",
               n_gpus=1, steps=args.steps, warmup=args.warmup, ms_per_step=g["ms_per_step"], higher_is_better=True,
               scaling="weak", vs_baseline=None, dtype="bf16", data="synthetic",
               config=dict(workload=wl.desc, global_batch=wl.global_batch, seq_len=wl.seq_len,
                           parallelism="single GPU"),
               roofline=roofline, tau=tau, prefill_s=wl.prefill_s, modes=modes, kernels=kernels)
    if calib is not None:
        out["calibration"] = calib
        # sequence determinism of the method at the benchmark's tau (the on-mismatch action)
        out["seq_det_at_tau"] = calib["repair_actions"]["actions"]["on_mismatch"]["seq_det"]
    if "off" in modes:
        t_off = modes["off"]["ms_per_step"]
        ov = {}
        for m in ("gated", "always", "gated_mfma", "always_mfma"):
            if m in modes:
                ov[f"inc_{m}"] = modes[m]["ms_per_step"] / t_off - 1
        if "inc_gated" in ov and "inc_always" in ov and ov["inc_gated"] > 0:
            ov["cut"] = ov["inc_always"] / ov["inc_gated"]
        if "inc_gated_mfma" in ov and "inc_always_mfma" in ov and ov["inc_gated_mfma"] > 0:
            ov["cut_mfma"] = ov["inc_always_mfma"] / ov["inc_gated_mfma"]
        out["verifier_overhead"] = ov
        # HBM roofline fraction of the fast forward alone (off) and of the verifier alone (its
        # algorithmic bytes per step over the time a mode adds to off)
        rf = {"fast_forward": modes["off"]["hbm_frac"]}
        for m in ("gated", "always", "gated_mfma", "always_mfma"):
            if m in modes and modes[m]["ms_per_step"] > t_off:
                rf[f"verifier_{m}"] = (modes[m]["verifier_bytes_per_step"] / ((modes[m]["ms_per_step"] - t_off) * 1e-3)
                                       / HBM_PEAK)
        out["hbm_frac"] = rf
    if cfg == "llama8b" and not args.no_extras:
        log("[bench] protected row alone (bs=1) vs inside the batch")
        out["bs1"] = bs1_leg(wl, args.warmup, args.steps, tau)
        log(f"[bench] bs=1: identical {out['bs1']['identical']}, first divergence "
            f"{out['bs1']['first_divergence']}, {out['bs1']['bs1']['ms_per_step']:.3f} ms/step")
        log("[bench] fast step at small batches")
        sb = small_batches(wl, (1, 8, 16, 32), args.warmup, min(args.steps, 32))
        if "off" in modes:
            sb[str(wl.global_batch)] = dict(ms_per_step=modes["off"]["ms_per_step"], tok_s=modes["off"]["tok_s"],
                                            hbm_frac=modes["off"]["hbm_frac"])
        out["fast_small_batch"] = sb
    if not args.no_cpu_baseline:
        log("[bench] cpu baseline (oracle)")
        rows = min(args.cpu_rows, wl.global_batch if cfg != "longctx" else 2)
        steps = args.cpu_steps if cfg != "longctx" else 1
        out["cpu_baseline"] = cpu_baseline(wl, np.arange(rows), steps)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
