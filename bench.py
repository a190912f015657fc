"""Benchmark of the MarginGate decode step on one MI355X.

Workload: a Llama-3.1-8B-shaped decoder (32 layers, d 4096, 32/8 heads, hd 128, FFN 14336,
vocab 128256, RoPE theta 5e5) with random-init N(0, 0.02) bf16 weights, batch 64, uniform
random 512-token prompts (canonical prefill, not timed), greedy decode.  Every row is
protected.  Three modes run from the same prefilled state:
  off     the BF16 fast path only (r_verify = 0)
  gated   MarginGate: verify rows whose top-1/top-2 margin is below tau
  always  the verifier on every row and step (the always-on baseline, r_verify = 1)
  gated_mfma, always_mfma  the same with the matrix-core verifier (fixed tiling,
          batch-invariant, tolerance parity) instead of the canonical one
tau is calibrated on the fast-path margins of an untimed run of the same length so that
the trigger rate matches the paper's Llama-3.1-8B operating point (18.56%); the measured
rate is reported.

One JSON line on stdout: value = gated decode tokens/s (B * steps / time of the timed
steps, inputs resident in HBM), plus the other modes, the verifier overhead
(inc_mode = T_mode / T_off - 1, cut = inc_always / inc_gated), the roofline of the
dominant kernel measured with HIP events over the timed region, the HBM roofline fraction
of each mode and of the fast forward and the verifier alone (algorithmic bytes: every
streamed weight once per forward, the live K/V of the rows involved, the fp32 logits), the
histogram of verified rows per step, and the CPU oracle baseline on a bounded sample.
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
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "{kernel}_traffic_llama8b_bs64.txt")


def attn_bytes(shape, rows, ctx):
    """Algorithmic HBM bytes of one layer's decode attention: K and V of `ctx` positions
    per row and KV head, the rotated query in and the attention output out."""
    kv = ctx * shape.n_kv_heads * shape.head_dim * 2 * 2
    qo = 2 * shape.n_q_heads * shape.head_dim * 2
    return rows * (kv + qo)


def streamed_weight_bytes(shape):
    """bf16 bytes of every weight a forward streams (the embedding is gathered, not streamed)."""
    return 2 * (shape.n_params() - shape.vocab * shape.d_model)


def forward_bytes(shape, rows, ctx):
    """Algorithmic HBM bytes of one forward over `rows` rows at context `ctx`: every streamed
    weight once, each layer's attention bytes, the fp32 logits written."""
    return streamed_weight_bytes(shape) + shape.n_layers * attn_bytes(shape, rows, ctx) + rows * shape.vocab * 4


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def run_mode(dec, mode, warmup, steps, state, kv_snap, eng, profile_kinds=(), profile_steps=32):
    # "<mode>_mfma": the same mode with the matrix-core verifier
    mode, _, ver = mode.partition("_")
    dec.verifier = "mfma" if ver == "mfma" else "canonical"
    eng.kv_pool.copy_(kv_snap)
    dec.set_state(*state)
    dec.n_repaired.zero_()
    for _ in range(warmup):
        dec.step(mode)
    torch.cuda.synchronize()
    dec.protected_row_steps = dec.verified_row_steps = 0
    dec.hist = []
    dec.n_repaired.zero_()
    prof_steps = min(steps, profile_steps)
    ctx0 = int(dec.positions.max().item()) + 1     # positions attended at the first timed step
    L = eng.shape.n_layers
    per_step = {mg.KIND_FAST_GEMM: 4 * L + 1, mg.KIND_CANON_GEMV: 4 * L + 1, mg.KIND_FAST_ATTN: L,
                mg.KIND_CANON_ATTN: L}
    for k in profile_kinds:
        eng.profile_begin(k, prof_steps * per_step[k])
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev[0].record()
    for s in range(steps):
        dec.step(mode)
        ev[s + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = np.array([ev[s].elapsed_time(ev[s + 1]) for s in range(steps)])
    prof = {k: eng.profile_end(k) for k in profile_kinds}
    B = dec.B
    # attention bytes are not known to the library (positions live on the device); every row
    # of this workload has the same position, so they follow from the step index.  A kind
    # records the launches of its first prof_steps steps that ran it (the verifier runs only
    # on steps with gated rows).
    for k, rows in ((mg.KIND_FAST_ATTN, [B] * steps), (mg.KIND_CANON_ATTN, dec.hist)):
        if k in prof:
            n, ms, b, f = prof[k]
            ran = [(s, r) for s, r in enumerate(rows) if r][:n // L]
            b = sum(L * attn_bytes(eng.shape, r, ctx0 + s) for s, r in ran)
            prof[k] = (n, ms, float(b), f)
    # algorithmic bytes of the timed steps: the fast forward of all rows, and the verifier's
    # forward of its rows on the steps that ran it (the weights are streamed again)
    fast_b = sum(forward_bytes(eng.shape, B, ctx0 + s) for s in range(steps))
    ver_b = sum(forward_bytes(eng.shape, r, ctx0 + s) for s, r in enumerate(dec.hist) if r)
    return dict(ms_per_step=wall * 1e3 / steps, tok_s=B * steps / wall, p50_ms=float(np.median(per)),
                p99_ms=float(np.percentile(per, 99)), r_verify=dec.r_verify, r_repair=dec.r_repair(),
                verified_rows_per_step=float(np.mean(dec.hist)),
                verified_rows_hist=np.bincount(np.asarray(dec.hist, dtype=np.int64), minlength=1).tolist(),
                fast_bytes_per_step=fast_b / steps, verifier_bytes_per_step=ver_b / steps,
                hbm_frac=(fast_b + ver_b) / wall / HBM_PEAK, prof=prof)


def calibrate_tau(dec, eng, state, kv_snap, steps, rate):
    eng.kv_pool.copy_(kv_snap)
    dec.set_state(*state)
    ms = []
    for _ in range(steps):
        dec.step("off")
        ms.append(dec.margin.cpu().numpy().copy())
    return float(np.quantile(np.concatenate(ms), rate))


def cpu_baseline(shape, weights, eng, pt, state, rows, steps):
    """The oracle (plain mode, as it stands) on host cores: `rows` rows x `steps` steps of the
    same workload, started from the GPU's prefilled cache of those rows."""
    from oracle import mgo
    last, pos = state
    wn = synth.weights_to_numpy(weights)
    maxp = pt.shape[1]
    n_pages = len(rows) * maxp
    om = mgo.OracleModel(shape, wn, len(rows), maxp, n_pages)
    kv = eng.kv_view()
    src_pages = torch.as_tensor(pt[rows].reshape(-1).astype(np.int64)).cuda()
    om.kv_view()[:] = kv[:, src_pages].cpu().numpy().view(np.uint16)
    ptl = np.arange(n_pages, dtype=np.int32).reshape(len(rows), maxp)
    toks, poss = last[rows].copy(), pos[rows].copy()
    t0 = time.perf_counter()
    for _ in range(steps):
        lg = om.decode_step(mgo.PLAIN, toks, poss, ptl)
        toks, poss = lg.argmax(1).astype(np.int32), poss + 1
    dt = time.perf_counter() - t0
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return dict(value=len(rows) * steps / dt, unit="tok/s", cores=threads, kind="oracle",
                sample=f"{len(rows)} rows x {steps} decode step(s) of the same workload (plain mode, context "
                       f"{int(pos[rows].min())}+), {dt:.1f} s")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=256)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--batch", type=int, default=64)
    ap.add_argument("--prompt", type=int, default=512)
    ap.add_argument("--modes", default="off,gated,always,gated_mfma,always_mfma")
    ap.add_argument("--always-steps", type=int, default=0, help="timed steps of the always mode (0 = --steps)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=4)
    ap.add_argument("--cpu-steps", type=int, default=2)
    ap.add_argument("--tau", type=float, default=None)
    ap.add_argument("--pareto-steps", type=int, default=None,
                    help="steps of the tau calibration recipe (reference decode, eps_pert, sweep; default --steps, "
                         "0 = skip)")
    ap.add_argument("--profile-steps", type=int, default=32,
                    help="timed gated steps (from the first) whose kernel launches are bracketed by HIP events")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run the plain copy kernel on MIB MiB five times (HBM counter scaling) and exit")
    ap.add_argument("--prefill", choices=("canonical", "fast"), default="canonical",
                    help="prompt prefill before the timed steps (not timed)")
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
    shape = synth.LLAMA8B
    B, P = args.batch, args.prompt
    always_steps = args.always_steps or args.steps
    ctx_cap = P + args.warmup + max(args.steps, always_steps) + 16
    maxp = -(-ctx_cap // shape.page_size)
    pt, n_pages = synth.make_page_table([ctx_cap] * B, shape.page_size, maxp, seed=5)
    log(f"[bench] weights {shape.name} on GPU (seed 0)")
    weights = synth.make_weights(shape, seed=0, device="cuda")
    eng = mg.Engine(shape, weights, B, maxp, n_pages, max_prefill=1024)
    prompts = synth.make_prompts(B, [P] * B, shape.vocab, seed=1)
    log(f"[bench] {args.prefill} prefill {B} x {P - 1} tokens")
    t0 = time.perf_counter()
    last, pos0 = (prefill_rows if args.prefill == "canonical" else prefill_fast)(eng, prompts, pt)
    prefill_s = time.perf_counter() - t0
    log(f"[bench] prefill {prefill_s:.1f} s")
    kv_snap = eng.kv_pool.clone()
    state = (last, pos0)
    dec = GatedDecoder(eng, pt, None, tau=0.0)
    # tau: the 18.56% quantile of the fast-path margins over as many steps as a timed run
    tau = args.tau if args.tau is not None else calibrate_tau(dec, eng, state, kv_snap, args.warmup + args.steps,
                                                              PAPER_TRIGGER)
    dec.tau = tau
    log(f"[bench] tau = {tau:.5f}")
    # the paper's threshold recipe (Sec. 3.1, Appendix A): eps_pert against the deterministic
    # reference, a sweep over 2 max(eps) x {1/8 .. 4}, tau_100
    pareto_steps = args.steps if args.pareto_steps is None else args.pareto_steps
    calib = None
    if pareto_steps > 0:
        log(f"[bench] tau calibration recipe over {pareto_steps} steps")
        calib = calibrate.calibrate(dec, state, kv_snap, pareto_steps)
        dec.tau = tau
        log(f"[bench] eps median {calib['eps_median']:.4f} max {calib['eps_max']:.4f}, tau_100 {calib['tau_100']}")
        # the repair actions of the commit at the benchmark's tau, against the same reference
        calib["repair_actions"] = calibrate.repair_actions(dec, state, kv_snap, pareto_steps, tau,
                                                           reference=calib.pop("reference"), t_off=calib.pop("t_off"))
        log("[bench] repair actions: " + ", ".join(f"{k} seq_det {v['seq_det']:.3f} first div {v['first_divergence_mean']:.1f}"
                                                     for k, v in calib["repair_actions"]["actions"].items()))
        # the divergence diagnostics of Sec. 2 (Obs. 1-3) and the oracle-position repair
        div, ref = diagnostics.flip_study(dec, state, kv_snap, pareto_steps, tau)
        div["oracle_repair"] = diagnostics.oracle_position_repair(dec, state, kv_snap, pareto_steps, ref)
        calib["divergence"] = div
        log(f"[bench] flips: rate {div['flips']['rate']:.4f} ({div['flips']['events']} events), K spike "
            f"{div['kv']['k_spike']}, oracle-position repairs/seq {div['oracle_repair']['repairs_per_sequence']:.2f} "
            f"seq_det {div['oracle_repair']['seq_det']:.3f}")
    modes = {}
    for mode in args.modes.split(","):
        steps = always_steps if mode.startswith("always") else args.steps
        kinds = (mg.KIND_FAST_GEMM, mg.KIND_CANON_GEMV, mg.KIND_FAST_ATTN, mg.KIND_CANON_ATTN) \
            if mode == "gated" and args.profile_steps > 0 else ()
        log(f"[bench] mode {mode}: {args.warmup} warmup + {steps} timed steps")
        modes[mode] = run_mode(dec, mode, args.warmup, steps, state, kv_snap, eng, kinds, args.profile_steps)
        log(f"[bench] mode {mode}: {modes[mode]['ms_per_step']:.3f} ms/step, {modes[mode]['tok_s']:.0f} tok/s, "
            f"r_verify {modes[mode]['r_verify']:.4f}")
    dec.verifier = "canonical"
    g = modes.get("gated") or next(iter(modes.values()))
    prof = g.pop("prof")
    for m in modes.values():
        m.pop("prof", None)
    # roofline of the dominant kernel of the gated step
    names = {mg.KIND_FAST_GEMM: "fast_gemm", mg.KIND_CANON_GEMV: "canon_gemv", mg.KIND_FAST_ATTN: "fast_attention",
             mg.KIND_CANON_ATTN: "canon_attention"}
    kernels = {}
    for k, (n, ms, b, f) in prof.items():
        kernels[names[k]] = dict(launches=n, total_ms=ms, avg_us=1e3 * ms / max(n, 1), algo_bytes=b, algo_flops=f,
                                 gbps=b / (ms * 1e-3) / 1e9 if ms > 0 else 0.0,
                                 tflops=f / (ms * 1e-3) / 1e12 if ms > 0 else 0.0)
    roofline = None
    if kernels:
        dom = max(kernels, key=lambda k: kernels[k]["total_ms"])
        kd = kernels[dom]
        sec = kd["total_ms"] * 1e-3
        hbm = kd["algo_bytes"] / sec
        alu = kd["algo_flops"] / sec
        # HBM bytes per launch from the committed FETCH_SIZE / WRITE_SIZE summary, if it was
        # taken on the kernel's current source
        traffic = None
        if dom in profsum.SOURCES:
            t = profsum.read_traffic(TRAFFIC_SUMMARY.format(kernel=dom))
            if t and t[1] == profsum.source_sha(dom):
                traffic = t[0]
        common = dict(kernel=dom, traffic=traffic, traffic_unit="bytes/launch", launches=kd["launches"],
                      algo_bytes_per_launch=kd["algo_bytes"] / max(kd["launches"], 1), avg_us=kd["avg_us"])
        # the bound follows the arithmetic intensity of the launches against the ridge point
        if dom == "canon_gemv" and kd["algo_flops"] / kd["algo_bytes"] > FP32_VECTOR_PEAK / HBM_PEAK:
            roofline = dict(bound="alu", achieved=alu / 1e12, peak=FP32_VECTOR_PEAK / 1e12, unit="TFLOP/s",
                            frac=alu / FP32_VECTOR_PEAK, **common)
        else:
            roofline = dict(bound="hbm", achieved=hbm / 1e9, peak=HBM_PEAK / 1e9, unit="GB/s",
                            frac=hbm / HBM_PEAK, **common)
    out = dict(metric=METRIC, value=g["tok_s"], unit="tok/s", n_gpus=1, steps=args.steps, warmup=args.warmup,
               ms_per_step=g["ms_per_step"], higher_is_better=True, scaling="weak", vs_baseline=None, dtype="bf16",
               data="synthetic",
               config=dict(workload=f"Llama-3.1-8B-shaped random-init decoder, batch {B}, uniform random {P}-token "
                                    f"prompts, gated greedy decode (all rows protected, tau for an 18.56% trigger)",
                           global_batch=B, seq_len=P, parallelism="single GPU"),
               roofline=roofline, tau=tau, prefill=args.prefill, prefill_s=prefill_s, modes=modes, kernels=kernels)
    if calib is not None:
        out["calibration"] = calib
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
                rf[f"verifier_{m}"] = modes[m]["verifier_bytes_per_step"] / ((modes[m]["ms_per_step"] - t_off) * 1e-3) / HBM_PEAK
        out["hbm_frac"] = rf
    if not args.no_cpu_baseline:
        log("[bench] cpu baseline (oracle)")
        eng.kv_pool.copy_(kv_snap)
        out["cpu_baseline"] = cpu_baseline(shape, weights, eng, pt, state, np.arange(args.cpu_rows), args.cpu_steps)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
