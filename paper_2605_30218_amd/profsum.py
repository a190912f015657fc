"""Summaries of rocprofv3 output for profiles/: kernel-trace statistics and HBM traffic.

    python -m paper_2605_30218_amd.profsum trace <kernel_trace.csv> <out.txt> "<command>" [modes]
    python -m paper_2605_30218_amd.profsum traffic <kernel> <fetch_csv> <write_csv> <copy_fetch_csv> \
        <copy_write_csv> <copy_bytes> <out.txt> "<command>" "<copy command>"
    python -m paper_2605_30218_amd.profsum util <counter_collection.csv> <out.txt> "<command>" <k1,k2,..>
    python -m paper_2605_30218_amd.profsum shapes <csv1,csv2,..> <out.txt> "<command>" <k1,k2,..>

Both summaries cover the decode window only: the dispatches from the first fast-path
residual/RMSNorm kernel on (the canonical prompt prefill before it uses other kernels).
The benchmark restores the KV cache from its snapshot (one copy of more than 1 ms) before
each mode, so the trace summary also splits the window at those copies into the tau
calibration steps, the runs of the threshold recipe, and the modes named by [modes]
(comma separated, benchmark order; they are the last windows).
The traffic summary scales FETCH_SIZE and WRITE_SIZE (KiB per dispatch) by what each
counter reads for a plain copy kernel of known size, and records the sha256 of the
kernel's source file so that a later change of the kernel makes the figure stale.
"""
from __future__ import annotations

import collections
import csv
import hashlib
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
# kernel name prefix -> source files (bench names: fast_gemm, canon_gemv; the canonical GEMV
# has a vector-fma kernel and a matrix-core kernel, canon_gemv_kernel and canon_gemv_mfma_kernel)
SOURCES = {"fast_gemm": ("k_gemm.hip",), "canon_gemv": ("k_gemv.hip", "k_gemv_mfma.hip")}
DECODE_START = "resid_norm_kernel"


def source_sha(kernel: str) -> str:
    h = hashlib.sha256()
    for f in SOURCES[kernel]:
        h.update(open(os.path.join(HERE, "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def _decode_window(rows, key):
    rows.sort(key=lambda r: int(r[key]))
    for i, r in enumerate(rows):
        if DECODE_START in r["Kernel_Name"]:
            return rows[i:]
    return rows


def _short(name: str) -> str:
    n = name.split("(")[0]
    return n.replace("void ", "").replace("mg::", "")


MODE_KERNELS = ("fast_gemm_kernel", "canon_gemv", "attn_fast_fused_kernel", "attn_canon_kernel")


def _mode_tables(rows, modes):
    cuts = [i for i, r in enumerate(rows) if "copyBuffer" in r["Kernel_Name"]
            and int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) > 1_000_000]
    bounds = [0] + cuts + [len(rows)]
    # windows that run decode steps (copies after the last mode, e.g. for the CPU baseline,
    # leave windows without any); the modes are the last of them, before them the quantile
    # tau calibration and the runs of the threshold recipe (reference decode, fast run, one
    # run per tau)
    segs = [rows[bounds[w]:bounds[w + 1]] for w in range(len(bounds) - 1)]
    segs = [seg for seg in segs if any(MODE_KERNELS[0] in r["Kernel_Name"] for r in seg)]
    nrec = max(0, len(segs) - 1 - len(modes))
    names = ["tau calibration"] + [f"recipe run {k}" for k in range(1, nrec + 1)] + modes
    lines = ["", "per mode (windows split at the KV snapshot restores; warmup steps included):",
             f"{'mode':16s} {'kernel':22s} {'calls':>7s} {'avg_us':>9s} {'total_ms':>9s}"]
    for w in range(min(len(names), len(segs))):
        seg = segs[w]
        for kn in MODE_KERNELS:
            d = [int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in seg if kn in r["Kernel_Name"]]
            if d:
                lines.append(f"{names[w]:16s} {kn:22s} {len(d):7d} {sum(d) / len(d) / 1e3:9.1f} {sum(d) / 1e6:9.2f}")
    return lines


def trace(trace_csv: str, out: str, command: str, modes: str = "") -> None:
    rows = _decode_window(list(csv.DictReader(open(trace_csv))), "Start_Timestamp")
    by = collections.defaultdict(list)
    shape = collections.defaultdict(list)
    for r in rows:
        d = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
        by[_short(r["Kernel_Name"])].append(d)
        grid = (r["Grid_Size_X"], r["Grid_Size_Y"], r["Grid_Size_Z"])
        shape[(_short(r["Kernel_Name"]), grid)].append(d)
    tot = sum(sum(v) for v in by.values())
    lines = [f"command: {command}", "window: decode steps (from the first fast-path resid_norm dispatch)",
             f"dispatches: {len(rows)}  total kernel time: {tot / 1e6:.2f} ms", "",
             f"{'kernel':60s} {'calls':>7s} {'avg_us':>9s} {'total_ms':>9s} {'pct':>6s}"]
    for k, v in sorted(by.items(), key=lambda kv: -sum(kv[1]))[:24]:
        lines.append(f"{k[:60]:60s} {len(v):7d} {sum(v) / len(v) / 1e3:9.1f} {sum(v) / 1e6:9.2f} "
                     f"{100 * sum(v) / tot:6.1f}")
    lines += ["", "per launch shape (grid x,y,z in threads) of the weight-streaming kernels:",
              f"{'kernel':44s} {'grid':>22s} {'calls':>7s} {'avg_us':>9s}"]
    for (k, g), v in sorted(shape.items(), key=lambda kv: -sum(kv[1])):
        if "fast_gemm" in k or "canon_gemv" in k:
            lines.append(f"{k[:44]:44s} {','.join(g):>22s} {len(v):7d} {sum(v) / len(v) / 1e3:9.1f}")
    lines.append("")
    for kn in SOURCES:
        fg = [d for k, v in by.items() if k.startswith(kn) for d in v]
        if fg:
            lines.append(f"{kn} kernels, all shapes: {len(fg)} launches, average {sum(fg) / len(fg) / 1e3:.1f} us")
    if modes:
        lines += _mode_tables(rows, modes.split(","))
    open(out, "w").write("\n".join(lines) + "\n")


def _per_dispatch(path: str, filt: str, window: bool = True):
    out = collections.defaultdict(list)
    rows = list(csv.DictReader(open(path)))
    rows = _decode_window(rows, "Dispatch_Id") if window else rows
    for r in rows:
        if filt in r["Kernel_Name"]:
            out[int(r["Grid_Size"])].append(float(r["Counter_Value"]) * 1024.0)
    return out


def traffic(kernel, fetch_csv, write_csv, copy_fetch_csv, copy_write_csv, copy_bytes, out, command, copy_command):
    copy_bytes = float(copy_bytes)
    cf = [v for vs in _per_dispatch(copy_fetch_csv, "copy16", False).values() for v in vs]
    cw = [v for vs in _per_dispatch(copy_write_csv, "copy16", False).values() for v in vs]
    f_scale = copy_bytes / (sum(cf[1:]) / len(cf[1:]) if len(cf) > 1 else cf[0])
    w_scale = copy_bytes / (sum(cw[1:]) / len(cw[1:]) if len(cw) > 1 else cw[0])
    fe = _per_dispatch(fetch_csv, kernel)
    wr = _per_dispatch(write_csv, kernel)
    lines = [f"kernel: {kernel} kernels (decode window)", f"command (FETCH_SIZE, then WRITE_SIZE): {command}",
             f"copy calibration: {copy_command}",
             f"copy kernel reads and writes {copy_bytes / 2**20:.0f} MiB: FETCH_SIZE scale {f_scale:.4f}, "
             f"WRITE_SIZE scale {w_scale:.4f}",
             f"source sha256[:16]: {source_sha(kernel)}", "",
             f"{'grid(threads)':>14s} {'launches':>9s} {'fetch_MB':>10s} {'write_MB':>10s}"]
    tot_b, tot_n = 0.0, 0
    for g in sorted(fe):
        f = sum(fe[g]) / len(fe[g]) * f_scale
        w = sum(wr.get(g, [0.0])) / max(len(wr.get(g, [])), 1) * w_scale
        lines.append(f"{g:14d} {len(fe[g]):9d} {f / 1e6:10.2f} {w / 1e6:10.2f}")
        tot_b += (f + w) * len(fe[g])
        tot_n += len(fe[g])
    lines += ["", f"traffic_bytes_per_launch: {tot_b / max(tot_n, 1):.0f}"]
    open(out, "w").write("\n".join(lines) + "\n")


def util(pmc_csv: str, out: str, command: str, kernels: str) -> None:
    """Mean of each collected counter (derived percentages such as MfmaUtil and VALUBusy)
    over the decode-window dispatches of each named kernel."""
    rows = _decode_window(list(csv.DictReader(open(pmc_csv))), "Dispatch_Id")
    agg = collections.defaultdict(lambda: collections.defaultdict(list))
    names = kernels.split(",")
    for r in rows:
        for k in names:
            if k in r["Kernel_Name"]:
                agg[k][r["Counter_Name"]].append(float(r["Counter_Value"]))
    counters = sorted({c for k in agg for c in agg[k]})
    lines = [f"command: {command}", "window: decode steps; mean over each kernel's dispatches", "",
             f"{'kernel':26s} {'dispatches':>10s} " + " ".join(f"{c:>12s}" for c in counters)]
    for k in names:
        if k in agg:
            n = max(len(v) for v in agg[k].values())
            lines.append(f"{k:26s} {n:10d} " + " ".join(
                f"{sum(agg[k][c]) / len(agg[k][c]):12.2f}" if agg[k][c] else f"{'-':>12s}" for c in counters))
    open(out, "w").write("\n".join(lines) + "\n")


def shapes(pmc_csvs: str, out: str, command: str, kernels: str) -> None:
    """Per launch shape (kernel instance and grid) of the named kernels: dispatches, mean
    duration and the mean of each SQ counter per dispatch (counter passes in separate CSVs),
    with the ratios that name a stall: the share of wave time waiting to issue (WAIT_INST_ANY),
    issuing VALU, LDS and vector memory instructions (ACTIVE_INST_*), LDS bank-conflict cycles
    per LDS instruction, and the matrix-core busy share of the launch's SIMD-cycles (256 CUs x
    4 SIMDs at 2.4 GHz)."""
    names = kernels.split(",")
    cnt = collections.defaultdict(lambda: collections.defaultdict(list))
    dur = collections.defaultdict(list)
    for path in pmc_csvs.split(","):
        rows = _decode_window(list(csv.DictReader(open(path))), "Dispatch_Id")
        seen = set()
        for r in rows:
            kn = r["Kernel_Name"]
            if not any(k in kn for k in names):
                continue
            key = (kn.replace("void ", "").replace("mg::", "").split("(")[0], int(r["Grid_Size"]))
            cnt[key][r["Counter_Name"]].append(float(r["Counter_Value"]))
            did = (path, r["Dispatch_Id"])
            if did not in seen:
                seen.add(did)
                dur[key].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1000.0)

    def mean(key, c):
        v = cnt[key].get(c)
        return sum(v) / len(v) if v else float("nan")

    lines = [f"command: {command}", "window: decode steps; per launch shape, mean over its dispatches",
             "ratios: wait, valu, lds, vmem = share of wave-cycles (SQ_WAVE_CYCLES) waiting to issue / issuing "
             "VALU / LDS / vector-memory instructions; conf = SQ_LDS_BANK_CONFLICT per SQ_INSTS_LDS; "
             "mfma = SQ_VALU_MFMA_BUSY_CYCLES over the launch's SIMD-cycles", "",
             f"{'kernel':58s} {'grid':>9s} {'n':>5s} {'us':>7s} {'wait':>6s} {'valu':>6s} {'lds':>6s} "
             f"{'vmem':>6s} {'conf':>6s} {'mfma':>6s}"]
    for key in sorted(cnt, key=lambda k: -sum(dur[k])):
        wc = mean(key, "SQ_WAVE_CYCLES")
        us = sum(dur[key]) / max(len(dur[key]), 1)
        ratio = lambda c: mean(key, c) / wc if wc == wc and wc > 0 else float("nan")
        conf = mean(key, "SQ_LDS_BANK_CONFLICT") / mean(key, "SQ_INSTS_LDS") if mean(key, "SQ_INSTS_LDS") else float("nan")
        mfma = mean(key, "SQ_VALU_MFMA_BUSY_CYCLES") / (us * 1e-6 * 2.4e9 * 1024) if us > 0 else float("nan")
        lines.append(f"{key[0][:58]:58s} {key[1]:9d} {len(dur[key]) // max(len(pmc_csvs.split(',')), 1):5d} {us:7.1f} "
                     f"{ratio('SQ_WAIT_INST_ANY'):6.2f} {ratio('SQ_ACTIVE_INST_VALU'):6.2f} "
                     f"{ratio('SQ_ACTIVE_INST_LDS'):6.2f} {ratio('SQ_ACTIVE_INST_VMEM'):6.2f} {conf:6.2f} {mfma:6.2f}")
    open(out, "w").write("\n".join(lines) + "\n")


def read_traffic(path: str):
    """(bytes per launch, source sha) from a traffic summary, or None."""
    if not os.path.exists(path):
        return None
    sha = per = None
    for line in open(path):
        if line.startswith("source sha256[:16]:"):
            sha = line[len("source sha256[:16]:"):].strip()
        if line.startswith("traffic_bytes_per_launch:"):
            per = float(line[len("traffic_bytes_per_launch:"):])
    return (per, sha) if per is not None and sha else None


if __name__ == "__main__":
    if sys.argv[1] == "trace":
        trace(*sys.argv[2:6])
    elif sys.argv[1] == "traffic":
        traffic(*sys.argv[2:11])
    elif sys.argv[1] == "util":
        util(*sys.argv[2:6])
    elif sys.argv[1] == "shapes":
        shapes(*sys.argv[2:6])
    else:
        raise SystemExit(__doc__)
