"""Host-side logic that is neither oracle nor kernel: the calibration recipe's statistics."""
import numpy as np
import pytest


def test_eps_pert_takes_the_reference_top50():
    """Host logic of the calibration recipe (Appendix A): eps is the l-infinity gap over the
    reference's top-50 entries only."""
    from paper_2605_30218_amd import calibrate
    ref = np.arange(100, dtype=np.float32)[None, :].repeat(2, 0)
    fast = ref.copy()
    fast[0, 10] += 5.0    # outside the top 50 (indices 50..99): ignored
    fast[0, 60] -= 0.25   # inside
    fast[1, 99] += 0.5
    np.testing.assert_allclose(calibrate.eps_pert(fast, ref), [0.25, 0.5])


def test_traffic_summary_round_trip(tmp_path):
    """The benchmark takes a kernel's HBM traffic from its committed summary only while the
    summary's recorded source hash matches the kernel's current source."""
    from paper_2605_30218_amd import profsum
    sha = profsum.source_sha("canon_gemv")
    p = tmp_path / "t.txt"
    p.write_text(f"kernel: canon_gemv_kernel\nsource sha256[:16]: {sha}\n\ntraffic_bytes_per_launch: 123456\n")
    assert profsum.read_traffic(str(p)) == (123456.0, sha)


def test_trace_mode_windows_are_named_from_the_last_decode_windows():
    """The kernel-trace summary splits the decode window at the long KV-restore copies; the
    modes are the last windows that run decode kernels (a restore after the last mode that
    runs none, like the CPU baseline's, is skipped).  The canonical GEMV's two kernels count
    as one kind."""
    from paper_2605_30218_amd import profsum
    t = [0]

    def row(name, dur=10):
        t[0] += 100
        return {"Kernel_Name": name, "Start_Timestamp": str(t[0]), "End_Timestamp": str(t[0] + dur)}

    def restore():
        return row("__amd_rocclr_copyBuffer", 2_000_000)

    rows = [row("resid_norm_kernel"), row("fast_gemm_kernel")]            # tau calibration
    rows += [restore(), row("canon_gemv_kernel"), row("fast_gemm_kernel")]  # recipe run 1
    rows += [restore(), row("fast_gemm_kernel")]                           # off
    rows += [restore(), row("fast_gemm_kernel"), row("canon_gemv_kernel", 30_000),
             row("canon_gemv_mfma_kernel", 50_000)]                       # gated
    rows += [restore(), row("fast_gemm_kernel"), row("canon_gemv_kernel", 70_000)]  # always
    rows += [restore(), row("copy_to_host")]                               # no decode kernels
    lines = profsum._mode_tables(rows, ["off", "gated", "always"])
    got = {(ln[:16].strip(), ln[17:39].strip()): float(ln.split()[-2]) for ln in lines[3:]}
    assert got[("gated", "canon_gemv")] == 40.0
    assert got[("always", "canon_gemv")] == 70.0
    assert ("off", "canon_gemv") not in got
    assert ("recipe run 1", "canon_gemv") in got


def test_forward_bytes_of_the_llama8b_shape():
    """The benchmark's algorithmic bytes: 7.505 B streamed parameters (embedding gathered, not
    streamed) and 128 KiB of K/V per token over all layers on the Llama-3.1-8B shape."""
    import bench
    from paper_2605_30218_amd import synth
    s = synth.LLAMA8B
    assert abs(bench.streamed_weight_bytes(s) / 2 - 7.505e9) < 0.001e9
    one = bench.forward_bytes(s, [1000]) - bench.forward_bytes(s, [999])
    assert one == 128 * 1024
    assert bench.forward_bytes(s, [10, 10]) - bench.forward_bytes(s, [10]) == \
        s.n_layers * bench.attn_bytes(s, [10]) + s.vocab * 4
    # ragged rows: the K/V bytes follow each row's own context
    assert bench.forward_bytes(s, [100, 300]) == bench.forward_bytes(s, [200, 200])
    assert bench.forward_bytes(s, []) == 0.0


def test_util_summary_means_per_kernel(tmp_path):
    """The counter-utilisation summary averages each counter over a kernel's dispatches in
    the decode window (dispatches before the first fast-path RMSNorm are prefill)."""
    from paper_2605_30218_amd import profsum
    p = tmp_path / "c.csv"
    rows = [("1", "prefill_kernel", "MfmaUtil", "99"), ("2", "resid_norm_kernel", "MfmaUtil", "0"),
            ("3", "fast_gemm_kernel<4>", "MfmaUtil", "10"), ("4", "fast_gemm_kernel<4>", "MfmaUtil", "30"),
            ("3", "fast_gemm_kernel<4>", "VALUBusy", "5"), ("5", "canon_gemv_kernel<2>", "VALUBusy", "80")]
    p.write_text("Dispatch_Id,Kernel_Name,Counter_Name,Counter_Value\n" + "".join(",".join(r) + "\n" for r in rows))
    out = tmp_path / "o.txt"
    profsum.util(str(p), str(out), "cmd", "fast_gemm_kernel,canon_gemv_kernel")
    lines = out.read_text().splitlines()
    fg = [ln for ln in lines if ln.startswith("fast_gemm_kernel")][0].split()
    assert fg[1] == "2" and float(fg[2]) == 20.0 and float(fg[3]) == 5.0
    cg = [ln for ln in lines if ln.startswith("canon_gemv_kernel")][0].split()
    assert cg[2] == "-" and float(cg[3]) == 80.0


def test_divergence_statistics():
    """Obs. 1-3 statistics (Sec. 2): events over synchronous samples, the K/V deviation aligned
    at the first divergent cache step (first divergent token + 1), the reference token's rank
    and the margin at each event."""
    from paper_2605_30218_amd import diagnostics
    steps = 10
    ref = np.arange(30, dtype=np.int32).reshape(3, steps)
    toks = ref.copy()
    toks[1, 4] += 1          # row 1 diverges at step 4
    toks[2, 0] += 1          # row 2 at step 0 (too early for the K/V window)
    margins = np.full((3, steps), 0.5, np.float32)
    margins[1, 4], margins[2, 0] = 0.01, 0.2
    ranks = np.zeros((3, steps), np.int64)
    ranks[1, 4], ranks[2, 0] = 1, 5
    ek = np.ones((3, steps))
    ek[1, 5:] = 50.0         # cache step 5 holds the first column from a divergent token
    ev = 2 * np.ones((3, steps))
    ev[1, 5:] = 40.0
    ncount = np.ones((3, steps, len(diagnostics.NEAR_TIE_DELTAS)), np.int64)
    ncount[1, 4] = [2, 2, 3, 5]  # the divergent steps
    ncount[2, 0] = [2, 4, 4, 7]
    ncount[0, 3] = [1, 1, 2, 3]  # one stable step of row 0
    ncount[1, 6] = 9             # after row 1's divergence: neither stable nor divergent
    st = diagnostics.divergence_stats(toks, ref, margins, ranks, ek, ev, tau=0.05, window=16, ncount=ncount)
    nc = st["near_tie_count"]
    # stable synchronous steps: row 0 all 10, row 1 steps 0..3, row 2 none -> 14 steps
    assert nc["0.25"] == dict(stable=1.0, divergent=2.0, ratio=2.0)
    assert nc["1.0"]["stable"] == (13 + 2) / 14 and nc["1.0"]["divergent"] == 3.5
    assert nc["2.0"]["stable"] == (13 + 3) / 14 and nc["2.0"]["divergent"] == 6.0
    assert st["flips"]["events"] == 2 and st["flips"]["synchronous_samples"] == 10 + 5 + 1
    assert st["kv"]["trials"] == 1
    assert st["kv"]["k_pre"] == 1.0 and st["kv"]["k_spike"] == 50.0
    assert st["kv"]["v_pre"] == 2.0 and st["kv"]["v_spike"] == 20.0
    assert abs(st["kv"]["k_slope_median"]) < 1e-12
    nt = st["near_tie"]
    assert (nt["top2"], nt["top3"], nt["top8"]) == (0.5, 0.5, 1.0)
    assert nt["gate_recall"] == 0.5 and nt["stable_trigger"] == 0.0


def test_step_position_guard():
    """The host guard of a step's device-trusted inputs: positions inside the page-table row,
    on a mapped page of the pool; everything else raises before any launch."""
    from paper_2605_30218_amd.runtime import check_positions
    pt = np.array([[3, 1, -1], [0, 2, 4]], np.int32)
    check_positions(pt, [0, 47], 16, 5)          # row 1's last slot
    check_positions(pt, [31, 16], 16, 5)         # row 0's last mapped slot
    for pos, what in (([32, 0], "maps to page -1"), ([0, 48], "outside"), ([-1, 0], "outside")):
        with pytest.raises(ValueError, match=what):
            check_positions(pt, pos, 16, 5)
    with pytest.raises(ValueError, match="not a page of the pool"):
        check_positions(pt, [0, 40], 16, 4)      # page id 4 in a pool of 4 pages
    with pytest.raises(ValueError, match="do not match"):
        check_positions(pt, [0], 16, 5)
