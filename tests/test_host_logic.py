"""Host-side logic that is neither oracle nor kernel: the calibration recipe's statistics."""
import numpy as np


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
    runs none, like the CPU baseline's, is skipped)."""
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
    rows += [restore(), row("fast_gemm_kernel"), row("canon_gemv_kernel", 30_000)]  # gated
    rows += [restore(), row("fast_gemm_kernel"), row("canon_gemv_kernel", 70_000)]  # always
    rows += [restore(), row("copy_to_host")]                               # no decode kernels
    lines = profsum._mode_tables(rows, ["off", "gated", "always"])
    got = {(ln[:16].strip(), ln[17:39].strip()): float(ln.split()[-2]) for ln in lines[3:]}
    assert got[("gated", "canon_gemv_kernel")] == 30.0
    assert got[("always", "canon_gemv_kernel")] == 70.0
    assert ("off", "canon_gemv_kernel") not in got
    assert ("recipe run 1", "canon_gemv_kernel") in got
