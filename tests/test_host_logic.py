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
