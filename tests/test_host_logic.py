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
