"""The restore-cost fit behind the OBR measurement (Eq. 2: T_load(n) =
n beta / B_eff + tau_load) recovers a known line exactly."""
import numpy as np

from paper_2609_33762_amd import drivers


def test_fit_recovers_bandwidth_and_overhead():
    beta = 24 * 1024
    n = np.array([16, 64, 256, 1024, 4096, 16384])
    B, tau = 55.0e9, 12.5e-6
    t = n * beta / B + tau
    b_fit, tau_fit, resid = drivers.fit_load_cost(n * beta, t)
    assert abs(b_fit / B - 1) < 1e-9 and abs(tau_fit - tau) < 1e-12 and resid < 1e-9
    # per-token cost of the appendix: beta / B_eff + tau / n
    assert abs((beta / b_fit + tau_fit / 4096) - t[-2] / 4096) < 1e-15
