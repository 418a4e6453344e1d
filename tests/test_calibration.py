"""Offline cost calibration (Sec. IV-A): the oracle's closed-form least
squares pinned by exact recovery, and the library's fits against it."""
import numpy as np
import pytest

import oracle
from paper_2606_29982_amd import calibrate as cal


def test_oracle_recovers_exact_line():
    S = np.array([1, 4, 16, 44, 88], dtype=np.float64) * 2 ** 20
    B = 64e3      # bytes per microsecond (64 GB/s)
    t = 1.25 * S / B + 7.5
    a, b = oracle.fit_alpha_beta(S, t, B)
    assert a == pytest.approx(1.25, rel=1e-12) and b == pytest.approx(7.5, rel=1e-12)


def test_oracle_grouped_recovers_exact_plane():
    m = np.repeat([8, 16, 32, 64], 3).astype(float)
    S = np.tile([1, 2, 4], 4) * 44040192.0
    B = 8e6       # bytes per microsecond (8 TB/s)
    t = 3.0 + m * (1.3 * S / B + 0.4)
    a, b, c0 = oracle.fit_grouped(m, S, t, B)
    assert (a, b, c0) == pytest.approx((1.3, 0.4, 3.0), rel=1e-10)


def test_oracle_rejects_one_size():
    with pytest.raises(ValueError):
        oracle.fit_alpha_beta([5.0, 5.0, 5.0], [1.0, 2.0, 3.0], 1.0)


@pytest.mark.parametrize("seed", range(3))
def test_link_fit_matches_oracle(seed):
    rng = np.random.default_rng(seed)
    S = rng.uniform(1, 100, 12) * 2 ** 20
    t = 1.1 * S / 64e3 + 4.0 + rng.normal(0, 2.0, 12)
    got = cal.fit_link(S, t, 64.0)
    a, b = oracle.fit_alpha_beta(S, t, 64e3)
    assert got.alpha == pytest.approx(a, rel=1e-9) and got.beta == pytest.approx(b, rel=1e-9, abs=1e-9)
    assert 0.0 < got.r2 <= 1.0


@pytest.mark.parametrize("seed", range(3))
def test_grouped_fit_matches_oracle(seed):
    rng = np.random.default_rng(seed)
    m = np.repeat([8, 16, 32, 64], 3).astype(float)
    S = np.tile([22020096.0, 44040192.0, 88080384.0], 4)
    t = 20.0 + m * (1.25 * S / 8e6 + 0.3) + rng.normal(0, 1.0, m.size)
    got = cal.fit_grouped(m, S, t, 8000.0)
    a, b, c0 = oracle.fit_grouped(m, S, t, 8e6)
    assert (got.alpha, got.beta, got.c0_us) == pytest.approx((a, b, c0), rel=1e-8, abs=1e-8)


def test_cost_table_and_residency():
    model = cal.CostModel(alpha=1.2, beta=3.0, bandwidth_gbps=64.0, r2=1.0)
    c = cal.cost_table(model, 88080384, 8, resident=[True, False] * 4)
    want = oracle.cost_of([88080384], 1.2, 3.0, 64e3)[0]
    assert c.dtype == np.float32
    assert np.all(c[::2] == 0.0) and np.allclose(c[1::2], want, rtol=1e-6)
