"""The cost-model reporter against the paper's own algebra (Sec. 4): the
speedup condition of Eq. (8) equals a positive phase slack (Eq. (9), (14));
with W_prop = W_main it reduces to Eq. (11) and needs h > s (Eq. (12)); at
KV = KV_crit (Eq. (13)) the slack vanishes; k does not change the sign."""
import math

import numpy as np
import pytest

from paper_2607_24260_amd import costmodel as C


@pytest.mark.parametrize("seed", range(4))
def test_speedup_condition_is_positive_phase_slack(seed):
    rng = np.random.default_rng(seed)
    for _ in range(500):
        k = int(rng.integers(1, 9))
        h, s = rng.random(), rng.random()
        Wm, Wp, KV = rng.random() * 10, rng.random() * 10, rng.random() * 100
        faster = C.cost_plan(k, s, Wp, Wm, KV) < C.cost_base(k, h, Wm, KV)
        assert faster == (C.phase_slack(h, s, Wp, Wm, KV) > 0)
        assert faster == ((h - s) * KV > Wp - h * Wm)


def test_self_speculation_boundary():
    rng = np.random.default_rng(9)
    for _ in range(300):
        h, s = rng.random(), rng.random()
        Wm, KV = rng.random() * 10, rng.random() * 100
        d = C.phase_slack(h, s, Wm, Wm, KV)
        assert math.isclose(d, (h - s) * KV - (1 - h) * Wm, rel_tol=1e-12, abs_tol=1e-12)
        if h <= s:
            assert d <= 0 and C.kv_crit(h, s, Wm) == math.inf
        else:
            kc = C.kv_crit(h, s, Wm)
            assert abs(C.phase_slack(h, s, Wm, Wm, kc)) < 1e-9 * max(1.0, kc)


def test_proposal_length_cancels_from_the_sign():
    for k in range(1, 9):
        assert (C.cost_plan(k, 0.1, 1, 1, 50) < C.cost_base(k, 0.3, 1, 50)) == \
               (C.phase_slack(0.3, 0.1, 1, 1, 50) > 0)


def test_expected_acceptance_closed_form():
    # E[min(X, g)] / g for P(X = j) = 0.6 * 0.4^j: 0.28, 0.1624, 0.0833 for g = 2, 4, 8
    assert math.isclose(C.expected_acceptance(2), 0.28)
    assert math.isclose(C.expected_acceptance(4), 0.4 * (1 - 0.4 ** 4) / 0.6 / 4)
    assert abs(C.expected_acceptance(8) - 0.0833) < 1e-3
    rng = np.random.default_rng(1)
    x = rng.geometric(0.6, 400000) - 1
    assert abs(np.minimum(x, 4).mean() / 4 - C.expected_acceptance(4)) < 2e-3


def test_measured_report_attention_only():
    r = C.measured(4, 0.1624, 0.055, T_view=25.0, T_full=330.0, T_verify=330.0)
    assert math.isclose(r.ideal_ratio, (4 * 0.055 + 1) / (1 + 4 * 0.1624))
    assert math.isclose(r.measured_ratio, (4 * 25 + 330) / ((1 + 4 * 0.1624) * 330))
