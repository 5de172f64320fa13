"""CPU tests of the executor's acceptance bookkeeping and fallback triggers
(Sec. 3.2 "Runtime stability and fallback"; h per Eq. (5); h > s per
Eq. (12)). The thresholds (window of 4 cycles, switch when h <= s after the
first cycle, sticky) are this implementation's reading: parity with the paper
is unpinned, so these tests pin the stated rule with scripted sequences."""
import numpy as np

from paper_2607_24260_amd.executor import FULL, SELECTED, FallbackPolicy, accepted_counts


def test_accepted_counts_clip_to_window():
    assert list(accepted_counts([0, 1, 5, 9], 4)) == [0, 1, 4, 4]
    assert list(accepted_counts([3, 0], 2)) == [2, 0]


def test_plan_failure_starts_on_full_context():
    p = FallbackPolicy(np.array([0.1, 0.1]), np.array([True, False]))
    assert list(p.mode) == [SELECTED, FULL]
    assert list(p.flipped_at) == [-1, 0]


def test_low_acceptance_flips_after_first_cycle_and_is_sticky():
    p = FallbackPolicy(np.array([0.30, 0.30]), np.array([True, True]))
    # cycle 1: sequence 0 accepts nothing, but the first cycle never switches
    assert len(p.update([0, 4], 4)) == 0
    # cycle 2: h0 = 0/8 <= 0.30 -> FULL; h1 = 8/8 stays
    assert list(p.update([0, 4], 4)) == [0]
    assert list(p.mode) == [FULL, SELECTED]
    # sticky even if acceptance recovers
    for _ in range(6):
        p.update([4, 4], 4)
    assert p.mode[0] == FULL and p.flipped_at[0] == 2


def test_boundary_h_equal_s_falls_back():
    p = FallbackPolicy(np.array([0.25]), np.array([True]))
    p.update([1], 4)                 # h = 1/4 but first cycle
    assert list(p.update([1], 4)) == [0]   # h = 2/8 = 0.25 <= s = 0.25


def test_window_forgets_old_cycles():
    p = FallbackPolicy(np.array([0.2]), np.array([True]), window=4)
    for m in (4, 4, 4, 4):
        p.update([m], 4)
    # bad cycles replace good ones in the 4-cycle window: h = 0.75, 0.5, 0.25,
    # then 0 <= s = 0.2 on the fourth
    flips = []
    for expect_h in (0.75, 0.5, 0.25, 0.0):
        flips.append(len(p.update([0], 4)))
        assert abs(p.acceptance(0) - expect_h) < 1e-12
    assert flips == [0, 0, 0, 1]


def test_mixed_gamma_acceptance_is_token_weighted():
    p = FallbackPolicy(np.array([0.4]), np.array([True]))
    p.update([2], 2)                 # 2/2
    p.update([0], 8)                 # (2 + 0) / (2 + 8) = 0.2 <= 0.4
    assert p.mode[0] == FULL
    assert abs(p.acceptance(0) - 0.2) < 1e-12


def test_negative_draws_clamp_to_zero():
    assert list(accepted_counts([-3, 2], 4)) == [0, 2]


def test_host_policy_matches_the_oracle_on_random_streams():
    # the executor's host policy against the oracle's access_modes, cycle by
    # cycle, over random plans (some failed), windows, gammas and accepts
    from oracle import kap_oracle as O

    rng = np.random.default_rng(11)
    for trial in range(80):
        B = int(rng.integers(1, 9))
        C = int(rng.integers(0, 12))
        w = int(rng.integers(1, 7))
        L = rng.integers(1, 5000, B)
        V = np.minimum(rng.integers(0, 5000, B), L)
        st = np.where(rng.random(B) < 0.2, O.PLAN_OVER_CAPACITY, O.PLAN_OK)
        gam = rng.choice([0, 1, 2, 4, 8], C)
        acc = rng.integers(-1, 10, (C, B))
        want = O.access_modes(st, V, L, acc, gam, w)
        p = FallbackPolicy(V / L.astype(np.float64), st == O.PLAN_OK, window=w)
        assert np.array_equal(p.mode, want[0]), trial
        for c in range(C):
            p.update(accepted_counts(acc[c], gam[c]), int(gam[c]))
            assert np.array_equal(p.mode, want[c + 1]), (trial, c)
