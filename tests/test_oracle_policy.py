"""CPU pins for the oracle's access-mode policy (Sec. 3.2 "Runtime stability
and fallback"; h per Eq. (5), s per Eq. (4), the margin condition h > s of
Eq. (12)) and for the view rows each mode reads.

The paper names the fallback conditions but prints no thresholds or worked
cycle, so the rule these tests fix is the oracle's reading (window of the last
cycles, no switch before the second cycle, h <= s switches, sticky): the
vectors below were worked out by hand from that rule, and each is chosen so
that a plausible slip (no window, no first-cycle grace, no clamp of the accept
count, a strict h < s, 0/0 read as 0) changes an expected mode.
"""
from fractions import Fraction

import numpy as np
import pytest

from oracle import kap_oracle as O

S, F = O.SELECTED, O.FULL

# window 2; cycles speculate 4, 4, 0, 0, 8 tokens
VEC_WINDOW = 2
VEC_GAMMAS = [4, 4, 0, 0, 8]
#            L     view  status                  accepted (raw) per cycle
VEC_SEQS = [(400, 100, O.PLAN_OK, [0, 4, 3, 0, 2]),
            (160, 96, O.PLAN_OK, [3, 1, 0, 0, 8]),
            (64, 0, O.PLAN_OVER_CAPACITY, [4, 4, 0, 0, 8]),
            (1000, 100, O.PLAN_OK, [0, 4, 7, 0, 1]),
            (320, 160, O.PLAN_OK, [0, 9, 0, 0, 4])]
# Worked by hand (window = last two cycles; row c + 1 = after cycle c):
#  seq 0, s = 1/4: c0 (0/4) first cycle, no check; c1 (0+4)/(4+4) = 1/2;
#    c2 accepts min(3, 0) = 0: (4+0)/(4+0) = 1; c3 window speculated 0+0 = 0:
#    no decision; c4 (0+2)/(0+8) = 1/4 <= 1/4 -> FULL. (Over all five cycles
#    h would be 6/16 = 3/8 > 1/4: the window decides.)
#  seq 1, s = 96/160 = 3/5: c1 (3+1)/8 = 1/2 <= 3/5 -> FULL, then sticky.
#  seq 2: plan over capacity -> FULL from the start.
#  seq 3, s = 1/10: c0 alone would give 0 <= 1/10, but the first cycle never
#    switches; c1 1/2, c2 1 (7 clamped to 0), c3 no decision, c4 1/8 > 1/10.
#  seq 4, s = 1/2: c1 accepts min(9, 4) = 4: (0+4)/8 = 1/2 <= 1/2 -> FULL
#    (unclamped, 9/8 would keep the plan).
VEC_MODES = np.array([[S, S, F, S, S],
                      [S, S, F, S, S],
                      [S, F, F, S, F],
                      [S, F, F, S, F],
                      [S, F, F, S, F],
                      [F, F, F, S, F]])


def _vec():
    L = [s[0] for s in VEC_SEQS]
    V = [s[1] for s in VEC_SEQS]
    st = [s[2] for s in VEC_SEQS]
    acc = np.array([s[3] for s in VEC_SEQS]).T          # [C][B]
    return st, V, L, acc


def test_hand_vector_modes():
    st, V, L, acc = _vec()
    modes = O.access_modes(st, V, L, acc, VEC_GAMMAS, VEC_WINDOW)
    assert modes.shape == (len(VEC_GAMMAS) + 1, len(VEC_SEQS))
    assert np.array_equal(modes, VEC_MODES)


def test_hand_vector_window_matters():
    # with a window covering every cycle, sequence 0 keeps its plan (3/8 > 1/4)
    st, V, L, acc = _vec()
    modes = O.access_modes(st, V, L, acc, VEC_GAMMAS, window=5)
    assert modes[-1, 0] == S
    assert np.array_equal(modes[:, 1:], VEC_MODES[:, 1:])


def test_equality_switches_and_strict_margin_keeps():
    # h = s exactly switches (Eq. (12) asks for h > s); one accepted token
    # more keeps the plan
    for acc2, want in ((1, F), (2, S)):
        m = O.access_modes([O.PLAN_OK], [1], [4], [[1], [acc2]], [4, 4], window=4)
        # h = (1 + acc2) / 8 against s = 1/4
        assert m[-1, 0] == want, acc2


def test_exact_rational_comparison():
    # s = 1/3 from 100 / 300 and h = 1/3 from 1 / 3: equal rationals switch
    m = O.access_modes([O.PLAN_OK], [100], [300], [[0], [1]], [0, 3], window=2)
    assert m[-1, 0] == F
    assert Fraction(1, 3) == Fraction(100, 300)


@pytest.mark.parametrize("bad", [O.PLAN_OVER_CAPACITY, O.PLAN_BAD_SCORE, O.PLAN_BAD_PAGE,
                                 O.PLAN_BAD_LENGTH, O.PLAN_BAD_SPANS])
def test_every_failed_status_starts_on_full_context(bad):
    m = O.access_modes([bad, O.PLAN_OK], [0, 10], [100, 100], np.zeros((3, 2)), [2, 2, 2], 4)
    assert np.all(m[:, 0] == F)
    assert m[0, 1] == S


def test_no_cycles_gives_start_modes_only():
    m = O.access_modes([O.PLAN_OK, O.PLAN_OVER_CAPACITY], [5, 0], [50, 50],
                       np.zeros((0, 2)), [], 4)
    assert m.tolist() == [[S, F]]


def test_random_streams_against_a_brute_force_rereading():
    # an independent restatement of the same rule over whole histories: at
    # cycle c the sequence is FULL iff its plan failed or some earlier check
    # point j (1 <= j <= c, 0-based cycle index) had positive speculated sum and
    # accepted * L <= view * speculated over cycles max(0, j-w+1) .. j
    rng = np.random.default_rng(7)
    for trial in range(60):
        B = int(rng.integers(1, 6))
        C = int(rng.integers(0, 9))
        w = int(rng.integers(1, 5))
        L = rng.integers(1, 400, B)
        V = np.minimum(rng.integers(0, 400, B), L)
        st = np.where(rng.random(B) < 0.2, O.PLAN_OVER_CAPACITY, O.PLAN_OK)
        gam = rng.integers(0, 9, C)
        acc = rng.integers(-2, 11, (C, B))
        got = O.access_modes(st, V, L, acc, gam, w)
        for b in range(B):
            a = np.minimum(np.maximum(acc[:, b], 0), gam)
            for c in range(C):
                full = st[b] != O.PLAN_OK
                for j in range(1, c + 1):
                    lo = max(0, j - w + 1)
                    A, Sp = int(a[lo:j + 1].sum()), int(gam[lo:j + 1].sum())
                    full = full or (Sp > 0 and A * int(L[b]) <= int(V[b]) * Sp)
                assert got[c + 1, b] == (F if full else S), (trial, b, c)


# --------------------------------------------------------------------------
# active view rows
# --------------------------------------------------------------------------

C1_FBT = [7, 3, 9, 0, 5, 2, 8]
C1_SPANS = [(20, 10, 0.5), (40, 30, 0.9), (90, 5, 0.9), (0, 5, 0.1)]


def _c1_plan(token_granular=False):
    fn = O.compile_plan_tokens_one if token_granular else O.compile_plan_one
    return fn(100, C1_FBT, [s[0] for s in C1_SPANS], [s[1] for s in C1_SPANS],
              [s[2] for s in C1_SPANS], 16, 8, 60, O.SELECT_SKIP, 100, 64)


def test_active_view_selected_is_the_plan_row():
    bt, lb, n, mk = O.active_view(S, _c1_plan(), C1_FBT + [-1, -1], 100)
    assert (bt, lb, n, mk) == ([7, 3, 2, 8], [0, 1, 5, 6], 4, None)


def test_active_view_full_is_the_whole_table():
    # L = 100 -> 7 pages; entries past them are not part of the view
    bt, lb, n, mk = O.active_view(F, _c1_plan(), C1_FBT + [-1, -1], 100)
    assert (bt, lb, n, mk) == (C1_FBT, list(range(7)), 7, None)


def test_active_view_token_granular():
    plan = _c1_plan(token_granular=True)
    bt, lb, n, mk = O.active_view(S, plan, C1_FBT, 100)
    # the hand-worked token plan of the same vector: pages 0, 2, 3, 4, 5, 6
    assert lb == [0, 2, 3, 4, 5, 6] and bt == [7, 9, 0, 5, 2, 8]
    assert mk == [0xFFFF, 0xFF00, 0xFFFF, 0x003F, 0xFC00, 0x000F]
    bt, lb, n, mk = O.active_view(F, plan, C1_FBT, 100)
    assert n == 7 and mk == [0xFFFF] * 7 and lb == list(range(7))


def test_failed_plan_view_is_full_context():
    plan = O.compile_plan_one(100, C1_FBT, [0], [10], [0.5], 16, 8, 60, O.SELECT_SKIP, 100,
                              capacity=1)
    assert plan.status == O.PLAN_OVER_CAPACITY
    m = O.access_modes([plan.status], [plan.view_tokens], [100], np.zeros((0, 1)), [], 4)
    bt, lb, n, _ = O.active_view(int(m[0, 0]), plan, C1_FBT, 100)
    assert n == 7 and bt == C1_FBT


# --------------------------------------------------------------------------
# the hand vector catches plausible slips
# --------------------------------------------------------------------------

def _reread(st, V, L, acc, gammas, window, slip=None):
    """The rule restated over whole histories (as in the random test), with
    one optional slip planted: each slip must change some mode of the hand
    vector, or the vector would not pin that part of the rule."""
    C, B = len(gammas), len(L)
    out = np.zeros((C + 1, B), dtype=np.int64)
    gam = np.asarray(gammas, dtype=np.int64)
    for b in range(B):
        raw = np.asarray([acc[c][b] for c in range(C)], dtype=np.int64)
        a = raw if slip == "no_clamp" else np.minimum(np.maximum(raw, 0), gam)
        full = st[b] != O.PLAN_OK
        out[0, b] = F if full else S
        for c in range(C):
            first = 0 if slip == "no_grace" else 1
            if c >= first and not full:
                lo = 0 if slip == "no_window" else max(0, c - window + 1)
                A, Sp = int(a[lo:c + 1].sum()), int(gam[lo:c + 1].sum())
                if slip == "zero_over_zero":
                    full = Sp == 0 or A * L[b] <= V[b] * Sp
                elif slip == "strict":
                    full = Sp > 0 and A * L[b] < V[b] * Sp
                else:
                    full = Sp > 0 and A * L[b] <= V[b] * Sp
            out[c + 1, b] = F if full else S
    return out


def test_hand_vector_rereading_agrees():
    st, V, L, acc = _vec()
    assert np.array_equal(_reread(st, V, L, acc, VEC_GAMMAS, VEC_WINDOW), VEC_MODES)


@pytest.mark.parametrize("slip", ["no_window", "no_grace", "no_clamp", "strict",
                                  "zero_over_zero"])
def test_hand_vector_catches_slip(slip):
    st, V, L, acc = _vec()
    assert not np.array_equal(_reread(st, V, L, acc, VEC_GAMMAS, VEC_WINDOW, slip), VEC_MODES)
