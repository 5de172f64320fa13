"""GPU parity of kap_compile_plan against the oracle: bit-exact on every output
(status, logical pages, physical pages, counts, per-span selection flags)."""
import numpy as np
import pytest
import torch

from oracle import kap_oracle as O
from paper_2607_24260_amd import kap as K
from paper_2607_24260_amd.workloads import make_workload

from kap_testlib import assert_plan_equal, dev_i32, gpu_plan, oracle_plan

pytestmark = pytest.mark.gpu


def run_both(seq_lens, fbt, spans_per_seq, prefix, suffix, budget, policy=0, capacity=None,
             num_pages=None, num_spans_extra=0, offsets=None):
    """spans_per_seq: list of lists of (start, len, prior)."""
    B = len(seq_lens)
    fbt = np.asarray(fbt, dtype=np.int32).reshape(B, -1)
    st, ln, pr, offs = [], [], [], [0]
    for sp in spans_per_seq:
        for s in sp:
            st.append(s[0]); ln.append(s[1]); pr.append(s[2])
        offs.append(len(st))
    if offsets is not None:
        offs = offsets
    st = np.asarray(st + [0] * num_spans_extra, dtype=np.int32)
    ln = np.asarray(ln + [0] * num_spans_extra, dtype=np.int32)
    pr = np.asarray(pr + [0.0] * num_spans_extra, dtype=np.float32)
    cap = fbt.shape[1] if capacity is None else capacity
    npages = int(fbt.max()) + 1 if num_pages is None else num_pages
    gpu = K.compile_plan(
        dev_i32(seq_lens), dev_i32(fbt), dev_i32(offs), dev_i32(st), dev_i32(ln),
        torch.as_tensor(pr).cuda(), dev_i32(prefix), dev_i32(suffix), dev_i32(budget),
        num_pages=npages, view_capacity=cap, policy=policy)
    torch.cuda.synchronize()
    plans = O.compile_plan(seq_lens, fbt, offs, st, ln, pr, prefix, suffix, budget, policy,
                           npages, cap)
    assert_plan_equal(gpu, plans, offs)
    return gpu, plans


C1_FBT = [7, 3, 9, 0, 5, 2, 8]
C1_SPANS = [(20, 10, 0.5), (40, 30, 0.9), (90, 5, 0.9), (0, 5, 0.1)]


@pytest.mark.parametrize("policy", [0, 1])
@pytest.mark.parametrize("budget", [10, 36, 52, 60, 84, 100, 1000])
def test_hand_vector(policy, budget):
    _, plans = run_both([100], C1_FBT, [C1_SPANS], [16], [8], [budget], policy=policy)
    if budget == 60 and policy == 0:
        assert plans[0].block_table == [7, 3, 2, 8]


def test_error_statuses_match():
    fbt = np.array([C1_FBT + [0], [1, 2, 3, 4, 5, 6, 7, 99]], dtype=np.int32)
    # seq 0 needs 4 view blocks: over capacity at 3, fine at 8
    _, p = run_both([100, 100], fbt, [C1_SPANS, C1_SPANS], [16, 16], [8, 8], [60, 60],
                    capacity=3, num_pages=50)
    assert [x.status for x in p] == [O.PLAN_OVER_CAPACITY, O.PLAN_OVER_CAPACITY]
    # seq 1 selects page id 99 >= num_pages
    _, p = run_both([100, 128], fbt, [C1_SPANS, [(0, 128, 1.0)]], [16, 0], [8, 1], [60, 128],
                    capacity=8, num_pages=50)
    assert [x.status for x in p] == [O.PLAN_OK, O.PLAN_BAD_PAGE]
    nan = [(20, 10, float("nan"))] + C1_SPANS[1:]
    run_both([100, 100], [C1_FBT, C1_FBT], [nan, C1_SPANS], [16, 16], [8, 8], [60, 60])
    _, p = run_both([0, 145], [C1_FBT + [0, 0], C1_FBT + [0, 0]], [C1_SPANS, C1_SPANS],
                    [16, 16], [8, 8], [60, 60])
    assert [x.status for x in p] == [O.PLAN_BAD_LENGTH, O.PLAN_BAD_LENGTH]
    # malformed CSR bounds for the second sequence
    _, p = run_both([100, 100], [C1_FBT, C1_FBT], [C1_SPANS, C1_SPANS], [16, 16], [8, 8],
                    [60, 60], offsets=[0, 4, 99])
    assert [x.status for x in p] == [O.PLAN_OK, O.PLAN_BAD_SPANS]


def test_no_spans_and_empty_spans():
    run_both([100, 37], [C1_FBT, C1_FBT], [[], [(50, 10, 3.0), (-30, 10, 2.0)]], [0, 0],
             [1, 1], [100, 100])


@pytest.mark.parametrize("seed", range(30))
def test_random_small(seed):
    rng = np.random.default_rng(1000 + seed)
    B = int(rng.integers(1, 6))
    seq_lens = rng.integers(1, 700, B)
    stride = int(-(-seq_lens.max() // 16))
    fbt = np.stack([rng.permutation(stride * B)[:stride] for _ in range(B)])
    spans = []
    for b in range(B):
        n = int(rng.integers(0, 40))
        L = int(seq_lens[b])
        spans.append([(int(rng.integers(-50, L + 30)), int(rng.integers(-5, 200)),
                       float(rng.choice([0.0, -0.0, 0.5, rng.random(), np.inf, -np.inf])))
                      for _ in range(n)])
    prefix = rng.integers(-10, 100, B)
    suffix = rng.integers(-10, 100, B)
    budget = rng.integers(-5, 800, B)
    cap = int(rng.integers(1, stride + 1))
    run_both(seq_lens, fbt, spans, prefix, suffix, budget, policy=int(seed % 2), capacity=cap,
             num_pages=stride * B)


def test_many_spans_one_sequence():
    rng = np.random.default_rng(5)
    L = 65536
    stride = L // 16
    spans = [(int(rng.integers(0, L)), int(rng.integers(16, 600)), float(rng.random()))
             for _ in range(3000)]
    for s in range(0, 3000, 7):       # plenty of exact ties
        spans[s] = (spans[s][0], spans[s][1], 0.25)
    run_both([L], [rng.permutation(stride)], [spans], [512], [256], [9000])


@pytest.mark.parametrize("n", [200, 2500])
@pytest.mark.parametrize("policy", [0, 1])
def test_spans_with_equal_prior_and_start(n, policy):
    # many spans share both prior (0.0 and -0.0 are equal) and start (4
    # starts), so their order is decided by their index alone; the lengths
    # differ, and under STOP the reversed order gives other pages and other
    # selected spans (checked with the oracle). 2500 spans take the
    # multi-chunk ranking path.
    rng = np.random.default_rng(95 + n)
    L = 4000
    stride = L // 16
    starts = rng.choice(np.arange(0, 3600, 16), 4, replace=False)
    spans = [(int(rng.choice(starts)), int(rng.integers(16, 800)),
              float(rng.choice([0.0, -0.0, 1.0]))) for _ in range(n)]
    fbt = rng.permutation(stride)
    if policy == 1:
        fw = O.compile_plan_one(L, fbt, *zip(*spans), 0, 1, 1600, 1, stride, stride)
        rv = O.compile_plan_one(L, fbt, *zip(*spans[::-1]), 0, 1, 1600, 1, stride, stride)
        assert list(fw.logical_blocks) != list(rv.logical_blocks)
    run_both([L], [fbt], [spans], [0], [1], [1600], policy=policy)


@pytest.mark.parametrize("config", [1, 2, 3, 4, 5])
@pytest.mark.parametrize("policy", [0, 1])
def test_workload_plans(config, policy):
    w = make_workload(config, device="cuda", n_decode=1, n_verify=1, with_kv=False)
    gpu = gpu_plan(w, policy=policy)
    plans = oracle_plan(w, policy=policy)
    assert_plan_equal(gpu, plans, w.span_offsets)
    assert all(p.status == O.PLAN_OK for p in plans)
    s = np.array([p.view_tokens / L for p, L in zip(plans, w.seq_lens)])
    if config == 4 and policy == 0:
        assert np.all(s <= 0.055) and np.all(s > 0.05)


def test_all_blocks_budget_gives_full_table():
    w = make_workload(3, device="cuda", n_decode=1, n_verify=1, with_kv=False)
    gpu = gpu_plan(w, budget=w.seq_lens.copy())
    plans = oracle_plan(w, budget=w.seq_lens.copy())
    assert_plan_equal(gpu, plans, w.span_offsets)


def test_capacity_boundary():
    w = make_workload(2, device="cuda", n_decode=1, n_verify=1, with_kv=False)
    plans = oracle_plan(w)
    need = max(p.num_blocks for p in plans)
    for cap in (need - 1, need):
        gpu = gpu_plan(w, capacity=cap)
        assert_plan_equal(gpu, oracle_plan(w, capacity=cap), w.span_offsets)


def test_deterministic():
    w = make_workload(5, device="cuda", n_decode=1, n_verify=1, with_kv=False)
    a = gpu_plan(w)
    b = gpu_plan(w)
    for k in ("view_num_blocks", "view_tokens", "spans_taken", "plan_status", "span_selected"):
        assert torch.equal(a[k], b[k]), k
    nb = a["view_num_blocks"].cpu()
    for k in ("view_block_table", "view_logical_block"):   # entries past nblk are untouched
        for r in range(w.batch):
            assert torch.equal(a[k][r, :nb[r]], b[k][r, :nb[r]]), (k, r)


@pytest.mark.parametrize("policy", [0, 1])
@pytest.mark.parametrize("frac", [0.3, 0.7, 1.0])
def test_long_overlapping_spans_many_taken(policy, frac):
    # 131072 tokens, 150 spans of up to the whole sequence (a span then covers
    # up to 256 bitmap words), heavy overlap and many zero-cost spans; with a
    # budget of the whole sequence every span is taken (one round each)
    rng = np.random.default_rng(int(frac * 10) + 3 * policy)
    L = 131072
    stride = L // 16
    spans = [(int(rng.integers(-1000, L)), int(rng.integers(1, L)), float(rng.choice([0.2, 0.5, rng.random()])))
             for _ in range(150)]
    spans += [(int(rng.integers(0, L - 64)), 64, 0.9) for _ in range(20)]
    _, plans = run_both([L], [rng.permutation(stride)], [spans], [100], [50],
                        [int(frac * L)], policy=policy)
    if frac == 1.0 and policy == 0:
        assert plans[0].spans_taken == sum(1 for s, n, _ in spans if min(L, s + n) > max(0, s))


@pytest.mark.parametrize("policy", [0, 1])
def test_largest_supported_stride(policy):
    # fbt_stride = 262144 pages (4194304 tokens, a 32 KB page bitmap), one
    # full-length sequence under a permuted table: spans that end at L, are
    # clipped there or sit in the last bitmap words, and budgets whose views
    # stay within the 2048 pages staged in LDS before the table is read and
    # go past them (each page then mapped where it is found)
    rng = np.random.default_rng(9 + policy)
    stride = 262144
    L = stride * 16
    spans = [(int(rng.integers(0, L)), int(rng.integers(1, 20000)), float(rng.random()) * 0.9)
             for _ in range(300)]
    spans += [(L - 40, 40, 0.99), (L - 3, 10, 0.98), (L - 16 * 32 * 3 - 7, 5000, 0.97),
              (L - 1, 1, 0.96), (L - 16 * 70, 16 * 33, 0.95), (0, 16 * 5000, 0.5)]
    fbt = [rng.permutation(stride)]
    for budget in (20000, 400000, 2000000):
        _, plans = run_both([L], fbt, [spans], [1000], [300], [budget], policy=policy)
        assert plans[0].status == O.PLAN_OK
    assert plans[0].num_blocks > 2048
