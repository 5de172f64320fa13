"""GPU: kap_decode_schedule + kap_selected_decode_scheduled.

A schedule records, per workgroup, the work item the balanced split map
gives it and its wavefronts' first view entries, so that decode calls on an
unchanged view skip the map. The scheduled call must return exactly the
unscheduled call's results (same split assignment, same kernels): checked bit
for bit on the bf16 workloads, the ragged fp8 workload and a token-granular
view, reused over several proposal steps, under HIP-graph replay, and against
the oracle on one workload. Calls without a balanced map (the generic path,
or one split per (sequence, KV head)) take an empty schedule.
"""
import numpy as np
import pytest
import torch

from oracle import kap_oracle as O
from paper_2607_24260_amd import kap as K
from paper_2607_24260_amd.workloads import make_workload

from kap_testlib import (LSE_TOL, O_TOL, assert_close, dev_i32, gpu_plan, kv_of, oracle_plan,
                         oracle_pool, plan_view_arrays)

pytestmark = pytest.mark.gpu


def _view(w, token_granular=False):
    cap = w.max_pages_per_seq
    if not token_granular:
        plan = gpu_plan(w)
        return plan, cap, None
    plan = K.compile_plan(
        dev_i32(w.seq_lens), dev_i32(w.full_block_table), dev_i32(w.span_offsets),
        dev_i32(w.span_start), dev_i32(w.span_len),
        torch.as_tensor(np.asarray(w.span_prior, dtype=np.float32)).cuda(), dev_i32(w.prefix),
        dev_i32(w.suffix), dev_i32(w.budget), num_pages=w.num_pages, view_capacity=cap,
        token_granular=True)
    torch.cuda.synchronize()
    return plan, cap, plan["view_token_mask"]


def _pair(w, plan, cap, mask, steps):
    """(scheduled, unscheduled) outputs of the given decode steps."""
    kv = kv_of(w)
    sl = dev_i32(w.seq_lens)
    args = (sl, plan["view_block_table"], plan["view_logical_block"], plan["view_num_blocks"],
            cap)
    sched = K.decode_schedule(kv, *args, view_token_mask=mask)
    got = []
    for s in steps:
        q = w.q_decode[s]
        a = K.selected_decode(kv, q, *args, w.sm_scale, view_token_mask=mask, schedule=sched)
        b = K.selected_decode(kv, q, *args, w.sm_scale, view_token_mask=mask)
        got.append((a, b))
    torch.cuda.synchronize()
    return sched, got


@pytest.mark.parametrize("config,kw", [
    (2, {}), (3, {}), (4, dict(n_decode=4, n_verify=1)),
    (5, dict(n_decode=3, n_verify=1)),
])
def test_scheduled_equals_balanced(config, kw):
    w = make_workload(config, device="cuda", **kw)
    plan, cap, _ = _view(w)
    sched, got = _pair(w, plan, cap, None, range(min(3, w.q_decode.shape[0])))
    assert sched.numel() > 0            # these calls take the balanced map
    for s, ((o1, l1), (o2, l2)) in enumerate(got):
        assert torch.equal(o1, o2), f"out differs at step {s}"
        assert torch.equal(l1, l2), f"lse differs at step {s}"


@pytest.mark.parametrize("seed", range(16))
def test_random_batches_scheduled_equals_balanced(seed):
    # seeded random batches: 1-70 sequences (the map reads lengths 64 at a
    # time), lengths 1-4096, per-sequence budgets, bf16 or fp8, page- or
    # token-granular views; the scheduled call must equal the balanced one
    rng = np.random.default_rng(777 + seed)
    cfg = 2 if seed % 2 == 0 else 5
    B = int(rng.choice([1, 3, 8, 33, 64, 65, 70]))
    w = make_workload(cfg, device="cuda", batch=B, seq_len=4096 if cfg == 2 else 5000,
                      n_decode=2, n_verify=1, with_kv=True)
    w.seq_lens[:] = rng.integers(1, 4097, B).astype(np.int32)
    budget = np.array([int(rng.integers(0, int(L) + 1)) for L in w.seq_lens], dtype=np.int32)
    token = seed % 3 == 0
    cap = w.max_pages_per_seq
    plan = K.compile_plan(
        dev_i32(w.seq_lens), dev_i32(w.full_block_table), dev_i32(w.span_offsets),
        dev_i32(w.span_start), dev_i32(w.span_len),
        torch.as_tensor(np.asarray(w.span_prior, dtype=np.float32)).cuda(), dev_i32(w.prefix),
        dev_i32(w.suffix), dev_i32(budget), num_pages=w.num_pages, view_capacity=cap,
        token_granular=token)
    torch.cuda.synchronize()
    mask = plan["view_token_mask"] if token else None
    sched, got = _pair(w, plan, cap, mask, range(2))
    assert sched.numel() > 0
    for s, ((o1, l1), (o2, l2)) in enumerate(got):
        assert torch.equal(o1, o2), f"out differs at step {s} (B={B}, token={token})"
        assert torch.equal(l1, l2), f"lse differs at step {s} (B={B}, token={token})"


def test_scheduled_token_granular_view():
    w = make_workload(4, device="cuda", n_decode=2, n_verify=1)
    plan, cap, mask = _view(w, token_granular=True)
    _, got = _pair(w, plan, cap, mask, range(2))
    for (o1, l1), (o2, l2) in got:
        assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_scheduled_matches_oracle():
    w = make_workload(2, device="cuda", n_decode=2, n_verify=1)
    pool = oracle_pool(w)
    plan, cap, _ = _view(w)
    kv = kv_of(w)
    sl = dev_i32(w.seq_lens)
    args = (sl, plan["view_block_table"], plan["view_logical_block"], plan["view_num_blocks"],
            cap)
    sched = K.decode_schedule(kv, *args)
    vbt, vlb, nb = plan_view_arrays(oracle_plan(w), cap)
    for s in range(2):
        q = w.q_decode[s]
        o, lse = K.selected_decode(kv, q, *args, w.sm_scale, schedule=sched)
        torch.cuda.synchronize()
        eo, el = O.selected_decode(pool, q.float().cpu().numpy(), w.seq_lens, vbt, vlb, nb,
                                   w.sm_scale)
        assert_close("scheduled O", o.cpu().numpy(), eo, O_TOL)
        assert_close("scheduled LSE", lse.cpu().numpy(), el, LSE_TOL)


def test_schedule_follows_a_changed_view():
    # a new plan (another budget) needs a new schedule; the rebuilt one matches
    w = make_workload(3, device="cuda", n_decode=1, n_verify=1)
    kv = kv_of(w)
    sl = dev_i32(w.seq_lens)
    cap = w.max_pages_per_seq
    sched = None
    for budget in (w.budget, (w.budget * 3) // 2):
        plan = gpu_plan(w, budget=budget)
        args = (sl, plan["view_block_table"], plan["view_logical_block"],
                plan["view_num_blocks"], cap)
        sched = K.decode_schedule(kv, *args, out=sched)
        a = K.selected_decode(kv, w.q_decode[0], *args, w.sm_scale, schedule=sched)
        b = K.selected_decode(kv, w.q_decode[0], *args, w.sm_scale)
        torch.cuda.synchronize()
        assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


def test_graph_replays_of_scheduled_decode():
    w = make_workload(4, device="cuda", n_decode=2, n_verify=1)
    plan, cap, _ = _view(w)
    kv = kv_of(w)
    sl = dev_i32(w.seq_lens)
    args = (sl, plan["view_block_table"], plan["view_logical_block"], plan["view_num_blocks"],
            cap)
    B = w.batch
    ref = K.selected_decode(kv, w.q_decode[1], *args, w.sm_scale)
    torch.cuda.synchronize()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        sched = torch.empty(K.decode_schedule_bytes(kv, B, cap) // 4, dtype=torch.int32,
                            device="cuda")
        o = torch.empty((B, w.num_q_heads, w.head_dim), dtype=torch.float32, device="cuda")
        lse = torch.empty((B, w.num_q_heads), dtype=torch.float32, device="cuda")
        ws = torch.zeros(max(256, K.selected_decode_workspace_bytes(kv, B, cap)),
                         dtype=torch.uint8, device="cuda")
        mk = K.bind_selected_decode  # validates once (eagerly) before capture
        K.decode_schedule(kv, *args, out=sched, stream=s)
        call = mk(kv, w.q_decode[1], *args, w.sm_scale, o, lse, ws, schedule=sched, stream=s)
    s.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=s):
        K.decode_schedule(kv, *args, out=sched, stream=s)
        call()
    for _ in range(3):
        o.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(o, ref[0]) and torch.equal(lse, ref[1])


def test_empty_schedule_without_balanced_map():
    # fp32 goes through the generic path: no map, no schedule
    w = make_workload(1, device="cuda")
    kv = kv_of(w)
    plan, cap, _ = _view(w)
    sl = dev_i32(w.seq_lens)
    args = (sl, plan["view_block_table"], plan["view_logical_block"], plan["view_num_blocks"],
            cap)
    assert K.decode_schedule_bytes(kv, w.batch, cap) == 0
    sched = K.decode_schedule(kv, *args)
    assert sched.numel() == 0
    a = K.selected_decode(kv, w.q_decode[0], *args, w.sm_scale, schedule=sched)
    b = K.selected_decode(kv, w.q_decode[0], *args, w.sm_scale)
    torch.cuda.synchronize()
    assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


def test_scheduled_call_rejects_a_missing_schedule():
    w = make_workload(2, device="cuda", n_decode=1, n_verify=1)
    kv = kv_of(w)
    plan, cap, _ = _view(w)
    B = w.batch
    o = torch.empty((B, w.num_q_heads, w.head_dim), dtype=torch.float32, device="cuda")
    lse = torch.empty((B, w.num_q_heads), dtype=torch.float32, device="cuda")
    lib = K.load_library()
    st = lib.kap_selected_decode_scheduled(
        K.ctypes.byref(kv.struct), B, K._ptr(w.q_decode[0]), K._ptr(dev_i32(w.seq_lens)),
        K._ptr(plan["view_block_table"]), K._ptr(plan["view_logical_block"]), None, cap,
        K._ptr(plan["view_num_blocks"]), cap, None, 1.0, K._ptr(o), K._ptr(lse), None, 0, None)
    assert st == K.KAP_ERR_INVALID_ARGUMENT
