"""The device-side access-mode policy (kap_fallback_update) against the
oracle's access_modes / active_view (Sec. 3.2 "Runtime stability and
fallback"; Eq. (5), Eq. (12)), HIP-graph replays of a whole device-resident
stream against its eager run, and the device-resident stream against the
host-policy stream and the oracle."""
import numpy as np
import pytest
import torch

from oracle import kap_oracle as O
from paper_2607_24260_amd import kap as K
from paper_2607_24260_amd.executor import FULL, DeviceStream, run_stream
from paper_2607_24260_amd.workloads import make_workload

from kap_testlib import dev_i32, gpu_plan, kv_of, oracle_plan

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("window", [1, 4, 7])
def test_device_policy_matches_oracle(window):
    # 40 sequences with assorted s (including plan failures), 14 cycles of
    # random gammas and geometric(0.6) - 1 accept draws (some negative and
    # some above gamma, which both sides clamp); after the reset and after
    # every cycle the device's modes and active view rows must equal the
    # oracle's, and its cycle counters the number of cycles run
    rng = np.random.default_rng(window)
    B, C, stride, cap = 40, 14, 96, 64
    L = rng.integers(100, 1500, B).astype(np.int32)
    vtok = np.minimum(rng.integers(16, 800, B), L).astype(np.int32)
    status = np.where(rng.random(B) < 0.15, K.KAP_PLAN_OVER_CAPACITY,
                      K.KAP_PLAN_OK).astype(np.int32)
    sel_nb = np.minimum(-(-vtok // 16), cap).astype(np.int32)
    sel_bt = rng.integers(0, 5000, (B, cap)).astype(np.int32)
    sel_lb = rng.integers(0, 90, (B, cap)).astype(np.int32)
    fbt = rng.integers(0, 5000, (B, stride)).astype(np.int32)
    gammas = rng.choice([2, 4, 8], C)
    draws = (rng.geometric(0.6, (C, B)) - 1).astype(np.int32)
    draws[rng.random((C, B)) < 0.05] = -1

    plan = {"view_block_table": dev_i32(sel_bt), "view_logical_block": dev_i32(sel_lb),
            "view_num_blocks": dev_i32(sel_nb), "view_tokens": dev_i32(vtok),
            "plan_status": dev_i32(status)}
    hist = torch.zeros((B, window, 2), dtype=torch.int32, device="cuda")
    cyc = torch.zeros(B, dtype=torch.int32, device="cuda")
    mode = torch.zeros(B, dtype=torch.int32, device="cuda")
    vbt = torch.full((B, stride), -5, dtype=torch.int32, device="cuda")
    vlb = torch.full((B, stride), -5, dtype=torch.int32, device="cuda")
    vnb = torch.zeros(B, dtype=torch.int32, device="cuda")
    common = (plan["view_tokens"], dev_i32(L), plan["plan_status"], hist, cyc, mode,
              plan["view_block_table"], plan["view_logical_block"], plan["view_num_blocks"],
              dev_i32(fbt), vbt, vlb, vnb)
    K.bind_fallback_update(True, window, 0, None, *common)()

    # the oracle's view of the same plan rows (inputs, not outputs of the library)
    plans = [O.Plan(int(status[b]), list(sel_lb[b, :sel_nb[b]]), list(sel_bt[b, :sel_nb[b]]),
                    int(sel_nb[b]), int(vtok[b]), 0, []) for b in range(B)]
    want_modes = O.access_modes(status, vtok, L, draws, gammas, window)

    def check(tag, row):
        torch.cuda.synchronize()
        got_mode = mode.cpu().numpy()
        assert np.array_equal(got_mode, want_modes[row]), tag
        got_nb, got_bt, got_lb = vnb.cpu().numpy(), vbt.cpu().numpy(), vlb.cpu().numpy()
        for b in range(B):
            bt, lb, n, _ = O.active_view(int(want_modes[row, b]), plans[b], fbt[b], int(L[b]))
            assert got_nb[b] == n, (tag, b)
            assert np.array_equal(got_bt[b, :n], bt), (tag, b)
            assert np.array_equal(got_lb[b, :n], lb), (tag, b)

    check("reset", 0)
    for c in range(C):
        K.bind_fallback_update(False, window, int(gammas[c]), dev_i32(draws[c]), *common)()
        check(f"cycle {c}", c + 1)
    assert ((want_modes[0] == O.SELECTED) & (want_modes[-1] == O.FULL)).any(), \
        "no sequence switched during the cycles"
    assert np.array_equal(cyc.cpu().numpy(), np.full(B, C))


def _snapshot(ds):
    return ([t.clone() for pair in ds.ver_out for t in pair]
            + [ds.out.clone(), ds.lse.clone(), ds.mode.clone(), ds.vnb.clone()])


def test_graph_replays_equal_the_eager_stream():
    # 16 ragged fp8 sequences (4K..64K), 8 cycles with fallbacks: the eager
    # device-resident stream, then 3 replays of its HIP graph with eager work
    # and synchronisations between them, each checked against the eager run
    w = make_workload(5, device="cuda", batch=16, seq_len=65536, n_verify=8)
    kv = kv_of(w)
    plan = gpu_plan(w)
    ds = DeviceStream(w, kv, plan)
    ds.run()
    torch.cuda.synchronize()
    eager = _snapshot(ds)
    assert bool((ds.mode == FULL).any()), "the recipe's accept law should trigger fallbacks"
    g = ds.capture()
    scratch = torch.zeros(1 << 20, device="cuda")
    for rep in range(3):
        for t in (ds.out, ds.lse):
            t.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        got = _snapshot(ds)
        for i, (a, b) in enumerate(zip(got, eager)):
            assert torch.equal(a, b), f"replay {rep}: tensor {i} differs"
        scratch.add_(1.0)                      # eager work between replays
        torch.cuda.synchronize()


def test_device_stream_equals_host_policy_stream():
    # the same stream with the host policy (run_stream): identical verify
    # outputs call by call, identical last decode, and both policies' final
    # modes equal the oracle's (oracle plans, the workload's accept draws)
    w = make_workload(5, device="cuda", batch=16, seq_len=65536, n_verify=8)
    kv = kv_of(w)
    plan = gpu_plan(w)
    ds = DeviceStream(w, kv, plan)
    ds.run()
    torch.cuda.synchronize()
    last = w.q_decode.shape[0] - 1
    res = run_stream(w, kv, plan, keep_outputs={("verify", j) for j in range(len(w.q_verify))}
                     | {("decode", last)})
    torch.cuda.synchronize()
    plans = oracle_plan(w)
    gammas = [q.shape[1] - 1 for q in w.q_verify]
    want = O.access_modes([p.status for p in plans], [p.view_tokens for p in plans],
                          w.seq_lens, w.accept_draws, gammas, 4)
    assert np.array_equal(ds.mode.cpu().numpy(), want[-1])
    assert np.array_equal(res.policy.mode, want[-1])
    for j, o, l in res.verify_out:
        assert torch.equal(o, ds.ver_out[j][0]) and torch.equal(l, ds.ver_out[j][1]), j
    (idx, o, l, _), = res.decode_out
    assert idx == last and torch.equal(o, ds.out) and torch.equal(l, ds.lse)


def test_token_granular_device_stream():
    # the ragged fp8 stream over token-granular views (Sec. 3.1 mask in the
    # device-resident cycle): the modes equal the oracle's (oracle token
    # plans, the workload's accept draws); every active row equals the
    # oracle's active view (the plan's pages and masks, or the full table with
    # all-ones masks); the last decode equals, for sampled sequences, the
    # oracle's decode over the oracle's views
    from kap_testlib import LSE_TOL, O_TOL, assert_close, oracle_pool

    # 4 cycles: long enough for some sequences to fall back, short enough
    # that others keep their views under the recipe's accept law
    w = make_workload(5, device="cuda", batch=16, seq_len=65536, n_verify=4)
    kv = kv_of(w)
    cap = w.max_pages_per_seq
    plan = K.compile_plan(
        dev_i32(w.seq_lens), dev_i32(w.full_block_table), dev_i32(w.span_offsets),
        dev_i32(w.span_start), dev_i32(w.span_len),
        torch.as_tensor(np.asarray(w.span_prior, dtype=np.float32)).cuda(), dev_i32(w.prefix),
        dev_i32(w.suffix), dev_i32(w.budget), num_pages=w.num_pages, view_capacity=cap,
        token_granular=True)
    ds = DeviceStream(w, kv, plan)
    ds.run()
    torch.cuda.synchronize()
    L = np.asarray(w.seq_lens, dtype=np.int64)
    plans = O.compile_plan(w.seq_lens, w.full_block_table, w.span_offsets, w.span_start,
                           w.span_len, w.span_prior, w.prefix, w.suffix, w.budget,
                           O.SELECT_SKIP, w.num_pages, cap, token_granular=True)
    gammas = [q.shape[1] - 1 for q in w.q_verify]
    want = O.access_modes([p.status for p in plans], [p.view_tokens for p in plans], L,
                          w.accept_draws, gammas, 4)[-1]
    mode = ds.mode.cpu().numpy()
    assert np.array_equal(mode, want)
    assert (mode == 0).any() and (mode == FULL).any(), "want both access modes in the stream"
    vnb, vbt = ds.vnb.cpu().numpy(), ds.vbt.cpu().numpy()
    vlb, vmk = ds.vlb.cpu().numpy(), ds.vmask.cpu().numpy().astype(np.int64) & 0xFFFFFFFF
    B, stride = w.batch, vbt.shape[1]
    ebt = np.zeros((B, stride), np.int64)
    elb = np.zeros((B, stride), np.int64)
    emk = np.zeros((B, stride), np.int64)
    enb = np.zeros(B, np.int64)
    for b in range(B):
        bt, lb, n, mk = O.active_view(int(want[b]), plans[b], w.full_block_table[b], int(L[b]))
        ebt[b, :n], elb[b, :n], emk[b, :n], enb[b] = bt, lb, mk, n
        assert vnb[b] == n, b
        assert np.array_equal(vbt[b, :n], bt) and np.array_equal(vlb[b, :n], lb), b
        assert np.array_equal(vmk[b, :n], mk), b
    last = w.q_decode.shape[0] - 1
    sel = [b for b in range(B) if want[b] == 0][:2] + [b for b in range(B) if want[b] == FULL][:2]
    eo, el = O.selected_decode(oracle_pool(w), w.q_decode[last].float().cpu().numpy()[sel],
                               L[sel], ebt[sel], elb[sel], enb[sel], w.sm_scale,
                               view_token_mask=emk[sel])
    assert_close("token stream O", ds.out.cpu().numpy()[sel], eo, O_TOL)
    assert_close("token stream LSE", ds.lse.cpu().numpy()[sel], el, LSE_TOL)
