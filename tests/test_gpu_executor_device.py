"""The device-side access-mode policy (kap_fallback_update) against the host
FallbackPolicy / ViewBuilder (whose rule the CPU tests pin), and HIP-graph
replays of a whole device-resident stream against its eager run."""
import numpy as np
import pytest
import torch

from paper_2607_24260_amd import kap as K
from paper_2607_24260_amd.executor import (FULL, DeviceStream, FallbackPolicy, ViewBuilder,
                                           accepted_counts, run_stream)
from paper_2607_24260_amd.workloads import make_workload

from kap_testlib import dev_i32, gpu_plan, kv_of

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("window", [1, 4, 7])
def test_device_policy_matches_host(window):
    # 40 sequences with assorted s (including plan failures), 14 cycles of
    # random gammas and geometric(0.6) - 1 accept draws
    rng = np.random.default_rng(window)
    B, C, stride, cap = 40, 14, 96, 64
    L = rng.integers(100, 1500, B).astype(np.int32)
    npg = -(-L // 16)
    vtok = np.minimum(rng.integers(16, 800, B), L).astype(np.int32)
    status = np.where(rng.random(B) < 0.15, K.KAP_PLAN_OVER_CAPACITY, K.KAP_PLAN_OK).astype(np.int32)
    sel_nb = np.minimum(-(-vtok // 16), cap).astype(np.int32)
    sel_bt = rng.integers(0, 5000, (B, cap)).astype(np.int32)
    sel_lb = rng.integers(0, 90, (B, cap)).astype(np.int32)
    fbt = rng.integers(0, 5000, (B, stride)).astype(np.int32)
    gammas = rng.choice([2, 4, 8], C)
    draws = (rng.geometric(0.6, (C, B)) - 1).astype(np.int32)

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

    policy = FallbackPolicy(vtok / L.astype(np.float64), status == K.KAP_PLAN_OK, window=window)
    views = ViewBuilder(plan, dev_i32(fbt), L, cap)
    views.apply(policy.mode)

    def check(tag):
        torch.cuda.synchronize()
        assert np.array_equal(mode.cpu().numpy(), policy.mode), tag
        assert np.array_equal(vnb.cpu().numpy(), views.vnb.cpu().numpy()), tag
        got_bt, got_lb = vbt.cpu().numpy(), vlb.cpu().numpy()
        want_bt, want_lb = views.vbt.cpu().numpy(), views.vlb.cpu().numpy()
        for b in range(B):
            n = int(vnb[b])
            assert np.array_equal(got_bt[b, :n], want_bt[b, :n]), (tag, b)
            assert np.array_equal(got_lb[b, :n], want_lb[b, :n]), (tag, b)

    check("reset")
    for c in range(C):
        d = dev_i32(draws[c])
        K.bind_fallback_update(False, window, int(gammas[c]), d, *common)()
        policy.update(accepted_counts(draws[c], gammas[c]), int(gammas[c]))
        views.apply(policy.mode)
        check(f"cycle {c}")
    assert (policy.flipped_at >= 2).any(), "no sequence switched during the cycles"
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
    # the same stream with the host policy (run_stream): identical modes and
    # identical verify outputs, call by call
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
    assert np.array_equal(ds.mode.cpu().numpy(), res.policy.mode)
    for j, o, l in res.verify_out:
        assert torch.equal(o, ds.ver_out[j][0]) and torch.equal(l, ds.ver_out[j][1]), j
    (idx, o, l, _), = res.decode_out
    assert idx == last and torch.equal(o, ds.out) and torch.equal(l, ds.lse)


def test_token_granular_device_stream():
    # the ragged fp8 stream over token-granular views (Sec. 3.1 mask in the
    # device-resident cycle): modes follow the host policy with the token
    # plan's s; every active row holds the plan's pages and masks (mode 0) or
    # the full table with all-ones masks (mode 1); the last decode equals a
    # masked call over those rows and, for sampled sequences, the oracle
    from oracle import kap_oracle as O

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
    vt = plan["view_tokens"].cpu().numpy()
    ok = plan["plan_status"].cpu().numpy() == K.KAP_PLAN_OK
    policy = FallbackPolicy(vt / L.astype(np.float64), ok, window=4)
    draws = np.asarray(w.accept_draws)
    for c, q in enumerate(w.q_verify):
        g = q.shape[1] - 1
        policy.update(accepted_counts(draws[c], g), g)
    mode = ds.mode.cpu().numpy()
    assert np.array_equal(mode, policy.mode)
    assert (mode == 0).any() and (mode == FULL).any(), "want both access modes in the stream"
    vnb, vbt = ds.vnb.cpu().numpy(), ds.vbt.cpu().numpy()
    vlb, vmk = ds.vlb.cpu().numpy(), ds.vmask.cpu().numpy().astype(np.int64) & 0xFFFFFFFF
    pbt, plb = plan["view_block_table"].cpu().numpy(), plan["view_logical_block"].cpu().numpy()
    pmk = plan["view_token_mask"].cpu().numpy().astype(np.int64) & 0xFFFFFFFF
    pnb = plan["view_num_blocks"].cpu().numpy()
    fbt = np.asarray(w.full_block_table)
    for b in range(w.batch):
        n = int(vnb[b])
        if mode[b] == 0:
            assert n == pnb[b]
            assert np.array_equal(vbt[b, :n], pbt[b, :n]) and np.array_equal(vlb[b, :n], plb[b, :n])
            assert np.array_equal(vmk[b, :n], pmk[b, :n]), b
        else:
            assert n == -(-L[b] // 16)
            assert np.array_equal(vbt[b, :n], fbt[b, :n]) and np.all(vmk[b, :n] == 0xFFFF), b
    last = w.q_decode.shape[0] - 1
    o, l = K.selected_decode(kv, w.q_decode[last], ds.seq_lens, ds.vbt, ds.vlb, ds.vnb,
                             ds.vbt.shape[1], w.sm_scale, view_token_mask=ds.vmask)
    torch.cuda.synchronize()
    assert torch.equal(o, ds.out) and torch.equal(l, ds.lse)
    sel = [b for b in range(w.batch) if mode[b] == 0][:2] + [b for b in range(w.batch)
                                                              if mode[b] == FULL][:2]
    eo, el = O.selected_decode(oracle_pool(w), w.q_decode[last].float().cpu().numpy()[sel],
                               L[sel], vbt[sel], vlb[sel], vnb[sel], w.sm_scale,
                               view_token_mask=vmk[sel])
    assert_close("token stream O", o.cpu().numpy()[sel], eo, O_TOL)
    assert_close("token stream LSE", l.cpu().numpy()[sel], el, LSE_TOL)
