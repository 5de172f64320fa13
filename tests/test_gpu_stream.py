"""GPU run of the ragged fp8 workload's interleaved stream (proposal decode and
gamma in {2,4,8} verify windows, geometric(0.6) accept lengths, fallback to
full-context access) with outputs checked against the oracle: a decode step
after fallbacks (mixed selected / full views) and the last verify window."""
import numpy as np
import pytest
import torch

from oracle import kap_oracle as O
from paper_2607_24260_amd import kap as K
from paper_2607_24260_amd.executor import FULL, run_stream
from paper_2607_24260_amd.workloads import make_workload

from kap_testlib import LSE_TOL, O_TOL, assert_close, gpu_plan, kv_of, oracle_pool

pytestmark = pytest.mark.gpu


def oracle_views(w, plans, mode):
    B, cap = w.batch, w.fbt_stride
    vbt = np.zeros((B, cap), np.int64)
    vlb = np.zeros((B, cap), np.int64)
    nb = np.zeros(B, np.int64)
    for b, p in enumerate(plans):
        if mode[b] == FULL:
            n = -(-int(w.seq_lens[b]) // 16)
            vbt[b, :n] = w.full_block_table[b, :n]
            vlb[b, :n] = np.arange(n)
            nb[b] = n
        else:
            vbt[b, :p.num_blocks] = p.block_table
            vlb[b, :p.num_blocks] = p.logical_blocks
            nb[b] = p.num_blocks
    return vbt, vlb, nb


def test_config5_stream_with_fallback():
    # 16 sequences of the ragged fp8 recipe (lengths 4K..64K), 8 cycles
    w = make_workload(5, device="cuda", batch=16, seq_len=65536, n_verify=8)
    kv = kv_of(w)
    plan = gpu_plan(w)
    n_dec = w.q_decode.shape[0]
    res = run_stream(w, kv, plan, keep_outputs={("decode", i) for i in range(n_dec)} |
                     {("verify", len(w.q_verify) - 1)})
    torch.cuda.synchronize()
    assert (res.policy.mode == FULL).any(), "the recipe's accept law should trigger fallbacks"
    assert len(res.decode_out) == n_dec
    # steps to check: the first, the one with the most even selected/full mix, the last
    mixes = [abs(int((m == FULL).sum()) - w.batch // 2) for _, _, _, m in res.decode_out]
    picks = sorted({0, int(np.argmin(mixes)), n_dec - 1})
    pool = oracle_pool(w)
    plans = O.compile_plan(w.seq_lens, w.full_block_table, w.span_offsets, w.span_start,
                           w.span_len, w.span_prior, w.prefix, w.suffix, w.budget,
                           O.SELECT_SKIP, w.num_pages, w.max_pages_per_seq)
    for k in picks:
        idx, o, l, mode_then = res.decode_out[k]
        vbt, vlb, nb = oracle_views(w, plans, mode_then)
        qh = w.q_decode[idx].float().cpu().numpy()
        eo, el = O.selected_decode(pool, qh, w.seq_lens, vbt, vlb, nb, w.sm_scale)
        assert_close(f"stream decode {idx} O", o.cpu().numpy(), eo, O_TOL)
        assert_close(f"stream decode {idx} LSE", l.cpu().numpy(), el, LSE_TOL)
    mixed = res.decode_out[picks[len(picks) // 2]][3]
    assert 0 < int((mixed == FULL).sum()) < w.batch, "a checked step mixes both view kinds"
    # last verify window: sequences 0 and 7, all heads
    j, ov, lv = res.verify_out[0]
    ev, elv = O.verify(pool, w.q_verify[j].float().cpu().numpy(), w.seq_lens,
                       w.full_block_table, w.sm_scale, batches=[0, 7])
    assert_close("stream verify O", ov.cpu().numpy()[[0, 7]], ev[[0, 7]], O_TOL)
    assert_close("stream verify LSE", lv.cpu().numpy()[[0, 7]], elv[[0, 7]], LSE_TOL)
