"""kap_selected_decode_noalloc (the allocation-free decode entry point, for
callers that cannot allocate) against kap_selected_decode with a workspace:
two calls in a row through the C ABI, the second with a smaller input, each
matching the workspace call to the parity bar (and in fact bit for bit: the
same kernels run on the same inputs), plus a generic-path call and the size
limits."""
import numpy as np
import pytest
import torch

from paper_2607_24260_amd import kap as K
from paper_2607_24260_amd.workloads import make_workload

from kap_testlib import LSE_TOL, O_TOL, assert_close, dev_i32, gpu_plan, kv_of

pytestmark = pytest.mark.gpu


def _both(w, num_splits=0, step=0):
    kv = kv_of(w)
    plan = gpu_plan(w)
    cap = w.max_pages_per_seq
    args = (kv, w.q_decode[step], dev_i32(w.seq_lens), plan["view_block_table"],
            plan["view_logical_block"], plan["view_num_blocks"], cap, w.sm_scale)
    o1, l1 = K.selected_decode(*args, num_splits=num_splits)
    o2, l2 = K.selected_decode_noalloc(*args, num_splits=num_splits)
    torch.cuda.synchronize()
    assert_close("noalloc O", o2.cpu().numpy(), o1.cpu().numpy(), O_TOL)
    assert_close("noalloc LSE", l2.cpu().numpy(), l1.cpu().numpy(), LSE_TOL)
    assert torch.equal(o1, o2) and torch.equal(l1, l2)
    assert torch.isfinite(l2).all()


def test_two_calls_in_a_row_second_smaller():
    # 1: the 128K workload (4 sequences, 5.5% views; the balanced split map,
    #    arrival counters and ~4 MB of partials in the scratch)
    print("noalloc call 1: workload 4 (B=4, L=131072, bf16)", flush=True)
    w = make_workload(4, device="cuda", n_decode=1, n_verify=1)
    _both(w)
    del w
    torch.cuda.empty_cache()
    # 2: smaller -- 3 ragged fp8 sequences, three uniform splits
    print("noalloc call 2: workload 5 (B=3, fp8, num_splits=3)", flush=True)
    w = make_workload(5, device="cuda", batch=3, seq_len=6000, n_verify=1)
    _both(w, num_splits=3)


def test_generic_path_and_repeat():
    # head_dim 64 (generic kernel + separate merge, partials in the scratch),
    # twice, then the tuned path again: the scratch keeps nothing a call needs
    print("noalloc: generic path D=64, bf16", flush=True)
    w = make_workload(2, device="cuda", batch=3, seq_len=3000, n_decode=2, n_verify=1,
                      head_dim=64)
    _both(w, step=0)
    _both(w, step=1)
    print("noalloc: tuned path after the generic one", flush=True)
    w = make_workload(2, device="cuda", batch=2, seq_len=2000, n_decode=1, n_verify=1)
    _both(w)


def test_calls_beyond_the_scratch_are_refused_before_launch():
    # generic path (fp32): 8 sequences x 32 heads x 128 splits of partials
    # (> 16 MiB) -- refused; the pool and tables are tiny, nothing runs
    print("noalloc: size limits", flush=True)
    dev = "cuda"
    B, Hq, Hkv, D, cap = 8, 32, 8, 128, 8192
    k = torch.zeros((4, Hkv, D // 8, 16, 8), dtype=torch.float32, device=dev)
    v = torch.zeros((4, Hkv, D, 16), dtype=torch.float32, device=dev)
    kv = K.KVCache(k, v, Hq, torch.float32)
    q = torch.zeros((B, Hq, D), dtype=torch.float32, device=dev)
    tab = torch.zeros((B, cap), dtype=torch.int32, device=dev)
    n = torch.ones(B, dtype=torch.int32, device=dev)
    with pytest.raises(K.KapError) as e:
        K.selected_decode_noalloc(kv, q, n * 16, tab, tab, n, cap, 1.0)
    assert e.value.status == K.KAP_ERR_WORKSPACE_TOO_SMALL and "scratch" in str(e.value)
    # tuned path, uniform splits: 600 x 8 (sequence, KV head) units need more
    # arrival counters than the scratch holds
    B = 600
    kb = torch.zeros((4, Hkv, D // 8, 16, 8), dtype=torch.bfloat16, device=dev)
    vb = torch.zeros((4, Hkv, D, 16), dtype=torch.bfloat16, device=dev)
    kvb = K.KVCache(kb, vb, Hq, torch.bfloat16)
    qb = torch.zeros((B, Hq, D), dtype=torch.bfloat16, device=dev)
    tb = torch.zeros((B, 4), dtype=torch.int32, device=dev)
    nb = torch.ones(B, dtype=torch.int32, device=dev)
    with pytest.raises(K.KapError) as e:
        K.selected_decode_noalloc(kvb, qb, nb * 16, tb, tb, nb, 4, 1.0, num_splits=2)
    assert e.value.status == K.KAP_ERR_UNSUPPORTED and "counters" in str(e.value)
    # the same batch without split partials runs (one split per unit)
    o, l = K.selected_decode_noalloc(kvb, qb, nb * 16, tb, tb, nb, 4, 1.0, num_splits=1)
    torch.cuda.synchronize()
    assert torch.all(o == 0) and torch.isfinite(l).all()
