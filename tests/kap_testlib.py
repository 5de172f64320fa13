"""Helpers shared by the GPU parity tests: move a seeded workload to the GPU,
run the library through the Python binding (which calls the C ABI), and build
the oracle's view of the very same stored bits."""
from __future__ import annotations

import numpy as np
import torch

from oracle import kap_oracle as O
from paper_2607_24260_amd import kap as K

# Tolerances for bf16 / fp8 / fp32 inputs against the fp64 oracle.
O_TOL = 2e-3
LSE_TOL = 1e-3


def dev_i32(x, device="cuda"):
    return torch.as_tensor(np.asarray(x, dtype=np.int32)).to(device)


def kv_of(w, replica=0) -> K.KVCache:
    qdt = torch.float32 if w.q_dtype == "f32" else torch.bfloat16
    return K.KVCache(w.k_pages[replica], w.v_pages[replica], w.num_q_heads, qdt,
                     w.kv_scales[replica])


def oracle_pool(w, replica=0) -> O.KVPool:
    k, v, sc = w.host_kv(replica)
    return O.KVPool(k, v, w.kv_dtype, sc)


def gpu_plan(w, budget=None, policy=K.KAP_SELECT_SKIP, capacity=None):
    cap = w.max_pages_per_seq if capacity is None else capacity
    b = w.budget if budget is None else budget
    out = K.compile_plan(
        dev_i32(w.seq_lens), dev_i32(w.full_block_table), dev_i32(w.span_offsets),
        dev_i32(w.span_start), dev_i32(w.span_len),
        torch.as_tensor(np.asarray(w.span_prior, dtype=np.float32)).cuda(),
        dev_i32(w.prefix), dev_i32(w.suffix), dev_i32(b), num_pages=w.num_pages,
        view_capacity=cap, policy=policy)
    torch.cuda.synchronize()
    return out


def oracle_plan(w, budget=None, policy=O.SELECT_SKIP, capacity=None):
    cap = w.max_pages_per_seq if capacity is None else capacity
    b = w.budget if budget is None else budget
    return O.compile_plan(w.seq_lens, w.full_block_table, w.span_offsets, w.span_start,
                          w.span_len, w.span_prior, w.prefix, w.suffix, b, policy,
                          w.num_pages, cap)


def assert_plan_equal(gpu: dict, plans, span_offsets):
    """Bit-exact comparison of every plan output."""
    st = gpu["plan_status"].cpu().numpy()
    nb = gpu["view_num_blocks"].cpu().numpy()
    vt = gpu["view_tokens"].cpu().numpy()
    tk = gpu["spans_taken"].cpu().numpy()
    vbt = gpu["view_block_table"].cpu().numpy()
    vlb = gpu["view_logical_block"].cpu().numpy()
    sel = gpu["span_selected"].cpu().numpy()
    for b, p in enumerate(plans):
        assert st[b] == p.status, (b, st[b], p.status)
        assert nb[b] == p.num_blocks, (b, nb[b], p.num_blocks)
        assert vt[b] == p.view_tokens, (b, vt[b], p.view_tokens)
        assert tk[b] == p.spans_taken, (b, tk[b], p.spans_taken)
        n = p.num_blocks
        assert np.array_equal(vlb[b, :n], np.asarray(p.logical_blocks, dtype=np.int32)), b
        assert np.array_equal(vbt[b, :n], np.asarray(p.block_table, dtype=np.int32)), b
        if p.status != O.PLAN_BAD_SPANS:
            lo, hi = int(span_offsets[b]), int(span_offsets[b + 1])
            assert np.array_equal(sel[lo:hi], np.asarray(p.span_selected, dtype=np.int32)), b


def plan_view_arrays(plans, capacity):
    """Host view arrays from oracle plans (for feeding the decode oracle)."""
    B = len(plans)
    vbt = np.zeros((B, max(capacity, 1)), dtype=np.int64)
    vlb = np.zeros((B, max(capacity, 1)), dtype=np.int64)
    nb = np.zeros(B, dtype=np.int64)
    for b, p in enumerate(plans):
        nb[b] = p.num_blocks
        vbt[b, :p.num_blocks] = p.block_table
        vlb[b, :p.num_blocks] = p.logical_blocks
    return vbt, vlb, nb


def full_view(w):
    """All-blocks view (full-context decode) as device tensors."""
    B = w.batch
    stride = w.fbt_stride
    npg = np.array([-(-int(L) // 16) for L in w.seq_lens], dtype=np.int32)
    lblk = np.tile(np.arange(stride, dtype=np.int32), (B, 1))
    return (dev_i32(w.full_block_table), dev_i32(lblk), dev_i32(npg), int(npg.max()))


def assert_close(name, got, want, tol, mask=None):
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    if mask is not None:
        got, want = got[mask], want[mask]
    both_inf = np.isinf(got) & np.isinf(want) & (np.sign(got) == np.sign(want))
    with np.errstate(invalid="ignore"):          # inf - inf where both_inf masks it
        diff = np.where(both_inf, 0.0, np.abs(got - want))
    worst = float(np.nanmax(diff)) if diff.size else 0.0
    assert not np.isnan(diff).any(), f"{name}: NaN"
    assert worst <= tol, f"{name}: max abs err {worst:.3e} > {tol:.1e}"
    return worst
