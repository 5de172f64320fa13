"""GPU parity of kap_append_kv and kap_compact_view (bit-exact against the
oracle), and of the attention calls that read what they wrote: verify after
appending a window (the KV^{full,+} advance of Sec. 3.2) and decode over the
compact workspace (Sec. 3.1)."""
import numpy as np
import pytest
import torch

from oracle import kap_oracle as O
from paper_2607_24260_amd import kap as K
from paper_2607_24260_amd.workloads import kv_pool, make_workload, queries

from kap_testlib import (LSE_TOL, O_TOL, assert_close, dev_i32, gpu_plan, kv_of, oracle_plan,
                         oracle_pool, plan_view_arrays)

pytestmark = pytest.mark.gpu

_QDT = {"f32": torch.float32, "bf16": torch.bfloat16, "fp8": torch.bfloat16}


def small_pool(dtype, num_pages=37, Hkv=2, D=128, seed=5):
    k, v, sc = kv_pool(num_pages, Hkv, D, dtype, seed, "cuda")
    return K.KVCache(k, v, 4 * Hkv, _QDT[dtype], sc)


def host_pool(kv: K.KVCache, dtype):
    conv = lambda t: (t.cpu().view(torch.int16).numpy().view(np.uint16) if dtype == "bf16"
                      else t.cpu().numpy())
    sc = None if kv.kv_scales is None else kv.kv_scales.cpu().numpy()
    return O.KVPool(conv(kv.k_pages), conv(kv.v_pages), dtype, sc)


def new_tokens(n, Hkv, D, dtype, seed):
    g = torch.Generator(device="cuda").manual_seed(seed)
    x = torch.randn((n, Hkv, D), generator=g, device="cuda")
    if dtype == "f32":
        return x
    if dtype == "bf16":
        return x.to(torch.bfloat16)
    return (x * 16).clamp(-448, 448).to(torch.float8_e4m3fn).view(torch.uint8)


def to_host_bits(t, dtype):
    return t.cpu().view(torch.int16).numpy().view(np.uint16) if dtype == "bf16" else t.cpu().numpy()


@pytest.mark.parametrize("dtype", ["f32", "bf16", "fp8"])
def test_append_bit_exact(dtype):
    kv = small_pool(dtype)
    before = host_pool(kv, dtype)
    n = 45
    rng = np.random.default_rng(1)
    slots = rng.choice(37 * 16, size=n, replace=False).astype(np.int64)
    slots[[3, 17]] = -1                                  # padding
    slots[[8, 30]] = [37 * 16, 10**9]                    # past the pool: skipped, counted
    k_new, v_new = new_tokens(n, 2, 128, dtype, 2), new_tokens(n, 2, 128, dtype, 3)
    bad = torch.zeros(1, dtype=torch.int32, device="cuda")
    K.append_kv(kv, k_new, v_new, torch.as_tensor(slots).cuda(), bad)
    torch.cuda.synchronize()
    want, want_bad = O.append_kv(before, to_host_bits(k_new, dtype), to_host_bits(v_new, dtype),
                                 slots)
    got = host_pool(kv, dtype)
    assert int(bad.item()) == want_bad == 2
    assert np.array_equal(got.k_pages, want.k_pages)
    assert np.array_equal(got.v_pages, want.v_pages)


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
@pytest.mark.parametrize("q_len", [1, 5, 9])
def test_verify_after_appending_the_window(dtype, q_len):
    # ragged sequences of the fp8 recipe's lengths (bf16 or fp8 pools); the
    # window's K/V are appended at their slots, then verified on the GPU
    w = make_workload(5, device="cuda", batch=6, seq_len=9000, with_kv=True)
    if dtype == "bf16":
        k, v, _ = kv_pool(w.num_pages, 8, 128, "bf16", 77, "cuda")
        kv = K.KVCache(k, v, 32, torch.bfloat16)
    else:
        kv = kv_of(w)
    before = host_pool(kv, dtype)
    L = np.asarray(w.seq_lens, dtype=np.int64)
    fbt = np.asarray(w.full_block_table, dtype=np.int64)
    slots = np.concatenate([fbt[b, (L[b] - q_len + np.arange(q_len)) // 16] * 16
                            + (L[b] - q_len + np.arange(q_len)) % 16 for b in range(w.batch)])
    T = len(slots)
    k_new = new_tokens(T, 8, 128, dtype, 11)
    v_new = new_tokens(T, 8, 128, dtype, 12)
    K.append_kv(kv, k_new, v_new, torch.as_tensor(slots).cuda())
    q = queries((w.batch, q_len, 32, 128), "bf16", 128, 13, "cuda")
    o, lse = K.verify(kv, q, dev_i32(w.seq_lens), dev_i32(w.full_block_table), int(L.max()),
                      w.sm_scale)
    torch.cuda.synchronize()
    pool, _ = O.append_kv(before, to_host_bits(k_new, dtype), to_host_bits(v_new, dtype), slots)
    for b in (0, 3, 5):
        eo, el = O.verify(pool, q[b:b + 1].float().cpu().numpy(), L[b:b + 1], fbt[b:b + 1],
                          w.sm_scale)
        assert_close(f"verify b={b} O", o[b].cpu().numpy(), eo[0], O_TOL)
        assert_close(f"verify b={b} LSE", lse[b].cpu().numpy(), el[0], LSE_TOL)


@pytest.mark.parametrize("config,batch,seq_len,cap", [(2, 3, 4096, 64), (5, 8, 20000, 520)])
def test_compact_view_bit_exact_and_decode_unchanged(config, batch, seq_len, cap):
    w = make_workload(config, device="cuda", batch=batch, seq_len=seq_len)
    kv = kv_of(w)
    dtype = w.kv_dtype
    plan = gpu_plan(w)
    B = w.batch
    k = torch.zeros((B * cap,) + tuple(kv.k_pages.shape[1:]), dtype=kv.k_pages.dtype,
                    device="cuda")
    v = torch.zeros((B * cap,) + tuple(kv.v_pages.shape[1:]), dtype=kv.v_pages.dtype,
                    device="cuda")
    sc = None if kv.kv_scales is None else torch.zeros((B * cap, 2), device="cuda")
    dst = K.KVCache(k, v, kv.num_q_heads, kv.q_dtype, sc)
    table = K.compact_view(kv, plan["view_block_table"], plan["view_num_blocks"], cap, dst)
    torch.cuda.synchronize()
    nb = plan["view_num_blocks"].cpu().numpy()
    assert nb.max() <= cap, "the capacity is chosen to hold every view"
    want_pool, want_table = O.compact_view(host_pool(kv, dtype),
                                           plan["view_block_table"].cpu().numpy(), nb, cap)
    got_table = table.cpu().numpy()
    assert np.array_equal(got_table, want_table)
    got = host_pool(dst, dtype)
    assert np.array_equal(got.k_pages, want_pool.k_pages)
    assert np.array_equal(got.v_pages, want_pool.v_pages)
    if sc is not None:
        assert np.array_equal(got.scales, want_pool.scales)
    # decode over the compact workspace = decode over the zero-copy view
    q = w.q_decode[0]
    o1, l1 = K.selected_decode(kv, q, dev_i32(w.seq_lens), plan["view_block_table"],
                               plan["view_logical_block"], plan["view_num_blocks"],
                               w.max_pages_per_seq, w.sm_scale)
    lblk = plan["view_logical_block"][:, :cap].contiguous()
    o2, l2 = K.selected_decode(dst, q, dev_i32(w.seq_lens), table, lblk,
                               plan["view_num_blocks"], cap, w.sm_scale)
    torch.cuda.synchronize()
    assert_close("compact decode O", o2.cpu().numpy(), o1.cpu().numpy(), 1e-6)
    assert_close("compact decode LSE", l2.cpu().numpy(), l1.cpu().numpy(), 1e-6)
    # and against the oracle on the compact pool
    vbt, vlb, nbo = plan_view_arrays(oracle_plan(w), w.max_pages_per_seq)
    eo, el = O.selected_decode(want_pool, q.float().cpu().numpy(), w.seq_lens, want_table,
                               vlb[:, :cap], nbo, w.sm_scale)
    assert_close("compact decode vs oracle O", o2.cpu().numpy(), eo, O_TOL)
    assert_close("compact decode vs oracle LSE", l2.cpu().numpy(), el, LSE_TOL)


def test_compact_view_at_128k_pages_match_source():
    # the 128K workload's 5.5% views (<= 451 pages per sequence) into a
    # 512-page-per-sequence workspace: every copied page equals its source
    w = make_workload(4, device="cuda", n_decode=1, n_verify=1)
    kv = kv_of(w)
    plan = gpu_plan(w)
    cap = 512
    B = w.batch
    dst = K.KVCache(torch.empty((B * cap,) + tuple(kv.k_pages.shape[1:]), dtype=kv.k_pages.dtype,
                                device="cuda"),
                    torch.empty((B * cap,) + tuple(kv.v_pages.shape[1:]), dtype=kv.v_pages.dtype,
                                device="cuda"), 32, torch.bfloat16)
    table = K.compact_view(kv, plan["view_block_table"], plan["view_num_blocks"], cap, dst)
    torch.cuda.synchronize()
    nb = plan["view_num_blocks"].long()
    vbt = plan["view_block_table"].long()
    for b in range(B):
        n = int(nb[b])
        assert torch.equal(table[b, :n].long(), b * cap + torch.arange(n, device="cuda"))
        assert bool((table[b, n:] == -1).all())
        src = vbt[b, :n]
        assert torch.equal(dst.k_pages[b * cap:b * cap + n], kv.k_pages[src])
        assert torch.equal(dst.v_pages[b * cap:b * cap + n], kv.v_pages[src])
