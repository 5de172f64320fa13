"""CPU pins of the oracle's slot-mapped KV append and view compaction
(Sec. 3.1 slot mappings / compact workspace, Alg. 1 AssignCompactSlots and
BuildBlockTable; Sec. 3.2 KV^{full,+}).

The append is pinned through the attention it feeds: a verify window whose
K/V were written by ``append_kv`` must equal torch's scaled-dot-product
attention over the old logical sequence (read by torch's own decoders)
followed by the new tokens (decoded by torch from the raw input bits). The
compaction is pinned by decode invariance and by the table's closed form."""
import numpy as np
import pytest
import torch

from oracle import kap_oracle as O

from test_oracle_attention import logical_kv, make_pool, sdpa_rows

P = O.PAGE


def torch_tokens(bits, dtype, scale_rows=None):
    """Raw stored values [T][Hkv][D] -> fp64 via torch's decoders (per-token
    scale rows [T][Hkv] for fp8)."""
    t = torch.from_numpy(np.ascontiguousarray(bits))
    if dtype == "f32":
        x = t.to(torch.float64)
    elif dtype == "bf16":
        x = t.view(torch.int16).view(torch.bfloat16).to(torch.float64)
    else:
        x = t.view(torch.float8_e4m3fn).to(torch.float64)
    if scale_rows is not None:
        x = x * torch.as_tensor(scale_rows, dtype=torch.float64)[..., None]
    return x


def random_new_tokens(rng, n, Hkv, D, dtype):
    if dtype == "f32":
        return rng.standard_normal((n, Hkv, D)).astype(np.float32)
    x = torch.from_numpy(rng.standard_normal((n, Hkv, D)).astype(np.float32))
    if dtype == "bf16":
        return x.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    return (x * 16).clamp(-448, 448).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


@pytest.mark.parametrize("dtype", ["f32", "bf16", "fp8"])
@pytest.mark.parametrize("n_new", [1, 5, 17])
def test_appended_window_verify_matches_sdpa(dtype, n_new):
    rng = np.random.default_rng(100 + n_new)
    Hkv, G, D, L = 2, 4, 16, 70 + n_new
    npg = -(-L // P)
    pool = make_pool(npg + 3, Hkv, D, dtype, seed=7)
    fbt = rng.permutation(npg + 3)[:npg]
    k_new = random_new_tokens(rng, n_new, Hkv, D, dtype)
    v_new = random_new_tokens(rng, n_new, Hkv, D, dtype)
    pos = np.arange(L - n_new, L)
    slots = fbt[pos // P] * P + pos % P
    new_pool, bad = O.append_kv(pool, k_new, v_new, slots)
    assert bad == 0
    q = (rng.standard_normal((1, n_new, Hkv * G, D)) / 4).astype(np.float64)
    o, lse = O.verify(new_pool, q, [L], fbt[None], 1.0)

    # expected: the old sequence's first L - n_new tokens, then the new tokens
    K_old, V_old = logical_kv(pool, fbt, L - n_new)                  # [Hkv][L-n][D]
    srows = None
    if dtype == "fp8":
        srows = np.stack([pool.scales[fbt[pos // P], 0]] * Hkv, axis=1)
        vrows = np.stack([pool.scales[fbt[pos // P], 1]] * Hkv, axis=1)
    Kn = torch_tokens(k_new, dtype, srows).permute(1, 0, 2)
    Vn = torch_tokens(v_new, dtype, vrows if dtype == "fp8" else None).permute(1, 0, 2)
    K = torch.cat([K_old, Kn], 1).repeat_interleave(G, 0)
    V = torch.cat([V_old, Vn], 1).repeat_interleave(G, 0)
    mask = torch.arange(L)[None, :] <= (L - n_new + torch.arange(n_new))[:, None]
    eo, el = sdpa_rows(torch.as_tensor(q[0]).transpose(0, 1), K, V, mask, 1.0)
    np.testing.assert_allclose(o[0], eo.transpose(0, 1).numpy(), rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse[0], el.transpose(0, 1).numpy(), rtol=0, atol=1e-12)


def test_append_reads_back_through_the_layout():
    rng = np.random.default_rng(3)
    pool = make_pool(5, 3, 32, "bf16", seed=1)
    k_new = random_new_tokens(rng, 4, 3, 32, "bf16")
    v_new = random_new_tokens(rng, 4, 3, 32, "bf16")
    slots = np.array([0, 17, 79, 40])
    new_pool, _ = O.append_kv(pool, k_new, v_new, slots)
    for t, s in enumerate(slots):
        page, off = divmod(int(s), P)
        for g in range(3):
            # K chunk c of token off holds dims 8c..8c+7; V row d holds dim d
            for d in range(32):
                assert new_pool.k_pages[page, g, d // 8, off, d % 8] == k_new[t, g, d]
                assert new_pool.v_pages[page, g, d, off] == v_new[t, g, d]


def test_append_skips_padding_and_counts_out_of_range():
    rng = np.random.default_rng(4)
    pool = make_pool(3, 2, 16, "fp8", seed=2)
    k_new = random_new_tokens(rng, 3, 2, 16, "fp8")
    v_new = random_new_tokens(rng, 3, 2, 16, "fp8")
    new_pool, bad = O.append_kv(pool, k_new, v_new, [-1, 3 * P, 3 * P + 5])
    assert bad == 2
    assert np.array_equal(new_pool.k_pages, pool.k_pages)
    assert np.array_equal(new_pool.v_pages, pool.v_pages)
    assert np.array_equal(new_pool.scales, pool.scales)


def test_planted_append_layout_mistake_is_caught(monkeypatch):
    """A writer that stores K chunks transposed (dim 8e + c instead of 8c + e)
    must fail the SDPA pin."""
    def wrong_append(pool, k_new, v_new, slots):
        k = np.array(pool.k_pages, copy=True)
        v = np.array(pool.v_pages, copy=True)
        _, Hkv, C, _, E = k.shape
        for t, s in enumerate(slots):
            page, off = divmod(int(s), P)
            k[page, :, :, off, :] = np.asarray(k_new[t]).reshape(Hkv, E, C).transpose(0, 2, 1)
            v[page, :, :, off] = np.asarray(v_new[t])
        return O.KVPool(k, v, pool.dtype, pool.scales), 0
    monkeypatch.setattr(O, "append_kv", wrong_append)
    with pytest.raises(AssertionError):
        test_appended_window_verify_matches_sdpa("f32", 5)


def _plan_like_view(rng, B, npages, cap, L):
    vbt = np.full((B, cap + 4), -7, dtype=np.int64)
    vlb = np.zeros_like(vbt)
    nb = np.zeros(B, dtype=np.int64)
    for b in range(B):
        n = int(rng.integers(0, cap + 3))          # some views longer than the capacity
        lb = np.sort(rng.choice(-(-L // P), size=min(n, -(-L // P)), replace=False))
        nb[b] = len(lb)
        vlb[b, :len(lb)] = lb
        vbt[b, :len(lb)] = rng.integers(-1, npages + 1, len(lb))   # a few invalid ids
    return vbt, vlb, nb


@pytest.mark.parametrize("dtype", ["f32", "bf16", "fp8"])
def test_compact_view_table_and_bytes(dtype):
    rng = np.random.default_rng(11)
    pool = make_pool(12, 2, 16, dtype, seed=5)
    vbt, vlb, nb = _plan_like_view(rng, 4, 12, 6, 150)
    cpool, table = O.compact_view(pool, vbt, nb, 6)
    for b in range(4):
        for j in range(6):
            p = vbt[b, j] if j < nb[b] else -1
            if j < nb[b] and 0 <= p < 12:
                assert table[b, j] == b * 6 + j
                assert np.array_equal(cpool.k_pages[b * 6 + j], pool.k_pages[p])
                assert np.array_equal(cpool.v_pages[b * 6 + j], pool.v_pages[p])
                if dtype == "fp8":
                    assert np.array_equal(cpool.scales[b * 6 + j], pool.scales[p])
            else:
                assert table[b, j] == -1


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_decode_over_compact_view_is_identical(dtype):
    rng = np.random.default_rng(12)
    B, Hkv, G, D, L = 3, 2, 4, 16, 150
    pool = make_pool(20, Hkv, D, dtype, seed=6)
    vbt, vlb, nb = _plan_like_view(rng, B, 20, 8, L)
    nb = np.minimum(nb, 8)                        # views within the capacity
    q = rng.standard_normal((B, Hkv * G, D)) / 4
    seq = np.full(B, L)
    o1, l1 = O.selected_decode(pool, q, seq, vbt, vlb, nb, 1.0)
    cpool, table = O.compact_view(pool, vbt, nb, 8)
    o2, l2 = O.selected_decode(cpool, q, seq, table, vlb[:, :8], nb, 1.0)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)


def test_invalid_view_pages_contribute_nothing():
    """Decode over a view with out-of-pool page ids equals decode over the same
    view with those entries removed (the documented reading), and differs from
    reading a wrapped-around page."""
    rng = np.random.default_rng(13)
    pool = make_pool(9, 2, 16, "bf16", seed=8)
    vbt = np.array([[3, -1, 5, 9, 1]])
    vlb = np.array([[0, 1, 2, 3, 4]])
    q = rng.standard_normal((1, 8, 16)) / 4
    o1, l1 = O.selected_decode(pool, q, [80], vbt, vlb, [5], 1.0)
    o2, l2 = O.selected_decode(pool, q, [80], np.array([[3, 5, 1]]), np.array([[0, 2, 4]]), [3], 1.0)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)
    o3, _ = O.selected_decode(pool, q, [80], np.array([[3, 8, 5, 1]]), np.array([[0, 1, 2, 4]]), [4], 1.0)
    assert not np.allclose(o1, o3)
