"""CPU pins for the oracle's attention (selected-view decode, full-KV verify,
LSE merge) and its decoding of stored KV bits.

Pins, none of which reuse the oracle's own formulas:
* brute force through an independent route: the logical K/V sequence is
  rebuilt with torch indexing, visibility becomes a boolean mask over logical
  positions, and torch's fp64 scaled_dot_product_attention / logsumexp give
  the expected values;
* closed forms (one visible token, constant keys, two tokens);
* invariants of the definitions (all-blocks view = verify with one query,
  order of view pages, split + merge, GQA = replicated MHA, verify row i =
  decode over the first L - q_len + i + 1 tokens);
* torch's own bfloat16 / float8_e4m3fn decoders for every bit pattern;
* planted mistakes in a copy of the oracle must fail the brute-force pin.
"""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import kap_oracle as O

P = 16


# --------------------------------------------------------------------------
# tiny random pools
# --------------------------------------------------------------------------

def make_pool(num_pages, Hkv, D, dtype, seed):
    """Random pool in the stored layout: K [P][Hkv][D/8][16][8], V [P][Hkv][D][16]."""
    g = torch.Generator().manual_seed(seed)
    k = torch.randn((num_pages, Hkv, D // 8, P, 8), generator=g)
    v = torch.randn((num_pages, Hkv, D, P), generator=g)
    if dtype == "f32":
        return O.KVPool(k.numpy(), v.numpy(), "f32")
    if dtype == "bf16":
        kb = k.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        vb = v.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        return O.KVPool(kb, vb, "bf16")
    sk = k.abs().flatten(1).amax(dim=1) / 448.0
    sv = v.abs().flatten(1).amax(dim=1) / 448.0
    kq = (k / sk[:, None, None, None, None]).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    vq = (v / sv[:, None, None, None]).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    return O.KVPool(kq, vq, "fp8", torch.stack([sk, sv], 1).numpy())


def key_vec(pool, page, g, t):
    """Stored K of token t (float64), read from the chunked layout by hand."""
    return np.concatenate([pool.k_pages[page, g, c, t] for c in range(pool.k_pages.shape[2])]
                          ).astype(np.float64)


def torch_values(pool):
    """Pool contents as fp64 torch tensors via torch's own dtype decoders:
    K [pages][Hkv][P][D] (chunks merged back), V [pages][Hkv][P][D]
    (V transposed back)."""
    if pool.dtype == "f32":
        k, v = torch.from_numpy(pool.k_pages), torch.from_numpy(pool.v_pages)
    elif pool.dtype == "bf16":
        k = torch.from_numpy(pool.k_pages.view(np.int16)).view(torch.bfloat16)
        v = torch.from_numpy(pool.v_pages.view(np.int16)).view(torch.bfloat16)
    else:
        k = torch.from_numpy(pool.k_pages).view(torch.float8_e4m3fn)
        v = torch.from_numpy(pool.v_pages).view(torch.float8_e4m3fn)
    nP, H, C, T, E = k.shape
    k = k.to(torch.float64).permute(0, 1, 3, 2, 4).reshape(nP, H, T, C * E)
    v = v.to(torch.float64).transpose(2, 3)
    if pool.dtype == "fp8":
        sc = torch.from_numpy(pool.scales).to(torch.float64)
        k = k * sc[:, 0, None, None, None]
        v = v * sc[:, 1, None, None, None]
    return k, v


def logical_kv(pool, fbt_row, L):
    """Logical K/V sequence [Hkv][L][D] of one sequence."""
    k, v = torch_values(pool)
    npg = -(-L // P)
    idx = torch.as_tensor(np.asarray(fbt_row[:npg], dtype=np.int64))
    K = k[idx].permute(1, 0, 2, 3).reshape(k.shape[1], npg * P, -1)[:, :L]
    V = v[idx].permute(1, 0, 2, 3).reshape(v.shape[1], npg * P, -1)[:, :L]
    return K, V


def sdpa_rows(q, K, V, mask, scale):
    """q [Hq][R][D], K/V [Hq][L][D], mask [R][L] bool -> o [Hq][R][D], lse [Hq][R]."""
    o = F.scaled_dot_product_attention(q[None], K[None], V[None], attn_mask=mask[None, None],
                                       scale=scale)[0]
    z = scale * (q @ K.transpose(-1, -2))
    lse = torch.logsumexp(z.masked_fill(~mask[None], -math.inf), dim=-1)
    return o, lse


def brute_decode(pool, q, seq_lens, fbt, vbt_lb, sm_scale):
    """Expected decode via logical positions: a token is visible iff its
    logical page is in the view."""
    B, Hq, D = q.shape
    Hkv = pool.k_pages.shape[1]
    G = Hq // Hkv
    o = np.zeros((B, Hq, D))
    lse = np.zeros((B, Hq))
    for b in range(B):
        L = int(seq_lens[b])
        K, V = logical_kv(pool, fbt[b], L)
        K, V = K.repeat_interleave(G, 0), V.repeat_interleave(G, 0)
        vis = torch.zeros(L, dtype=torch.bool)
        for lb in vbt_lb[b]:
            vis[lb * P:min(L, (lb + 1) * P)] = True
        qq = torch.as_tensor(np.asarray(q[b], dtype=np.float64))[:, None, :]
        ob, lb_ = sdpa_rows(qq, K, V, vis[None, :], sm_scale)
        o[b] = ob[:, 0].numpy()
        lse[b] = lb_[:, 0].numpy()
    return o, lse


def brute_verify(pool, q, seq_lens, fbt, sm_scale):
    B, QL, Hq, D = q.shape
    Hkv = pool.k_pages.shape[1]
    G = Hq // Hkv
    o = np.zeros((B, QL, Hq, D))
    lse = np.zeros((B, QL, Hq))
    for b in range(B):
        L = int(seq_lens[b])
        K, V = logical_kv(pool, fbt[b], L)
        K, V = K.repeat_interleave(G, 0), V.repeat_interleave(G, 0)
        pos = torch.arange(L)
        mask = pos[None, :] <= (L - QL + torch.arange(QL))[:, None]
        qq = torch.as_tensor(np.asarray(q[b], dtype=np.float64)).transpose(0, 1)  # [Hq][QL][D]
        ob, lb = sdpa_rows(qq, K, V, mask, sm_scale)
        o[b] = ob.transpose(0, 1).numpy()
        lse[b] = lb.transpose(0, 1).numpy()
    return o, lse


def random_case(seed, dtype, D=16, Hkv=2, G=4, B=3, max_L=200):
    rng = np.random.default_rng(seed)
    seq_lens = rng.integers(1, max_L, B)
    npg = [-(-int(L) // P) for L in seq_lens]
    num_pages = sum(npg) + 3
    perm = rng.permutation(num_pages)
    fbt = np.full((B, max(npg)), -1, dtype=np.int64)
    off = 0
    for b, n in enumerate(npg):
        fbt[b, :n] = perm[off:off + n]
        off += n
    pool = make_pool(num_pages, Hkv, D, dtype, seed)
    views = []
    for b in range(B):
        n = npg[b]
        lbs = sorted(set(rng.choice(n, size=int(rng.integers(1, n + 1)), replace=False).tolist())
                     | {n - 1})
        views.append(lbs)
    q = rng.standard_normal((B, G * Hkv, D)) / math.sqrt(D)
    return pool, seq_lens, fbt, views, q


def view_arrays(fbt, views):
    B = len(views)
    cap = max(len(v) for v in views)
    vbt = np.full((B, cap), -1, dtype=np.int64)
    vlb = np.full((B, cap), -1, dtype=np.int64)
    nb = np.zeros(B, dtype=np.int64)
    for b, lbs in enumerate(views):
        nb[b] = len(lbs)
        vlb[b, :len(lbs)] = lbs
        vbt[b, :len(lbs)] = fbt[b, lbs]
    return vbt, vlb, nb


# --------------------------------------------------------------------------
# brute force
# --------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["f32", "bf16", "fp8"])
@pytest.mark.parametrize("seed", range(4))
def test_decode_matches_sdpa(dtype, seed):
    pool, seq_lens, fbt, views, q = random_case(seed, dtype)
    vbt, vlb, nb = view_arrays(fbt, views)
    o, lse = O.selected_decode(pool, q, seq_lens, vbt, vlb, nb, 0.7)
    eo, el = brute_decode(pool, q, seq_lens, fbt, views, 0.7)
    np.testing.assert_allclose(o, eo, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, el, rtol=0, atol=1e-12)


@pytest.mark.parametrize("dtype", ["f32", "bf16", "fp8"])
@pytest.mark.parametrize("q_len", [1, 2, 5, 9])
def test_verify_matches_sdpa(dtype, q_len):
    pool, seq_lens, fbt, _, _ = random_case(q_len, dtype, max_L=150)
    seq_lens = np.maximum(seq_lens, q_len)
    rng = np.random.default_rng(q_len)
    q = rng.standard_normal((len(seq_lens), q_len, 8, 16)) / 4
    o, lse = O.verify(pool, q, seq_lens, fbt, 0.9)
    eo, el = brute_verify(pool, q, seq_lens, fbt, 0.9)
    np.testing.assert_allclose(o, eo, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, el, rtol=0, atol=1e-12)


def test_decode_matches_sdpa_head_dim_128():
    pool, seq_lens, fbt, views, q = random_case(11, "bf16", D=128, Hkv=8, G=4, B=2, max_L=260)
    vbt, vlb, nb = view_arrays(fbt, views)
    o, lse = O.selected_decode(pool, q, seq_lens, vbt, vlb, nb, 1.0)
    eo, el = brute_decode(pool, q, seq_lens, fbt, views, 1.0)
    np.testing.assert_allclose(o, eo, rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse, el, rtol=0, atol=1e-12)


# --------------------------------------------------------------------------
# closed forms
# --------------------------------------------------------------------------

def test_single_visible_token():
    # L = 17: logical page 1 holds only token 16. A view of that page alone
    # shows one token, so o = v_16 and lse = z_16.
    pool = make_pool(4, 1, 8, "f32", 3)
    fbt = np.array([[2, 0]])
    q = np.random.default_rng(0).standard_normal((1, 1, 8))
    o, lse = O.selected_decode(pool, q, [17], [[0]], [[1]], [1], 0.5)
    k16 = key_vec(pool, 0, 0, 0)
    v16 = pool.v_pages[0, 0, :, 0].astype(np.float64)
    np.testing.assert_allclose(o[0, 0], v16, atol=1e-15)
    assert abs(lse[0, 0] - 0.5 * float(q[0, 0] @ k16)) < 1e-14
    del fbt


def test_constant_keys_give_mean():
    # All keys zero: every logit is 0, weights are uniform -> mean of the
    # visible values, lse = ln(n).
    pool = make_pool(3, 1, 8, "f32", 4)
    pool.k_pages[:] = 0.0
    L = 37
    o, lse = O.verify(pool, np.ones((1, 1, 1, 8)), [L], [[1, 2, 0]], 1.0)
    V = np.concatenate([pool.v_pages[p, 0].T for p in (1, 2, 0)])[:L].astype(np.float64)
    np.testing.assert_allclose(o[0, 0, 0], V.mean(0), atol=1e-14)
    assert abs(lse[0, 0, 0] - math.log(L)) < 1e-14


def test_two_tokens_sigmoid():
    pool = make_pool(1, 1, 8, "f32", 5)
    q = np.array([[[[0.3, -1.2, 0.7, 2.0, -0.4, 0.1, 0.9, -1.5]]]])
    o, lse = O.verify(pool, q, [2], [[0]], 1.3)
    k1, k2 = key_vec(pool, 0, 0, 0), key_vec(pool, 0, 0, 1)
    v1, v2 = pool.v_pages[0, 0, :, 0].astype(float), pool.v_pages[0, 0, :, 1].astype(float)
    z1, z2 = 1.3 * q[0, 0, 0] @ k1, 1.3 * q[0, 0, 0] @ k2
    sig = 1.0 / (1.0 + math.exp(-(z1 - z2)))
    np.testing.assert_allclose(o[0, 0, 0], sig * v1 + (1 - sig) * v2, atol=1e-14)
    assert abs(lse[0, 0, 0] - np.logaddexp(z1, z2)) < 1e-14


def test_empty_view_row():
    pool = make_pool(2, 1, 8, "f32", 6)
    o, lse = O.selected_decode(pool, np.ones((1, 1, 8)), [20], [[0]], [[0]], [0], 1.0)
    assert np.all(o == 0) and lse[0, 0] == -np.inf


# --------------------------------------------------------------------------
# invariants
# --------------------------------------------------------------------------

@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_all_blocks_view_equals_verify_one_query(dtype):
    pool, seq_lens, fbt, _, q = random_case(21, dtype)
    views = [list(range(-(-int(L) // P))) for L in seq_lens]
    vbt, vlb, nb = view_arrays(fbt, views)
    od, ld = O.selected_decode(pool, q, seq_lens, vbt, vlb, nb, 1.1)
    ov, lv = O.verify(pool, q[:, None], seq_lens, fbt, 1.1)
    np.testing.assert_allclose(od, ov[:, 0], atol=1e-13)
    np.testing.assert_allclose(ld, lv[:, 0], atol=1e-13)


def test_view_page_order_is_irrelevant():
    pool, seq_lens, fbt, views, q = random_case(22, "bf16")
    vbt, vlb, nb = view_arrays(fbt, views)
    o1, l1 = O.selected_decode(pool, q, seq_lens, vbt, vlb, nb, 1.0)
    rng = np.random.default_rng(0)
    for b in range(len(views)):
        perm = rng.permutation(int(nb[b]))
        vbt[b, :nb[b]] = vbt[b, perm]
        vlb[b, :nb[b]] = vlb[b, perm]
    o2, l2 = O.selected_decode(pool, q, seq_lens, vbt, vlb, nb, 1.0)
    np.testing.assert_allclose(o1, o2, atol=1e-12)
    np.testing.assert_allclose(l1, l2, atol=1e-12)


@pytest.mark.parametrize("seed", range(6))
def test_split_then_merge_equals_unsplit(seed):
    rng = np.random.default_rng(seed)
    T, D, R = int(rng.integers(1, 90)), 8, 3
    q = rng.standard_normal((R, D))
    k = rng.standard_normal((T, D)) * 2
    v = rng.standard_normal((T, D))
    cuts = sorted(rng.integers(0, T + 1, int(rng.integers(0, 7))).tolist())
    bounds = [0] + cuts + [T]                     # repeated cuts = empty parts
    o1, l1 = O.attend(q, k, v, [T] * R, 0.8)
    o2, l2 = O.split_attend(q, k, v, bounds, 0.8)
    np.testing.assert_allclose(o1, o2, atol=1e-13)
    np.testing.assert_allclose(l1, l2, atol=1e-13)


def test_merge_with_all_empty_parts():
    o, lse = O.lse_merge(np.zeros((3, 2, 4)), np.full((3, 2), -np.inf))
    assert np.all(o == 0) and np.all(lse == -np.inf)


def test_gqa_equals_replicated_mha():
    pool, seq_lens, fbt, views, q = random_case(23, "f32", Hkv=2, G=4)
    vbt, vlb, nb = view_arrays(fbt, views)
    o1, l1 = O.selected_decode(pool, q, seq_lens, vbt, vlb, nb, 1.0)
    rep = O.KVPool(np.repeat(pool.k_pages, 4, axis=1), np.repeat(pool.v_pages, 4, axis=1), "f32")
    o2, l2 = O.selected_decode(rep, q, seq_lens, vbt, vlb, nb, 1.0)
    np.testing.assert_allclose(o1, o2, atol=1e-14)
    np.testing.assert_allclose(l1, l2, atol=1e-14)


def test_verify_row_equals_truncated_decode():
    pool, seq_lens, fbt, _, _ = random_case(24, "bf16", max_L=120)
    QL = 4
    seq_lens = np.maximum(seq_lens, QL)
    rng = np.random.default_rng(1)
    q = rng.standard_normal((len(seq_lens), QL, 8, 16))
    ov, lv = O.verify(pool, q, seq_lens, fbt, 0.6)
    for i in range(QL):
        Li = seq_lens - QL + i + 1
        views = [list(range(-(-int(L) // P))) for L in Li]
        vbt, vlb, nb = view_arrays(fbt, views)
        od, ld = O.selected_decode(pool, q[:, i], Li, vbt, vlb, nb, 0.6)
        np.testing.assert_allclose(ov[:, i], od, atol=1e-13)
        np.testing.assert_allclose(lv[:, i], ld, atol=1e-13)


# --------------------------------------------------------------------------
# stored-bit decoders against torch
# --------------------------------------------------------------------------

def test_e4m3fn_all_codes_match_torch():
    codes = np.arange(256, dtype=np.uint8)
    mine = O.e4m3fn_to_f64(codes)
    ref = torch.from_numpy(codes).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    assert np.array_equal(np.isnan(mine), np.isnan(ref))
    assert np.sum(np.isnan(mine)) == 2                       # 0x7F and 0xFF
    ok = ~np.isnan(ref)
    assert np.array_equal(mine[ok], ref[ok])
    assert np.nanmax(mine) == 448.0 and np.nanmin(mine) == -448.0
    assert mine[1] == 2.0 ** -9                              # smallest subnormal


def test_bf16_all_patterns_match_torch():
    pats = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    mine = O.bf16_to_f64(pats)
    ref = torch.from_numpy(pats.view(np.int16)).view(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(np.isnan(mine), np.isnan(ref))
    ok = ~np.isnan(ref)
    assert np.array_equal(mine[ok], ref[ok])


# --------------------------------------------------------------------------
# planted mistakes must be caught by the brute-force pins
# --------------------------------------------------------------------------

def _decode_mismatch(monkeypatch, patch):
    pool, seq_lens, fbt, views, q = random_case(31, "bf16", B=2, max_L=180)
    vbt, vlb, nb = view_arrays(fbt, views)
    eo, el = brute_decode(pool, q, seq_lens, fbt, views, 1.0)
    with monkeypatch.context() as m:
        patch(m, pool)
        o, lse = O.selected_decode(pool, q, seq_lens, vbt, vlb, nb, 1.0)
    return max(np.abs(o - eo).max(), np.abs(lse - el).max())


def test_planted_untransposed_v_is_caught(monkeypatch):
    def patch(m, pool):
        m.setattr(O.KVPool, "values",
                  lambda self, pages, g: O.bf16_to_f64(self.v_pages[np.asarray(pages), g]
                                                       .reshape(len(pages), P, -1)))
    assert _decode_mismatch(monkeypatch, patch) > 1e-3


def test_planted_gqa_mapping_is_caught(monkeypatch):
    orig = O.KVPool.keys

    def patch(m, pool):
        Hkv = pool.k_pages.shape[1]
        m.setattr(O.KVPool, "keys", lambda self, pages, g: orig(self, pages, (g + 1) % Hkv))
    assert _decode_mismatch(monkeypatch, patch) > 1e-3


def test_planted_last_page_count_is_caught(monkeypatch):
    orig = O._view_tokens

    def patch(m, pool):
        m.setattr(O, "_view_tokens",
                  lambda pool_, g, L, pages, lblks, **kw: orig(pool_, g, L + 1, pages, lblks, **kw))
    assert _decode_mismatch(monkeypatch, patch) > 1e-3


def test_planted_missing_max_in_lse_is_caught(monkeypatch):
    orig = O.attend

    def bad_attend(q, k, v, n_visible, sm_scale):
        o, lse = orig(q, k, v, n_visible, sm_scale)
        zmax = np.array([(sm_scale * (k[:n] @ q[r])).max() if n else 0.0
                         for r, n in enumerate(n_visible)])
        return o, lse - zmax

    def patch(m, pool):
        m.setattr(O, "attend", bad_attend)
    assert _decode_mismatch(monkeypatch, patch) > 1e-3


def test_planted_causal_off_by_one_is_caught(monkeypatch):
    pool, seq_lens, fbt, _, _ = random_case(32, "f32", max_L=100)
    seq_lens = np.maximum(seq_lens, 3)
    q = np.random.default_rng(2).standard_normal((len(seq_lens), 3, 8, 16))
    eo, _ = brute_verify(pool, q, seq_lens, fbt, 1.0)
    orig = O.attend
    with monkeypatch.context() as m:
        m.setattr(O, "attend", lambda q_, k, v, nv, s: orig(q_, k, v, [n - 1 for n in nv], s))
        o, _ = O.verify(pool, q, seq_lens, fbt, 1.0)
    assert np.abs(o - eo).max() > 1e-3


# --------------------------------------------------------------------------
# page ids outside the pool contribute no keys
# --------------------------------------------------------------------------

def _masked_brute_verify(pool, q, seq_lens, fbt, sm_scale):
    """brute_verify with the positions of out-of-pool pages masked out (their
    ids replaced by page 0 only to gather something, then hidden)."""
    nP = pool.k_pages.shape[0]
    B, QL, Hq, D = q.shape
    G = Hq // pool.k_pages.shape[1]
    o = np.zeros((B, QL, Hq, D))
    lse = np.zeros((B, QL, Hq))
    for b in range(B):
        L = int(seq_lens[b])
        row = np.asarray(fbt[b], dtype=np.int64)
        bad = (row < 0) | (row >= nP)
        K, V = logical_kv(pool, np.where(bad, 0, row), L)
        K, V = K.repeat_interleave(G, 0), V.repeat_interleave(G, 0)
        pos = torch.arange(L)
        shown = ~torch.as_tensor(bad)[pos // P]
        mask = (pos[None, :] <= (L - QL + torch.arange(QL))[:, None]) & shown[None, :]
        qq = torch.as_tensor(np.asarray(q[b], dtype=np.float64)).transpose(0, 1)
        ob, lb = sdpa_rows(qq, K, V, mask, sm_scale)
        o[b] = ob.transpose(0, 1).nan_to_num(0.0).numpy()
        lse[b] = lb.transpose(0, 1).numpy()
    return o, lse


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_verify_out_of_pool_pages_contribute_no_keys(dtype):
    rng = np.random.default_rng(5)
    pool = make_pool(12, 2, 16, dtype, seed=9)
    seq_lens = np.array([70, 33, 20])
    fbt = rng.integers(0, 12, (3, 5))
    fbt[0, 1], fbt[0, 4] = 12, -1          # an inner page and the last page
    fbt[1, 0] = 40                          # the first page
    fbt[2, 1] = -7                          # the last page: the window's own keys
    q = rng.standard_normal((3, 4, 8, 16))
    eo, el = O.verify(pool, q, seq_lens, fbt, 0.3)
    bo, bl = _masked_brute_verify(pool, q, seq_lens, fbt, 0.3)
    assert np.abs(eo - bo).max() < 1e-12
    fin = np.isfinite(bl)
    assert np.array_equal(fin, np.isfinite(el)) and np.abs(el[fin] - bl[fin]).max() < 1e-12
    # sequence 2's last page (tokens 16..19) is out of the pool: every row sees
    # exactly tokens 0..15, as a one-page sequence of 16 tokens whose window
    # rows all see the whole page
    assert np.all(fin[2])
    for i in range(4):
        one = O.selected_decode(pool, q[2, i][None], [16], [[fbt[2, 0]]], [[0]], [1], 0.3)
        assert np.abs(eo[2, i] - one[0][0]).max() < 1e-12


def test_decode_out_of_pool_pages_contribute_no_keys():
    pool = make_pool(6, 2, 16, "bf16", seed=2)
    q = np.random.default_rng(1).standard_normal((1, 8, 16))
    full = O.selected_decode(pool, q, [40], [[3, 1, 5]], [[0, 1, 2]], [3], 0.5)
    part = O.selected_decode(pool, q, [40], [[3, 9, 5, -2]], [[0, 1, 2, 1]], [4], 0.5)
    only = O.selected_decode(pool, q, [40], [[3, 5]], [[0, 2]], [2], 0.5)
    assert np.abs(part[0] - only[0]).max() < 1e-15 and np.abs(full[0] - only[0]).max() > 1e-3
