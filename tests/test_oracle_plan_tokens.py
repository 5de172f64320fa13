"""CPU pins of the token-granular plan (visibility mask at token resolution,
Sec. 3.1) and of decode over a masked view: a hand-worked vector, an
independent replay with boolean token arrays, invariants, and torch's
scaled-dot-product attention with a token-level visibility mask."""
import numpy as np
import pytest
import torch

from oracle import kap_oracle as O

from test_oracle_attention import logical_kv, make_pool, sdpa_rows

P = O.PAGE
C1 = dict(seq_len=100, fbt_row=[7, 3, 9, 0, 5, 2, 8], starts=[20, 40, 90, 0], lens=[10, 30, 5, 5],
          priors=[0.5, 0.9, 0.9, 0.1], prefix=16, suffix=8, budget=60, num_pages=10, capacity=8)


@pytest.mark.parametrize("policy", [O.SELECT_SKIP, O.SELECT_STOP])
def test_hand_worked_vector(policy):
    # mandatory tokens [0,16) + [92,100): 24; rank: span 1, span 2, span 0, span 3.
    # span 1 [40,70): +30 -> 54; span 2 [90,95): +2 (90, 91) -> 56; span 0
    # [20,30): +10 does not fit (SKIP goes on, STOP ends); span 3 [0,5): +0.
    p = O.compile_plan_tokens_one(**C1, policy=policy)
    assert p.status == O.PLAN_OK
    assert p.logical_blocks == [0, 2, 3, 4, 5, 6]
    assert p.block_table == [7, 9, 0, 5, 2, 8]
    assert p.token_masks == [0xFFFF, 0xFF00, 0xFFFF, 0x003F, 0xFC00, 0x000F]
    assert p.view_tokens == 56
    if policy == O.SELECT_SKIP:
        assert p.spans_taken == 3 and p.span_selected == [0, 1, 1, 1]
    else:
        assert p.spans_taken == 2 and p.span_selected == [0, 1, 1, 0]


def replay_with_arrays(L, starts, lens, priors, prefix, suffix, budget, policy):
    """The same rule through boolean token arrays and numpy's lexsort."""
    vis = np.zeros(L, dtype=bool)
    vis[:min(max(prefix, 0), L)] = True
    vis[max(0, L - max(suffix, 1)):] = True
    order = np.lexsort((np.arange(len(starts)), np.asarray(starts), -np.asarray(priors, float)))
    flags = np.zeros(len(starts), dtype=int)
    for i in order:
        x, e = max(0, starts[i]), min(L, starts[i] + lens[i])
        if e <= x:
            continue
        span = np.zeros(L, dtype=bool)
        span[x:e] = True
        cost = int((span & ~vis).sum())
        if vis.sum() + cost <= budget:
            vis |= span
            flags[i] = 1
        elif policy == O.SELECT_STOP:
            break
    pages = np.unique(np.nonzero(vis)[0] // P)
    masks = [int(sum(1 << t for t in range(P) if p * P + t < L and vis[p * P + t])) for p in pages]
    return list(pages), masks, int(vis.sum()), list(flags)


@pytest.mark.parametrize("seed", range(40))
def test_matches_boolean_array_replay(seed):
    rng = np.random.default_rng(seed)
    L = int(rng.integers(1, 700))
    n = int(rng.integers(0, 12))
    starts = [int(x) for x in rng.integers(-40, L + 40, n)]
    lens = [int(x) for x in rng.integers(0, 200, n)]
    priors = [float(x) for x in rng.choice([0.1, 0.3, 0.3, 0.9], n)]
    prefix, suffix = int(rng.integers(0, 80)), int(rng.integers(0, 80))
    budget = int(rng.integers(0, L + 50))
    policy = int(rng.integers(0, 2))
    npg = -(-L // P)
    fbt = list(rng.permutation(npg + 5)[:npg])
    p = O.compile_plan_tokens_one(L, fbt, starts, lens, priors, prefix, suffix, budget, policy,
                                  npg + 5, npg)
    pages, masks, used, flags = replay_with_arrays(L, starts, lens, priors, prefix, suffix,
                                                   budget, policy)
    assert p.status == O.PLAN_OK
    assert p.logical_blocks == pages and p.token_masks == masks
    assert p.view_tokens == used and p.span_selected == flags
    assert p.block_table == [fbt[j] for j in pages]
    # invariants: masks are the visible tokens; mandatory tokens visible;
    # the budget holds unless the mandatory tokens alone exceed it
    assert sum(bin(m).count("1") for m in masks) == used
    mandatory = min(max(prefix, 0), L) + min(max(suffix, 1), L) - max(
        0, min(max(prefix, 0), L) - max(0, L - max(suffix, 1)))
    assert used <= budget or used == mandatory


def test_budget_at_least_the_length_sees_every_token():
    p = O.compile_plan_tokens_one(100, list(range(7)), [0], [100], [0.5], 0, 1, 100, 0, 7, 7)
    assert p.view_tokens == 100 and p.logical_blocks == list(range(7))
    assert p.token_masks == [0xFFFF] * 6 + [0x000F]


@pytest.mark.parametrize("dtype", ["bf16", "fp8"])
def test_masked_decode_matches_sdpa(dtype):
    rng = np.random.default_rng(5)
    Hkv, G, D, L = 2, 4, 16, 150
    npg = -(-L // P)
    pool = make_pool(npg + 2, Hkv, D, dtype, seed=9)
    fbt = rng.permutation(npg + 2)[:npg]
    p = O.compile_plan_tokens_one(L, list(fbt), [20, 70, 121], [15, 33, 9], [0.9, 0.5, 0.7],
                                  5, 3, 80, 0, npg + 2, npg)
    q = rng.standard_normal((1, Hkv * G, D)) / 4
    o, lse = O.selected_decode(pool, q, [L], [p.block_table], [p.logical_blocks],
                               [p.num_blocks], 1.0, view_token_mask=[p.token_masks])
    K, V = logical_kv(pool, fbt, L)
    K, V = K.repeat_interleave(G, 0), V.repeat_interleave(G, 0)
    vis = torch.zeros(L, dtype=torch.bool)
    for j, m in zip(p.logical_blocks, p.token_masks):
        for t in range(P):
            if (m >> t) & 1 and j * P + t < L:
                vis[j * P + t] = True
    assert int(vis.sum()) == p.view_tokens
    eo, el = sdpa_rows(torch.as_tensor(q[0])[:, None, :], K, V, vis[None, :], 1.0)
    np.testing.assert_allclose(o[0], eo[:, 0].numpy(), rtol=0, atol=1e-12)
    np.testing.assert_allclose(lse[0], el[:, 0].numpy(), rtol=0, atol=1e-12)


def test_full_masks_equal_page_granular_decode():
    rng = np.random.default_rng(6)
    pool = make_pool(12, 2, 16, "bf16", seed=3)
    q = rng.standard_normal((1, 8, 16)) / 4
    vbt, vlb = [[3, 7, 1]], [[0, 2, 5]]
    o1, l1 = O.selected_decode(pool, q, [90], vbt, vlb, [3], 1.0)
    o2, l2 = O.selected_decode(pool, q, [90], vbt, vlb, [3], 1.0, view_token_mask=[[0xFFFF] * 3])
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2)
