"""GPU parity of kap_selected_decode and kap_verify against the fp64 oracle.

Tolerances (bf16 / fp8 / fp32 inputs, fp32 outputs): max |O - O_ref| <= 2e-3,
max |LSE - LSE_ref| <= 1e-3, both sides reading the same stored KV bits.
Small and mid-size workloads are checked on every step; the 128K workload and
the 64-sequence fp8 workload on seeded subsets of steps / sequences / KV heads
(the subsets are named in each test), in the launch configuration bench.py
times.
"""
import numpy as np
import pytest
import torch

from oracle import kap_oracle as O
from paper_2607_24260_amd import kap as K
from paper_2607_24260_amd.workloads import make_workload

from kap_testlib import (LSE_TOL, O_TOL, assert_close, dev_i32, full_view, gpu_plan, kv_of,
                         oracle_plan, oracle_pool, plan_view_arrays)

pytestmark = pytest.mark.gpu

_CACHE = {}


def workload(config, **kw):
    key = (config, tuple(sorted(kw.items())))
    if key not in _CACHE:
        _CACHE.clear()
        torch.cuda.empty_cache()
        w = make_workload(config, device="cuda", **kw)
        _CACHE[key] = (w, oracle_pool(w))
    return _CACHE[key]


def decode_check(w, pool, steps, budget=None, num_splits=0, batches=None):
    plan = gpu_plan(w, budget=budget)
    plans = oracle_plan(w, budget=budget)
    cap = w.max_pages_per_seq
    vbt, vlb, nb = plan_view_arrays(plans, cap)
    kv = kv_of(w)
    worst = [0.0, 0.0]
    for s in steps:
        q = w.q_decode[s]
        o, lse = K.selected_decode(kv, q, dev_i32(w.seq_lens), plan["view_block_table"],
                                   plan["view_logical_block"], plan["view_num_blocks"], cap,
                                   w.sm_scale, num_splits=num_splits)
        torch.cuda.synchronize()
        qh = q.float().cpu().numpy()
        sel = list(range(w.batch)) if batches is None else batches
        eo, el = O.selected_decode(pool, qh[sel], w.seq_lens[sel], vbt[sel], vlb[sel], nb[sel],
                                   w.sm_scale)
        worst[0] = max(worst[0], assert_close(f"O step {s}", o.cpu().numpy()[sel], eo, O_TOL))
        worst[1] = max(worst[1], assert_close(f"LSE step {s}", lse.cpu().numpy()[sel], el,
                                              LSE_TOL))
    return worst


def verify_check(w, pool, calls, num_splits=0, batches=None, kv_heads=None):
    kv = kv_of(w)
    Hkv, G = w.num_kv_heads, w.num_q_heads // w.num_kv_heads
    for c in calls:
        q = w.q_verify[c]
        o, lse = K.verify(kv, q, dev_i32(w.seq_lens), dev_i32(w.full_block_table),
                          int(w.seq_lens.max()), w.sm_scale, num_splits=num_splits)
        torch.cuda.synchronize()
        eo, el = O.verify(pool, q.float().cpu().numpy(), w.seq_lens, w.full_block_table,
                          w.sm_scale, batches=batches, kv_heads=kv_heads)
        bs = list(range(w.batch)) if batches is None else batches
        hs = list(range(Hkv)) if kv_heads is None else kv_heads
        heads = [g * G + j for g in hs for j in range(G)]
        on, ln = o.cpu().numpy(), lse.cpu().numpy()
        assert_close(f"verify O call {c}", on[np.ix_(bs, range(q.shape[1]), heads)],
                     eo[np.ix_(bs, range(q.shape[1]), heads)], O_TOL)
        assert_close(f"verify LSE call {c}", ln[np.ix_(bs, range(q.shape[1]), heads)],
                     el[np.ix_(bs, range(q.shape[1]), heads)], LSE_TOL)


# --------------------------------------------------------------------------
# the five workloads
# --------------------------------------------------------------------------

def test_config1_fp32():
    w, pool = workload(1)
    decode_check(w, pool, [0])
    verify_check(w, pool, [0])


def test_config2_decode_all_steps():
    w, pool = workload(2)
    decode_check(w, pool, range(32))


def test_config2_verify_all_calls():
    w, pool = workload(2)
    verify_check(w, pool, range(8))


@pytest.mark.parametrize("first", [0, 8, 16, 24])
def test_config3_decode_all_steps(first):
    w, pool = workload(3)
    decode_check(w, pool, range(first, first + 8))


def test_config3_all_blocks_plan_equals_full_decode():
    """The all-blocks plan (the full block table as the view, what fallback
    uses) must equal full decode: checked against the oracle, against verify
    with a one-token window, and built by the plan kernel from a span that
    covers the whole sequence."""
    w, pool = workload(3)
    kv = kv_of(w)
    fbt, lblk, npg, mx = full_view(w)
    full_b = np.asarray(w.full_block_table, dtype=np.int64)
    full_l = np.tile(np.arange(w.fbt_stride), (w.batch, 1))
    for s in (0, 31):
        q = w.q_decode[s]
        o, lse = K.selected_decode(kv, q, dev_i32(w.seq_lens), fbt, lblk, npg, mx, 1.0)
        ov, lv = K.verify(kv, q[:, None].contiguous(), dev_i32(w.seq_lens), fbt, mx * 16, 1.0)
        torch.cuda.synchronize()
        eo, el = O.selected_decode(pool, q.float().cpu().numpy(), w.seq_lens, full_b, full_l,
                                   npg.cpu().numpy(), 1.0)
        assert_close("full-view O", o.cpu().numpy(), eo, O_TOL)
        assert_close("full-view LSE", lse.cpu().numpy(), el, LSE_TOL)
        assert (o - ov[:, 0]).abs().max().item() <= O_TOL
        assert (lse - lv[:, 0]).abs().max().item() <= LSE_TOL
    # budget = L plus one span over [0, L): the plan kernel emits the full table
    B = w.batch
    offs = np.arange(B + 1, dtype=np.int32)
    plan = K.compile_plan(dev_i32(w.seq_lens), fbt, dev_i32(offs), dev_i32(np.zeros(B)),
                          dev_i32(w.seq_lens), torch.ones(B, device="cuda"),
                          dev_i32(w.prefix), dev_i32(w.suffix), dev_i32(w.seq_lens),
                          num_pages=w.num_pages, view_capacity=w.fbt_stride)
    torch.cuda.synchronize()
    assert torch.equal(plan["view_block_table"], fbt)
    assert torch.equal(plan["view_num_blocks"], npg)
    assert torch.equal(plan["view_tokens"], dev_i32(w.seq_lens))


def test_config3_verify():
    w, pool = workload(3)
    verify_check(w, pool, [0, 7], batches=[0, 5, 15])


def test_config4_decode_sampled_steps():
    # steps 0, 21, 42, 63 of 64, every sequence and head
    w, pool = workload(4, n_verify=2)
    decode_check(w, pool, [0, 21, 42, 63])


def test_config4_verify_sampled():
    # verify call 0 and 1; sequences {0, 3} x KV heads {0, 7}
    w, pool = workload(4, n_verify=2)
    verify_check(w, pool, [0, 1], batches=[0, 3], kv_heads=[0, 7])


def test_config4_verify_full_width():
    # one whole 128K verify call: all 4 sequences x 8 KV heads x 4 query
    # heads x 5 window rows against the oracle
    w, pool = workload(4, n_verify=2)
    verify_check(w, pool, [1])


def test_config5_fp8_decode():
    # decode steps 0 and last, all 64 ragged sequences on the GPU; the oracle
    # checks every fourth sequence (0, 4, ..., 60)
    w, pool = workload(5)
    decode_check(w, pool, [0, w.q_decode.shape[0] - 1], batches=list(range(0, 64, 4)))


def test_config5_fp8_verify_each_window_size():
    # one verify call per distinct gamma; sequences 0, 17, 63 x KV heads 0, 5
    w, pool = workload(5)
    gammas = [q.shape[1] - 1 for q in w.q_verify]
    first = {g: c for c, g in reversed(list(enumerate(gammas)))}
    verify_check(w, pool, sorted(first.values()), batches=[0, 17, 63], kv_heads=[0, 5])


def test_balanced_map_beyond_64_sequences():
    # 100 ragged fp8 sequences of 4K-16K tokens (800 (sequence, KV head) units:
    # the balanced split map, which takes two passes over the batch); the
    # oracle checks sequences 0, 63, 64, 65, 99 (decode) and 0, 64, 99 x KV
    # heads 0, 7 (verify)
    w, pool = workload(5, batch=100, seq_len=16384)
    decode_check(w, pool, [0], batches=[0, 63, 64, 65, 99])
    verify_check(w, pool, [0], batches=[0, 64, 99], kv_heads=[0, 7])


@pytest.mark.parametrize("seq_len,frac", [(4096, 0.401), (16384, 0.242), (65536, 0.108)])
def test_table2_context_buckets(seq_len, frac):
    # the bench's context sweep shapes (B = 4, the bucket's retained ratio as
    # the budget): decode on every sequence, verify on sequences {0, 3} x KV
    # heads {0, 4}
    w, pool = workload(4, seq_len=seq_len, budget_frac=frac, n_decode=1, n_verify=1)
    decode_check(w, pool, [0])
    verify_check(w, pool, [0], batches=[0, 3], kv_heads=[0, 4])


def test_head_split_share():
    # one GPU's share of a 4-way head split at 128K: 8 query / 2 KV heads
    w, pool = workload(4, num_q_heads=8, num_kv_heads=2, n_decode=1, n_verify=1)
    decode_check(w, pool, [0])
    verify_check(w, pool, [0], batches=[1, 2])


# --------------------------------------------------------------------------
# cross-checks and edge cases on small shapes (several tiles + ragged tails)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
def test_split_count_does_not_change_result(kv_dtype):
    cfg = 2 if kv_dtype == "bf16" else 5
    kw = dict(batch=3, seq_len=5000, n_decode=1, n_verify=1)
    w, pool = workload(cfg, **kw)
    for ns in (1, 3, 10_000):
        decode_check(w, pool, [0], num_splits=ns)
        verify_check(w, pool, [0], num_splits=ns)


@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
def test_split_merge_of_long_windows(kv_dtype):
    # 16-token windows: 64 rows, so the last workgroup merges 2048 (row, 4-dim)
    # items, several per thread and in several passes; with the maximum split
    # count every item folds in more than eight partials (several load batches)
    cfg = 2 if kv_dtype == "bf16" else 5
    w, pool = workload(cfg, batch=3, seq_len=5000, n_decode=1, n_verify=1)
    orig = w.q_verify
    try:
        w.q_verify = [_window(w, 16, seed=16)]
        for ns in (3, 10_000):
            verify_check(w, pool, [0], num_splits=ns)
    finally:
        w.q_verify = orig


@pytest.mark.parametrize("kv_dtype,q_len", [("bf16", 5), ("bf16", 11), ("fp8", 5), ("fp8", 9),
                                             ("fp8", 11), ("fp8", 12), ("fp8", 13)])
def test_combined_tile_stores_at_every_split_count(kv_dtype, q_len):
    # After the wavefronts combine, a verify workgroup writes each row tile
    # either from every thread or staged through LDS by one wavefront (the
    # kernel instance decides), as the final output (one split) or as its
    # split's partial for the merge: each way at 1, 3 and the maximum number
    # of splits, on ragged lengths with a sequence shorter than the window.
    cfg = 2 if kv_dtype == "bf16" else 5
    w, pool = _ragged(cfg, 3, 4096 if cfg == 2 else 5000, [2500, 777, q_len - 1])
    q = _window(w, q_len, 700 + q_len)
    for ns in (1, 3, 10_000):
        o, lse = K.verify(kv_of(w), q, dev_i32(w.seq_lens), dev_i32(w.full_block_table),
                          2500, 1.0, num_splits=ns)
        torch.cuda.synchronize()
        eo, el = O.verify(pool, q.float().cpu().numpy(), w.seq_lens, w.full_block_table, 1.0)
        assert_close(f"verify O (q_len={q_len}, splits={ns})", o.cpu().numpy(), eo, O_TOL)
        assert_close(f"verify LSE (q_len={q_len}, splits={ns})", lse.cpu().numpy(), el, LSE_TOL)


def test_view_order_does_not_matter():
    w, pool = workload(2, batch=2, seq_len=4000, n_decode=1, n_verify=1)
    plan = gpu_plan(w)
    kv = kv_of(w)
    args = (dev_i32(w.seq_lens),)
    o1, l1 = K.selected_decode(kv, w.q_decode[0], *args, plan["view_block_table"],
                               plan["view_logical_block"], plan["view_num_blocks"],
                               w.max_pages_per_seq, 1.0)
    vbt = plan["view_block_table"].clone()
    vlb = plan["view_logical_block"].clone()
    g = torch.Generator(device="cpu").manual_seed(3)
    for b in range(w.batch):
        n = int(plan["view_num_blocks"][b])
        perm = torch.randperm(n, generator=g).cuda()
        vbt[b, :n] = vbt[b, :n][perm]
        vlb[b, :n] = vlb[b, :n][perm]
    o2, l2 = K.selected_decode(kv, w.q_decode[0], *args, vbt, vlb, plan["view_num_blocks"],
                               w.max_pages_per_seq, 1.0)
    torch.cuda.synchronize()
    assert (o1 - o2).abs().max().item() <= 1e-5
    assert (l1 - l2).abs().max().item() <= 1e-5


def test_verify_one_token_equals_all_blocks_decode():
    w, pool = workload(2, batch=3, seq_len=3000, n_decode=1, n_verify=1)
    kv = kv_of(w)
    fbt, lblk, npg, mx = full_view(w)
    q = w.q_decode[0]
    od, ld = K.selected_decode(kv, q, dev_i32(w.seq_lens), fbt, lblk, npg, mx, 1.0)
    ov, lv = K.verify(kv, q[:, None].contiguous(), dev_i32(w.seq_lens), fbt, mx * 16, 1.0)
    torch.cuda.synchronize()
    assert (od - ov[:, 0]).abs().max().item() <= 2e-3
    assert (ld - lv[:, 0]).abs().max().item() <= 1e-3


@pytest.mark.parametrize("q_len", [1, 2, 3, 4, 5, 8, 9, 13, 16])
def test_verify_window_sizes_ragged(q_len):
    # ragged lengths (not multiples of 16), windows from 1 to 16 query tokens
    w, pool = workload(2, batch=4, seq_len=1000, n_decode=1, n_verify=1)
    w.seq_lens[:] = [1000, 999, 37, q_len]
    g = torch.Generator(device="cuda").manual_seed(q_len)
    q = (torch.randn((4, q_len, 32, 128), generator=g, device="cuda") / 11.3).to(torch.bfloat16)
    kv = kv_of(w)
    o, lse = K.verify(kv, q, dev_i32(w.seq_lens), dev_i32(w.full_block_table), 1000, 1.0)
    torch.cuda.synchronize()
    eo, el = O.verify(pool, q.float().cpu().numpy(), w.seq_lens, w.full_block_table, 1.0)
    assert_close("O", o.cpu().numpy(), eo, O_TOL)
    assert_close("LSE", lse.cpu().numpy(), el, LSE_TOL)


@pytest.mark.parametrize("q_len", [1, 2, 3, 5, 8, 9, 12, 13, 16])
def test_verify_window_sizes_ragged_fp8(q_len):
    # fp8 pools (per-page scales), ragged lengths with partial last pages and a
    # sequence as short as the window: one to four row tiles, each with its own
    # ring depth and wavefronts per SIMD, and the whole-row V^T loads
    w, pool = workload(5, batch=4, seq_len=5000, n_decode=1, n_verify=1)
    lens = np.array([4000, 3999, 37, q_len], dtype=np.int32)
    assert np.all((w.full_block_table >= 0).sum(1) * 16 >= lens)
    g = torch.Generator(device="cuda").manual_seed(100 + q_len)
    q = (torch.randn((4, q_len, 32, 128), generator=g, device="cuda") / 11.3).to(torch.bfloat16)
    o, lse = K.verify(kv_of(w), q, dev_i32(lens), dev_i32(w.full_block_table), 4000, 1.0)
    torch.cuda.synchronize()
    eo, el = O.verify(pool, q.float().cpu().numpy(), lens, w.full_block_table, 1.0)
    assert_close("O", o.cpu().numpy(), eo, O_TOL)
    assert_close("LSE", lse.cpu().numpy(), el, LSE_TOL)


@pytest.mark.parametrize("q_len", [1, 5, 9, 13, 16])
def test_fp8_page_scales_of_any_sign_and_size(q_len):
    """Per-page fp8 scales are plain floats: a negative K scale flips a page's
    logits, a zero K scale makes them 0 and a zero V scale blanks the page's
    values; K scales up to 16x and V scales down to 2^-8 of the quantiser's.
    Pages of different sign and size share a page pair, so the fold of the
    scales into logits and weights is checked per page -- also in the
    gathered last row tile of 1-, 5-, 9- and 13-token windows."""
    w, _ = workload(5, batch=4, seq_len=5000, n_decode=1, n_verify=1)
    _CACHE.clear()                  # the workload's scales are changed below
    sc = w.kv_scales[0]
    gen = torch.Generator(device="cuda").manual_seed(1000 + q_len)
    kf = torch.tensor([1.0, -1.0, 0.0, 0.25, 4.0, 16.0, -3.0], device="cuda")
    vf = torch.tensor([1.0, -1.0, 0.0, 0.25, 2.0 ** -8, 4.0, -2.0], device="cuda")
    n = sc.shape[0]
    sc[:, 0] *= kf[torch.randint(0, len(kf), (n,), generator=gen, device="cuda")]
    sc[:, 1] *= vf[torch.randint(0, len(vf), (n,), generator=gen, device="cuda")]
    torch.cuda.synchronize()
    pool = oracle_pool(w)
    lens = np.array([4000, 3999, 37, q_len], dtype=np.int32)
    g = torch.Generator(device="cuda").manual_seed(200 + q_len)
    q = (torch.randn((4, q_len, 32, 128), generator=g, device="cuda") / 11.3).to(torch.bfloat16)
    o, lse = K.verify(kv_of(w), q, dev_i32(lens), dev_i32(w.full_block_table), 4000, 1.0)
    torch.cuda.synchronize()
    eo, el = O.verify(pool, q.float().cpu().numpy(), lens, w.full_block_table, 1.0)
    assert_close("verify O", o.cpu().numpy(), eo, O_TOL)
    assert_close("verify LSE", lse.cpu().numpy(), el, LSE_TOL)
    if q_len == 1:
        decode_check(w, pool, [0])
        decode_check(w, pool, [0], num_splits=3)


@pytest.mark.parametrize("seed", range(32))
def test_random_shapes(seed):
    """Seeded random batches: 1-6 sequences of 1-4096 tokens (partial pages,
    sequences shorter than the window), random budgets per sequence, windows
    of 1-16 tokens, bf16 or fp8, balanced or forced split counts; decode over
    the plan's view and verify over the full table against the oracle."""
    rng = np.random.default_rng(4242 + seed)
    kv_dtype = "bf16" if seed % 2 == 0 else "fp8"
    cfg = 2 if kv_dtype == "bf16" else 5
    B = int(rng.integers(1, 7))
    lens = [int(x) for x in rng.integers(1, 4097, B)]
    w, pool = _ragged(cfg, B, 4096 if cfg == 2 else 5000, lens)
    budget = np.array([int(rng.integers(0, L + 1)) for L in lens], dtype=np.int32)
    ns = int(rng.choice([0, 0, 1, 2, 7, 10_000]))
    decode_check(w, pool, [0], budget=budget, num_splits=ns)
    q_len = int(rng.integers(1, 17))
    q = _window(w, q_len, 900 + seed)
    o, lse = K.verify(kv_of(w), q, dev_i32(w.seq_lens), dev_i32(w.full_block_table),
                      int(max(lens)), 1.0, num_splits=ns)
    torch.cuda.synchronize()
    eo, el = O.verify(pool, q.float().cpu().numpy(), w.seq_lens, w.full_block_table, 1.0)
    assert_close(f"verify O (B={B}, q_len={q_len}, splits={ns})", o.cpu().numpy(), eo, O_TOL)
    assert_close(f"verify LSE (B={B}, q_len={q_len}, splits={ns})", lse.cpu().numpy(), el, LSE_TOL)


def test_window_longer_than_sequence_gives_empty_rows():
    w, pool = workload(2, batch=2, seq_len=100, n_decode=1, n_verify=1)
    w.seq_lens[:] = [3, 100]
    q = w.q_verify[0]                                      # q_len 5 > L = 3 for sequence 0
    o, lse = K.verify(kv_of(w), q, dev_i32(w.seq_lens), dev_i32(w.full_block_table), 100, 1.0)
    torch.cuda.synchronize()
    eo, el = O.verify(pool, q.float().cpu().numpy(), w.seq_lens, w.full_block_table, 1.0)
    assert np.all(np.isneginf(lse.cpu().numpy()[0, :2]))
    assert np.all(o.cpu().numpy()[0, :2] == 0)
    assert_close("O", o.cpu().numpy(), eo, O_TOL)
    assert_close("LSE", lse.cpu().numpy(), el, LSE_TOL)


def test_empty_view_gives_zero_and_neg_inf():
    w, _ = workload(2, batch=2, seq_len=500, n_decode=1, n_verify=1)
    plan = gpu_plan(w)
    nb = plan["view_num_blocks"].clone()
    nb[1] = 0
    o, lse = K.selected_decode(kv_of(w), w.q_decode[0], dev_i32(w.seq_lens),
                               plan["view_block_table"], plan["view_logical_block"], nb,
                               w.max_pages_per_seq, 1.0)
    torch.cuda.synchronize()
    assert torch.all(o[1] == 0) and torch.all(torch.isneginf(lse[1]))
    assert torch.all(torch.isfinite(lse[0]))


@pytest.mark.parametrize("alpha", [8.0, 16.0])
@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
def test_peaky_planted_keys(alpha, kv_dtype):
    """Plant K_t = alpha q_h / |q_h|^2 (then stored in the KV dtype) at a few
    selected positions so one logit per head dominates: stresses the max
    subtraction, the split merge and the rounding of P."""
    cfg = 2 if kv_dtype == "bf16" else 5
    w, _ = workload(cfg, batch=2, seq_len=6000, n_decode=1, n_verify=1)
    plans = oracle_plan(w)
    rng = np.random.default_rng(int(alpha))
    k = w.k_pages[0]
    q = w.q_decode[0].float()
    for b, p in enumerate(plans):
        for _ in range(3):
            kk = int(rng.integers(0, p.num_blocks))
            page, lb = p.block_table[kk], p.logical_blocks[kk]
            slot = int(rng.integers(0, min(16, int(w.seq_lens[b]) - 16 * lb)))
            for g in range(w.num_kv_heads):
                h = g * 4 + int(rng.integers(0, 4))
                vec = alpha * q[b, h] / (q[b, h] @ q[b, h])
                vec = vec.view(-1, 8)                       # K pages hold 8-dim chunks
                if kv_dtype == "bf16":
                    k[page, g, :, slot] = vec.to(torch.bfloat16)
                else:
                    sc = float(w.kv_scales[0][page, 0])
                    k[page, g, :, slot] = (vec / sc).clamp(-448, 448).to(
                        torch.float8_e4m3fn).view(torch.uint8)
    pool = oracle_pool(w)
    _CACHE.clear()
    decode_check(w, pool, [0])
    decode_check(w, pool, [0], num_splits=1)
    # the planted keys also sit in the full KV the verify window reads
    qv = w.q_decode[0][:, None].repeat(1, 3, 1, 1).contiguous()
    w.q_verify = [qv]
    verify_check(w, pool, [0])


# --------------------------------------------------------------------------
# every geometry the ABI accepts: the generic path (any GQA ratio, head_dim
# 64 / 128 / 256) for bf16 and fp8 pools, one and several key splits
# --------------------------------------------------------------------------

def _ragged(cfg, batch, seq_len, lens, **kw):
    """Workload with its lengths replaced by the (shorter) ragged ones."""
    w, _ = workload(cfg, batch=batch, seq_len=seq_len, n_decode=1, n_verify=1, **kw)
    lens = np.asarray(lens, dtype=np.int32)
    assert np.all((w.full_block_table >= 0).sum(1) * 16 >= lens)
    w.seq_lens[:] = lens
    _CACHE.clear()
    return w, oracle_pool(w)


def _window(w, q_len, seed):
    g = torch.Generator(device="cuda").manual_seed(seed)
    x = torch.randn((w.batch, q_len, w.num_q_heads, w.head_dim), generator=g, device="cuda")
    return (x / float(np.sqrt(w.head_dim))).to(torch.bfloat16)


@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
@pytest.mark.parametrize("D,Hq,Hkv", [(64, 8, 4), (256, 16, 2), (128, 16, 8), (128, 32, 4)])
@pytest.mark.parametrize("L,num_splits", [(900, 0), (3000, 0), (3000, 7)])
def test_generic_path_geometries(kv_dtype, D, Hq, Hkv, L, num_splits):
    # lengths L, L - 1 and 37 (partial last pages); with this few query rows
    # the generic path splits the keys into pieces of 4 pages and more (9-15
    # splits at 900 tokens, 9-47 at 3000, by call); num_splits = 7 asks for
    # at least seven
    cfg = 2 if kv_dtype == "bf16" else 5
    # (the ragged fp8 recipe draws its lengths from [4096, seq_len])
    w, pool = _ragged(cfg, 3, max(L, 1000) if cfg == 2 else 5000, [L, L - 1, 37],
                      num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D)
    decode_check(w, pool, [0], num_splits=num_splits)
    q = _window(w, 5, D + Hq + L)
    o, lse = K.verify(kv_of(w), q, dev_i32(w.seq_lens), dev_i32(w.full_block_table), L, 1.0,
                      num_splits=num_splits)
    torch.cuda.synchronize()
    eo, el = O.verify(pool, q.float().cpu().numpy(), w.seq_lens, w.full_block_table, 1.0)
    assert_close("generic verify O", o.cpu().numpy(), eo, O_TOL)
    assert_close("generic verify LSE", lse.cpu().numpy(), el, LSE_TOL)


# --------------------------------------------------------------------------
# page ids outside [0, num_pages) contribute no keys
# --------------------------------------------------------------------------

@pytest.mark.parametrize("kv_dtype,D", [("bf16", 128), ("fp8", 128), ("bf16", 64), ("fp8", 256)])
def test_out_of_pool_page_ids_contribute_no_keys(kv_dtype, D):
    # the library is told the pool holds fewer pages than the tensors do, so
    # the ids past that count name allocated memory that must still not be
    # read; views and tables also carry negative ids. D = 128 runs the tuned
    # kernels, D = 64 / 256 the generic path.
    cfg = 2 if kv_dtype == "bf16" else 5
    w, _ = workload(cfg, batch=3, seq_len=5000, n_decode=1, n_verify=1, head_dim=D)
    small = w.num_pages - w.num_pages // 4
    sc = w.kv_scales[0]
    kv = K.KVCache(w.k_pages[0][:small], w.v_pages[0][:small], w.num_q_heads, torch.bfloat16,
                   None if sc is None else sc[:small].contiguous())
    k, v, hsc = w.host_kv()
    pool = O.KVPool(k[:small], v[:small], w.kv_dtype, None if hsc is None else hsc[:small])
    fbt = np.array(w.full_block_table)
    fbt[0, 3] = -1
    fbt[1, 0] = -100000
    assert (fbt >= small).any() and ((fbt >= 0) & (fbt < small)).any()
    plans = oracle_plan(w)          # compiled against the whole pool
    cap = w.max_pages_per_seq
    vbt, vlb, nb = plan_view_arrays(plans, cap)
    vbt[2, 0] = -3
    seq = dev_i32(w.seq_lens)
    for ns in (0, 3):
        o, lse = K.selected_decode(kv, w.q_decode[0], seq, dev_i32(vbt), dev_i32(vlb),
                                   dev_i32(nb), cap, 1.0, num_splits=ns)
        torch.cuda.synchronize()
        eo, el = O.selected_decode(pool, w.q_decode[0].float().cpu().numpy(), w.seq_lens, vbt,
                                   vlb, nb, 1.0)
        assert_close("decode O", o.cpu().numpy(), eo, O_TOL)
        assert_close("decode LSE", lse.cpu().numpy(), el, LSE_TOL)
        q = _window(w, 5, 77 + ns)
        ov, lv = K.verify(kv, q, seq, dev_i32(fbt), int(w.seq_lens.max()), 1.0, num_splits=ns)
        torch.cuda.synchronize()
        ev, elv = O.verify(pool, q.float().cpu().numpy(), w.seq_lens, fbt, 1.0)
        assert_close("verify O", ov.cpu().numpy(), ev, O_TOL)
        assert_close("verify LSE", lv.cpu().numpy(), elv, LSE_TOL)


# --------------------------------------------------------------------------
# the workspace contract: all zero between calls, shareable by any sequence
# of decode and verify calls
# --------------------------------------------------------------------------

@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8"])
def test_shared_workspace(kv_dtype):
    # one workspace serves decode and verify calls of the tuned kernels
    # (balanced and uniform splits) and of the generic path in turn, so each
    # call finds the previous calls' partials in it; after every call
    # its arrival-counter block is zero again, and every result equals the
    # same call's result with a fresh workspace
    cfg = 2 if kv_dtype == "bf16" else 5
    w, _ = workload(cfg, batch=3, seq_len=6000, n_decode=1, n_verify=1)
    # (the same batch for every call: the counter block grows with batch * Hkv)
    w64, _ = _ragged(cfg, 3, 6000 if cfg == 5 else 3000, [2500, 700, 37], head_dim=64)
    kv, kv64 = kv_of(w), kv_of(w64)
    plan = gpu_plan(w)
    cap = w.max_pages_per_seq
    seq = dev_i32(w.seq_lens)
    fbt = dev_i32(w.full_block_table)
    L = int(w.seq_lens.max())
    qv = _window(w, 5, 11)
    fbt64 = dev_i32(w64.full_block_table)
    qv64 = _window(w64, 3, 12)
    need = max(K.selected_decode_workspace_bytes(kv, 3, cap, ns) for ns in (0, 3))
    need = max(need, *(K.verify_workspace_bytes(kv, 3, 5, L, ns) for ns in (0, 5)),
               K.verify_workspace_bytes(kv64, 3, 3, 2500, 0))
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda")
    # everything past the counters is scratch: start it as random bytes (words
    # that decode as records of an earlier call included)
    ctr = 64 * 3 * 8
    g = torch.Generator(device="cuda").manual_seed(5)
    ws[ctr:] = torch.randint(0, 256, (need - ctr,), generator=g, device="cuda",
                             dtype=torch.int32).to(torch.uint8)
    calls = [
        ("decode auto", lambda **k: K.selected_decode(
            kv, w.q_decode[0], seq, plan["view_block_table"], plan["view_logical_block"],
            plan["view_num_blocks"], cap, 1.0, **k)),
        ("verify auto", lambda **k: K.verify(kv, qv, seq, fbt, L, 1.0, **k)),
        ("generic verify", lambda **k: K.verify(kv64, qv64, dev_i32(w64.seq_lens), fbt64, 2500,
                                                1.0, **k)),
        ("decode 3 splits", lambda **k: K.selected_decode(
            kv, w.q_decode[0], seq, plan["view_block_table"], plan["view_logical_block"],
            plan["view_num_blocks"], cap, 1.0, num_splits=3, **k)),
        ("verify 5 splits", lambda **k: K.verify(kv, qv, seq, fbt, L, 1.0, num_splits=5, **k)),
    ]
    for rep in range(2):
        for name, fn in calls:
            o, l = fn(workspace=ws)
            torch.cuda.synchronize()
            assert int(torch.count_nonzero(ws[:ctr])) == 0, f"{name}: counters not zero"
            o2, l2 = fn()
            torch.cuda.synchronize()
            assert torch.equal(o, o2) and torch.equal(l, l2), name
