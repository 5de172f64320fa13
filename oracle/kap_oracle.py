"""Plain fp64 CPU oracle for the KAP / GraphSpec selected-KV hot path.

TEST INFRASTRUCTURE. This module is the oracle, not the product: only the
test suite, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import or call it. It shares no code, tables or helpers with
the HIP library or its Python binding, and imports neither.

Paper: "KAP: Bridging the Knowledge Selection--Runtime Consumption Gap in LLM
Systems" (arXiv 2607.24260). What is computed, and where it is defined:

* ``compile_plan`` -- Alg. 1 (GraphSpecCompile), the steps that select evidence
  under a budget, resolve it to KV pages, keep logical positions and build the
  block table (Sec. 3.1, "Evidence-to-runtime compilation" and "Selected-KV
  view materialization"); the plan fields follow Eq. (1).
* ``selected_decode`` -- Sec. 3.2, "Selected-KV proposal": one query token per
  step attends only to the prompt-side KV pages the plan exposes.
* ``verify`` -- Sec. 3.2, "Full-context verification" and Eq. (2): a window of
  k+1 query tokens attends causally to the full KV cache.
* ``append_kv`` / ``compact_view`` -- Sec. 3.1 slot mappings and compact
  workspace (Alg. 1, AssignCompactSlots / BuildBlockTable): placing new
  tokens into their KV slots, and copying a view's pages into a compact
  workspace of fixed capacity.
* ``accept_top_k`` -- Sec. 3.2 target-guided tolerant verification (the
  Top-3 rule): accepted prefix length and the verifier's carry token.
* ``access_modes`` / ``active_view`` -- Sec. 3.2, "Runtime stability and
  fallback": per cycle, whether a sequence's proposal steps read its plan's
  view or the full context (h from Eq. (5) against s from Eq. (4), the
  margin condition h > s of Eq. (12)), and the view rows that mode reads.
* ``lse_merge`` -- the exact softmax identity used to combine attention over
  disjoint key sets (a standard identity, not stated in the paper).
* ``e4m3fn_to_f64`` / ``bf16_to_f64`` -- decoding of stored KV bits (OCP 8-bit
  float E4M3 "FN" encoding; bfloat16 = upper half of an IEEE binary32).

Attention is the plain definition softmax(z) V with z = sm_scale * K q,
computed in fp64. Where the paper is silent this oracle reads it as follows:
visibility is page-granular; view pages are listed in ascending logical order;
the budget counts visible tokens of selected pages, mandatory prefix/suffix
included; a span that does not fit is skipped (or, under the STOP policy, ends
selection); ranking is a total order (prior desc, start asc, index asc);
spans are clipped to [0, L); LSE is the natural log of the scaled logits; the
verify window is the last q_len cached tokens; query head h reads KV head
h // (Hq / Hkv).

Parity status: every function here is pinned by a CPU test against something
other than itself (hand-worked vectors, closed forms, brute force, torch
library routines, invariants); see tests/test_oracle_*.py. The access-mode
policy's window length, its first-cycle grace and its stickiness are this
oracle's reading (the paper names the fallback conditions but gives no
thresholds): its pins fix that stated rule, and parity with the paper's own
thresholds is unpinned.
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from fractions import Fraction
from typing import Optional, Sequence

import numpy as np

PAGE = 16  # tokens per KV page

# Per-sequence plan status codes (reading of the fallback triggers of Sec. 3.2,
# "Runtime stability and fallback": a plan that does not fit the compact
# workspace, or that cannot be executed, is reported so the executor falls back
# to full-context access).
PLAN_OK = 0
PLAN_OVER_CAPACITY = 1
PLAN_BAD_SCORE = 2
PLAN_BAD_PAGE = 3
PLAN_BAD_LENGTH = 4
PLAN_BAD_SPANS = 5

SELECT_SKIP = 0
SELECT_STOP = 1


# --------------------------------------------------------------------------
# Decoding of stored KV bits
# --------------------------------------------------------------------------

def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> exact float64.

    A bfloat16 value is the upper 16 bits of an IEEE-754 binary32 value, so the
    pattern shifted left by 16 is that binary32 value exactly.
    """
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    with np.errstate(invalid="ignore"):        # NaN patterns stay NaN
        return b.view(np.float32).astype(np.float64)


def e4m3fn_to_f64(bits: np.ndarray) -> np.ndarray:
    """OCP FP8 E4M3FN bit patterns (uint8) -> exact float64.

    Encoding: 1 sign bit, 4 exponent bits with bias 7, 3 mantissa bits.
    Exponent field 0 encodes subnormals m/8 * 2^-6; otherwise (1 + m/8) *
    2^(e-7). The patterns S.1111.111 are NaN; there is no infinity, so the
    largest finite magnitude is 1.75 * 2^8 = 448.
    """
    b = np.asarray(bits, dtype=np.uint8).astype(np.int64)
    sign = np.where((b >> 7) & 1, -1.0, 1.0)
    exp = (b >> 3) & 0xF
    man = (b & 0x7).astype(np.float64)
    normal = (1.0 + man / 8.0) * np.exp2(exp.astype(np.float64) - 7.0)
    subnormal = (man / 8.0) * 2.0 ** -6
    mag = np.where(exp == 0, subnormal, normal)
    out = sign * mag
    out = np.where((b & 0x7F) == 0x7F, np.nan, out)
    return out


@dataclass
class KVPool:
    """Stored KV bits, as the GPU library reads them.

    k_pages: [num_pages][Hkv][D/8][PAGE][8]: each page's K tile in 8-dim
             chunks; element [p][g][c][t][e] is dim 8c+e of token t.
    v_pages: [num_pages][Hkv][D][PAGE], dim-major within a page (each page's
             V tile is stored transposed).
    dtype:   'f32' (float32 arrays), 'bf16' (uint16 bit arrays) or
             'fp8' (uint8 E4M3FN bit arrays, with per-page scales).
    scales:  [num_pages][2] float32 (K scale, V scale) for 'fp8', else None.
    """

    k_pages: np.ndarray
    v_pages: np.ndarray
    dtype: str
    scales: Optional[np.ndarray] = None

    def _decode(self, raw: np.ndarray) -> np.ndarray:
        if self.dtype == "f32":
            return np.asarray(raw, dtype=np.float32).astype(np.float64)
        if self.dtype == "bf16":
            return bf16_to_f64(raw)
        if self.dtype == "fp8":
            return e4m3fn_to_f64(raw)
        raise ValueError(f"unknown KV dtype {self.dtype!r}")

    def keys(self, pages: np.ndarray, g: int) -> np.ndarray:
        """K values of the given physical pages for KV head g: [n][PAGE][D]."""
        pages = np.asarray(pages, dtype=np.int64)
        raw = self.k_pages[pages, g]                       # [n][D/8][PAGE][8]
        n, C, T, E = raw.shape
        k = self._decode(raw).transpose(0, 2, 1, 3).reshape(n, T, C * E)
        if self.dtype == "fp8":
            k = k * self.scales[pages, 0].astype(np.float64)[:, None, None]
        return k

    def values(self, pages: np.ndarray, g: int) -> np.ndarray:
        """V values of the given physical pages for KV head g: [n][PAGE][D]."""
        pages = np.asarray(pages, dtype=np.int64)
        v = self._decode(self.v_pages[pages, g]).transpose(0, 2, 1)
        if self.dtype == "fp8":
            v = v * self.scales[pages, 1].astype(np.float64)[:, None, None]
        return v


# --------------------------------------------------------------------------
# Plan compilation (Alg. 1)
# --------------------------------------------------------------------------

@dataclass
class Plan:
    status: int
    logical_blocks: list        # ascending logical page indices (lblk)
    block_table: list           # physical page of each view block (vbt)
    num_blocks: int
    view_tokens: int            # visible tokens of the selected pages
    spans_taken: int
    span_selected: list         # per input span: 1 if selected, else 0
    token_masks: Optional[list] = None   # token-granular plans: visible-token bits per view page


def _pages_of(x: int, e: int) -> set:
    """Logical pages touched by the token range [x, e)."""
    if e <= x:
        return set()
    return set(range(x // PAGE, -(-e // PAGE)))


def compile_plan_one(seq_len: int, fbt_row: Sequence[int], starts: Sequence[int],
                     lens: Sequence[int], priors: Sequence[float], prefix: int,
                     suffix: int, budget: int, policy: int, num_pages: int,
                     capacity: int) -> Plan:
    """Compile the runtime access plan of one sequence (Alg. 1).

    Steps, in the algorithm's order:
      SelectEvidenceUnderBudget -- rank the evidence spans by prior and keep
        them greedily while the visible-token count stays within the budget;
        the mandatory prefix and suffix pages (the suffix always includes the
        page of the current token) are kept first and are never dropped.
      ResolveSelectedKVObjects / PreserveLogicalPositions -- the selected
        spans become the set of logical KV pages they touch, listed in
        ascending logical order (the logical positions).
      BuildBlockTable -- each view block maps to its physical page through the
        sequence's full block table.
    Readings where the paper is silent: see the module docstring.
    """
    n = len(starts)
    L = int(seq_len)
    fail = Plan(PLAN_OK, [], [], 0, 0, 0, [0] * n)

    if L < 1 or -(-L // PAGE) > len(fbt_row):
        fail.status = PLAN_BAD_LENGTH
        return fail
    if any(math.isnan(float(p)) for p in priors):
        fail.status = PLAN_BAD_SCORE
        return fail

    def valid(j: int) -> int:            # tokens of logical page j below L
        return min(PAGE, L - PAGE * j)

    # Mandatory context: the prefix, and a suffix of at least one token so the
    # decoding token's own page is always visible.
    sel = _pages_of(0, min(max(prefix, 0), L))
    sel |= _pages_of(max(0, L - max(suffix, 1)), L)
    used = sum(valid(j) for j in sel)

    # Rank: prior descending, then span start ascending, then input index.
    order = sorted(range(n), key=lambda i: (-float(priors[i]), int(starts[i]), i))

    taken = 0
    flags = [0] * n
    for i in order:
        x = max(0, int(starts[i]))
        e = min(L, int(starts[i]) + int(lens[i]))
        if e <= x:                       # empty after clipping: ignored
            continue
        new = _pages_of(x, e) - sel
        cost = sum(valid(j) for j in new)
        if used + cost <= budget:
            sel |= new
            used += cost
            taken += 1
            flags[i] = 1
        elif policy == SELECT_STOP:
            break

    lblk = sorted(sel)
    if len(lblk) > capacity:
        fail.status = PLAN_OVER_CAPACITY
        return fail
    vbt = [int(fbt_row[j]) for j in lblk]
    if any(p < 0 or p >= num_pages for p in vbt):
        fail.status = PLAN_BAD_PAGE
        return fail
    return Plan(PLAN_OK, lblk, vbt, len(lblk), used, taken, flags)


def compile_plan_tokens_one(seq_len: int, fbt_row: Sequence[int], starts: Sequence[int],
                            lens: Sequence[int], priors: Sequence[float], prefix: int,
                            suffix: int, budget: int, policy: int, num_pages: int,
                            capacity: int) -> Plan:
    """``compile_plan_one`` with token-granular visibility (the visibility mask
    of Sec. 3.1 at token resolution): the selection, the budget and the
    mandatory prefix / suffix are counted in tokens, a span costs the tokens
    it adds, and the view lists every logical page holding a visible token,
    with a 16-bit mask of its visible tokens (bit t = token t of the page).
    Ranking, the SKIP / STOP rule and the status codes are as for pages."""
    n = len(starts)
    L = int(seq_len)
    fail = Plan(PLAN_OK, [], [], 0, 0, 0, [0] * n, [])
    if L < 1 or -(-L // PAGE) > len(fbt_row):
        fail.status = PLAN_BAD_LENGTH
        return fail
    if any(math.isnan(float(p)) for p in priors):
        fail.status = PLAN_BAD_SCORE
        return fail

    sel = set(range(0, min(max(prefix, 0), L)))
    sel |= set(range(max(0, L - max(suffix, 1)), L))
    order = sorted(range(n), key=lambda i: (-float(priors[i]), int(starts[i]), i))
    taken = 0
    flags = [0] * n
    for i in order:
        x = max(0, int(starts[i]))
        e = min(L, int(starts[i]) + int(lens[i]))
        if e <= x:
            continue
        new = set(range(x, e)) - sel
        if len(sel) + len(new) <= budget:
            sel |= new
            taken += 1
            flags[i] = 1
        elif policy == SELECT_STOP:
            break

    lblk = sorted({t // PAGE for t in sel})
    if len(lblk) > capacity:
        fail.status = PLAN_OVER_CAPACITY
        return fail
    vbt = [int(fbt_row[j]) for j in lblk]
    if any(p < 0 or p >= num_pages for p in vbt):
        fail.status = PLAN_BAD_PAGE
        return fail
    masks = [sum(1 << (t - PAGE * j) for t in sel if t // PAGE == j) for j in lblk]
    return Plan(PLAN_OK, lblk, vbt, len(lblk), len(sel), taken, flags, masks)


def compile_plan(seq_lens, full_block_table, span_offsets, span_start, span_len,
                 span_prior, prefix, suffix, budget, policy, num_pages,
                 capacity, token_granular: bool = False) -> list:
    """Batched ``compile_plan_one`` over CSR span arrays; returns a list of Plan.

    Sequence b owns spans span_offsets[b] .. span_offsets[b+1]-1. Malformed CSR
    bounds give PLAN_BAD_SPANS for that sequence. ``token_granular`` selects
    ``compile_plan_tokens_one``.
    """
    out = []
    total = len(span_start)
    for b in range(len(seq_lens)):
        lo, hi = int(span_offsets[b]), int(span_offsets[b + 1])
        if lo < 0 or hi < lo or hi > total:
            out.append(Plan(PLAN_BAD_SPANS, [], [], 0, 0, 0, [],
                            [] if token_granular else None))
            continue
        one = compile_plan_tokens_one if token_granular else compile_plan_one
        out.append(one(
            int(seq_lens[b]), full_block_table[b], span_start[lo:hi],
            span_len[lo:hi], span_prior[lo:hi], int(prefix[b]), int(suffix[b]),
            int(budget[b]), policy, num_pages, capacity))
    return out


# --------------------------------------------------------------------------
# Attention
# --------------------------------------------------------------------------

def attend(q: np.ndarray, k: np.ndarray, v: np.ndarray, n_visible: Sequence[int],
           sm_scale: float):
    """Softmax attention of query rows over a visible prefix of a key list.

    q: [R][D], k and v: [T][D] (float64). Row r sees keys 0 .. n_visible[r]-1.
    Returns o [R][D] and natural-log lse [R] of the scaled logits
    z = sm_scale * k q. A row with no visible key gives o = 0, lse = -inf.
    """
    q = np.asarray(q, dtype=np.float64)
    R, D = q.shape
    o = np.zeros((R, D), dtype=np.float64)
    lse = np.full(R, -np.inf, dtype=np.float64)
    for r in range(R):
        n = int(max(0, min(int(n_visible[r]), k.shape[0])))
        if n == 0:
            continue
        z = sm_scale * (k[:n] @ q[r])
        m = z.max()
        w = np.exp(z - m)
        den = w.sum()
        o[r] = (w @ v[:n]) / den
        lse[r] = m + math.log(den)
    return o, lse


def _view_tokens(pool: KVPool, g: int, seq_len: int, pages, lblks, skip_invalid: bool = True,
                 masks=None):
    """K and V of the visible tokens of a list of (physical, logical) pages.

    A view entry whose page id lies outside the pool contributes no keys (the
    reading the boundary documents for ids kap_compile_plan would report as
    KAP_PLAN_BAD_PAGE)."""
    pages = np.asarray(pages, dtype=np.int64)
    lblks = np.asarray(lblks, dtype=np.int64)
    masks = (np.full(len(pages), 0xFFFF, dtype=np.int64) if masks is None
             else np.asarray(masks, dtype=np.int64))
    if skip_invalid:
        ok = (pages >= 0) & (pages < pool.k_pages.shape[0])
        pages, lblks, masks = pages[ok], lblks[ok], masks[ok]
    if len(pages) == 0:
        D = pool.v_pages.shape[2]
        return np.zeros((0, D)), np.zeros((0, D))
    nvalid = np.clip(seq_len - PAGE * lblks, 0, PAGE)
    t = np.arange(PAGE)[None, :]
    mask = (t < nvalid[:, None]) & (((masks[:, None] >> t) & 1) == 1)   # [n][PAGE]
    k = pool.keys(pages, g)[mask]
    v = pool.values(pages, g)[mask]
    return k, v


def selected_decode(pool: KVPool, q: np.ndarray, seq_lens, view_block_table,
                    view_logical_block, view_num_blocks, sm_scale: float,
                    view_token_mask=None):
    """One proposal step over the selected-KV view (Sec. 3.2, q_prop = 1).

    q: [B][Hq][D] (any float dtype; promoted to fp64). Sequence b sees the
    first view_num_blocks[b] view blocks; block k is physical page
    view_block_table[b][k] holding logical page view_logical_block[b][k], whose
    tokens below seq_lens[b] are visible. Query head h uses KV head
    h // (Hq / Hkv). With ``view_token_mask`` [B][cap] (token-granular
    plans), token t of view block k is visible only if bit t of its mask is
    set. Returns o [B][Hq][D] and lse [B][Hq] in float64.
    """
    q = np.asarray(q, dtype=np.float64)
    B, Hq, D = q.shape
    Hkv = pool.k_pages.shape[1]
    G = Hq // Hkv
    o = np.zeros((B, Hq, D))
    lse = np.full((B, Hq), -np.inf)
    for b in range(B):
        nb = int(view_num_blocks[b])
        pages = np.asarray(view_block_table[b])[:nb]
        lblks = np.asarray(view_logical_block[b])[:nb]
        masks = None if view_token_mask is None else np.asarray(view_token_mask[b])[:nb]
        for g in range(Hkv):
            k, v = _view_tokens(pool, g, int(seq_lens[b]), pages, lblks, masks=masks)
            rows = q[b, g * G:(g + 1) * G]
            ob, lb = attend(rows, k, v, [k.shape[0]] * G, sm_scale)
            o[b, g * G:(g + 1) * G] = ob
            lse[b, g * G:(g + 1) * G] = lb
    return o, lse


def full_tokens(pool: KVPool, g: int, seq_len: int, fbt_row):
    """K, V and logical positions of the tokens 0 .. seq_len-1 of one
    sequence, in logical order. A page whose id lies outside the pool
    contributes no keys (as for views), so its positions are absent."""
    npages = -(-int(seq_len) // PAGE)
    pages = np.asarray(fbt_row, dtype=np.int64)[:npages]
    k, v = _view_tokens(pool, g, int(seq_len), pages, np.arange(npages))
    ok = (pages >= 0) & (pages < pool.k_pages.shape[0])
    grid = PAGE * np.arange(npages)[:, None] + np.arange(PAGE)[None, :]   # [page][token]
    pos = grid[ok[:, None] & (grid < int(seq_len))]                        # row-major: ascending
    return k, v, pos


def verify(pool: KVPool, q: np.ndarray, seq_lens, full_block_table,
           sm_scale: float, batches: Optional[Sequence[int]] = None,
           kv_heads: Optional[Sequence[int]] = None):
    """Full-context verification attention (Sec. 3.2, Eq. (2)).

    q: [B][q_len][Hq][D]: the carry token and the k proposed tokens. Their K/V
    are the last q_len tokens of the cache, so seq_lens[b] counts them. Window
    row i sees the keys at logical positions 0 .. seq_lens[b] - q_len + i
    (causal among the window). Returns o [B][q_len][Hq][D] and lse
    [B][q_len][Hq] in float64. ``batches`` / ``kv_heads`` restrict the work to
    a subset (other entries are left as o = 0, lse = -inf).
    """
    q = np.asarray(q, dtype=np.float64)
    B, QL, Hq, D = q.shape
    Hkv = pool.k_pages.shape[1]
    G = Hq // Hkv
    o = np.zeros((B, QL, Hq, D))
    lse = np.full((B, QL, Hq), -np.inf)
    for b in (range(B) if batches is None else batches):
        L = int(seq_lens[b])
        for g in (range(Hkv) if kv_heads is None else kv_heads):
            k, v, pos = full_tokens(pool, g, L, full_block_table[b])
            # keys are in ascending position: row i sees a prefix of them
            nvis = [int(np.sum(pos <= L - QL + i)) for i in range(QL)]
            for h in range(g * G, (g + 1) * G):
                ob, lb = attend(q[b, :, h], k, v, nvis, sm_scale)
                o[b, :, h] = ob
                lse[b, :, h] = lb
    return o, lse


def lse_merge(o_parts: np.ndarray, lse_parts: np.ndarray):
    """Combine attention over disjoint key sets.

    o_parts: [S][R][D], lse_parts: [S][R]; part s is softmax attention over
    key set s with log-sum-exp lse_parts[s]. The attention over the union has
    lse = log sum_s exp(lse_s) and o = sum_s exp(lse_s - lse) o_s. Parts with
    lse = -inf (no keys) contribute nothing.
    """
    o_parts = np.asarray(o_parts, dtype=np.float64)
    lse_parts = np.asarray(lse_parts, dtype=np.float64)
    S, R, D = o_parts.shape
    o = np.zeros((R, D))
    lse = np.full(R, -np.inf)
    for r in range(R):
        finite = [s for s in range(S) if np.isfinite(lse_parts[s, r])]
        if not finite:
            continue
        m = max(lse_parts[s, r] for s in finite)
        tot = sum(math.exp(lse_parts[s, r] - m) for s in finite)
        lse[r] = m + math.log(tot)
        for s in finite:
            o[r] += math.exp(lse_parts[s, r] - lse[r]) * o_parts[s, r]
    return o, lse


def split_attend(q: np.ndarray, k: np.ndarray, v: np.ndarray, bounds: Sequence[int],
                 sm_scale: float):
    """Attention over keys split at ``bounds`` and recombined by ``lse_merge``.

    bounds: non-decreasing cut points 0 = c_0 <= c_1 <= ... <= c_S = T; part s
    covers keys [c_s, c_{s+1}) (possibly empty). All rows see every key.
    """
    parts_o, parts_l = [], []
    R = q.shape[0]
    for s in range(len(bounds) - 1):
        lo, hi = bounds[s], bounds[s + 1]
        ob, lb = attend(q, k[lo:hi], v[lo:hi], [hi - lo] * R, sm_scale)
        parts_o.append(ob)
        parts_l.append(lb)
    return lse_merge(np.stack(parts_o), np.stack(parts_l))


# --------------------------------------------------------------------------
# KV maintenance: slot-mapped append and view compaction
# --------------------------------------------------------------------------

def append_kv(pool: KVPool, k_new: np.ndarray, v_new: np.ndarray, slot_mapping):
    """Place new tokens' stored K/V values into their physical slots.

    Sec. 3.1 ("Selected-KV view materialization"): slot mappings place newly
    scheduled tokens into their KV slots; Sec. 3.2 ("Full-context
    verification"): this is how the full-context state KV^{full,+} advances.

    k_new / v_new: [T][Hkv][D] in the pool's storage dtype. Token t goes to
    slot s = slot_mapping[t] = page * PAGE + offset: dim d of KV head g is
    element [page][g][d // 8][offset][d % 8] of k_pages and [page][g][d][offset]
    of v_pages. Negative slots are skipped; slots past the pool are skipped
    and counted. Returns (new pool, number of out-of-range slots).
    """
    k = np.array(pool.k_pages, copy=True)
    v = np.array(pool.v_pages, copy=True)
    P, Hkv, C, _, E = k.shape
    bad = 0
    for t, s in enumerate(np.asarray(slot_mapping, dtype=np.int64)):
        s = int(s)
        if s < 0:
            continue
        if s >= P * PAGE:
            bad += 1
            continue
        page, off = divmod(s, PAGE)
        k[page, :, :, off, :] = np.asarray(k_new[t]).reshape(Hkv, C, E)
        v[page, :, :, off] = np.asarray(v_new[t])
    return KVPool(k, v, pool.dtype, pool.scales), bad


def compact_view(pool: KVPool, view_block_table, view_num_blocks, capacity: int):
    """Copy each sequence's selected pages into a compact workspace.

    Alg. 1, AssignCompactSlots and BuildBlockTable; Sec. 3.1: the selected
    pages are compacted in access order into a workspace of fixed capacity.
    View entry k < min(view_num_blocks[b], capacity) of sequence b (a valid
    page id) goes to compact page b * capacity + k (K, V and fp8 scales);
    the compact block table holds that page, or -1. Compact pages that receive
    nothing are left zero. Returns (compact pool, table [B][capacity]).
    """
    vbt = np.asarray(view_block_table, dtype=np.int64)
    nb = np.asarray(view_num_blocks, dtype=np.int64)
    B = len(nb)
    P = pool.k_pages.shape[0]
    k = np.zeros((B * capacity,) + pool.k_pages.shape[1:], dtype=pool.k_pages.dtype)
    v = np.zeros((B * capacity,) + pool.v_pages.shape[1:], dtype=pool.v_pages.dtype)
    sc = None if pool.scales is None else np.zeros((B * capacity, 2), dtype=np.float32)
    table = np.full((B, capacity), -1, dtype=np.int64)
    for b in range(B):
        for j in range(min(int(nb[b]), capacity)):
            p = int(vbt[b, j])
            if not 0 <= p < P:
                continue
            dst = b * capacity + j
            k[dst] = pool.k_pages[p]
            v[dst] = pool.v_pages[p]
            if sc is not None:
                sc[dst] = pool.scales[p]
            table[b, j] = dst
    return KVPool(k, v, pool.dtype, sc), table


# --------------------------------------------------------------------------
# Access mode per cycle: the selected view or full-context fallback
# --------------------------------------------------------------------------

SELECTED = 0   # proposal steps read the plan's selected-KV view
FULL = 1       # proposal steps read the whole context


def access_modes(plan_status, view_tokens, seq_lens, accepted, gammas, window: int):
    """Access mode of every sequence at the start and after each cycle.

    Sec. 3.2 ("Runtime stability and fallback") has the executor read the
    full context instead of the plan when the plan cannot be executed (it
    exceeds the compact workspace, or is otherwise unusable) or when the
    observed acceptance is low for the KV the plan retains. The quantities
    are s, the retained ratio of Eq. (4) -- here view_tokens[b] / seq_lens[b],
    the proposal path's visible tokens over the full context's -- and h, the
    acceptance rate of Eq. (5), accepted over speculated proposed tokens;
    Eq. (12) gives h > s as the condition for a positive KV-access margin.

    Reading used (the paper names the conditions, not thresholds):
      * a sequence starts on its plan (SELECTED) iff plan_status[b] is OK
        (0), else on the full context (FULL);
      * cycle c speculates gammas[c] tokens per sequence, of which
        min(max(accepted[c][b], 0), gammas[c]) are accepted;
      * once a sequence has completed at least two cycles, h is taken over
        its last ``window`` cycles (sum accepted / sum speculated); if that
        sum speculated is positive and h <= s, the sequence switches to FULL;
      * FULL is kept for the rest of the run.
    h and s are compared as exact rationals.

    accepted: [C][B] integers, gammas: [C]. Returns an int64 array
    [C + 1][B]: row 0 holds the modes before the first cycle, row c + 1 the
    modes after cycle c.
    """
    B = len(seq_lens)
    C = len(gammas)
    modes = np.zeros((C + 1, B), dtype=np.int64)
    for b in range(B):
        mode = SELECTED if int(plan_status[b]) == PLAN_OK else FULL
        modes[0, b] = mode
        history = []                     # (accepted, speculated) per cycle
        s = Fraction(int(view_tokens[b]), int(seq_lens[b])) if int(seq_lens[b]) > 0 else None
        for c in range(C):
            g = int(gammas[c])
            a = min(max(int(accepted[c][b]), 0), g)
            history.append((a, g))
            if mode == SELECTED and len(history) >= 2 and s is not None:
                recent = history[-window:]
                acc = sum(x for x, _ in recent)
                spec = sum(y for _, y in recent)
                if spec > 0 and Fraction(acc, spec) <= s:
                    mode = FULL
            modes[c + 1, b] = mode
    return modes


def active_view(mode: int, plan: Plan, full_block_table_row, seq_len: int):
    """The view rows a proposal step of one sequence reads in a given mode.

    SELECTED: the plan's view (its physical pages, logical pages and, for a
    token-granular plan, its token masks). FULL: every page of the context
    that the full block table holds, in logical order, each with all 16
    tokens marked visible. Returns (block_table, logical_blocks, num_blocks,
    token_masks) as lists; token_masks is None for a page-granular plan.
    """
    masked = plan.token_masks is not None
    if mode == SELECTED:
        n = plan.num_blocks
        masks = list(plan.token_masks[:n]) if masked else None
        return list(plan.block_table[:n]), list(plan.logical_blocks[:n]), n, masks
    row = list(full_block_table_row)
    n = min(-(-int(seq_len) // PAGE), len(row)) if seq_len > 0 else 0
    return row[:n], list(range(n)), n, ([0xFFFF] * n if masked else None)


# --------------------------------------------------------------------------
# Tolerant acceptance of a verify window
# --------------------------------------------------------------------------

def token_rank(row: np.ndarray, d: int) -> int:
    """Rank of token d in a logits row: the number of tokens that come before
    it when the row is ordered by logit (largest first), ties broken by the
    lower token index."""
    x = np.asarray(row, dtype=np.float64)
    idx = np.arange(len(x))
    return int(np.sum((x > x[d]) | ((x == x[d]) & (idx < d))))


def accept_top_k(logits: np.ndarray, drafts: np.ndarray, top_k: int = 3):
    """Sec. 3.2 ("Full-context verification"): the verifier accepts a proposed
    token when it lies within its top candidates under the full context (the
    paper's Top-3 rule); the accepted count m is the number of leading
    accepted proposals, and the verifier's next (carry) token is its choice at
    position m.

    logits [B][window][vocab]: the verifier's logits at the window positions;
    drafts [B][window-1]: proposed tokens (draft i is scored in row i).
    Returns (m [B], carry [B]); carry = argmax of row m (lowest index among
    equal maxima). A draft outside [0, vocab) is never accepted."""
    logits = np.asarray(logits, dtype=np.float64)
    B, Wn, V = logits.shape
    m = np.zeros(B, dtype=np.int64)
    carry = np.zeros(B, dtype=np.int64)
    for b in range(B):
        i = 0
        while i < Wn - 1:
            d = int(drafts[b][i])
            if not 0 <= d < V or token_rank(logits[b, i], d) >= top_k:
                break
            i += 1
        m[b] = i
        carry[b] = int(np.argmax(logits[b, i]))
    return m, carry
