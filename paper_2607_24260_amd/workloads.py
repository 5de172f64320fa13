"""Seeded synthetic inputs for the selected-KV decode / verify path.

This module only draws inputs: KV pools, query tokens, page tables, evidence
spans with prior scores, budgets, proposal lengths and accept-length draws. It
holds none of the method's arithmetic (no selection, no attention), so both the
GPU path and the CPU checker can consume what it produces.

Shapes follow the paper's workloads: a nested long-context sweep from 4K to
128K tokens (Sec. 5.1, "Context-length control"), a 5.5% retained-KV ratio at 128K
(Table 2), bf16 KV (Sec. 5.1, "Model and serving backend"), self-speculation with a k+1 verify window
(Sec. 3.2). The model, the dataset and the Graph-RAG frontend are not
available, so everything here is synthetic:

* K, V and Q are iid N(0, 1); Q is pre-scaled by 1/sqrt(head_dim) and stored
  in the query dtype, so the softmax scale passed to the kernels is 1.
* Physical KV pages are a seeded random permutation of one pool shared by the
  whole batch (a shuffled physical page order).
* Evidence spans have seeded starts and lengths; prior scores are
  Dirichlet(0.5) (or derived from a parent span for the graph-expansion
  workload) and stored as float32.
* Budgets are integers floor(frac * L), computed here in float64.
* fp8 KV: each page's K (and V) is divided by amax(page)/448 and rounded to
  OCP E4M3FN by torch; the per-page scales are stored in float32.

KV layout (as stored for the library):
  k_pages [num_pages][Hkv][D/8][16][8]  8-dim chunks, then tokens, within a page
  v_pages [num_pages][Hkv][D][16]       dim-major within a page
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np
import torch

PAGE = 16
SEED_BASE = 20261202

KV_STORAGE = {"f32": torch.float32, "bf16": torch.bfloat16, "fp8": torch.uint8}
Q_STORAGE = {"f32": torch.float32, "bf16": torch.bfloat16}


@dataclass
class Workload:
    name: str
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    kv_dtype: str
    q_dtype: str
    seq_lens: np.ndarray            # int32 [B]
    num_pages: int
    full_block_table: np.ndarray    # int32 [B][stride], -1 past each sequence
    span_offsets: np.ndarray        # int32 [B+1]
    span_start: np.ndarray          # int32 [S]
    span_len: np.ndarray            # int32 [S]
    span_prior: np.ndarray          # float32 [S]
    prefix: np.ndarray              # int32 [B]
    suffix: np.ndarray              # int32 [B]
    budget: np.ndarray              # int32 [B]
    sm_scale: float
    k_pages: List[torch.Tensor]     # one pool per replica
    v_pages: List[torch.Tensor]
    kv_scales: List[Optional[torch.Tensor]]
    q_decode: torch.Tensor          # [n_decode][B][Hq][D]
    q_verify: List[torch.Tensor]    # per verify call: [B][q_len][Hq][D]
    schedule: List[tuple] = field(default_factory=list)   # ('decode', i) / ('verify', j)
    accept_draws: Optional[np.ndarray] = None             # [n_verify][B], geometric - 1
    notes: str = ""

    @property
    def fbt_stride(self) -> int:
        return int(self.full_block_table.shape[1])

    @property
    def max_pages_per_seq(self) -> int:
        return int(-(-int(self.seq_lens.max()) // PAGE))

    def host_kv(self, replica: int = 0):
        """Raw KV bits on the host: (k, v, scales) as numpy arrays.

        bf16 is returned as uint16 bit patterns and fp8 as uint8 bit patterns.
        """
        k = self.k_pages[replica].cpu()
        v = self.v_pages[replica].cpu()
        if self.kv_dtype == "bf16":
            k, v = k.view(torch.int16), v.view(torch.int16)
            kn, vn = k.numpy().view(np.uint16), v.numpy().view(np.uint16)
        else:
            kn, vn = k.numpy(), v.numpy()
        sc = self.kv_scales[replica]
        return kn, vn, (None if sc is None else sc.cpu().numpy())


def config_seed(config: int) -> int:
    return SEED_BASE + 1000 * config


# --------------------------------------------------------------------------
# building blocks
# --------------------------------------------------------------------------

def page_tables(seq_lens: np.ndarray, rng: np.random.Generator, spare_pages: int = 0):
    """Shuffled physical pages for every sequence of a batch.

    Returns (num_pages, full_block_table [B][max_pages] int32, -1 padded).
    """
    npg = [-(-int(L) // PAGE) for L in seq_lens]
    total = int(sum(npg)) + int(spare_pages)
    perm = rng.permutation(total).astype(np.int32)
    stride = max(npg) if npg else 1
    fbt = np.full((len(seq_lens), max(stride, 1)), -1, dtype=np.int32)
    off = 0
    for b, n in enumerate(npg):
        fbt[b, :n] = perm[off:off + n]
        off += n
    return total, fbt


def kv_pool(num_pages: int, Hkv: int, D: int, dtype: str, seed: int, device):
    """iid N(0,1) K and V pools in the library's page layout."""
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    store = KV_STORAGE[dtype]
    k = torch.empty((num_pages, Hkv, D // 8, PAGE, 8), dtype=store, device=device)
    v = torch.empty((num_pages, Hkv, D, PAGE), dtype=store, device=device)
    scales = (torch.empty((num_pages, 2), dtype=torch.float32, device=device)
              if dtype == "fp8" else None)
    chunk = max(1, (64 << 20) // (Hkv * PAGE * D * 4))
    for which, dst in ((0, k), (1, v)):
        for p0 in range(0, num_pages, chunk):
            p1 = min(num_pages, p0 + chunk)
            x = torch.randn(dst[p0:p1].shape, generator=gen, device=device,
                            dtype=torch.float32)
            if dtype == "f32":
                dst[p0:p1] = x
            elif dtype == "bf16":
                dst[p0:p1] = x.to(torch.bfloat16)
            else:
                amax = x.abs().flatten(1).amax(dim=1)
                sc = amax / 448.0
                y = (x / sc.view(-1, *([1] * (x.dim() - 1)))).clamp_(-448.0, 448.0)
                dst[p0:p1] = y.to(torch.float8_e4m3fn).view(torch.uint8)
                scales[p0:p1, which] = sc
    return k, v, scales


def queries(shape, q_dtype: str, head_dim: int, seed: int, device):
    """iid N(0,1) queries pre-scaled by 1/sqrt(head_dim), in the query dtype."""
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    x = torch.randn(shape, generator=gen, device=device, dtype=torch.float32)
    x = x * (1.0 / math.sqrt(head_dim))
    return x.to(Q_STORAGE[q_dtype])


def ranked_spans(rng: np.random.Generator, L: int, n: int, len_lo: int, len_hi: int):
    """n candidate spans with lengths 16*round(U[len_lo, len_hi]/16) and uniform
    (not page-aligned) starts; prior scores Dirichlet(0.5)."""
    lens = (PAGE * np.round(rng.uniform(len_lo, len_hi, n) / PAGE)).astype(np.int64)
    lens = np.clip(lens, PAGE, max(PAGE, L))
    starts = np.array([rng.integers(0, max(1, L - int(l)) + 1) for l in lens], dtype=np.int64)
    prior = rng.dirichlet(np.full(n, 0.5)).astype(np.float32)
    return starts.astype(np.int32), lens.astype(np.int32), prior


def graph_spans(rng: np.random.Generator, L: int, n_seeds: int = 40):
    """Graph-expansion candidates: seed spans with Dirichlet(0.5) priors, each
    with 0..3 neighbouring spans within +-2048 tokens whose prior is the parent's
    times U(0.1, 0.9)."""
    s_start, s_len, s_prior = ranked_spans(rng, L, n_seeds, 64, 512)
    starts, lens, pri = list(s_start), list(s_len), list(s_prior)
    for i in range(n_seeds):
        for _ in range(int(rng.integers(0, 4))):
            ln = int(PAGE * np.round(rng.uniform(64, 512) / PAGE))
            st = int(s_start[i]) + int(rng.integers(-2048, 2049))
            st = min(max(st, 0), max(0, L - 1))
            starts.append(st)
            lens.append(ln)
            pri.append(np.float32(s_prior[i] * rng.uniform(0.1, 0.9)))
    return (np.asarray(starts, dtype=np.int32), np.asarray(lens, dtype=np.int32),
            np.asarray(pri, dtype=np.float32))


def budget_tokens(frac, seq_lens) -> np.ndarray:
    return np.array([math.floor(float(f) * int(L)) for f, L in
                     zip(np.broadcast_to(frac, len(seq_lens)), seq_lens)], dtype=np.int32)


def _csr(per_seq):
    offs = [0]
    st, ln, pr = [], [], []
    for s, l, p in per_seq:
        st.append(s); ln.append(l); pr.append(p)
        offs.append(offs[-1] + len(s))
    cat = (lambda xs, dt: np.concatenate(xs).astype(dt) if xs else np.zeros(0, dt))
    return (np.asarray(offs, dtype=np.int32), cat(st, np.int32), cat(ln, np.int32),
            cat(pr, np.float32))


# --------------------------------------------------------------------------
# the five workloads
# --------------------------------------------------------------------------

DESCRIPTIONS = {
    1: "tiny: B=1, L=4096, fp32 KV, 64+8x128+64-token plan (28.125%), 1 decode + 1 verify(q=5)",
    2: "B=8, L=16384, bf16 KV, 15% budget, 32 decode + 8 verify(gamma=4)",
    3: "B=16, L=32768, bf16 KV, 10% graph-expansion plan (+ all-blocks plan), 32 decode + 8 verify(gamma=4)",
    4: "B=4, L=131072, bf16 KV, 5.5% plan, 64 decode + 16 verify(gamma=4)",
    5: "64 ragged seqs, L log-uniform in [4096,131072], fp8 E4M3FN KV + per-page scales, "
       "budgets U[3%,30%], gamma in {2,4,8}, geometric(0.6) accepts",
}


def make_workload(config: int, device="cpu", replicas: int = 1, batch: Optional[int] = None,
                  seq_len: Optional[int] = None, seed: Optional[int] = None,
                  n_decode: Optional[int] = None, n_verify: Optional[int] = None,
                  num_q_heads: int = 32, num_kv_heads: int = 8, head_dim: int = 128,
                  with_kv: bool = True, budget_frac: Optional[float] = None) -> Workload:
    """Build workload ``config`` (1..5). ``batch`` / ``seq_len`` / step counts may
    be shrunk for tests; the recipe is otherwise unchanged. ``with_kv=False``
    skips drawing the KV pools (plan-only use). ``budget_frac`` replaces the
    budget fraction of workloads 2-4 (for sweeps over the retained ratio)."""
    seed = config_seed(config) if seed is None else seed
    rng = np.random.Generator(np.random.PCG64(seed))
    Hq, Hkv, D = num_q_heads, num_kv_heads, head_dim
    q_dtype = "bf16"
    gammas = None
    accept = None

    if config == 1:
        B = batch or 1
        L = seq_len or 4096
        kv_dtype, q_dtype = "f32", "f32"
        seq_lens = np.full(B, L, dtype=np.int32)
        per = []
        for _ in range(B):
            units = (L - 128) // PAGE            # 16-token units in [64, L-64)
            free = units - 8 * 8
            gaps = np.sort(rng.integers(0, free + 1, 8))
            starts = (64 + PAGE * (gaps + 8 * np.arange(8))).astype(np.int32)
            per.append((starts, np.full(8, 128, np.int32),
                        rng.dirichlet(np.full(8, 0.5)).astype(np.float32)))
        prefix = np.full(B, 64, np.int32)
        suffix = np.full(B, 64, np.int32)
        budget = seq_lens.copy()
        nd, nv, qlen = 1, 1, 5
    elif config == 2:
        B = batch or 8
        L = seq_len or 16384
        kv_dtype = "bf16"
        seq_lens = np.full(B, L, dtype=np.int32)
        per = [ranked_spans(rng, L, 128, 32, 512) for _ in range(B)]
        prefix = np.full(B, 256, np.int32)
        suffix = np.full(B, 128, np.int32)
        budget = budget_tokens(0.15, seq_lens)
        nd, nv, qlen = 32, 8, 5
    elif config == 3:
        B = batch or 16
        L = seq_len or 32768
        kv_dtype = "bf16"
        seq_lens = np.full(B, L, dtype=np.int32)
        per = [graph_spans(rng, L) for _ in range(B)]
        prefix = np.full(B, 256, np.int32)
        suffix = np.full(B, 128, np.int32)
        budget = budget_tokens(0.10, seq_lens)
        nd, nv, qlen = 32, 8, 5
    elif config == 4:
        B = batch or 4
        L = seq_len or 131072
        kv_dtype = "bf16"
        seq_lens = np.full(B, L, dtype=np.int32)
        per = [ranked_spans(rng, L, 128, 64, 1024) for _ in range(B)]
        prefix = np.full(B, 512, np.int32)
        suffix = np.full(B, 256, np.int32)
        budget = budget_tokens(0.055, seq_lens)
        nd, nv, qlen = 64, 16, 5
    elif config == 5:
        B = batch or 64
        lo, hi = math.log(4096), math.log(seq_len or 131072)
        seq_lens = np.array([int(round(math.exp(rng.uniform(lo, hi)))) for _ in range(B)],
                            dtype=np.int32)
        kv_dtype = "fp8"
        per = [ranked_spans(rng, int(L), 128, 64, 1024) for L in seq_lens]
        prefix = np.full(B, 256, np.int32)
        suffix = np.full(B, 128, np.int32)
        budget = budget_tokens(rng.uniform(0.03, 0.30, B), seq_lens)
        cycles = n_verify or 16
        gammas = [int(g) for g in rng.choice([2, 4, 8], size=cycles)]
        accept = (rng.geometric(0.6, size=(cycles, B)) - 1).astype(np.int32)
        nd = int(sum(gammas))
        nv = cycles
        qlen = None
    else:
        raise ValueError(f"unknown workload {config}")

    if budget_frac is not None and config in (2, 3, 4):
        budget = budget_tokens(budget_frac, seq_lens)
    if n_decode is not None and config != 5:
        nd = n_decode
    if n_verify is not None and config != 5:
        nv = n_verify

    num_pages, fbt = page_tables(seq_lens, rng)
    offs, st, ln, pr = _csr(per)

    ks, vs, scs = [], [], []
    for r in range(replicas if with_kv else 0):
        k, v, sc = kv_pool(num_pages, Hkv, D, kv_dtype, seed + 17 + 7919 * r, device)
        ks.append(k); vs.append(v); scs.append(sc)

    qd = queries((nd, B, Hq, D), q_dtype, D, seed + 101, device)
    if config == 5:
        qv = [queries((B, g + 1, Hq, D), q_dtype, D, seed + 211 + c, device)
              for c, g in enumerate(gammas)]
        sched = []
        di = 0
        for c, g in enumerate(gammas):
            for _ in range(g):
                sched.append(("decode", di)); di += 1
            sched.append(("verify", c))
    else:
        qv = [queries((B, qlen, Hq, D), q_dtype, D, seed + 211 + j, device) for j in range(nv)]
        sched = []
        if nv > 0 and nd >= nv:
            per_cycle = nd // nv
            di = 0
            for j in range(nv):
                for _ in range(per_cycle):
                    sched.append(("decode", di)); di += 1
                sched.append(("verify", j))
            while di < nd:
                sched.append(("decode", di)); di += 1
        else:
            sched = [("decode", i) for i in range(nd)] + [("verify", j) for j in range(nv)]

    return Workload(
        name=f"config{config}", batch=B, num_q_heads=Hq, num_kv_heads=Hkv, head_dim=D,
        kv_dtype=kv_dtype, q_dtype=q_dtype, seq_lens=seq_lens, num_pages=num_pages,
        full_block_table=fbt, span_offsets=offs, span_start=st, span_len=ln,
        span_prior=pr, prefix=prefix, suffix=suffix, budget=budget, sm_scale=1.0,
        k_pages=ks, v_pages=vs, kv_scales=scs, q_decode=qd, q_verify=qv,
        schedule=sched, accept_draws=accept, notes=DESCRIPTIONS[config])
