"""Throughput of the KAP selected-KV hot path on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config 4]

A step is one pass of the whole hot path over one batch: kap_compile_plan,
kap_decode_schedule (the decode calls' split assignment for the plan's view,
written once), then the proposal / verify schedule of the workload (for the 128K
workload: 64 selected-view decode calls and 16 verify calls with a gamma = 4
window, interleaved 4 : 1). Every call reads the KV pool of its own "layer replica";
the replicas rotate so that the bytes touched between two reads of the same
buffer far exceed the 256 MB Infinity Cache -- the numbers are HBM numbers.

Printed: one JSON line (rank 0). `value` is effective KV GB/s of the whole
step (algorithmic bytes / step time); decode steps/s, verify calls/s, the
roofline of the dominant call (kap_verify) and of decode, and `per_config`:
plan / decode / verify per call for every workload (1-3 timed here, 5 from its
device-resident stream), each beside the fp64 oracle's median-of-3 call times
on the host cores (bounded samples, scaled by KV bytes; workload 1 also on one
thread). `cpu_baseline` is the oracle's rate on the 128K step. Diagnostics go
to stderr.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "effective KV GB/s (% of HBM peak) + decode steps/s at 128K, 5.5% plan"
HBM_PEAK_GBS = 8000.0
BYTES_PER_TOKEN = {"bf16": 2 * 8 * 128 * 2, "fp8": 2 * 8 * 128, "f32": 2 * 8 * 128 * 4}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def algorithmic_bytes(w, view_tokens, view_blocks, kind, q_len=1):
    """Bytes the method itself must move for one call (KV, scales, Q, O, LSE,
    tables); split partials are overhead and are not counted."""
    B, Hq, D = w.batch, w.num_q_heads, w.head_dim
    qb = 4 if w.q_dtype == "f32" else 2
    per_tok = BYTES_PER_TOKEN[w.kv_dtype]
    if kind == "decode":
        kv = int(np.sum(view_tokens)) * per_tok
        pages = int(np.sum(view_blocks))
        tables = pages * 8 + B * 8
        scales = pages * 8 if w.kv_dtype == "fp8" else 0
        return kv + scales + tables + B * Hq * D * (qb + 4) + B * Hq * 4
    L = np.asarray(w.seq_lens, dtype=np.int64)
    pages = int(np.sum(-(-L // 16)))
    kv = int(L.sum()) * per_tok
    scales = pages * 8 if w.kv_dtype == "fp8" else 0
    return kv + scales + pages * 4 + B * 4 + B * q_len * Hq * (D * (qb + 4) + 4)


def plan_bytes(w, view_blocks):
    B = w.batch
    S = len(w.span_start)
    return (B * w.fbt_stride * 4 + S * 12 + (B + 1) * 4 + B * 16 + S * 4 * 2
            + int(np.sum(view_blocks)) * 8 + B * 16)


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "kap_128k_5p5pct_hbm_traffic.txt")
KERNEL_SOURCES = {
    "verify_mfma_kernel": ["paper_2607_24260_amd/csrc/verify_mfma.hip",
                           "paper_2607_24260_amd/csrc/kap_internal.h"],
    "decode_fast_kernel": ["paper_2607_24260_amd/csrc/decode_fast.hip",
                           "paper_2607_24260_amd/csrc/kap_internal.h"],
}


def counter_traffic(kernel):
    """HBM bytes per dispatch of `kernel` from the committed rocprofv3 counter
    summary, or None when the kernel's sources changed since the counters were
    taken (or the summary is missing)."""
    import hashlib
    try:
        lines = open(TRAFFIC_FILE).read().splitlines()
    except OSError:
        return None
    vals = {}
    for ln in lines:
        parts = ln.split()
        if len(parts) == 4 and parts[2] == "=" and parts[1] == kernel:
            vals[parts[0]] = parts[3]
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        h.update(open(os.path.join(ROOT, f), "rb").read())
    if vals.get("source_sha256") != h.hexdigest() or "traffic_bytes" not in vals:
        return None
    return int(vals["traffic_bytes"])


def time_loop(fn, n, reps, torch):
    """Median over `reps` of the mean time per call of `n` back-to-back calls,
    bracketed by HIP events on the current stream."""
    out = []
    for _ in range(reps):
        s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s.record()
        for i in range(n):
            fn(i)
        e.record()
        e.synchronize()
        out.append(s.elapsed_time(e) / n)
    return statistics.median(out)


def _host_info():
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        blas_threads = 1
    aff = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else os.cpu_count()
    model = ""
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                model = ln.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"host_cpus": os.cpu_count(), "affinity_cpus": aff, "blas_threads": int(blas_threads),
            "cpu_model": model}


def _median_s(fn, reps):
    ts = []
    for _ in range(reps):
        t0 = time.perf_counter()
        fn()
        ts.append(time.perf_counter() - t0)
    return statistics.median(ts)


def oracle_call_times(w, dec_seqs=None, ver_heads=1, reps=3):
    """The fp64 oracle on the host cores, median of `reps` runs each, for one
    plan compile, one decode step and one verify call of workload `w` (KV of
    replica 0, the first decode / verify queries).

    Bounded samples: decode runs over the first `dec_seqs` sequences (all when
    None); verify over sequence 0 with KV heads 0 .. ver_heads - 1 (every
    (sequence, KV head) unit of verify is independent and reads its own KV).
    Each sample time is scaled to the whole call by the KV bytes it reads
    (decode: view tokens; verify: sequence length x KV heads), and GB/s is the
    call's algorithmic bytes over that scaled time."""
    from oracle import kap_oracle as O
    k, v, sc = w.host_kv(0)
    pool = O.KVPool(k, v, w.kv_dtype, sc)
    B, Hkv = w.batch, w.num_kv_heads

    def compile_():
        return O.compile_plan(w.seq_lens, w.full_block_table, w.span_offsets, w.span_start,
                              w.span_len, w.span_prior, w.prefix, w.suffix, w.budget, 0,
                              w.num_pages, w.max_pages_per_seq)

    t_plan = _median_s(compile_, reps)
    plans = compile_()
    vbt = np.zeros((B, w.max_pages_per_seq), np.int64)
    vlb = np.zeros_like(vbt)
    for b, p in enumerate(plans):
        vbt[b, :p.num_blocks] = p.block_table
        vlb[b, :p.num_blocks] = p.logical_blocks
    nb = np.array([p.num_blocks for p in plans], dtype=np.int64)
    vt = np.array([p.view_tokens for p in plans], dtype=np.int64)

    nd = B if dec_seqs is None else min(B, dec_seqs)
    qd = w.q_decode[0].float().cpu().numpy()[:nd]
    t_dec_s = _median_s(lambda: O.selected_decode(pool, qd, w.seq_lens[:nd], vbt[:nd], vlb[:nd],
                                                  nb[:nd], w.sm_scale), reps)
    t_dec = t_dec_s * float(vt.sum()) / max(float(vt[:nd].sum()), 1.0)

    qv = w.q_verify[0].float().cpu().numpy()
    nh = min(Hkv, ver_heads)
    t_ver_s = _median_s(lambda: O.verify(pool, qv, w.seq_lens, w.full_block_table, w.sm_scale,
                                         batches=[0], kv_heads=range(nh)), reps)
    L = np.asarray(w.seq_lens, dtype=np.float64)
    t_ver = t_ver_s * float(L.sum()) * Hkv / (float(L[0]) * nh)

    dec_b = algorithmic_bytes(w, vt, nb, "decode")
    ver_b = algorithmic_bytes(w, vt, nb, "verify", qv.shape[1])
    return {
        "compile_s": round(t_plan, 4),
        "decode_call_s": round(t_dec, 4), "decode_sample_s": round(t_dec_s, 4),
        "decode_sample": f"{nd} of {B} sequences, all {Hkv} KV heads",
        "decode_gbs": round(dec_b / t_dec / 1e9, 4),
        "verify_call_s": round(t_ver, 4), "verify_sample_s": round(t_ver_s, 4),
        "verify_sample": f"sequence 0 ({int(L[0])} tokens), {nh} of {Hkv} KV heads, "
                         f"q_len {qv.shape[1]}",
        "verify_gbs": round(ver_b / t_ver / 1e9, 4),
        "reps": reps,
    }


def cpu_baseline(w, n_dec, n_ver, step_b, oracle):
    """The oracle's rate on the bench step of workload `w` (1 compile, n_dec
    decode and n_ver verify calls), from the per-call medians of
    oracle_call_times: algorithmic bytes of the step / the oracle's time for
    it."""
    t_step = oracle["compile_s"] + n_dec * oracle["decode_call_s"] + n_ver * oracle["verify_call_s"]
    info = _host_info()
    return {
        "value": round(step_b / t_step / 1e9, 4), "unit": "GB/s", "cores": info["blas_threads"],
        "kind": "oracle",
        "sample": (f"median of {oracle['reps']} runs each of 1 plan compile, 1 decode step "
                   f"({oracle['decode_sample']}) and 1 verify call ({oracle['verify_sample']}), "
                   f"each scaled to its whole call by KV bytes, combined as the step's "
                   f"1 + {n_dec} + {n_ver} calls; fp64 numpy"),
        "seconds_step_estimate": round(t_step, 3),
        **info,
    }


def stream_read_ceiling(torch, K, dev):
    """kap_stream_read (a plain coalesced read kernel) at the decode call's size
    (118 MB, 10 rotating buffers) and the verify call's size (2 GiB, 2 buffers):
    the practical HBM read rate the attention kernels are compared with."""
    out = {}
    for name, nbytes, nbuf, n in (("decode_size", 118 << 20, 10, 200), ("verify_size", 2 << 30, 2, 16)):
        bufs = [torch.ones(nbytes, dtype=torch.uint8, device=dev) for _ in range(nbuf)]
        sink = torch.zeros(1, dtype=torch.int32, device=dev)
        t = time_loop(lambda i: K.stream_read(bufs[i % nbuf], sink), n, 5, torch)
        out[name] = {"bytes": nbytes, "us_per_call": round(t * 1e3, 2),
                     "gbs": round(nbytes / (t * 1e-3) / 1e9, 1)}
        del bufs
    torch.cuda.empty_cache()
    return out


# Context buckets of the paper's Table 2: length, retained ratio s, Top-3 acceptance h
TAB2 = [(4096, 0.401, 0.958), (8192, 0.344, 0.957), (16384, 0.242, 0.957),
        (32768, 0.161, 0.956), (65536, 0.108, 0.962), (131072, 0.055, 0.953)]


def _attention_calls(torch, K, w, R, dev):
    """Bound plan, view decode, all-blocks decode and verify calls of workload
    `w` over R KV replicas; returns the timings (ms) and the plan's s."""
    i32 = lambda x: torch.as_tensor(np.asarray(x, dtype=np.int32)).to(dev)
    B, Hq, D, cap = w.batch, w.num_q_heads, w.head_dim, w.max_pages_per_seq
    kvs = [K.KVCache(w.k_pages[r], w.v_pages[r], Hq, torch.bfloat16) for r in range(R)]
    seq_lens, fbt = i32(w.seq_lens), i32(w.full_block_table)
    plan = K.compile_plan(seq_lens, fbt, i32(w.span_offsets), i32(w.span_start),
                          i32(w.span_len), torch.as_tensor(w.span_prior).to(dev), i32(w.prefix),
                          i32(w.suffix), i32(w.budget), num_pages=w.num_pages,
                          view_capacity=cap)
    torch.cuda.synchronize()
    assert np.all(plan["plan_status"].cpu().numpy() == 0)
    s = plan["view_tokens"].cpu().numpy() / w.seq_lens
    q_len = w.q_verify[0].shape[1]
    o = torch.empty((B, Hq, D), dtype=torch.float32, device=dev)
    l = torch.empty((B, Hq), dtype=torch.float32, device=dev)
    ov = torch.empty((B, q_len, Hq, D), dtype=torch.float32, device=dev)
    lv = torch.empty((B, q_len, Hq), dtype=torch.float32, device=dev)
    lblk_f = torch.arange(fbt.shape[1], dtype=torch.int32, device=dev).repeat(B, 1)
    nb_f = i32(-(-np.asarray(w.seq_lens, dtype=np.int64) // 16))
    Lmax = int(w.seq_lens.max())
    ws_d = torch.zeros(max(256, K.selected_decode_workspace_bytes(kvs[0], B, fbt.shape[1])),
                       dtype=torch.uint8, device=dev)
    ws_v = torch.zeros(max(256, K.verify_workspace_bytes(kvs[0], B, q_len, Lmax)),
                       dtype=torch.uint8, device=dev)
    sv = K.decode_schedule(kvs[0], seq_lens, plan["view_block_table"],
                           plan["view_logical_block"], plan["view_num_blocks"], cap)
    sf = K.decode_schedule(kvs[0], seq_lens, fbt, lblk_f, nb_f, fbt.shape[1])
    view = [K.bind_selected_decode(kvs[r], w.q_decode[0], seq_lens, plan["view_block_table"],
                                   plan["view_logical_block"], plan["view_num_blocks"], cap,
                                   w.sm_scale, o, l, ws_d, schedule=sv) for r in range(R)]
    full = [K.bind_selected_decode(kvs[r], w.q_decode[0], seq_lens, fbt, lblk_f, nb_f,
                                   fbt.shape[1], w.sm_scale, o, l, ws_d, schedule=sf)
            for r in range(R)]
    ver = [K.bind_verify(kvs[r], w.q_verify[0], seq_lens, fbt, Lmax, w.sm_scale, ov, lv, ws_v)
           for r in range(R)]
    t_view = time_loop(lambda i: view[i % R](), max(64, 3 * R), 5, torch)
    t_full = time_loop(lambda i: full[i % R](), max(12, R), 3, torch)
    t_ver = time_loop(lambda i: ver[i % R](), max(12, R), 3, torch)
    return t_view, t_full, t_ver, s


def config_figures(torch, K, dev, cfg, with_cpu):
    """GPU figures of workload `cfg` (1-3) with the oracle beside them: plan
    compile, selected-view decode and verify per call (decode and verify
    rotating over R KV replicas, R x the decode call's KV >= 1 GiB); for
    workload 3 also its all-blocks plan (budget = L and one span over the
    whole sequence, so the view is the full block table) and the decode over
    it, which is full-context decode."""
    from paper_2607_24260_amd.workloads import DESCRIPTIONS, make_workload
    R = {1: 32, 2: 14, 3: 5}[cfg]
    w = make_workload(cfg, device=dev, replicas=R)
    i32 = lambda x: torch.as_tensor(np.asarray(x, dtype=np.int32)).to(dev)
    B, Hq, D, cap = w.batch, w.num_q_heads, w.head_dim, w.max_pages_per_seq
    qdt = torch.float32 if w.q_dtype == "f32" else torch.bfloat16
    kvs = [K.KVCache(w.k_pages[r], w.v_pages[r], Hq, qdt, w.kv_scales[r]) for r in range(R)]
    seq_lens, fbt = i32(w.seq_lens), i32(w.full_block_table)
    Lmax = int(w.seq_lens.max())
    q_len = w.q_verify[0].shape[1]
    nq, nv = w.q_decode.shape[0], len(w.q_verify)

    def plan_for(span_offsets, span_start, span_len, prior, budget):
        out = {
            "view_block_table": torch.zeros((B, cap), dtype=torch.int32, device=dev),
            "view_logical_block": torch.zeros((B, cap), dtype=torch.int32, device=dev),
            "view_num_blocks": torch.zeros(B, dtype=torch.int32, device=dev),
            "view_tokens": torch.zeros(B, dtype=torch.int32, device=dev),
            "spans_taken": torch.zeros(B, dtype=torch.int32, device=dev),
            "plan_status": torch.zeros(B, dtype=torch.int32, device=dev),
            "span_selected": torch.zeros(len(span_start), dtype=torch.int32, device=dev),
        }
        ws = torch.empty(max(K.compile_plan_workspace_bytes(B, len(span_start), w.fbt_stride),
                             256), dtype=torch.uint8, device=dev)
        call = K.bind_compile_plan(seq_lens, fbt, i32(span_offsets), i32(span_start),
                                   i32(span_len), torch.as_tensor(prior).to(dev), i32(w.prefix),
                                   i32(w.suffix), i32(budget), num_pages=w.num_pages,
                                   view_capacity=cap, out=out, workspace=ws)
        torch.cuda.synchronize()
        assert np.all(out["plan_status"].cpu().numpy() == 0)
        t = time_loop(lambda i: call(), 50, 3, torch)
        return out, t

    def decode_figures(plan):
        vt = plan["view_tokens"].cpu().numpy()
        vb = plan["view_num_blocks"].cpu().numpy()
        o = torch.empty((B, Hq, D), dtype=torch.float32, device=dev)
        l = torch.empty((B, Hq), dtype=torch.float32, device=dev)
        ws = torch.zeros(max(256, K.selected_decode_workspace_bytes(kvs[0], B, cap)),
                         dtype=torch.uint8, device=dev)
        sch = K.decode_schedule(kvs[0], seq_lens, plan["view_block_table"],
                                plan["view_logical_block"], plan["view_num_blocks"], cap)
        calls = [[K.bind_selected_decode(kvs[r], w.q_decode[s], seq_lens,
                                         plan["view_block_table"], plan["view_logical_block"],
                                         plan["view_num_blocks"], cap, w.sm_scale, o, l, ws,
                                         schedule=sch)
                  for s in range(nq)] for r in range(R)]
        t = time_loop(lambda i: calls[i % R][i % nq](), max(200, 3 * R), 5, torch)
        nbytes = algorithmic_bytes(w, vt, vb, "decode")
        gbs = nbytes / (t * 1e-3) / 1e9
        return {"us_per_call": round(t * 1e3, 3), "steps_per_s": round(1e3 / t, 1),
                "effective_gbs": round(gbs, 1), "pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
                "algorithmic_bytes": nbytes, "view_tokens": int(vt.sum()),
                "retained_ratio_s_mean": round(float(np.mean(vt / w.seq_lens)), 4)}

    plan, t_plan = plan_for(w.span_offsets, w.span_start, w.span_len, w.span_prior, w.budget)
    dec = decode_figures(plan)
    ov = torch.empty((B, q_len, Hq, D), dtype=torch.float32, device=dev)
    lv = torch.empty((B, q_len, Hq), dtype=torch.float32, device=dev)
    ws_v = torch.zeros(max(256, K.verify_workspace_bytes(kvs[0], B, q_len, Lmax)),
                       dtype=torch.uint8, device=dev)
    ver_calls = [[K.bind_verify(kvs[r], w.q_verify[j], seq_lens, fbt, Lmax, w.sm_scale, ov, lv,
                                ws_v) for j in range(nv)] for r in range(R)]
    t_ver = time_loop(lambda i: ver_calls[i % R][i % nv](), max(24, 3 * R), 3, torch)
    ver_b = algorithmic_bytes(w, None, None, "verify", q_len)
    ver_gbs = ver_b / (t_ver * 1e-3) / 1e9
    out = {
        "workload": f"config{cfg}: {DESCRIPTIONS[cfg]}", "kv_replicas": R,
        "kv_dtype": w.kv_dtype, "q_dtype": w.q_dtype,
        "plan_us_per_call": round(t_plan * 1e3, 2),
        "decode": dec,
        "verify": {"us_per_call": round(t_ver * 1e3, 2), "q_len": q_len,
                   "effective_gbs": round(ver_gbs, 1),
                   "pct_hbm_peak": round(100 * ver_gbs / HBM_PEAK_GBS, 2),
                   "algorithmic_bytes": ver_b},
    }
    if cfg == 3:
        offs = np.arange(B + 1, dtype=np.int32)
        full, t_full_plan = plan_for(offs, np.zeros(B, np.int32), w.seq_lens,
                                     np.ones(B, np.float32), w.seq_lens)
        assert torch.equal(full["view_num_blocks"].cpu(),
                           torch.as_tensor(-(-np.asarray(w.seq_lens, np.int64) // 16)).int())
        out["all_blocks_plan"] = {"plan_us_per_call": round(t_full_plan * 1e3, 2),
                                  "decode": decode_figures(full)}
    if with_cpu:
        out["oracle"] = oracle_call_times(w, ver_heads=1 if cfg > 1 else w.num_kv_heads)
        if cfg == 1:
            from threadpoolctl import threadpool_limits
            with threadpool_limits(limits=1):
                out["oracle_1_thread"] = oracle_call_times(w, ver_heads=w.num_kv_heads)
    log(f"config {cfg}: {out}")
    del w, kvs
    torch.cuda.empty_cache()
    return out


def rq1_sweep(torch, K, dev):
    """Kernel-level analog of the paper's Table 2: B = 4 sequences per context
    bucket with the bucket's retained ratio s as the budget; selected-view
    decode against all-blocks decode (ideal ratio 1/s), and the attention-only
    cost ratio of Eq. (6)-(7) with k = 4 and the bucket's h."""
    from paper_2607_24260_amd import costmodel
    from paper_2607_24260_amd.workloads import make_workload
    rows = []
    for L, s_paper, h in TAB2:
        kv_bytes = 4 * L * BYTES_PER_TOKEN["bf16"]
        R = int(min(64, max(2, math.ceil((1 << 30) / (s_paper * kv_bytes)))))
        w = make_workload(4, device=dev, replicas=R, seq_len=L, n_decode=1, n_verify=1,
                          budget_frac=s_paper)
        t_view, t_full, t_ver, s = _attention_calls(torch, K, w, R, dev)
        rep_ = costmodel.measured(4, h, float(np.mean(s)), t_view, t_full, t_ver)
        vt = float(np.sum(s * w.seq_lens))
        rows.append({
            "seq_len": L, "s_paper": s_paper, "s_plan": round(float(np.mean(s)), 4), "h_paper": h,
            "decode_view_us": round(t_view * 1e3, 2), "decode_all_blocks_us": round(t_full * 1e3, 2),
            "verify_us": round(t_ver * 1e3, 2),
            "access_reduction_measured": round(t_full / t_view, 2),
            "access_reduction_ideal": round(1.0 / float(np.mean(s)), 2),
            "decode_view_gbs": round(vt * BYTES_PER_TOKEN["bf16"] / (t_view * 1e-3) / 1e9, 1),
            "attention_speedup_measured": round(1.0 / rep_.measured_ratio, 3),
            "attention_speedup_ideal": round(1.0 / rep_.ideal_ratio, 3),
            "kv_replicas": R})
        log(f"sweep L={L}: {rows[-1]}")
        del w
        torch.cuda.empty_cache()
    return rows


def tp4_share(torch, K, dev):
    """One GPU's share of the 128K workload under a 4-way head split (the
    paper's TP = 4): 8 query heads over 2 KV heads of every page."""
    from paper_2607_24260_amd.workloads import make_workload
    R = 36
    w = make_workload(4, device=dev, replicas=R, n_decode=1, n_verify=1, num_q_heads=8,
                      num_kv_heads=2)
    t_view, t_full, t_ver, s = _attention_calls(torch, K, w, R, dev)
    per_tok = 2 * 2 * 128 * 2
    dec_b = float(np.sum(s * w.seq_lens)) * per_tok
    ver_b = float(np.sum(w.seq_lens)) * per_tok
    out = {"heads": "8 query / 2 KV heads (1/4 of 32 / 8)", "kv_replicas": R,
           "decode_us_per_call": round(t_view * 1e3, 2),
           "decode_gbs": round(dec_b / (t_view * 1e-3) / 1e9, 1),
           "verify_us_per_call": round(t_ver * 1e3, 2),
           "verify_gbs": round(ver_b / (t_ver * 1e-3) / 1e9, 1),
           "all_blocks_decode_us": round(t_full * 1e3, 2)}
    del w
    torch.cuda.empty_cache()
    return out


def verify_windows(torch, K, dev, windows=(3, 5, 9, 13, 16), calls=12):
    """kap_verify alone on the ragged fp8 workload's KV (64 sequences of 4K..128K
    tokens, fp8 E4M3FN with per-page scales; the pool far exceeds the
    Infinity Cache) for each verify window size: the gamma = 2, 4, 8 windows
    of that workload and the largest the tuned kernel takes. Each window size
    runs its own kernel instance (row tiles of 16 = 4 heads x 4 tokens)."""
    from paper_2607_24260_amd.workloads import make_workload
    w = make_workload(5, device=dev, n_decode=1, n_verify=1)
    B, Hq, D = w.batch, w.num_q_heads, w.head_dim
    kv = K.KVCache(w.k_pages[0], w.v_pages[0], Hq, torch.bfloat16, w.kv_scales[0])
    seq_lens = torch.as_tensor(np.asarray(w.seq_lens, dtype=np.int32)).to(dev)
    fbt = torch.as_tensor(np.asarray(w.full_block_table, dtype=np.int32)).to(dev)
    Lmax = int(w.seq_lens.max())
    pages = -(-np.asarray(w.seq_lens, dtype=np.int64) // 16)
    pairs = int(np.sum(-(-pages // 2))) * w.num_kv_heads
    gen = torch.Generator(device=dev)
    gen.manual_seed(20261202)
    out = {"workload": "config5 KV (64 ragged sequences, fp8 E4M3FN + per-page scales)",
           "page_pairs_per_call": pairs, "windows": []}
    for ql in windows:
        q = (torch.randn((B, ql, Hq, D), generator=gen, device=dev) / math.sqrt(D)).to(torch.bfloat16)
        o = torch.empty((B, ql, Hq, D), dtype=torch.float32, device=dev)
        l = torch.empty((B, ql, Hq), dtype=torch.float32, device=dev)
        ws = torch.zeros(max(256, K.verify_workspace_bytes(kv, B, ql, Lmax)), dtype=torch.uint8,
                         device=dev)
        call = K.bind_verify(kv, q, seq_lens, fbt, Lmax, w.sm_scale, o, l, ws)
        t = time_loop(lambda i: call(), calls, 3, torch)
        nbytes = algorithmic_bytes(w, None, None, "verify", ql)
        gbs = nbytes / (t * 1e-3) / 1e9
        out["windows"].append({"q_len": ql, "row_tiles": (4 * ql + 15) // 16,
                               "us_per_call": round(t * 1e3, 2), "effective_gbs": round(gbs, 1),
                               "pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2)})
        log(f"fp8 verify window {ql}: {out['windows'][-1]}")
    del w, kv
    torch.cuda.empty_cache()
    return out


def ragged_stream(torch, K, dev, reps=3, with_cpu=False):
    """The ragged fp8 workload (64 sequences of 4K..128K tokens, fp8 KV with
    per-page scales, budgets 3%..30%) run device-resident, as
    executor.DeviceStream runs it: one plan compile, then 16 cycles of gamma in
    {2, 4, 8} proposal decode calls and one verify window each, with seeded
    accept lengths and the h <= s fallback to full-context access decided and
    applied on the device (kap_fallback_update). Timed with HIP events over
    whole streams, launched eagerly and as one HIP graph replay; rate =
    algorithmic bytes / time (the bytes follow the host FallbackPolicy, which
    makes the same decisions)."""
    from paper_2607_24260_amd.executor import (FULL, DeviceStream, FallbackPolicy,
                                               accepted_counts)
    from paper_2607_24260_amd.workloads import DESCRIPTIONS, make_workload

    w = make_workload(5, device=dev)
    B, Hq, D = w.batch, w.num_q_heads, w.head_dim
    i32 = lambda x: torch.as_tensor(np.asarray(x, dtype=np.int32)).to(dev)
    kv = K.KVCache(w.k_pages[0], w.v_pages[0], Hq, torch.bfloat16, w.kv_scales[0])
    seq_lens, fbt = i32(w.seq_lens), i32(w.full_block_table)
    cap = w.max_pages_per_seq
    plan = {
        "view_block_table": torch.zeros((B, cap), dtype=torch.int32, device=dev),
        "view_logical_block": torch.zeros((B, cap), dtype=torch.int32, device=dev),
        "view_num_blocks": torch.zeros(B, dtype=torch.int32, device=dev),
        "view_tokens": torch.zeros(B, dtype=torch.int32, device=dev),
        "spans_taken": torch.zeros(B, dtype=torch.int32, device=dev),
        "plan_status": torch.zeros(B, dtype=torch.int32, device=dev),
        "span_selected": torch.zeros(len(w.span_start), dtype=torch.int32, device=dev),
    }
    ds_stream = torch.cuda.Stream(device=dev)
    ws_plan = torch.empty(max(K.compile_plan_workspace_bytes(B, len(w.span_start), w.fbt_stride),
                              256), dtype=torch.uint8, device=dev)
    plan_call = K.bind_compile_plan(seq_lens, fbt, i32(w.span_offsets), i32(w.span_start),
                                    i32(w.span_len), torch.as_tensor(w.span_prior).to(dev),
                                    i32(w.prefix), i32(w.suffix), i32(w.budget),
                                    num_pages=w.num_pages, view_capacity=cap, out=plan,
                                    workspace=ws_plan, stream=ds_stream)
    ds_stream.synchronize()
    ds = DeviceStream(w, kv, plan, plan_call=plan_call, stream=ds_stream)
    status = plan["plan_status"].cpu().numpy()
    vtok = plan["view_tokens"].cpu().numpy().astype(np.int64)
    vblk = plan["view_num_blocks"].cpu().numpy().astype(np.int64)
    L = np.asarray(w.seq_lens, dtype=np.int64)
    pages_full = -(-L // 16)
    gammas = [q.shape[1] - 1 for q in w.q_verify]

    # algorithmic bytes of one stream, following the (identical) host policy
    policy = FallbackPolicy(vtok / L, status == K.KAP_PLAN_OK)
    dec_bytes = ver_bytes = n_dec = n_ver = 0
    for kind, idx in w.schedule:
        if kind == "decode":
            full = policy.mode == FULL
            tok = np.where(full, L, vtok)
            pages = np.where(full, pages_full, vblk)
            dec_bytes += (int(tok.sum()) * 2048 + int(pages.sum()) * 16 + B * 8
                          + B * Hq * (D * 6 + 4))
            n_dec += 1
        else:
            ver_bytes += algorithmic_bytes(w, None, None, "verify", gammas[idx] + 1)
            policy.update(accepted_counts(w.accept_draws[idx], gammas[idx]), gammas[idx])
            n_ver += 1
    nbytes = plan_bytes(w, vblk) + dec_bytes + ver_bytes
    flips = int((policy.mode == FULL).sum())

    def timed(launch, stream):
        out = []
        for _ in range(reps):
            s_ev, e_ev = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            s_ev.record(stream)
            launch()
            e_ev.record(stream)
            e_ev.synchronize()
            out.append(s_ev.elapsed_time(e_ev))
        return statistics.median(out)

    ds.run()
    ds_stream.synchronize()
    ms_eager = timed(ds.run, ds_stream)
    graph = ds.capture()
    cur = torch.cuda.current_stream()
    graph.replay()
    torch.cuda.synchronize()
    ms_graph = timed(graph.replay, cur)

    # decode / verify split of one eager stream (events between the calls)
    ev = []
    t0 = torch.cuda.Event(enable_timing=True)
    t0.record(ds_stream)
    plan_call()
    ds.reset()
    for kind, idx in w.schedule:
        if kind == "decode":
            ds.decode[idx]()
        else:
            ds.verify[idx]()
        e = torch.cuda.Event(enable_timing=True)
        e.record(ds_stream)
        ev.append((kind, e))
        if kind == "verify":
            ds.update[idx]()
    ds_stream.synchronize()
    dt = {"decode": 0.0, "verify": 0.0}
    prev = t0
    for kind, e in ev:
        dt[kind] += prev.elapsed_time(e)
        prev = e
    gbs = nbytes / (ms_graph * 1e-3) / 1e9
    dec_gbs = dec_bytes / (dt["decode"] * 1e-3) / 1e9
    ver_gbs = ver_bytes / (dt["verify"] * 1e-3) / 1e9
    oracle = None
    if with_cpu:
        oracle = oracle_call_times(w, dec_seqs=2, ver_heads=1)
    return {
        "workload": f"config5: {DESCRIPTIONS[5]}",
        "ms_per_stream_graph": round(ms_graph, 3), "ms_per_stream_eager": round(ms_eager, 3),
        "algorithmic_gb": round(nbytes / 1e9, 3),
        "effective_gbs": round(gbs, 1), "pct_hbm_peak": round(100 * gbs / HBM_PEAK_GBS, 2),
        "decode_calls": n_dec, "verify_calls": n_ver,
        "decode_us_mean": round(1e3 * dt["decode"] / max(n_dec, 1), 2),
        "verify_us_mean": round(1e3 * dt["verify"] / max(n_ver, 1), 2),
        "decode_effective_gbs": round(dec_gbs, 1),
        "decode_pct_hbm_peak": round(100 * dec_gbs / HBM_PEAK_GBS, 2),
        "verify_effective_gbs": round(ver_gbs, 1),
        "verify_pct_hbm_peak": round(100 * ver_gbs / HBM_PEAK_GBS, 2),
        "oracle": oracle,
        "sequences_on_full_context_at_end": flips,
        "kv_dtype": "fp8-e4m3fn + per-page fp32 scales",
        "note": "device-resident stream (plan compile, decode/verify calls, device-side "
                "fallback updates) captured in one HIP graph; effective_gbs uses the graph time",
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", type=int, default=4)
    ap.add_argument("--replicas", type=int, default=0, help="KV layer replicas (0 = auto)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-ragged", action="store_true",
                    help="skip the ragged fp8 stream measurement")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the stream-read ceiling, the context sweep and the TP-share run")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the per-call figures of workloads 1-3")
    ap.add_argument("--profile", action="store_true",
                    help="only the timed steps (for rocprofv3 runs)")
    ap.add_argument("--ragged-only", action="store_true",
                    help="only the ragged fp8 stream (for rocprofv3 runs of that workload); "
                         "prints its JSON object")
    ap.add_argument("--verify-windows-only", action="store_true",
                    help="only fp8 verify per window size on the ragged workload's KV (for "
                         "rocprofv3 runs); prints its JSON object")
    ap.add_argument("--calibrate", action="store_true",
                    help="also run a 1 GiB device-to-device copy (known bytes for scaling "
                         "FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: the library has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2607_24260_amd import kap as K
    from paper_2607_24260_amd.workloads import DESCRIPTIONS, make_workload

    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    if args.ragged_only:
        print(json.dumps(ragged_stream(torch, K, dev)), flush=True)
        return
    if args.verify_windows_only:
        print(json.dumps(verify_windows(torch, K, dev)), flush=True)
        return
    cfg = args.config
    if cfg == 5:
        print("the ragged fp8 workload is driven by its own accept/fallback schedule; "
              "bench.py times workloads 1-4", file=sys.stderr)
        sys.exit(2)

    # replicas: >= 1 GiB of KV between two reads of the same decode buffer
    R = args.replicas if args.replicas > 0 else (9 if cfg == 4 else 4)
    t0 = time.time()
    w = make_workload(cfg, device=dev, replicas=R)
    torch.cuda.synchronize()
    log(f"workload {cfg}: {DESCRIPTIONS[cfg]}; {R} KV replicas "
        f"({R * w.k_pages[0].numel() * w.k_pages[0].element_size() * 2 / 2**30:.1f} GiB) "
        f"built in {time.time() - t0:.1f}s")

    i32 = lambda x: torch.as_tensor(np.asarray(x, dtype=np.int32)).to(dev)
    B = w.batch
    cap = w.max_pages_per_seq
    qdt = torch.float32 if w.q_dtype == "f32" else torch.bfloat16
    kvs = [K.KVCache(w.k_pages[r], w.v_pages[r], w.num_q_heads, qdt, w.kv_scales[r])
           for r in range(R)]
    seq_lens = i32(w.seq_lens)
    fbt = i32(w.full_block_table)
    plan_in = (seq_lens, fbt, i32(w.span_offsets), i32(w.span_start), i32(w.span_len),
               torch.as_tensor(w.span_prior).to(dev), i32(w.prefix), i32(w.suffix),
               i32(w.budget))
    plan_out = {
        "view_block_table": torch.zeros((B, cap), dtype=torch.int32, device=dev),
        "view_logical_block": torch.zeros((B, cap), dtype=torch.int32, device=dev),
        "view_num_blocks": torch.zeros(B, dtype=torch.int32, device=dev),
        "view_tokens": torch.zeros(B, dtype=torch.int32, device=dev),
        "spans_taken": torch.zeros(B, dtype=torch.int32, device=dev),
        "plan_status": torch.zeros(B, dtype=torch.int32, device=dev),
        "span_selected": torch.zeros(len(w.span_start), dtype=torch.int32, device=dev),
    }
    ws_plan = torch.empty(max(K.compile_plan_workspace_bytes(B, len(w.span_start), w.fbt_stride),
                              256), dtype=torch.uint8, device=dev)
    plan_call = K.bind_compile_plan(*plan_in, num_pages=w.num_pages, view_capacity=cap,
                                    out=plan_out, workspace=ws_plan)
    torch.cuda.synchronize()
    view_tokens = plan_out["view_tokens"].cpu().numpy()
    view_blocks = plan_out["view_num_blocks"].cpu().numpy()
    assert np.all(plan_out["plan_status"].cpu().numpy() == 0)
    s_ratio = view_tokens / w.seq_lens

    # outputs per replica; workspaces shared (calls are stream-ordered)
    q_len = w.q_verify[0].shape[1]
    Hq, D = w.num_q_heads, w.head_dim
    ws_dec = torch.zeros(max(K.selected_decode_workspace_bytes(kvs[0], B, cap), 256),
                         dtype=torch.uint8, device=dev)
    ws_ver = torch.zeros(max(K.verify_workspace_bytes(kvs[0], B, q_len, int(w.seq_lens.max())),
                             256), dtype=torch.uint8, device=dev)
    outs = [(torch.empty((B, Hq, D), dtype=torch.float32, device=dev),
             torch.empty((B, Hq), dtype=torch.float32, device=dev),
             torch.empty((B, q_len, Hq, D), dtype=torch.float32, device=dev),
             torch.empty((B, q_len, Hq), dtype=torch.float32, device=dev)) for _ in range(R)]

    # the decode calls' split assignment, written once per plan (kap_decode_schedule)
    view_args = (seq_lens, plan_out["view_block_table"], plan_out["view_logical_block"],
                 plan_out["view_num_blocks"], cap)
    dsched = K.decode_schedule(kvs[0], *view_args)
    sched_call = K.bind_decode_schedule(kvs[0], *view_args, dsched)

    def bind_decodes(stream, schedule):
        return [[K.bind_selected_decode(kvs[r], w.q_decode[s], *view_args, w.sm_scale,
                                        outs[r][0], outs[r][1], ws_dec, schedule=schedule,
                                        stream=stream)
                 for s in range(w.q_decode.shape[0])] for r in range(R)]

    def bind_calls(stream):
        dcs, vcs = bind_decodes(stream, dsched), []
        for r in range(R):
            o, l, ov, lv = outs[r]
            vcs.append([K.bind_verify(kvs[r], w.q_verify[j], seq_lens, fbt,
                                      int(w.seq_lens.max()), w.sm_scale, ov, lv, ws_ver,
                                      stream=stream)
                        for j in range(len(w.q_verify))])
        return dcs, vcs

    dec_calls, ver_calls = bind_calls(None)

    sched = w.schedule
    n_dec = sum(1 for k, _ in sched if k == "decode")
    n_ver = len(sched) - n_dec

    def step_with(pc, sc, dcs, vcs):
        pc()
        sc()
        for c, (kind, i) in enumerate(sched):
            r = c % R
            if kind == "decode":
                dcs[r][i]()
            else:
                vcs[r][i]()

    def step(_):
        step_with(plan_call, sched_call, dec_calls, ver_calls)

    dec_b = algorithmic_bytes(w, view_tokens, view_blocks, "decode")
    ver_b = algorithmic_bytes(w, view_tokens, view_blocks, "verify", q_len)
    step_b = plan_bytes(w, view_blocks) + n_dec * dec_b + n_ver * ver_b

    if args.calibrate:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(2):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    for _ in range(args.warmup):
        step(0)
    torch.cuda.synchronize()
    s_ev, e_ev = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    s_ev.record()
    for k in range(args.steps):
        step(k)
    e_ev.record()
    torch.cuda.synchronize()
    ms_step = s_ev.elapsed_time(e_ev) / args.steps
    value = step_b / (ms_step * 1e-3) / 1e9
    log(f"step: {ms_step:.3f} ms, {step_b / 1e9:.3f} GB algorithmic -> {value:.1f} GB/s")
    if args.profile:
        return

    # the same step captured as one HIP graph: the calls bound to a side
    # stream (binding runs each once there), captured, and replayed on it
    gs = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(gs):
        g_plan = K.bind_compile_plan(*plan_in, num_pages=w.num_pages, view_capacity=cap,
                                     out=plan_out, workspace=ws_plan, stream=gs)
        g_sched = K.bind_decode_schedule(kvs[0], *view_args, dsched, stream=gs)
        g_dec, g_ver = bind_calls(gs)
    gs.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=gs):
        step_with(g_plan, g_sched, g_dec, g_ver)
    with torch.cuda.stream(gs):
        for _ in range(max(args.warmup, 1)):
            graph.replay()
        gs.synchronize()
        gs_ev, ge_ev = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        gs_ev.record(gs)
        for _ in range(args.steps):
            graph.replay()
        ge_ev.record(gs)
    torch.cuda.synchronize()
    ms_step_graph = gs_ev.elapsed_time(ge_ev) / args.steps
    log(f"step as one HIP graph: {ms_step_graph:.3f} ms ({len(sched) + 2} launches per step)")
    del graph

    # per-call rates, rotating replicas (HBM) and on one buffer (cache-hot, context)
    nq = w.q_decode.shape[0]
    t_dec = time_loop(lambda i: dec_calls[i % R][i % nq](), 256, 5, torch)
    dec_bal = bind_decodes(None, None)      # the same calls computing the split map themselves
    t_dec_bal = time_loop(lambda i: dec_bal[i % R][i % nq](), 256, 5, torch)
    t_sched = time_loop(lambda i: sched_call(), 50, 3, torch)
    t_dec_hot = time_loop(lambda i: dec_calls[0][i % nq](), 256, 5, torch)
    t_ver = time_loop(lambda i: ver_calls[i % R][i % len(w.q_verify)](), 48, 3, torch)
    t_plan = time_loop(lambda i: plan_call(), 50, 3, torch)
    dec_gbs = dec_b / (t_dec * 1e-3) / 1e9
    ver_gbs = ver_b / (t_ver * 1e-3) / 1e9
    log(f"decode: {t_dec * 1e3:.2f} us/call ({dec_gbs:.0f} GB/s, {1e3 / t_dec:.0f} steps/s); "
        f"cache-hot {t_dec_hot * 1e3:.2f} us; verify: {t_ver * 1e3:.1f} us/call "
        f"({ver_gbs:.0f} GB/s); plan: {t_plan * 1e3:.1f} us")

    # compaction into a compact workspace (the paper's materialised view) against
    # the zero-copy view, and the slot-mapped append of one verify window
    maint = None
    if cfg == 4:
        cap_c = 512
        kv0 = kvs[0]
        comp = [K.KVCache(torch.empty((B * cap_c,) + tuple(kv0.k_pages.shape[1:]),
                                      dtype=kv0.k_pages.dtype, device=dev),
                          torch.empty((B * cap_c,) + tuple(kv0.v_pages.shape[1:]),
                                      dtype=kv0.v_pages.dtype, device=dev), Hq, qdt)
                for _ in range(R)]
        ctab = torch.empty((B, cap_c), dtype=torch.int32, device=dev)
        vbt_, vnb_ = plan_out["view_block_table"], plan_out["view_num_blocks"]
        t_comp = time_loop(lambda i: K.compact_view(kvs[i % R], vbt_, vnb_, cap_c, comp[i % R],
                                                    out=ctab), 45, 3, torch)
        lblk_c = plan_out["view_logical_block"][:, :cap_c].contiguous()
        o_c = torch.empty((B, Hq, D), dtype=torch.float32, device=dev)
        l_c = torch.empty((B, Hq), dtype=torch.float32, device=dev)
        ws_c = torch.zeros(max(256, K.selected_decode_workspace_bytes(comp[0], B, cap_c)),
                           dtype=torch.uint8, device=dev)
        s_c = K.decode_schedule(comp[0], seq_lens, ctab, lblk_c, plan_out["view_num_blocks"],
                                cap_c)
        dec_c = [K.bind_selected_decode(comp[c], w.q_decode[0], seq_lens, ctab, lblk_c,
                                        plan_out["view_num_blocks"], cap_c, w.sm_scale, o_c, l_c,
                                        ws_c, schedule=s_c) for c in range(R)]
        t_dec_c = time_loop(lambda i: dec_c[i % R](), 256, 5, torch)
        win = q_len * B
        Lh = np.asarray(w.seq_lens, dtype=np.int64)
        fbh = np.asarray(w.full_block_table, dtype=np.int64)
        pos = [Lh[b] - q_len + np.arange(q_len) for b in range(B)]
        slots = torch.as_tensor(np.concatenate([fbh[b, p // 16] * 16 + p % 16
                                                for b, p in enumerate(pos)])).to(dev)
        k_win = torch.randn((win, w.num_kv_heads, D), device=dev).to(kv0.k_pages.dtype)
        v_win = torch.randn((win, w.num_kv_heads, D), device=dev).to(kv0.k_pages.dtype)
        t_app = time_loop(lambda i: K.append_kv(kvs[i % R], k_win, v_win, slots), 200, 3, torch)
        comp_bytes = 2 * (int(np.sum(view_blocks)) * 16 * BYTES_PER_TOKEN[w.kv_dtype])
        maint = {
            "compact_view_us": round(t_comp * 1e3, 2),
            "compact_view_gbs": round(comp_bytes / (t_comp * 1e-3) / 1e9, 1),
            "compact_view_bytes": comp_bytes,
            "decode_on_compact_us": round(t_dec_c * 1e3, 2),
            "zero_copy_decode_us": round(t_dec * 1e3, 2),
            "append_window_us": round(t_app * 1e3, 2),
            "append_window_tokens": win,
        }
        log(f"kv maintenance: {maint}")

    # full-context decode (the same batch on every page) for the cost model,
    # and the Top-3 acceptance of 64 gamma = 4 windows over a 151936-token vocabulary
    phase = accept = None
    if cfg == 4:
        from paper_2607_24260_amd import costmodel
        lblk_f = torch.arange(fbt.shape[1], dtype=torch.int32, device=dev).repeat(B, 1)
        nb_f = torch.as_tensor(-(-np.asarray(w.seq_lens, dtype=np.int64) // 16)).int().to(dev)
        ws_f = torch.zeros(max(256, K.selected_decode_workspace_bytes(kvs[0], B, fbt.shape[1])),
                           dtype=torch.uint8, device=dev)
        o_f = torch.empty((B, Hq, D), dtype=torch.float32, device=dev)
        l_f = torch.empty((B, Hq), dtype=torch.float32, device=dev)
        s_f = K.decode_schedule(kvs[0], seq_lens, fbt, lblk_f, nb_f, fbt.shape[1])
        dec_f = [K.bind_selected_decode(kvs[r], w.q_decode[0], seq_lens, fbt, lblk_f, nb_f,
                                        fbt.shape[1], w.sm_scale, o_f, l_f, ws_f, schedule=s_f)
                 for r in range(R)]
        t_full = time_loop(lambda i: dec_f[i % R](), 27, 3, torch)
        rep_ = costmodel.measured(q_len - 1, costmodel.expected_acceptance(q_len - 1),
                                  float(np.mean(s_ratio)), t_dec, t_full, t_ver)
        phase = {**rep_.as_dict(), "full_context_decode_us": round(t_full * 1e3, 2),
                 "h_source": "E[min(X, gamma)]/gamma of the recipe's accept law"}
        log(f"phase: {phase}")
        aB, aW, aV, nrep = 64, 5, 151936, 4
        lg = [torch.randn((aB, aW, aV), device=dev).to(torch.bfloat16) for _ in range(nrep)]
        dr = torch.randint(0, aV, (aB, aW - 1), dtype=torch.int32, device=dev)
        acc_m = torch.empty(aB, dtype=torch.int32, device=dev)
        acc_c = torch.empty(aB, dtype=torch.int32, device=dev)
        acc_ws = torch.zeros(K.load_library().kap_accept_top3_workspace_bytes(aB, aW),
                             dtype=torch.uint8, device=dev)
        t_acc = time_loop(lambda i: K.accept_top3(lg[i % nrep], dr, 3, acc_m, acc_c, acc_ws),
                          40, 3, torch)
        accept = {"shape": f"{aB} windows x {aW} positions x {aV} vocab, bf16 logits",
                  "us_per_call": round(t_acc * 1e3, 2),
                  "gbs": round(aB * aW * aV * 2 / (t_acc * 1e-3) / 1e9, 1)}
        log(f"accept_top3: {accept}")
        del lg

    # token-granular visibility (Sec. 3.1 mask at token resolution): the same
    # spans and budgets, plan in token mode, decode with per-page token masks
    tokmode = None
    if cfg == 4:
        plan_tok = {k: torch.zeros_like(v) for k, v in plan_out.items()}
        plan_tok["view_token_mask"] = torch.zeros((B, cap), dtype=torch.int32, device=dev)
        plan_tok_call = K.bind_compile_plan(*plan_in, num_pages=w.num_pages, view_capacity=cap,
                                            out=plan_tok, workspace=ws_plan, token_granular=True)
        torch.cuda.synchronize()
        assert np.all(plan_tok["plan_status"].cpu().numpy() == 0)
        vt_tok = plan_tok["view_tokens"].cpu().numpy()
        vb_tok = plan_tok["view_num_blocks"].cpu().numpy()
        o_t = torch.empty((B, Hq, D), dtype=torch.float32, device=dev)
        l_t = torch.empty((B, Hq), dtype=torch.float32, device=dev)
        s_t = K.decode_schedule(kvs[0], seq_lens, plan_tok["view_block_table"],
                                plan_tok["view_logical_block"], plan_tok["view_num_blocks"], cap,
                                view_token_mask=plan_tok["view_token_mask"])
        dec_t = [K.bind_selected_decode(kvs[r], w.q_decode[0], seq_lens,
                                        plan_tok["view_block_table"],
                                        plan_tok["view_logical_block"],
                                        plan_tok["view_num_blocks"], cap, w.sm_scale, o_t, l_t,
                                        ws_dec, view_token_mask=plan_tok["view_token_mask"],
                                        schedule=s_t)
                 for r in range(R)]
        t_dec_t = time_loop(lambda i: dec_t[i % R](), 256, 5, torch)
        t_plan_t = time_loop(lambda i: plan_tok_call(), 50, 3, torch)
        read_b = int(np.sum(vb_tok)) * 16 * BYTES_PER_TOKEN[w.kv_dtype]
        tokmode = {
            "plan_us_per_call": round(t_plan_t * 1e3, 2),
            "decode_us_per_call": round(t_dec_t * 1e3, 3),
            "visible_tokens": int(np.sum(vt_tok)),
            "view_pages": int(np.sum(vb_tok)),
            "retained_ratio_s_mean": round(float(np.mean(vt_tok / w.seq_lens)), 5),
            "page_mode_visible_tokens": int(np.sum(view_tokens)),
            "page_mode_view_pages": int(np.sum(view_blocks)),
            "decode_page_read_gbs": round(read_b / (t_dec_t * 1e-3) / 1e9, 1),
        }
        log(f"token-granular: {tokmode}")

    ceiling = sweep = share = None
    if cfg == 4 and not args.no_sweep:
        ceiling = stream_read_ceiling(torch, K, dev)
        log(f"stream-read ceiling: {ceiling}")
        sweep = rq1_sweep(torch, K, dev)
        share = tp4_share(torch, K, dev)
        log(f"tp4 share: {share}")

    others = {}
    if cfg == 4 and not args.no_configs:
        for c in (1, 2, 3):
            others[f"config{c}"] = config_figures(torch, K, dev, c, not args.no_cpu)

    windows = None
    if not args.no_ragged and cfg == 4:
        windows = verify_windows(torch, K, dev)

    ragged = None
    if not args.no_ragged and cfg == 4:
        ragged = ragged_stream(torch, K, dev, with_cpu=not args.no_cpu)
        log(f"ragged fp8 stream: {ragged}")

    cpu = oracle = None
    if not args.no_cpu:
        oracle = oracle_call_times(w, ver_heads=1)
        cpu = cpu_baseline(w, n_dec, n_ver, step_b, oracle)
        log(f"cpu oracle: {cpu}")
    per_config = None
    if others:
        per_config = {**others, f"config{cfg}": {
            "workload": f"config{cfg}: {DESCRIPTIONS[cfg]}", "kv_replicas": R,
            "plan_us_per_call": round(t_plan * 1e3, 2),
            "decode": {"us_per_call": round(t_dec * 1e3, 3), "steps_per_s": round(1e3 / t_dec, 1),
                       "effective_gbs": round(dec_gbs, 1),
                       "pct_hbm_peak": round(100 * dec_gbs / HBM_PEAK_GBS, 2),
                       "algorithmic_bytes": dec_b},
            "verify": {"us_per_call": round(t_ver * 1e3, 2), "q_len": q_len,
                       "effective_gbs": round(ver_gbs, 1),
                       "pct_hbm_peak": round(100 * ver_gbs / HBM_PEAK_GBS, 2),
                       "algorithmic_bytes": ver_b},
            "oracle": oracle}}
        if ragged is not None:
            per_config["config5"] = {k: ragged[k] for k in (
                "workload", "decode_us_mean", "decode_effective_gbs", "decode_pct_hbm_peak",
                "verify_us_mean", "verify_effective_gbs", "verify_pct_hbm_peak", "oracle")}

    res = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "ms_per_step_graph": round(ms_step_graph, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": {"bf16": "bf16", "fp8": "fp8-e4m3fn(kv)/bf16(q)", "f32": "f32"}[w.kv_dtype],
        "data": "synthetic",
        "config": {
            "workload": f"config{cfg}: {DESCRIPTIONS[cfg]}",
            "batch": int(B), "seq_len": int(w.seq_lens.max()), "q_heads": Hq,
            "kv_heads": w.num_kv_heads, "head_dim": D, "page_tokens": 16,
            "kv_dtype": w.kv_dtype, "plan_budget_tokens": [int(x) for x in w.budget],
            "retained_ratio_s": [round(float(x), 5) for x in s_ratio],
            "decode_calls_per_step": n_dec, "verify_calls_per_step": n_ver,
            "verify_q_len": q_len, "kv_layer_replicas": R,
        },
        "pct_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2),
        "decode_steps_per_s": round(1e3 / t_dec, 1),
        "decode_tokens_per_s": round(B * 1e3 / t_dec, 1),
        "decode_us_per_call": round(t_dec * 1e3, 3),
        "decode_effective_gbs": round(dec_gbs, 1),
        "decode_pct_hbm_peak": round(100 * dec_gbs / HBM_PEAK_GBS, 2),
        "decode_cache_hot_us_per_call": round(t_dec_hot * 1e3, 3),
        "decode_unscheduled_us_per_call": round(t_dec_bal * 1e3, 3),
        "decode_schedule_us_per_call": round(t_sched * 1e3, 2),
        "verify_calls_per_s": round(1e3 / t_ver, 1),
        "verify_us_per_call": round(t_ver * 1e3, 2),
        "verify_effective_gbs": round(ver_gbs, 1),
        "plan_us_per_call": round(t_plan * 1e3, 2),
        "algorithmic_bytes": {"decode_call": dec_b, "verify_call": ver_b, "step": step_b},
        "roofline": {
            "kernel": "kap_verify (verify_mfma_kernel, splits merged in-kernel)",
            "bound": "hbm", "achieved": round(ver_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(ver_gbs / HBM_PEAK_GBS, 4),
            "traffic": counter_traffic("verify_mfma_kernel") if cfg == 4 else None,
        },
        "decode_roofline": {
            "kernel": "kap_selected_decode (decode_fast_kernel, splits merged in-kernel)",
            "bound": "hbm", "achieved": round(dec_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(dec_gbs / HBM_PEAK_GBS, 4),
            "traffic": counter_traffic("decode_fast_kernel") if cfg == 4 else None,
        },
        "token_granular_view": tokmode,
        "stream_read_ceiling": ceiling,
        # the same calls against a plain streaming read of their size
        "frac_of_read_ceiling": None if ceiling is None else {
            "verify": round(ceiling["verify_size"]["us_per_call"] / (t_ver * 1e3)
                            * ver_b / ceiling["verify_size"]["bytes"], 4),
            "decode": round(ceiling["decode_size"]["us_per_call"] / (t_dec * 1e3)
                            * dec_b / ceiling["decode_size"]["bytes"], 4)},
        "context_sweep_table2": sweep,
        "tp4_per_gpu_share": share,
        "kv_maintenance": maint,
        "accept_top3": accept,
        "phase_cost_model": phase,
        "ragged_fp8_stream": ragged,
        "fp8_verify_windows": windows,
        "per_config": per_config,
        "cpu_baseline": cpu,
    }
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
