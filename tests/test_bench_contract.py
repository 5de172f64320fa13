"""bench.py's measurement definitions, checked without a GPU: the one-GPU
guard, and the algorithmic bytes of the 128K workload's calls against their
closed forms (KV bytes of the visible / full context, plus Q, O, LSE and the
tables; split partials are not counted)."""
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from oracle import kap_oracle as O  # noqa: E402
from paper_2607_24260_amd.workloads import make_workload  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=60)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_algorithmic_bytes_of_the_128k_workload():
    w = make_workload(4, n_decode=1, n_verify=1, with_kv=False)
    plans = O.compile_plan(w.seq_lens, w.full_block_table, w.span_offsets, w.span_start,
                           w.span_len, w.span_prior, w.prefix, w.suffix, w.budget, 0,
                           w.num_pages, w.max_pages_per_seq)
    vt = np.array([p.view_tokens for p in plans])
    nb = np.array([p.num_blocks for p in plans])
    B, Hq, D = 4, 32, 128
    # decode: visible tokens x 4096 B (bf16 K + V, 8 KV heads x 128 dims), the
    # view tables (2 x int32 per entry), seq_len + view length, Q (bf16),
    # O (fp32) and LSE (fp32)
    want_dec = int(vt.sum()) * 4096 + int(nb.sum()) * 8 + B * 8 + B * Hq * D * (2 + 4) + B * Hq * 4
    assert bench.algorithmic_bytes(w, vt, nb, "decode") == want_dec
    assert 117e6 < want_dec < 118.2e6          # <= 118.1 MB at 5.5% of 128K
    # verify (q_len 5): every token of the 4 x 131072 context, the block table,
    # seq_len, Q / O / LSE of the window rows
    want_ver = 4 * 131072 * 4096 + 4 * 8192 * 4 + B * 4 + B * 5 * Hq * (D * 6 + 4)
    assert bench.algorithmic_bytes(w, vt, nb, "verify", 5) == want_ver
    assert abs(want_ver / 2**31 - 1.0) < 2e-3   # 2 GiB of KV plus metadata
