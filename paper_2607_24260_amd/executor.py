"""Host-side executor cycle: proposal steps over the selected-KV view, a
verify window over the full KV, acceptance bookkeeping and fallback.

Paper: Sec. 3.2 ("Selected-KV proposal", "Full-context verification",
"Runtime stability and fallback"); acceptance rate h = accepted / speculated
(Eq. (5)); retained ratio s (Eq. (4)); the self-speculation margin condition
h > s (Eq. (12)).

The policy here is a minimal reading of the paper's qualitative fallback list
(the thresholds are this implementation's, not the paper's):
* a sequence whose plan could not be compiled (any non-OK plan status, e.g.
  the view exceeds the compact capacity) uses full-context access from the
  start;
* after its first cycle, a sequence falls back to full-context access once its
  acceptance rate over the last `window` cycles is not above its retained
  ratio s (h <= s violates Eq. (12));
* fallback is sticky for the rest of the run.

Accepted counts come from the caller (here: seeded draws, so the whole stream
can be enqueued without reading GPU results back). All attention runs in the
HIP library through the binding.
"""
from __future__ import annotations

from collections import deque
from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np

SELECTED = 0
FULL = 1


@dataclass
class FallbackPolicy:
    """Per-sequence access mode (SELECTED / FULL) driven by acceptance."""

    retained: np.ndarray                       # s_b = view_tokens_b / L_b (float64)
    plan_ok: np.ndarray                        # bool per sequence
    window: int = 4
    mode: np.ndarray = field(init=False)
    history: List[deque] = field(init=False)
    cycles: np.ndarray = field(init=False)
    flipped_at: np.ndarray = field(init=False)

    def __post_init__(self):
        B = len(self.retained)
        self.retained = np.asarray(self.retained, dtype=np.float64)
        self.mode = np.where(np.asarray(self.plan_ok, dtype=bool), SELECTED, FULL).astype(np.int32)
        self.history = [deque(maxlen=self.window) for _ in range(B)]
        self.cycles = np.zeros(B, dtype=np.int64)
        self.flipped_at = np.where(self.mode == FULL, 0, -1).astype(np.int64)

    def acceptance(self, b: int) -> float:
        """h over the last `window` cycles (Eq. (5)); nan before any cycle."""
        acc = sum(a for a, _ in self.history[b])
        spec = sum(s for _, s in self.history[b])
        return acc / spec if spec > 0 else float("nan")

    def update(self, accepted: np.ndarray, speculated: np.ndarray) -> np.ndarray:
        """Record one cycle for every sequence and return the sequences that
        switch to full-context access now."""
        accepted = np.asarray(accepted)
        speculated = np.broadcast_to(np.asarray(speculated), accepted.shape)
        flips = []
        for b in range(len(self.retained)):
            self.history[b].append((int(accepted[b]), int(speculated[b])))
            self.cycles[b] += 1
            if self.mode[b] == FULL or self.cycles[b] < 2:
                continue
            if self.acceptance(b) <= self.retained[b]:
                self.mode[b] = FULL
                self.flipped_at[b] = self.cycles[b]
                flips.append(b)
        return np.asarray(flips, dtype=np.int64)


def accepted_counts(draws: np.ndarray, gamma: int) -> np.ndarray:
    """m = min(max(X, 0), gamma) for accept draws X (m in {0, ..., gamma},
    Eq. (2)); the device policy clamps the same way."""
    return np.clip(np.asarray(draws, dtype=np.int64), 0, int(gamma))


class ViewBuilder:
    """Device view arrays for a batch whose sequences are either on their
    compiled selected view or on the full block table (fallback)."""

    def __init__(self, plan: dict, full_block_table, seq_lens_host, capacity: int):
        import torch
        self.torch = torch
        dev = full_block_table.device
        B, stride = full_block_table.shape
        self.stride = max(int(stride), int(capacity))
        self.B = B
        self.sel_bt = torch.zeros((B, self.stride), dtype=torch.int32, device=dev)
        self.sel_lb = torch.zeros((B, self.stride), dtype=torch.int32, device=dev)
        self.sel_bt[:, :capacity] = plan["view_block_table"]
        self.sel_lb[:, :capacity] = plan["view_logical_block"]
        self.sel_nb = plan["view_num_blocks"].clone()
        self.full_bt = torch.zeros((B, self.stride), dtype=torch.int32, device=dev)
        self.full_bt[:, :stride] = full_block_table
        self.full_lb = torch.arange(self.stride, dtype=torch.int32, device=dev).repeat(B, 1)
        npg = [-(-int(L) // 16) for L in seq_lens_host]
        self.full_nb = torch.as_tensor(np.asarray(npg, dtype=np.int32)).to(dev)
        self.max_blocks = int(self.stride)
        self.vbt = self.sel_bt.clone()
        self.vlb = self.sel_lb.clone()
        self.vnb = self.sel_nb.clone()

    def apply(self, mode: np.ndarray):
        """Rebuild the active view from the per-sequence modes (device copies)."""
        torch = self.torch
        full = torch.as_tensor(np.asarray(mode) == FULL).to(self.vbt.device)
        self.vbt.copy_(torch.where(full[:, None], self.full_bt, self.sel_bt))
        self.vlb.copy_(torch.where(full[:, None], self.full_lb, self.sel_lb))
        self.vnb.copy_(torch.where(full, self.full_nb, self.sel_nb))


@dataclass
class StreamResult:
    policy: FallbackPolicy
    decode_out: list            # per decode call: (out, lse, mode snapshot)
    verify_out: list            # per verify call: (out, lse)
    accepted: np.ndarray        # [cycles][B]
    gammas: list


def run_stream(w, kv, plan: dict, *, window: int = 4, keep_outputs: Optional[set] = None,
               stream=None) -> StreamResult:
    """Run the workload's interleaved schedule (gamma proposal steps, then a
    verify window of gamma + 1 tokens, per cycle) through the library.

    `plan` holds the compiled plan tensors (see kap.compile_plan). The plan's
    view_tokens are read back once to form s_b. Outputs of the calls named in
    keep_outputs ({('decode', i), ('verify', j)}) are kept (cloned).

    With ``stream``, everything -- the library calls, the view switches and
    the output copies -- is enqueued on that stream (it becomes torch's
    current stream for the run), so the host-side tensor work stays ordered
    with the kernels."""
    import torch

    from . import kap as K

    if stream is not None:
        with torch.cuda.stream(stream):
            return run_stream(w, kv, plan, window=window, keep_outputs=keep_outputs)

    dev = kv.device
    i32 = lambda x: torch.as_tensor(np.asarray(x, dtype=np.int32)).to(dev)
    seq_lens = i32(w.seq_lens)
    fbt = i32(w.full_block_table)
    cap = plan["view_block_table"].shape[1]
    status = plan["plan_status"].cpu().numpy()
    s = plan["view_tokens"].cpu().numpy().astype(np.float64) / np.asarray(w.seq_lens)
    policy = FallbackPolicy(s, status == K.KAP_PLAN_OK, window=window)
    views = ViewBuilder(plan, fbt, w.seq_lens, cap)
    views.apply(policy.mode)
    keep = keep_outputs or set()
    B, Hq, D = w.batch, w.num_q_heads, w.head_dim
    out = torch.empty((B, Hq, D), dtype=torch.float32, device=dev)
    lse = torch.empty((B, Hq), dtype=torch.float32, device=dev)
    ws_dec = torch.zeros(max(256, K.selected_decode_workspace_bytes(kv, B, views.max_blocks)),
                         dtype=torch.uint8, device=dev)
    max_len = int(np.max(w.seq_lens))
    dec_res, ver_res, acc_all = [], [], []
    gammas = [q.shape[1] - 1 for q in w.q_verify]
    cycle = 0
    for kind, idx in w.schedule:
        if kind == "decode":
            K.selected_decode(kv, w.q_decode[idx], seq_lens, views.vbt, views.vlb, views.vnb,
                              views.max_blocks, w.sm_scale, out=out, lse=lse, workspace=ws_dec)
            if ("decode", idx) in keep:
                dec_res.append((idx, out.clone(), lse.clone(), policy.mode.copy()))
        else:
            q = w.q_verify[idx]
            ov, lv = K.verify(kv, q, seq_lens, fbt, max_len, w.sm_scale)
            if ("verify", idx) in keep:
                ver_res.append((idx, ov, lv))
            g = gammas[idx]
            m = accepted_counts(w.accept_draws[cycle], g)
            acc_all.append(m)
            flips = policy.update(m, g)
            if len(flips):
                views.apply(policy.mode)
            cycle += 1
    return StreamResult(policy, dec_res, ver_res, np.asarray(acc_all), gammas)


class DeviceStream:
    """The workload's interleaved schedule with the access-mode policy on the
    device (kap_fallback_update, Sec. 3.2 "Runtime stability and fallback"):
    a cycle is kernel launches only, all on one stream, so a whole stream can
    be captured in a HIP graph (``capture``) and replayed. The policy is the
    one of FallbackPolicy (window, h <= s after the first cycle, sticky,
    failed plans start on full context); h <= s is compared exactly in
    integers on the device.

    Accept lengths per cycle come in as device arrays uploaded once (here the
    seeded draws; the kernel clamps them to gamma). ``plan`` holds the
    compiled plan tensors; ``plan_call``, if given, recompiles the plan at
    the start of every stream. A token-granular plan (one with
    ``view_token_mask``, Sec. 3.1's visibility mask at token resolution) runs
    with masked decode calls and a masked fallback switch."""

    def __init__(self, w, kv, plan: dict, *, window: int = 4, plan_call=None, stream=None):
        import torch

        from . import kap as K

        self.torch = torch
        dev = kv.device
        self.stream = stream if stream is not None else torch.cuda.Stream(device=dev)
        # the inputs were made on the current stream; everything allocated
        # here is made (and zero-filled) on self.stream, where the bound
        # calls run -- binding validates each call by launching it once
        self.stream.wait_stream(torch.cuda.current_stream(dev))
        with torch.cuda.stream(self.stream):
            i32 = lambda x: torch.as_tensor(np.asarray(x, dtype=np.int32)).to(dev)
            B = w.batch
            self.w = w
            self.plan_call = plan_call
            self.seq_lens = i32(w.seq_lens)
            self.fbt = i32(w.full_block_table)
            cap = plan["view_block_table"].shape[1]
            stride = max(int(self.fbt.shape[1]), int(cap))
            self.vbt = torch.zeros((B, stride), dtype=torch.int32, device=dev)
            self.vlb = torch.zeros((B, stride), dtype=torch.int32, device=dev)
            self.vnb = torch.zeros(B, dtype=torch.int32, device=dev)
            tok = "view_token_mask" in plan
            self.vmask = torch.zeros((B, stride), dtype=torch.int32, device=dev) if tok else None
            masks = dict(sel_token_mask=plan["view_token_mask"], view_token_mask=self.vmask) \
                if tok else {}
            self.history = torch.zeros((B, window, 2), dtype=torch.int32, device=dev)
            self.cycles = torch.zeros(B, dtype=torch.int32, device=dev)
            self.mode = torch.zeros(B, dtype=torch.int32, device=dev)
            self.draws = i32(w.accept_draws)                        # [cycles][B]
            self.gammas = [q.shape[1] - 1 for q in w.q_verify]
            common = (plan["view_tokens"], self.seq_lens, plan["plan_status"], self.history,
                      self.cycles, self.mode, plan["view_block_table"],
                      plan["view_logical_block"], plan["view_num_blocks"], self.fbt, self.vbt,
                      self.vlb, self.vnb)
            s = self.stream
            self.reset = K.bind_fallback_update(True, window, 0, None, *common, stream=s, **masks)
            self.update = [K.bind_fallback_update(False, window, g, self.draws[c], *common,
                                                  stream=s, **masks)
                           for c, g in enumerate(self.gammas)]
            Hq, D = w.num_q_heads, w.head_dim
            self.out = torch.empty((B, Hq, D), dtype=torch.float32, device=dev)
            self.lse = torch.empty((B, Hq), dtype=torch.float32, device=dev)
            ws = torch.zeros(max(256, K.selected_decode_workspace_bytes(kv, B, stride)),
                             dtype=torch.uint8, device=dev)
            self.decode = [K.bind_selected_decode(kv, w.q_decode[i], self.seq_lens, self.vbt,
                                                  self.vlb, self.vnb, stride, w.sm_scale,
                                                  self.out, self.lse, ws,
                                                  view_token_mask=self.vmask, stream=s)
                           for i in range(w.q_decode.shape[0])]
            max_len = int(np.max(w.seq_lens))
            self.ver_out, self.verify = [], []
            for q in w.q_verify:
                ql = q.shape[1]
                ov = torch.empty((B, ql, Hq, D), dtype=torch.float32, device=dev)
                lv = torch.empty((B, ql, Hq), dtype=torch.float32, device=dev)
                wv = torch.zeros(max(256, K.verify_workspace_bytes(kv, B, ql, max_len)),
                                 dtype=torch.uint8, device=dev)
                self.ver_out.append((ov, lv))
                self.verify.append(K.bind_verify(kv, q, self.seq_lens, self.fbt, max_len,
                                                 w.sm_scale, ov, lv, wv, stream=s))

    def run(self):
        """Enqueue one whole stream on self.stream (no host synchronisation)."""
        if self.plan_call is not None:
            self.plan_call()
        self.reset()
        for kind, idx in self.w.schedule:
            if kind == "decode":
                self.decode[idx]()
            else:
                self.verify[idx]()
                self.update[idx]()

    def capture(self):
        """A HIP graph of one whole stream (run)."""
        torch = self.torch
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=self.stream):
            self.run()
        return g
