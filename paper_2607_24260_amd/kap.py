"""Python binding of the kap.h C ABI (argument marshalling only).

Every function here checks tensor placement, dtype and shape, allocates
outputs / workspace with torch when the caller does not pass them, and calls
the matching ``kap_*`` entry point of ``libkap.so`` on the given stream
(torch's current HIP stream by default). Tensors allocated here are allocated,
and zero-filled where needed, on that same stream, so they are ordered with
the launch and the caching allocator reuses them only after it. All
computation happens in the library's HIP kernels; there is no CPU path. A
missing library or a CPU tensor raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libkap.so")

KAP_OK = 0
KAP_ERR_INVALID_ARGUMENT = 1
KAP_ERR_UNSUPPORTED = 2
KAP_ERR_WORKSPACE_TOO_SMALL = 3
KAP_ERR_HIP = 4

KAP_DT_F32 = 0
KAP_DT_BF16 = 1
KAP_DT_FP8_E4M3FN = 2

KAP_SELECT_SKIP = 0
KAP_SELECT_STOP = 1

KAP_PLAN_OK = 0
KAP_PLAN_OVER_CAPACITY = 1
KAP_PLAN_BAD_SCORE = 2
KAP_PLAN_BAD_PAGE = 3
KAP_PLAN_BAD_LENGTH = 4
KAP_PLAN_BAD_SPANS = 5

PAGE = 16

EXPORTS = (
    "kap_compile_plan", "kap_compile_plan_workspace_bytes", "kap_compile_plan_masked",
    "kap_selected_decode", "kap_selected_decode_workspace_bytes", "kap_selected_decode_masked",
    "kap_selected_decode_noalloc", "kap_decode_schedule_bytes", "kap_decode_schedule",
    "kap_selected_decode_scheduled",
    "kap_verify", "kap_verify_workspace_bytes",
    "kap_append_kv", "kap_compact_view", "kap_fallback_update", "kap_fallback_update_masked",
    "kap_accept_top3", "kap_accept_top3_workspace_bytes",
    "kap_status_string", "kap_last_error", "kap_abi_version",
    "kap_stream_read",
)


class KapError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(message)
        self.status = status


class KVCacheStruct(ctypes.Structure):
    _fields_ = [
        ("num_q_heads", ctypes.c_int32),
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("page_size", ctypes.c_int32),
        ("kv_dtype", ctypes.c_int32),
        ("q_dtype", ctypes.c_int32),
        ("k_pages", ctypes.c_void_p),
        ("v_pages", ctypes.c_void_p),
        ("kv_scales", ctypes.c_void_p),
        ("num_pages", ctypes.c_int64),
    ]


_lib = None
_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_SZ = ctypes.c_size_t
_F = ctypes.c_float


def load_library(path: str = LIB_PATH):
    """Load libkap.so once; raise if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"libkap.so not found at {path}; build it with "
                          f"`python -m paper_2607_24260_amd.build`")
    lib = ctypes.CDLL(path)
    lib.kap_compile_plan.restype = _I32
    lib.kap_compile_plan.argtypes = [
        _I32, _P, _P, _I32, _P, _I32, _P, _P, _P, _P, _P, _P, _I32, _I64, _I32,
        _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]
    lib.kap_compile_plan_masked.restype = _I32
    lib.kap_compile_plan_masked.argtypes = [
        _I32, _P, _P, _I32, _P, _I32, _P, _P, _P, _P, _P, _P, _I32, _I64, _I32,
        _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P]
    lib.kap_compile_plan_workspace_bytes.restype = _SZ
    lib.kap_compile_plan_workspace_bytes.argtypes = [_I32, _I32, _I32]
    lib.kap_selected_decode.restype = _I32
    lib.kap_selected_decode.argtypes = [
        ctypes.POINTER(KVCacheStruct), _I32, _P, _P, _P, _P, _I32, _P, _I32, _F, _I32,
        _P, _P, _P, _SZ, _P]
    lib.kap_selected_decode_masked.restype = _I32
    lib.kap_selected_decode_masked.argtypes = [
        ctypes.POINTER(KVCacheStruct), _I32, _P, _P, _P, _P, _P, _I32, _P, _I32, _F, _I32,
        _P, _P, _P, _SZ, _P]
    lib.kap_selected_decode_noalloc.restype = _I32
    lib.kap_selected_decode_noalloc.argtypes = [
        ctypes.POINTER(KVCacheStruct), _I32, _P, _P, _P, _P, _I32, _P, _I32, _F, _I32,
        _P, _P, _P]
    lib.kap_decode_schedule_bytes.restype = _SZ
    lib.kap_decode_schedule_bytes.argtypes = [ctypes.POINTER(KVCacheStruct), _I32, _I32]
    lib.kap_decode_schedule.restype = _I32
    lib.kap_decode_schedule.argtypes = [
        ctypes.POINTER(KVCacheStruct), _I32, _P, _P, _P, _P, _I32, _P, _I32, _P, _SZ, _P]
    lib.kap_selected_decode_scheduled.restype = _I32
    lib.kap_selected_decode_scheduled.argtypes = [
        ctypes.POINTER(KVCacheStruct), _I32, _P, _P, _P, _P, _P, _I32, _P, _I32, _P, _F,
        _P, _P, _P, _SZ, _P]
    lib.kap_selected_decode_workspace_bytes.restype = _SZ
    lib.kap_selected_decode_workspace_bytes.argtypes = [
        ctypes.POINTER(KVCacheStruct), _I32, _I32, _I32]
    lib.kap_verify.restype = _I32
    lib.kap_verify.argtypes = [
        ctypes.POINTER(KVCacheStruct), _I32, _I32, _P, _P, _P, _I32, _I32, _F, _I32,
        _P, _P, _P, _SZ, _P]
    lib.kap_verify_workspace_bytes.restype = _SZ
    lib.kap_verify_workspace_bytes.argtypes = [
        ctypes.POINTER(KVCacheStruct), _I32, _I32, _I32, _I32]
    lib.kap_append_kv.restype = _I32
    lib.kap_append_kv.argtypes = [ctypes.POINTER(KVCacheStruct), _I32, _P, _P, _P, _P, _P]
    lib.kap_compact_view.restype = _I32
    lib.kap_compact_view.argtypes = [
        ctypes.POINTER(KVCacheStruct), _I32, _P, _I32, _P, _I32, ctypes.POINTER(KVCacheStruct),
        _P, _P]
    lib.kap_fallback_update.restype = _I32
    lib.kap_fallback_update.argtypes = [
        _I32, _I32, _I32, _I32, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _I32, _P, _I32,
        _P, _P, _P, _I32, _P]
    lib.kap_fallback_update_masked.restype = _I32
    lib.kap_fallback_update_masked.argtypes = [
        _I32, _I32, _I32, _I32, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _I32, _P, _I32,
        _P, _P, _P, _P, _I32, _P]
    lib.kap_accept_top3.restype = _I32
    lib.kap_accept_top3.argtypes = [_I32, _I32, _I32, _P, _I32, _P, _I32, _P, _P, _P, _SZ, _P]
    lib.kap_accept_top3_workspace_bytes.restype = _SZ
    lib.kap_accept_top3_workspace_bytes.argtypes = [_I32, _I32]
    lib.kap_stream_read.restype = _I32
    lib.kap_stream_read.argtypes = [_P, _SZ, _P, _P]
    lib.kap_status_string.restype = ctypes.c_char_p
    lib.kap_status_string.argtypes = [_I32]
    lib.kap_last_error.restype = ctypes.c_char_p
    lib.kap_last_error.argtypes = []
    lib.kap_abi_version.restype = _I32
    lib.kap_abi_version.argtypes = []
    _lib = lib
    return lib


def _check(status: int):
    if status != KAP_OK:
        lib = load_library()
        raise KapError(status, f"{lib.kap_status_string(status).decode()}: "
                               f"{lib.kap_last_error().decode()}")


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dev(t: torch.Tensor, name: str, dtype=None, ndim=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor (got {t.device}); libkap has no CPU path")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must have {ndim} dims, got {tuple(t.shape)}")
    return t


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _workspace(nbytes: int, device, workspace: Optional[torch.Tensor]):
    """Caller's workspace, or a zero-filled temporary (the arrival counters
    must start at 0). Call under ``torch.cuda.stream(launch stream)``."""
    if nbytes == 0:
        return workspace, 0
    if workspace is None:
        workspace = torch.zeros(nbytes, dtype=torch.uint8, device=device)
    _dev(workspace, "workspace")
    have = workspace.numel() * workspace.element_size()
    return workspace, have


# --------------------------------------------------------------------------
# KV cache descriptor
# --------------------------------------------------------------------------

_KV_DT = {torch.float32: KAP_DT_F32, torch.bfloat16: KAP_DT_BF16, torch.uint8: KAP_DT_FP8_E4M3FN,
          torch.float8_e4m3fn: KAP_DT_FP8_E4M3FN}
_Q_DT = {torch.float32: KAP_DT_F32, torch.bfloat16: KAP_DT_BF16}


@dataclass
class KVCache:
    """Paged KV pool: k_pages [P][Hkv][D/8][16][8] (8-dim chunks, then
    tokens), v_pages [P][Hkv][D][16]; fp8 pools are uint8 (E4M3FN codes) with
    kv_scales [P][2] float32."""
    k_pages: torch.Tensor
    v_pages: torch.Tensor
    num_q_heads: int
    q_dtype: torch.dtype
    kv_scales: Optional[torch.Tensor] = None

    def __post_init__(self):
        _dev(self.k_pages, "k_pages", ndim=5)
        _dev(self.v_pages, "v_pages", ndim=4)
        P, Hkv, C, page, E = self.k_pages.shape
        D = C * E
        if E != 8:
            raise ValueError("k_pages must be [P][Hkv][D/8][page][8]")
        if tuple(self.v_pages.shape) != (P, Hkv, D, page):
            raise ValueError(f"v_pages must be [P][Hkv][D][page] = {(P, Hkv, D, page)}, "
                             f"got {tuple(self.v_pages.shape)}")
        if self.k_pages.dtype != self.v_pages.dtype or self.k_pages.dtype not in _KV_DT:
            raise TypeError("k_pages / v_pages must share a float32, bfloat16 or uint8 dtype")
        if self.q_dtype not in _Q_DT:
            raise TypeError("q_dtype must be float32 or bfloat16")
        if _KV_DT[self.k_pages.dtype] == KAP_DT_FP8_E4M3FN:
            if self.kv_scales is None:
                raise ValueError("fp8 KV needs kv_scales [P][2]")
            _dev(self.kv_scales, "kv_scales", torch.float32)
            if tuple(self.kv_scales.shape) != (P, 2):
                raise ValueError("kv_scales must be [num_pages][2]")
        self.num_kv_heads = Hkv
        self.head_dim = D
        self.page_size = page
        self.num_pages = P
        self.struct = KVCacheStruct(
            self.num_q_heads, Hkv, D, page, _KV_DT[self.k_pages.dtype], _Q_DT[self.q_dtype],
            self.k_pages.data_ptr(), self.v_pages.data_ptr(),
            self.kv_scales.data_ptr() if self.kv_scales is not None else None, P)

    @property
    def device(self):
        return self.k_pages.device


# --------------------------------------------------------------------------
# kap_append_kv / kap_compact_view
# --------------------------------------------------------------------------

def append_kv(kv: KVCache, k_new, v_new, slot_mapping, bad_slots=None, stream=None):
    """Write new tokens' stored K/V ([T][Hkv][D], the pool's storage dtype)
    into their slots (page * 16 + offset; negative = padding) of ``kv``, in
    place. ``bad_slots`` (int32 [1], zeroed by the caller) counts slots past
    the pool."""
    lib = load_library()
    T = int(slot_mapping.shape[0])
    _dev(slot_mapping, "slot_mapping", torch.int64, 1)
    shape = (T, kv.num_kv_heads, kv.head_dim)
    for name, t in (("k_new", k_new), ("v_new", v_new)):
        _dev(t, name, kv.k_pages.dtype)
        if tuple(t.shape) != shape:
            raise ValueError(f"{name} must be {shape}, got {tuple(t.shape)}")
    if bad_slots is not None:
        _dev(bad_slots, "bad_slots", torch.int32)
    _check(lib.kap_append_kv(ctypes.byref(kv.struct), T, _ptr(k_new), _ptr(v_new),
                             _ptr(slot_mapping), _ptr(bad_slots), _stream(stream)))


def compact_view(src: KVCache, view_block_table, view_num_blocks, view_capacity: int,
                 dst: KVCache, out=None, stream=None) -> torch.Tensor:
    """Copy each sequence's first min(view_num_blocks[b], view_capacity) view
    pages of ``src`` to pages b * view_capacity + k of ``dst``; returns the
    compact block table [B][view_capacity] (int32, -1 where nothing was
    copied)."""
    lib = load_library()
    _dev(view_block_table, "view_block_table", torch.int32, 2)
    _dev(view_num_blocks, "view_num_blocks", torch.int32, 1)
    B = int(view_num_blocks.shape[0])
    if view_block_table.shape[0] != B:
        raise ValueError("view_block_table and view_num_blocks disagree on the batch")
    if out is None:
        with torch.cuda.stream(stream):
            out = torch.empty((B, view_capacity), dtype=torch.int32, device=src.device)
    _dev(out, "out", torch.int32, 2)
    if tuple(out.shape) != (B, view_capacity):
        raise ValueError(f"out must be {(B, view_capacity)}")
    _check(lib.kap_compact_view(ctypes.byref(src.struct), B, _ptr(view_block_table),
                                view_block_table.shape[1], _ptr(view_num_blocks),
                                int(view_capacity), ctypes.byref(dst.struct), _ptr(out),
                                _stream(stream)))
    return out


# --------------------------------------------------------------------------
# kap_fallback_update
# --------------------------------------------------------------------------

def bind_fallback_update(reset: bool, window: int, gamma: int, accepted, view_tokens, seq_lens,
                         plan_status, history, cycles, mode, sel_block_table, sel_logical_block,
                         sel_num_blocks, full_block_table, view_block_table, view_logical_block,
                         view_num_blocks, sel_token_mask=None, view_token_mask=None,
                         stream=None) -> "BoundCall":
    """One cycle of the device-side access-mode policy (kap_fallback_update),
    marshalled once; see kap.h. All arrays int32 on the GPU; history
    [B][window][2], the tables [B][stride]. With the two token-mask tables
    (token-granular views, shaped like the sel_ / view_ tables) it calls
    kap_fallback_update_masked."""
    lib = load_library()
    B = int(seq_lens.shape[0])
    named = dict(view_tokens=view_tokens, seq_lens=seq_lens, plan_status=plan_status,
                 cycles=cycles, mode=mode, sel_num_blocks=sel_num_blocks,
                 view_num_blocks=view_num_blocks)
    for name, t in named.items():
        _dev(t, name, torch.int32, 1)
        if t.shape[0] != B:
            raise ValueError(f"{name} must have {B} entries")
    if not reset or accepted is not None:
        _dev(accepted, "accepted", torch.int32, 1)
        if accepted.shape[0] != B:
            raise ValueError(f"accepted must have {B} entries")
    _dev(history, "history", torch.int32, 3)
    if tuple(history.shape) != (B, window, 2):
        raise ValueError(f"history must be {(B, window, 2)}")
    for name, t in (("sel_block_table", sel_block_table), ("sel_logical_block", sel_logical_block),
                    ("full_block_table", full_block_table), ("view_block_table", view_block_table),
                    ("view_logical_block", view_logical_block)):
        _dev(t, name, torch.int32, 2)
        if t.shape[0] != B:
            raise ValueError(f"{name} must have {B} rows")
    if sel_logical_block.shape != sel_block_table.shape or \
            view_logical_block.shape != view_block_table.shape:
        raise ValueError("block and logical-block tables must have the same shape")
    masked = sel_token_mask is not None or view_token_mask is not None
    if masked:
        for name, t, like in (("sel_token_mask", sel_token_mask, sel_block_table),
                              ("view_token_mask", view_token_mask, view_block_table)):
            _dev(t, name, torch.int32, 2)
            if t.shape != like.shape:
                raise ValueError(f"{name} must be shaped like its block table")
    mask = lambda t: (_ptr(t),) if masked else ()
    args = (B, int(bool(reset)), int(window), int(gamma), _ptr(accepted), _ptr(view_tokens),
            _ptr(seq_lens), _ptr(plan_status), _ptr(history), _ptr(cycles), _ptr(mode),
            _ptr(sel_block_table), _ptr(sel_logical_block), *mask(sel_token_mask),
            _ptr(sel_num_blocks), sel_block_table.shape[1], _ptr(full_block_table),
            full_block_table.shape[1], _ptr(view_block_table), _ptr(view_logical_block),
            *mask(view_token_mask), _ptr(view_num_blocks), view_block_table.shape[1],
            _stream(stream))
    # not run here: the call updates state (errors surface when it is called)
    fn = lib.kap_fallback_update_masked if masked else lib.kap_fallback_update
    return BoundCall(fn, args,
                     (accepted, view_tokens, seq_lens, plan_status, history, cycles, mode,
                      sel_block_table, sel_logical_block, sel_num_blocks, full_block_table,
                      view_block_table, view_logical_block, view_num_blocks, sel_token_mask,
                      view_token_mask))


# --------------------------------------------------------------------------
# kap_accept_top3
# --------------------------------------------------------------------------

def accept_top3(logits, draft_tokens, top_k: int = 3, accepted=None, carry=None,
                workspace=None, stream=None):
    """Tolerant acceptance of verify windows: logits [B][window][vocab]
    (float32 / bfloat16), draft_tokens [B][window-1] int32. Returns
    (accepted [B], carry_token [B]) int32 tensors; see kap.h."""
    lib = load_library()
    _dev(logits, "logits", None, 3)
    if logits.dtype not in (torch.float32, torch.bfloat16):
        raise TypeError("logits must be float32 or bfloat16")
    B, Wn, V = logits.shape
    _dev(draft_tokens, "draft_tokens", torch.int32, 2)
    if tuple(draft_tokens.shape) != (B, Wn - 1):
        raise ValueError(f"draft_tokens must be {(B, Wn - 1)}")
    dev = logits.device
    with torch.cuda.stream(stream):
        if accepted is None:
            accepted = torch.empty(B, dtype=torch.int32, device=dev)
        if carry is None:
            carry = torch.empty(B, dtype=torch.int32, device=dev)
        workspace, have = _workspace(int(lib.kap_accept_top3_workspace_bytes(B, Wn)), dev,
                                     workspace)
    _dev(accepted, "accepted", torch.int32, 1)
    _dev(carry, "carry", torch.int32, 1)
    dt = KAP_DT_F32 if logits.dtype == torch.float32 else KAP_DT_BF16
    _check(lib.kap_accept_top3(B, Wn, V, _ptr(logits), dt, _ptr(draft_tokens), int(top_k),
                               _ptr(accepted), _ptr(carry), _ptr(workspace), have,
                               _stream(stream)))
    return accepted, carry


# --------------------------------------------------------------------------
# kap_compile_plan
# --------------------------------------------------------------------------

def compile_plan_workspace_bytes(batch: int, num_spans: int, fbt_stride: int) -> int:
    return int(load_library().kap_compile_plan_workspace_bytes(batch, num_spans, fbt_stride))


def _plan_call(seq_lens, full_block_table, span_offsets, span_start, span_len, span_prior,
               prefix_tokens, suffix_tokens, budget_tokens, num_pages, view_capacity, policy,
               out, workspace, token_granular, stream):
    """Validate and marshal one kap_compile_plan[_masked] call: returns
    (function, ctypes arguments, out)."""
    lib = load_library()
    i32 = torch.int32
    _dev(seq_lens, "seq_lens", i32, 1)
    B = seq_lens.shape[0]
    _dev(full_block_table, "full_block_table", i32, 2)
    if full_block_table.shape[0] != B:
        raise ValueError("full_block_table must have one row per sequence")
    _dev(span_offsets, "span_offsets", i32, 1)
    if span_offsets.shape[0] != B + 1:
        raise ValueError("span_offsets must have batch+1 entries")
    for name, t, dt in (("span_start", span_start, i32), ("span_len", span_len, i32),
                        ("span_prior", span_prior, torch.float32)):
        _dev(t, name, dt, 1)
    S = span_start.shape[0]
    if span_len.shape[0] != S or span_prior.shape[0] != S:
        raise ValueError("span arrays must have equal length")
    for name, t in (("prefix_tokens", prefix_tokens), ("suffix_tokens", suffix_tokens),
                    ("budget_tokens", budget_tokens)):
        _dev(t, name, i32, 1)
        if t.shape[0] != B:
            raise ValueError(f"{name} must have batch entries")
    dev = seq_lens.device
    with torch.cuda.stream(stream):
        if out is None:
            cap = max(int(view_capacity), 0)
            out = {
                "view_block_table": torch.empty((B, cap), dtype=i32, device=dev),
                "view_logical_block": torch.empty((B, cap), dtype=i32, device=dev),
                "view_num_blocks": torch.empty(B, dtype=i32, device=dev),
                "view_tokens": torch.empty(B, dtype=i32, device=dev),
                "spans_taken": torch.empty(B, dtype=i32, device=dev),
                "plan_status": torch.empty(B, dtype=i32, device=dev),
                "span_selected": torch.empty(S, dtype=i32, device=dev),
            }
            if token_granular:
                out["view_token_mask"] = torch.empty((B, cap), dtype=i32, device=dev)
        need = compile_plan_workspace_bytes(B, S, full_block_table.shape[1])
        workspace, have = _workspace(need, dev, workspace)
    tables = ("view_block_table", "view_logical_block") + (
        ("view_token_mask",) if token_granular else ())
    for name in tables:
        if name not in out:
            raise ValueError(f"out needs {name}")
        _dev(out[name], name, i32, 2)
        if out[name].shape != (B, view_capacity):
            raise ValueError(f"{name} must be [batch][view_capacity]")
    head = (B, _ptr(seq_lens), _ptr(full_block_table), full_block_table.shape[1],
            _ptr(span_offsets), S, _ptr(span_start), _ptr(span_len), _ptr(span_prior),
            _ptr(prefix_tokens), _ptr(suffix_tokens), _ptr(budget_tokens), int(policy),
            int(num_pages), int(view_capacity), _ptr(out["view_block_table"]),
            _ptr(out["view_logical_block"]))
    mask = (_ptr(out["view_token_mask"]),) if token_granular else ()
    tail = (_ptr(out["view_num_blocks"]), _ptr(out["view_tokens"]), _ptr(out["spans_taken"]),
            _ptr(out["plan_status"]), _ptr(out.get("span_selected")), _ptr(workspace), have,
            _stream(stream))
    fn = lib.kap_compile_plan_masked if token_granular else lib.kap_compile_plan
    keep = (seq_lens, full_block_table, span_offsets, span_start, span_len, span_prior,
            prefix_tokens, suffix_tokens, budget_tokens, out, workspace)
    return fn, head + mask + tail, out, keep


def compile_plan(seq_lens, full_block_table, span_offsets, span_start, span_len, span_prior,
                 prefix_tokens, suffix_tokens, budget_tokens, *, num_pages: int,
                 view_capacity: int, policy: int = KAP_SELECT_SKIP, out: Optional[dict] = None,
                 workspace: Optional[torch.Tensor] = None, token_granular: bool = False,
                 stream=None) -> dict:
    """Runtime access plan of every sequence (Alg. 1). Returns a dict of GPU
    tensors: view_block_table, view_logical_block [B][view_capacity],
    view_num_blocks, view_tokens, spans_taken, plan_status [B], span_selected [S];
    with ``token_granular`` (kap_compile_plan_masked) also view_token_mask
    [B][view_capacity] (int32 holding the 16-bit masks)."""
    fn, args, out, _ = _plan_call(seq_lens, full_block_table, span_offsets, span_start,
                                  span_len, span_prior, prefix_tokens, suffix_tokens,
                                  budget_tokens, num_pages, view_capacity, policy, out,
                                  workspace, token_granular, stream)
    _check(fn(*args))
    return out


# --------------------------------------------------------------------------
# kap_selected_decode / kap_verify
# --------------------------------------------------------------------------

def selected_decode_workspace_bytes(kv: KVCache, batch: int, max_view_blocks: int,
                                    num_splits: int = 0) -> int:
    return int(load_library().kap_selected_decode_workspace_bytes(
        ctypes.byref(kv.struct), batch, max_view_blocks, num_splits))


def verify_workspace_bytes(kv: KVCache, batch: int, q_len: int, max_seq_len: int,
                           num_splits: int = 0) -> int:
    return int(load_library().kap_verify_workspace_bytes(
        ctypes.byref(kv.struct), batch, q_len, max_seq_len, num_splits))


def _outputs(shape, dev, out, lse):
    if out is None:
        out = torch.empty(shape, dtype=torch.float32, device=dev)
    if lse is None:
        lse = torch.empty(shape[:-1], dtype=torch.float32, device=dev)
    _dev(out, "out", torch.float32)
    _dev(lse, "lse", torch.float32)
    if tuple(out.shape) != tuple(shape) or tuple(lse.shape) != tuple(shape[:-1]):
        raise ValueError(f"out must be {tuple(shape)} and lse {tuple(shape[:-1])}")
    return out, lse


def _decode_call(kv: KVCache, q, seq_lens, view_block_table, view_logical_block,
                 view_num_blocks, max_view_blocks, sm_scale, num_splits, out, lse, workspace,
                 view_token_mask, stream, noalloc=False, schedule=None):
    """Validate and marshal one kap_selected_decode[_masked] call, or with
    ``schedule`` (from decode_schedule) a kap_selected_decode_scheduled one."""
    lib = load_library()
    _dev(q, "q", kv.q_dtype, 3)
    B = q.shape[0]
    if tuple(q.shape[1:]) != (kv.num_q_heads, kv.head_dim):
        raise ValueError("q must be [batch][num_q_heads][head_dim]")
    _dev(seq_lens, "seq_lens", torch.int32, 1)
    _dev(view_num_blocks, "view_num_blocks", torch.int32, 1)
    _dev(view_block_table, "view_block_table", torch.int32, 2)
    _dev(view_logical_block, "view_logical_block", torch.int32, 2)
    if view_block_table.shape != view_logical_block.shape or view_block_table.shape[0] != B:
        raise ValueError("view tables must both be [batch][view_stride]")
    if view_token_mask is not None:
        _dev(view_token_mask, "view_token_mask", torch.int32, 2)
        if view_token_mask.shape != view_block_table.shape:
            raise ValueError("view_token_mask must be shaped like the view tables")
    if seq_lens.shape[0] != B or view_num_blocks.shape[0] != B:
        raise ValueError("seq_lens / view_num_blocks must have batch entries")
    if schedule is not None:
        if num_splits != 0:
            raise ValueError("a scheduled decode takes num_splits = 0")
        nbytes = decode_schedule_bytes(kv, B, max_view_blocks)
        if nbytes:
            _dev(schedule, "schedule", torch.int32, 1)
        if schedule.numel() * 4 < nbytes:
            raise ValueError(f"schedule of {nbytes} bytes required")
    need = 0 if noalloc else selected_decode_workspace_bytes(kv, B, max_view_blocks, num_splits)
    with torch.cuda.stream(stream):
        out, lse = _outputs((B, kv.num_q_heads, kv.head_dim), q.device, out, lse)
        workspace, have = _workspace(need, q.device, workspace)
    head = (ctypes.byref(kv.struct), B, _ptr(q), _ptr(seq_lens), _ptr(view_block_table),
            _ptr(view_logical_block))
    mask = () if view_token_mask is None else (_ptr(view_token_mask),)
    tail = (view_block_table.shape[1], _ptr(view_num_blocks), int(max_view_blocks),
            float(sm_scale), int(num_splits), _ptr(out), _ptr(lse), _ptr(workspace), have,
            _stream(stream))
    keep = (kv, q, seq_lens, view_block_table, view_logical_block, view_num_blocks,
            view_token_mask, out, lse, workspace, schedule)
    if schedule is not None:
        args = head + (_ptr(view_token_mask), view_block_table.shape[1], _ptr(view_num_blocks),
                       int(max_view_blocks),
                       _ptr(schedule) if schedule.numel() else None, float(sm_scale),
                       _ptr(out), _ptr(lse), _ptr(workspace), have, _stream(stream))
        return lib.kap_selected_decode_scheduled, args, (out, lse), keep
    fn = lib.kap_selected_decode if view_token_mask is None else lib.kap_selected_decode_masked
    return fn, head + mask + tail, (out, lse), keep


def selected_decode(kv: KVCache, q, seq_lens, view_block_table, view_logical_block,
                    view_num_blocks, max_view_blocks: int, sm_scale: float, *,
                    num_splits: int = 0, out=None, lse=None, workspace=None,
                    view_token_mask=None, schedule=None, stream=None):
    """One proposal step over the selected-KV view. q [B][Hq][D]; returns
    (out [B][Hq][D] float32, lse [B][Hq] float32). ``view_token_mask``
    [B][view_stride] (a token-granular plan's masks) calls
    kap_selected_decode_masked; ``schedule`` (decode_schedule's output for
    this view) calls kap_selected_decode_scheduled."""
    fn, args, res, _ = _decode_call(kv, q, seq_lens, view_block_table, view_logical_block,
                                    view_num_blocks, max_view_blocks, sm_scale, num_splits,
                                    out, lse, workspace, view_token_mask, stream,
                                    schedule=schedule)
    _check(fn(*args))
    return res


def decode_schedule_bytes(kv: KVCache, batch: int, max_view_blocks: int) -> int:
    return int(load_library().kap_decode_schedule_bytes(ctypes.byref(kv.struct), int(batch),
                                                        int(max_view_blocks)))


def _schedule_call(kv: KVCache, seq_lens, view_block_table, view_logical_block,
                   view_num_blocks, max_view_blocks, view_token_mask, out, stream):
    """Validate and marshal one kap_decode_schedule call: (args, out)."""
    _dev(seq_lens, "seq_lens", torch.int32, 1)
    _dev(view_num_blocks, "view_num_blocks", torch.int32, 1)
    _dev(view_block_table, "view_block_table", torch.int32, 2)
    _dev(view_logical_block, "view_logical_block", torch.int32, 2)
    B = seq_lens.shape[0]
    if view_block_table.shape != view_logical_block.shape or view_block_table.shape[0] != B:
        raise ValueError("view tables must both be [batch][view_stride]")
    if view_token_mask is not None:
        _dev(view_token_mask, "view_token_mask", torch.int32, 2)
        if view_token_mask.shape != view_block_table.shape:
            raise ValueError("view_token_mask must be shaped like the view tables")
    nbytes = decode_schedule_bytes(kv, B, max_view_blocks)
    with torch.cuda.stream(stream):
        if out is None:
            out = torch.empty(nbytes // 4, dtype=torch.int32, device=seq_lens.device)
    if nbytes:
        _dev(out, "out", torch.int32, 1)
    if out.numel() * 4 < nbytes:
        raise ValueError(f"out must hold {nbytes} bytes")
    args = (ctypes.byref(kv.struct), B, _ptr(seq_lens), _ptr(view_block_table),
            _ptr(view_logical_block), _ptr(view_token_mask), view_block_table.shape[1],
            _ptr(view_num_blocks), int(max_view_blocks), _ptr(out) if out.numel() else None,
            out.numel() * 4, _stream(stream))
    return args, out


def decode_schedule(kv: KVCache, seq_lens, view_block_table, view_logical_block,
                    view_num_blocks, max_view_blocks: int, *, view_token_mask=None, out=None,
                    stream=None):
    """kap_decode_schedule: the balanced split assignment of decode calls on
    this view, computed once. Returns an int32 tensor to pass as ``schedule``
    (empty when these calls take no balanced map); written into ``out`` when
    given."""
    args, out = _schedule_call(kv, seq_lens, view_block_table, view_logical_block,
                               view_num_blocks, max_view_blocks, view_token_mask, out, stream)
    _check(load_library().kap_decode_schedule(*args))
    return out


def bind_decode_schedule(kv: KVCache, seq_lens, view_block_table, view_logical_block,
                         view_num_blocks, max_view_blocks: int, out, view_token_mask=None,
                         stream=None) -> "BoundCall":
    """decode_schedule pre-marshalled (and run once here) for tight loops and
    graph capture; each call rewrites ``out`` from the view arrays' current
    contents."""
    args, out = _schedule_call(kv, seq_lens, view_block_table, view_logical_block,
                               view_num_blocks, max_view_blocks, view_token_mask, out, stream)
    lib = load_library()
    _check(lib.kap_decode_schedule(*args))
    return BoundCall(lib.kap_decode_schedule, args,
                     (kv, seq_lens, view_block_table, view_logical_block, view_num_blocks,
                      view_token_mask, out))


def selected_decode_noalloc(kv: KVCache, q, seq_lens, view_block_table, view_logical_block,
                            view_num_blocks, max_view_blocks: int, sm_scale: float, *,
                            num_splits: int = 0, out=None, lse=None, stream=None):
    """kap_selected_decode_noalloc: selected_decode without a workspace (the
    library's per-GPU scratch holds the split partials). Returns (out, lse);
    outputs not passed are allocated here, on the launch stream."""
    lib = load_library()
    fn, args, res, _ = _decode_call(kv, q, seq_lens, view_block_table, view_logical_block,
                                    view_num_blocks, max_view_blocks, sm_scale, num_splits,
                                    out, lse, None, None, stream, noalloc=True)
    del fn
    # kap_selected_decode's arguments without (workspace, workspace_bytes)
    _check(lib.kap_selected_decode_noalloc(*args[:-3], args[-1]))
    return res


def verify(kv: KVCache, q, seq_lens, full_block_table, max_seq_len: int, sm_scale: float, *,
           num_splits: int = 0, out=None, lse=None, workspace=None, stream=None):
    """Causal attention of the verify window over the full KV. q [B][q_len][Hq][D];
    returns (out [B][q_len][Hq][D] float32, lse [B][q_len][Hq] float32)."""
    lib = load_library()
    _dev(q, "q", kv.q_dtype, 4)
    B, q_len = q.shape[0], q.shape[1]
    if tuple(q.shape[2:]) != (kv.num_q_heads, kv.head_dim):
        raise ValueError("q must be [batch][q_len][num_q_heads][head_dim]")
    _dev(seq_lens, "seq_lens", torch.int32, 1)
    _dev(full_block_table, "full_block_table", torch.int32, 2)
    if seq_lens.shape[0] != B or full_block_table.shape[0] != B:
        raise ValueError("seq_lens / full_block_table must have batch rows")
    need = verify_workspace_bytes(kv, B, q_len, max_seq_len, num_splits)
    with torch.cuda.stream(stream):
        out, lse = _outputs((B, q_len, kv.num_q_heads, kv.head_dim), q.device, out, lse)
        workspace, have = _workspace(need, q.device, workspace)
    st = lib.kap_verify(
        ctypes.byref(kv.struct), B, q_len, _ptr(q), _ptr(seq_lens), _ptr(full_block_table),
        full_block_table.shape[1], int(max_seq_len), float(sm_scale), int(num_splits),
        _ptr(out), _ptr(lse), _ptr(workspace), have, _stream(stream))
    _check(st)
    return out, lse


def stream_read(buf, sink, stream=None):
    """kap_stream_read (measurement helper): read every byte of the device
    tensor ``buf`` once with a plain streaming kernel, XOR-folding its words
    into the int32 device scalar ``sink``."""
    _dev(buf, "buf")
    _dev(sink, "sink", torch.int32)
    if not buf.is_contiguous():
        raise ValueError("buf must be contiguous")
    _check(load_library().kap_stream_read(_ptr(buf), buf.numel() * buf.element_size(),
                                          _ptr(sink), _stream(stream)))


def abi_version() -> int:
    return int(load_library().kap_abi_version())


# --------------------------------------------------------------------------
# pre-marshalled calls (for tight loops and graph capture)
# --------------------------------------------------------------------------

class BoundCall:
    """A kap_* call whose ctypes arguments were marshalled once. Calling it
    re-issues the same launch on the stream captured at bind time; the caller
    keeps every tensor named at bind time alive."""

    def __init__(self, fn, args, keep):
        self._fn = fn
        self._args = args
        self._keep = keep

    def __call__(self):
        _check(self._fn(*self._args))


def bind_selected_decode(kv: KVCache, q, seq_lens, view_block_table, view_logical_block,
                         view_num_blocks, max_view_blocks: int, sm_scale: float, out, lse,
                         workspace=None, num_splits: int = 0, view_token_mask=None,
                         schedule=None, stream=None) -> BoundCall:
    need = selected_decode_workspace_bytes(kv, q.shape[0], max_view_blocks, num_splits)
    have = 0 if workspace is None else workspace.numel() * workspace.element_size()
    if need > have:
        raise ValueError(f"workspace of {need} bytes required")
    fn, args, _, keep = _decode_call(kv, q, seq_lens, view_block_table, view_logical_block,
                                     view_num_blocks, max_view_blocks, sm_scale, num_splits,
                                     out, lse, workspace, view_token_mask, stream,
                                     schedule=schedule)
    _check(fn(*args))                                             # validates once
    return BoundCall(fn, args, keep)


def bind_verify(kv: KVCache, q, seq_lens, full_block_table, max_seq_len: int, sm_scale: float,
                out, lse, workspace=None, num_splits: int = 0, stream=None) -> BoundCall:
    lib = load_library()
    verify(kv, q, seq_lens, full_block_table, max_seq_len, sm_scale, num_splits=num_splits,
           out=out, lse=lse, workspace=workspace, stream=stream)
    need = verify_workspace_bytes(kv, q.shape[0], q.shape[1], max_seq_len, num_splits)
    have = 0 if workspace is None else workspace.numel() * workspace.element_size()
    if need > have:
        raise ValueError(f"workspace of {need} bytes required")
    args = (ctypes.byref(kv.struct), q.shape[0], q.shape[1], _ptr(q), _ptr(seq_lens),
            _ptr(full_block_table), full_block_table.shape[1], int(max_seq_len),
            float(sm_scale), int(num_splits), _ptr(out), _ptr(lse), _ptr(workspace), have,
            _stream(stream))
    return BoundCall(lib.kap_verify, args,
                     (kv, q, seq_lens, full_block_table, out, lse, workspace))


def bind_compile_plan(seq_lens, full_block_table, span_offsets, span_start, span_len,
                      span_prior, prefix_tokens, suffix_tokens, budget_tokens, *, num_pages: int,
                      view_capacity: int, out: dict, workspace=None,
                      policy: int = KAP_SELECT_SKIP, token_granular: bool = False,
                      stream=None) -> BoundCall:
    B, S = seq_lens.shape[0], span_start.shape[0]
    need = compile_plan_workspace_bytes(B, S, full_block_table.shape[1])
    have = 0 if workspace is None else workspace.numel() * workspace.element_size()
    if need > have:
        raise ValueError(f"workspace of {need} bytes required")
    fn, args, out, keep = _plan_call(seq_lens, full_block_table, span_offsets, span_start,
                                     span_len, span_prior, prefix_tokens, suffix_tokens,
                                     budget_tokens, num_pages, view_capacity, policy, out,
                                     workspace, token_granular, stream)
    _check(fn(*args))                                             # validates once
    return BoundCall(fn, args, keep)
