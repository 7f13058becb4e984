"""ctypes binding of libckv.so (include/ckv.h). Argument marshalling only.

Every function keeps the C name and contract; torch tensors stand in for device
pointers. Errors come back as :class:`CkvError` carrying the status code.
There is no fallback: if libckv.so is missing or fails to load, every call
raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libckv.so")

# status codes and enums (mirror include/ckv.h)
CKV_OK = 0
CKV_ERR_INVALID_ARG = -1
CKV_ERR_UNSUPPORTED = -2
CKV_ERR_BUDGET = -3
CKV_ERR_MASK = -4
CKV_ERR_WORKSPACE = -5
CKV_ERR_HIP = -6
CKV_BF16, CKV_F16, CKV_F32 = 0, 1, 2
CKV_POOL_AVG, CKV_POOL_MAX = 0, 1
CKV_KEEP_WINDOW = 1
CKV_SHARE_LAYER = 2
CKV_MAX_SEQS = 16
CKV_STACK_LAYERS_PER_LAUNCH = 3
CKV_STACK_CHUNK_TOKENS = 98304


def stack_layers_per_launch(seq_lens) -> int:
    """Layers per K-pass launch of ckv_compress_stack for prompts of these
    lengths (the rule stated in include/ckv.h)."""
    tokens = sum(int(x) for x in seq_lens)
    return max(1, min(CKV_STACK_LAYERS_PER_LAUNCH, CKV_STACK_CHUNK_TOKENS // max(tokens, 1)))
CKV_NOALLOC_MAX_WORKSPACE_BYTES = 64 << 20

EXPORTED = ("ckv_workspace_bytes", "ckv_score", "ckv_select", "ckv_gather", "ckv_compress_layer",
            "ckv_compress_stack", "ckv_allocate_budgets", "ckv_status_string",
            "ckv_last_hip_error", "ckv_set_stage_events", "ckv_set_stack_stage_events",
            "ckv_decode_workspace_bytes", "ckv_decode_attention", "ckv_layer_error_workspace_bytes",
            "ckv_layer_error", "ckv_normalize_errors", "ckv_decode_batch_workspace_bytes",
            "ckv_decode_attention_batch", "ckv_streaming_select", "ckv_compress_layer_noalloc")

_DTYPE_CODE = {torch.bfloat16: CKV_BF16, torch.float16: CKV_F16, torch.float32: CKV_F32}


class ckv_layer_desc(ctypes.Structure):
    _fields_ = [("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("window", ctypes.c_int32),
                ("dtype", ctypes.c_int32), ("scale", ctypes.c_float),
                ("pool", ctypes.c_int32), ("pool_kernel", ctypes.c_int32),
                ("flags", ctypes.c_uint32), ("reserved", ctypes.c_int32)]


class ckv_seq(ctypes.Structure):
    _fields_ = [("q_win", ctypes.c_void_p), ("q_stride_head", ctypes.c_int64),
                ("q_stride_row", ctypes.c_int64), ("k", ctypes.c_void_p), ("v", ctypes.c_void_p),
                ("kv_stride_head", ctypes.c_int64), ("kv_stride_tok", ctypes.c_int64),
                ("seq_len", ctypes.c_int64), ("budget", ctypes.c_int32),
                ("reserved", ctypes.c_int32), ("scores", ctypes.c_void_p),
                ("idx", ctypes.c_void_p), ("k_out", ctypes.c_void_p), ("v_out", ctypes.c_void_p),
                ("lse", ctypes.c_void_p), ("lse_stride_head", ctypes.c_int64)]


class ckv_attn_desc(ctypes.Structure):
    _fields_ = [("num_q_heads", ctypes.c_int32), ("num_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("scale", ctypes.c_float), ("reserved", ctypes.c_int32)]


class ckv_kv_cache(ctypes.Structure):
    _fields_ = [("k", ctypes.c_void_p), ("v", ctypes.c_void_p), ("stride_head", ctypes.c_int64),
                ("stride_tok", ctypes.c_int64), ("n", ctypes.c_int64)]


class ckv_decode_seq(ctypes.Structure):
    _fields_ = [("q", ctypes.c_void_p), ("q_stride_t", ctypes.c_int64),
                ("q_stride_h", ctypes.c_int64), ("T", ctypes.c_int32), ("reserved", ctypes.c_int32),
                ("cache", ckv_kv_cache), ("out", ctypes.c_void_p)]


class CkvError(RuntimeError):
    def __init__(self, status: int, what: str):
        msg = "%s: %s (status %d)" % (what, status_string(status), status)
        if status == CKV_ERR_HIP:
            msg += ", hipError %d" % ckv_last_hip_error()
        super().__init__(msg)
        self.status = status


_lib = None


def load() -> ctypes.CDLL:
    """Load libckv.so; raise if it is not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libckv.so is not built (%s); run __graft_entry__.build()" % LIB_PATH)
        lib = ctypes.CDLL(LIB_PATH)
        P, vp = ctypes.POINTER, ctypes.c_void_p
        D, S = P(ckv_layer_desc), P(ckv_seq)
        lib.ckv_workspace_bytes.argtypes = [D, S, ctypes.c_int32]
        lib.ckv_workspace_bytes.restype = ctypes.c_size_t
        lib.ckv_score.argtypes = [D, P(ctypes.c_uint8), S, ctypes.c_int32, vp, ctypes.c_size_t, vp]
        lib.ckv_select.argtypes = [D, S, ctypes.c_int32, vp, ctypes.c_size_t, vp]
        lib.ckv_gather.argtypes = [D, S, ctypes.c_int32, vp]
        lib.ckv_compress_layer.argtypes = [D, P(ctypes.c_uint8), S, ctypes.c_int32, vp,
                                           ctypes.c_size_t, vp]
        lib.ckv_compress_layer_noalloc.argtypes = [D, P(ctypes.c_uint8), S, ctypes.c_int32, vp]
        lib.ckv_compress_stack.argtypes = [D, ctypes.c_int32, P(ctypes.c_uint8), S, ctypes.c_int32,
                                           vp, ctypes.c_size_t, vp, vp]
        lib.ckv_set_stack_stage_events.argtypes = [P(vp), P(vp), ctypes.c_int32]
        lib.ckv_allocate_budgets.argtypes = [P(ctypes.c_double), ctypes.c_int32, ctypes.c_int64,
                                             ctypes.c_int32, ctypes.c_int32, P(ctypes.c_int32)]
        AD, KC = P(ckv_attn_desc), P(ckv_kv_cache)
        lib.ckv_decode_workspace_bytes.argtypes = [AD, ctypes.c_int32, ctypes.c_int64]
        lib.ckv_decode_workspace_bytes.restype = ctypes.c_size_t
        lib.ckv_decode_attention.argtypes = [AD, vp, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                             KC, vp, vp, ctypes.c_size_t, vp]
        lib.ckv_layer_error_workspace_bytes.argtypes = [AD, ctypes.c_int32, ctypes.c_int64,
                                                        ctypes.c_int64, ctypes.c_int32]
        lib.ckv_layer_error_workspace_bytes.restype = ctypes.c_size_t
        lib.ckv_layer_error.argtypes = [AD, vp, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32, KC,
                                        KC, vp, ctypes.c_int64, ctypes.c_int32, ctypes.c_float,
                                        vp, vp, vp, ctypes.c_size_t, vp]
        lib.ckv_normalize_errors.argtypes = [P(ctypes.c_double), ctypes.c_int32, ctypes.c_int32,
                                             P(ctypes.c_double)]
        lib.ckv_streaming_select.argtypes = [D, S, ctypes.c_int32, ctypes.c_int32, vp]
        lib.ckv_streaming_select.restype = ctypes.c_int
        DS = P(ckv_decode_seq)
        lib.ckv_decode_batch_workspace_bytes.argtypes = [AD, DS, ctypes.c_int32]
        lib.ckv_decode_batch_workspace_bytes.restype = ctypes.c_size_t
        lib.ckv_decode_attention_batch.argtypes = [AD, DS, ctypes.c_int32, vp, ctypes.c_size_t, vp]
        for name in ("ckv_decode_attention", "ckv_layer_error", "ckv_normalize_errors",
                     "ckv_decode_attention_batch", "ckv_streaming_select", "ckv_compress_layer_noalloc"):
            getattr(lib, name).restype = ctypes.c_int
        lib.ckv_status_string.argtypes = [ctypes.c_int]
        lib.ckv_status_string.restype = ctypes.c_char_p
        lib.ckv_last_hip_error.argtypes = []
        lib.ckv_set_stage_events.argtypes = [P(vp), P(vp)]
        for name in ("ckv_score", "ckv_select", "ckv_gather", "ckv_compress_layer",
                     "ckv_compress_stack", "ckv_allocate_budgets", "ckv_last_hip_error",
                     "ckv_set_stage_events", "ckv_set_stack_stage_events"):
            getattr(lib, name).restype = ctypes.c_int
        _lib = lib
    return _lib


def status_string(status: int) -> str:
    return load().ckv_status_string(status).decode()


ckv_status_string = status_string


def ckv_last_hip_error() -> int:
    return load().ckv_last_hip_error()


# --------------------------------------------------------------------------
# marshalling helpers
# --------------------------------------------------------------------------
def layer_desc(num_q_heads: int, num_kv_heads: int, head_dim: int, window: int,
               dtype: torch.dtype = torch.bfloat16, scale: float = 0.0, pool: int = CKV_POOL_MAX,
               pool_kernel: int = 7, flags: int = CKV_KEEP_WINDOW) -> ckv_layer_desc:
    code = _DTYPE_CODE[dtype] if isinstance(dtype, torch.dtype) else int(dtype)
    return ckv_layer_desc(num_q_heads, num_kv_heads, head_dim, window, code, scale, pool,
                          pool_kernel, flags, 0)


@dataclass
class Seq:
    """One prompt. q_win [H, w, d], k/v [n_kv, L, d] (last axis contiguous),
    outputs as in include/ckv.h (None where a call does not need them). lse
    [H, w] fp32 (window axis contiguous) optionally carries the window rows'
    log-sum-exp from the caller's prefill attention."""
    q_win: Optional[torch.Tensor]
    k: Optional[torch.Tensor]
    v: Optional[torch.Tensor]
    budget: int
    scores: Optional[torch.Tensor] = None
    idx: Optional[torch.Tensor] = None
    k_out: Optional[torch.Tensor] = None
    v_out: Optional[torch.Tensor] = None
    seq_len: Optional[int] = None
    lse: Optional[torch.Tensor] = None


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _seq_array(seqs: Sequence[Seq]):
    arr = (ckv_seq * len(seqs))()
    for i, s in enumerate(seqs):
        c = arr[i]
        if s.q_win is not None:
            c.q_win = s.q_win.data_ptr()
            c.q_stride_head, c.q_stride_row = s.q_win.stride(0), s.q_win.stride(1)
        kv = s.k if s.k is not None else s.v
        if s.k is not None:
            c.k = s.k.data_ptr()
        if s.v is not None:
            c.v = s.v.data_ptr()
            if s.k is not None and s.v.stride()[:2] != s.k.stride()[:2]:
                raise ValueError("k and v must share strides")
        if kv is not None:
            c.kv_stride_head, c.kv_stride_tok = kv.stride(0), kv.stride(1)
            c.seq_len = kv.shape[1]
        if s.seq_len is not None:
            c.seq_len = s.seq_len
        c.budget = int(s.budget)
        c.scores, c.idx = _ptr(s.scores), _ptr(s.idx)
        c.k_out, c.v_out = _ptr(s.k_out), _ptr(s.v_out)
        if s.lse is not None:
            if s.lse.dtype != torch.float32 or s.lse.dim() != 2 or s.lse.stride(1) != 1:
                raise ValueError("lse must be fp32 [H, w] with the window axis contiguous")
            c.lse, c.lse_stride_head = s.lse.data_ptr(), s.lse.stride(0)
    return arr


def _mask(head_mask) -> ctypes.Array:
    m = np.ascontiguousarray(np.asarray(head_mask, dtype=np.uint8))
    return (ctypes.c_uint8 * m.size).from_buffer_copy(m.tobytes())


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream if torch.cuda.is_available() else None
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _check(status: int, what: str) -> None:
    if status != CKV_OK:
        raise CkvError(status, what)


# --------------------------------------------------------------------------
# the C entry points
# --------------------------------------------------------------------------
def ckv_workspace_bytes(desc: ckv_layer_desc, seqs: Sequence[Seq]) -> int:
    arr = _seq_array(seqs)
    return load().ckv_workspace_bytes(ctypes.byref(desc), arr, len(seqs))


def ckv_score(desc, head_mask, seqs: Sequence[Seq], workspace: torch.Tensor, stream=None) -> None:
    arr = _seq_array(seqs)
    _check(load().ckv_score(ctypes.byref(desc), _mask(head_mask), arr, len(seqs),
                            workspace.data_ptr(), workspace.numel() * workspace.element_size(),
                            _stream(stream)), "ckv_score")


def ckv_select(desc, seqs: Sequence[Seq], workspace: Optional[torch.Tensor] = None,
               stream=None) -> None:
    arr = _seq_array(seqs)
    ws_ptr = workspace.data_ptr() if workspace is not None else None
    ws_n = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(load().ckv_select(ctypes.byref(desc), arr, len(seqs), ws_ptr, ws_n, _stream(stream)),
           "ckv_select")


def ckv_gather(desc, seqs: Sequence[Seq], stream=None) -> None:
    arr = _seq_array(seqs)
    _check(load().ckv_gather(ctypes.byref(desc), arr, len(seqs), _stream(stream)), "ckv_gather")


def ckv_streaming_select(desc, seqs: Sequence[Seq], n_sink: int, stream=None) -> None:
    """StreamingLLM-style preset: keep the first n_sink and the most recent tokens."""
    arr = _seq_array(seqs)
    _check(load().ckv_streaming_select(ctypes.byref(desc), arr, len(seqs), int(n_sink),
                                       _stream(stream)), "ckv_streaming_select")


def snapkv_mask(num_q_heads: int) -> np.ndarray:
    """SnapKV-style preset for ckv_compress_layer: every query head chosen."""
    return np.ones(num_q_heads, dtype=np.uint8)


def ckv_compress_layer(desc, head_mask, seqs: Sequence[Seq], workspace: torch.Tensor,
                       stream=None) -> None:
    arr = _seq_array(seqs)
    _check(load().ckv_compress_layer(ctypes.byref(desc), _mask(head_mask), arr, len(seqs),
                                     workspace.data_ptr(),
                                     workspace.numel() * workspace.element_size(),
                                     _stream(stream)), "ckv_compress_layer")


def ckv_compress_layer_noalloc(desc, head_mask, seqs: Sequence[Seq], stream=None) -> None:
    arr = _seq_array(seqs)
    _check(load().ckv_compress_layer_noalloc(ctypes.byref(desc), _mask(head_mask), arr,
                                             len(seqs), _stream(stream)),
           "ckv_compress_layer_noalloc")


def ckv_compress_stack(desc, head_masks, seqs: Sequence[Sequence[Seq]], workspace: torch.Tensor,
                       stream=None, side_stream=None) -> None:
    """head_masks [n_layers][H]; seqs[l] is layer l's list of prompts (the same
    lengths in every layer). The workspace holds at least one layer slot
    (ckv_workspace_bytes of one layer); with a side stream, consecutive
    layers' K passes alternate between the two streams."""
    n_layers = len(seqs)
    num_seqs = len(seqs[0]) if n_layers else 0
    if any(len(x) != num_seqs for x in seqs):
        raise ValueError("ckv_compress_stack: every layer needs the same number of prompts")
    flat = [s for layer in seqs for s in layer]
    arr = _seq_array(flat)
    m = np.ascontiguousarray(np.asarray(head_masks, dtype=np.uint8)).reshape(-1)
    if m.size != n_layers * desc.num_q_heads:
        raise ValueError("ckv_compress_stack: head_masks must be [n_layers][H]")
    masks = (ctypes.c_uint8 * m.size).from_buffer_copy(m.tobytes())
    side = None if side_stream is None else _stream(side_stream)
    _check(load().ckv_compress_stack(ctypes.byref(desc), n_layers, masks, arr, num_seqs,
                                     workspace.data_ptr(),
                                     workspace.numel() * workspace.element_size(),
                                     _stream(stream), side), "ckv_compress_stack")


def ckv_allocate_budgets(err_norm, total: int, m: int, M: int):
    """Algorithm 1 on the host. Returns (budgets int32 array, status)."""
    e = np.ascontiguousarray(np.asarray(err_norm, dtype=np.float64))
    out = np.zeros(e.shape[0], dtype=np.int32)
    st = load().ckv_allocate_budgets(e.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                                     e.shape[0], int(total), int(m), int(M),
                                     out.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)))
    if st not in (CKV_OK, CKV_ERR_BUDGET):
        raise CkvError(st, "ckv_allocate_budgets")
    return out, st


CKV_NUM_STAGES = 5
STAGE_NAMES = ("rowstats", "score", "pool", "select", "gather")


def ckv_set_stage_events(begin, end) -> None:
    """begin/end: sequences of CKV_NUM_STAGES raw hipEvent_t handles (None entries
    leave that stage untimed), or None to stop."""
    if begin is None or end is None:
        _check(load().ckv_set_stage_events(None, None), "ckv_set_stage_events")
        return
    if len(begin) != CKV_NUM_STAGES or len(end) != CKV_NUM_STAGES:
        raise ValueError("ckv_set_stage_events: need %d begin and end events" % CKV_NUM_STAGES)
    b = (ctypes.c_void_p * CKV_NUM_STAGES)(*begin)
    e = (ctypes.c_void_p * CKV_NUM_STAGES)(*end)
    _check(load().ckv_set_stage_events(b, e), "ckv_set_stage_events")


_stack_events = None  # keeps the arrays passed to ckv_set_stack_stage_events alive


def ckv_set_stack_stage_events(begin, end) -> None:
    """begin/end: [n_layers][CKV_NUM_STAGES] raw hipEvent_t handles (None entries
    untimed) for the layers of the following ckv_compress_stack calls, or None
    to stop."""
    global _stack_events
    if begin is None or end is None:
        _check(load().ckv_set_stack_stage_events(None, None, 0), "ckv_set_stack_stage_events")
        _stack_events = None
        return
    n = len(begin)
    if len(end) != n or any(len(x) != CKV_NUM_STAGES for x in list(begin) + list(end)):
        raise ValueError("ckv_set_stack_stage_events: need [n_layers][%d] events" % CKV_NUM_STAGES)
    b = (ctypes.c_void_p * (n * CKV_NUM_STAGES))(*[x for row in begin for x in row])
    e = (ctypes.c_void_p * (n * CKV_NUM_STAGES))(*[x for row in end for x in row])
    _stack_events = (b, e)
    _check(load().ckv_set_stack_stage_events(b, e, n), "ckv_set_stack_stage_events")


# --------------------------------------------------------------------------
# output allocation (plumbing)
# --------------------------------------------------------------------------
def alloc_outputs(desc: ckv_layer_desc, s: Seq, with_scores: bool = True) -> Seq:
    """Allocate scores/idx/k_out/v_out for one prompt on the device of s.k
    (one score row and one index row under CKV_SHARE_LAYER; score rows of L - w
    with CKV_KEEP_WINDOW, of L without)."""
    L = s.k.shape[1] if s.seq_len is None else s.seq_len
    n_kv, d = desc.num_kv_heads, desc.head_dim
    n_sg = 1 if desc.flags & CKV_SHARE_LAYER else n_kv
    n_ret = min(int(s.budget), L)
    dev = s.k.device
    tail = desc.window if desc.flags & CKV_KEEP_WINDOW else 0  # tokens kept by rule, unscored
    if with_scores:
        s.scores = torch.empty((n_sg, L - tail), dtype=torch.float32, device=dev)
    s.idx = torch.empty((n_sg, n_ret), dtype=torch.int32, device=dev)
    s.k_out = torch.empty((n_kv, n_ret, d), dtype=s.k.dtype, device=dev)
    s.v_out = torch.empty((n_kv, n_ret, d), dtype=s.k.dtype, device=dev)
    return s


def alloc_workspace(desc: ckv_layer_desc, seqs: Sequence[Seq], device) -> torch.Tensor:
    n = ckv_workspace_bytes(desc, seqs)
    if n == 0:
        raise CkvError(CKV_ERR_INVALID_ARG, "ckv_workspace_bytes")
    return torch.empty(n, dtype=torch.uint8, device=device)


# --------------------------------------------------------------------------
# compression-error profile (decode attention, layer error, normalisation)
# --------------------------------------------------------------------------
def attn_desc(num_q_heads: int, num_kv_heads: int, head_dim: int,
              dtype: torch.dtype = torch.bfloat16, scale: float = 0.0) -> ckv_attn_desc:
    code = _DTYPE_CODE[dtype] if isinstance(dtype, torch.dtype) else int(dtype)
    return ckv_attn_desc(num_q_heads, num_kv_heads, head_dim, code, scale, 0)


def kv_cache(k: torch.Tensor, v: torch.Tensor) -> ckv_kv_cache:
    """k, v [n_kv, n, d] with the same strides and d contiguous."""
    if k.stride() != v.stride() or k.shape != v.shape or k.stride(2) != 1:
        raise ValueError("k and v must be [n_kv, n, d] with equal strides, d contiguous")
    return ckv_kv_cache(k.data_ptr(), v.data_ptr(), k.stride(0), k.stride(1), k.shape[1])


def ckv_decode_workspace_bytes(desc: ckv_attn_desc, T: int, n: int) -> int:
    return load().ckv_decode_workspace_bytes(ctypes.byref(desc), int(T), int(n))


def ckv_decode_attention(desc: ckv_attn_desc, q: torch.Tensor, cache: ckv_kv_cache,
                         out: torch.Tensor, workspace: torch.Tensor, stream=None) -> None:
    """q [T, H, d] (d contiguous), out [T, H, d] fp32 contiguous."""
    if out.dtype != torch.float32 or not out.is_contiguous():
        raise ValueError("out must be contiguous fp32 [T, H, d]")
    _check(load().ckv_decode_attention(ctypes.byref(desc), q.data_ptr(), q.stride(0), q.stride(1),
                                       q.shape[0], ctypes.byref(cache), out.data_ptr(),
                                       workspace.data_ptr(),
                                       workspace.numel() * workspace.element_size(),
                                       _stream(stream)), "ckv_decode_attention")


def decode_seq(q: torch.Tensor, cache: ckv_kv_cache, out: torch.Tensor) -> ckv_decode_seq:
    """One prompt of a decode batch: q [T, H, d] (d contiguous), out [T, H, d] fp32 contiguous."""
    if out.dtype != torch.float32 or not out.is_contiguous():
        raise ValueError("out must be contiguous fp32 [T, H, d]")
    return ckv_decode_seq(q.data_ptr(), q.stride(0), q.stride(1), q.shape[0], 0, cache,
                          out.data_ptr())


def _decode_seq_array(seqs):
    arr = (ckv_decode_seq * max(len(seqs), 1))()
    for i, s in enumerate(seqs):
        arr[i] = s
    return arr


def ckv_decode_batch_workspace_bytes(desc: ckv_attn_desc, seqs) -> int:
    return load().ckv_decode_batch_workspace_bytes(ctypes.byref(desc), _decode_seq_array(seqs),
                                                   len(seqs))


def ckv_decode_attention_batch(desc: ckv_attn_desc, seqs, workspace: torch.Tensor,
                               stream=None) -> None:
    """Decode attention of every prompt in seqs (ckv_decode_seq, e.g. from decode_seq())."""
    _check(load().ckv_decode_attention_batch(ctypes.byref(desc), _decode_seq_array(seqs),
                                             len(seqs), workspace.data_ptr(),
                                             workspace.numel() * workspace.element_size(),
                                             _stream(stream)), "ckv_decode_attention_batch")


def ckv_layer_error_workspace_bytes(desc: ckv_attn_desc, T: int, n_full: int, n_comp: int,
                                    D: int) -> int:
    return load().ckv_layer_error_workspace_bytes(ctypes.byref(desc), int(T), int(n_full),
                                                  int(n_comp), int(D))


def ckv_layer_error(desc: ckv_attn_desc, q: torch.Tensor, full: ckv_kv_cache, comp: ckv_kv_cache,
                    w_o: torch.Tensor, eps: float, ratio: torch.Tensor, e: torch.Tensor,
                    workspace: torch.Tensor, stream=None) -> None:
    """q [T, H, d]; w_o [D, H*d] (rows contiguous); ratio [T] and e [1] fp32 on the device."""
    if w_o.stride(1) != 1:
        raise ValueError("w_o rows must be contiguous")
    _check(load().ckv_layer_error(ctypes.byref(desc), q.data_ptr(), q.stride(0), q.stride(1),
                                  q.shape[0], ctypes.byref(full), ctypes.byref(comp),
                                  w_o.data_ptr(), w_o.stride(0), w_o.shape[0], float(eps),
                                  ratio.data_ptr(), e.data_ptr(), workspace.data_ptr(),
                                  workspace.numel() * workspace.element_size(), _stream(stream)),
           "ckv_layer_error")


def ckv_normalize_errors(e) -> np.ndarray:
    """Eq. 10-12 on the host: e [n_sets, n_layers] -> e_tilde [n_layers] (float64)."""
    a = np.ascontiguousarray(np.atleast_2d(np.asarray(e, dtype=np.float64)))
    out = np.zeros(a.shape[1], dtype=np.float64)
    _check(load().ckv_normalize_errors(a.ctypes.data_as(ctypes.POINTER(ctypes.c_double)),
                                       a.shape[0], a.shape[1],
                                       out.ctypes.data_as(ctypes.POINTER(ctypes.c_double))),
           "ckv_normalize_errors")
    return out
