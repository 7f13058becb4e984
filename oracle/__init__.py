"""fp64 CPU oracle of CompressKV's prefill-end token selection.

TEST INFRASTRUCTURE ONLY: the parity reference for the HIP library. Only the
tests, ``__graft_entry__.smoke()`` and the benchmark's ``cpu_baseline`` leg may
import this package. It shares no code with ``paper_2508_02401_amd``; its C
source is ``ckv_oracle.c`` next to this file (plain loops, fp64).

Paper: CompressKV (arXiv 2508.02401). Sec. 3.3 defines the token selection
(window sums of the chosen heads' attention scores, pooling, head mean, top-N,
retain/evict); Eq. 2 the attention scores; Algorithm 1 (appendix "More
Implementation Details") the layer budgets.

Parity pins: every function here is pinned by tests in ``tests/test_oracle_*.py``
(hand-worked exact examples, closed forms, invariants, library routines and
brute force on tiny inputs). None is "parity unpinned".
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ckv_oracle.c")
_LIB = os.path.join(_HERE, "libckv_oracle.so")

POOL_AVG = 0
POOL_MAX = 1

OK = 0
EINVAL = -1
EBUDGET = -3
EMASK = -4


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (fp64, OpenMP). Returns the library path."""
    if not force and os.path.exists(_LIB) and os.path.getmtime(_LIB) >= os.path.getmtime(_SRC):
        return _LIB
    tmp = _LIB + ".tmp%d" % os.getpid()
    cmd = ["gcc", "-O2", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", "-shared",
           "-fPIC", "-std=c11", _SRC, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        lib = ctypes.CDLL(_LIB)
        P = ctypes.POINTER
        d = ctypes.c_double
        i32, i64 = ctypes.c_int32, ctypes.c_int64
        lib.ckvo_attention_row.argtypes = [P(d), P(d), i64, i32, d, P(d)]
        lib.ckvo_attention_row.restype = ctypes.c_int
        lib.ckvo_window_sums.argtypes = [P(d), i32, P(d), i64, i32, i32, d, P(d)]
        lib.ckvo_window_sums.restype = ctypes.c_int
        lib.ckvo_window_lse.argtypes = [P(d), i32, P(d), i64, i32, i32, d, P(d)]
        lib.ckvo_window_lse.restype = ctypes.c_int
        lib.ckvo_pool.argtypes = [P(d), i64, i32, i32, P(d)]
        lib.ckvo_pool.restype = ctypes.c_int
        lib.ckvo_select_tokens.argtypes = [P(d), i64, i32, i64, P(i32)]
        lib.ckvo_select_tokens.restype = i64
        lib.ckvo_gather_rows.argtypes = [ctypes.c_void_p, i64, P(i32), i64, ctypes.c_void_p]
        lib.ckvo_gather_rows.restype = ctypes.c_int
        lib.ckvo_select_group.argtypes = [P(d), i32, P(d), i64, i32, i32, d, i32, i32, i64,
                                          P(d), P(d), P(i32)]
        lib.ckvo_select_group.restype = i64
        lib.ckvo_select_layer.argtypes = [P(d), P(ctypes.c_uint8), i32, i32, P(d), i64, i32,
                                          i32, d, i32, i32, i64, P(d), P(i32), i32]
        lib.ckvo_select_layer.restype = i64
        lib.ckvo_select_layer_shared.argtypes = lib.ckvo_select_layer.argtypes
        lib.ckvo_select_tokens_all.argtypes = [P(d), i64, i64, P(i32)]
        lib.ckvo_select_tokens_all.restype = i64
        lib.ckvo_select_group_all.argtypes = [P(d), i32, P(d), i64, i32, i32, d, i32, i32, i64,
                                              P(d), P(i32)]
        lib.ckvo_select_group_all.restype = i64
        lib.ckvo_select_layer_shared_all.argtypes = [P(d), P(ctypes.c_uint8), i32, i32, P(d), i64,
                                                     i32, i32, d, i32, i32, i64, P(d), P(i32)]
        lib.ckvo_select_layer_shared_all.restype = i64
        lib.ckvo_select_layer_shared.restype = i64
        lib.ckvo_decode_attention.argtypes = [P(d), P(d), P(d), i32, i32, i64, i32, d, P(d)]
        lib.ckvo_decode_attention.restype = ctypes.c_int
        lib.ckvo_layer_error.argtypes = [P(d), i32, i32, i32, i32, P(d), P(d), i64, P(d), P(d),
                                         i64, P(d), i32, d, d, P(d), P(d)]
        lib.ckvo_layer_error.restype = ctypes.c_int
        lib.ckvo_normalize_errors.argtypes = [P(d), i32, i32, P(d)]
        lib.ckvo_normalize_errors.restype = ctypes.c_int
        lib.ckvo_allocate_budgets.argtypes = [P(d), i32, i64, i64, i64, P(i64)]
        lib.ckvo_allocate_budgets.restype = ctypes.c_int
        _lib = lib
    return _lib


def _f64(x) -> np.ndarray:
    a = np.ascontiguousarray(np.asarray(x, dtype=np.float64))
    return a


def _ptr(a: np.ndarray, ct):
    return a.ctypes.data_as(ctypes.POINTER(ct))


class OracleError(RuntimeError):
    def __init__(self, code: int, what: str):
        super().__init__("%s failed with oracle status %d" % (what, code))
        self.code = code


def attention_row(q, k, n_visible: int, scale: float) -> np.ndarray:
    """Row softmax of scale * q . k_j over keys j < n_visible (Eq. 2)."""
    q, k = _f64(q), _f64(k)
    p = np.empty(n_visible, dtype=np.float64)
    rc = _load().ckvo_attention_row(_ptr(q, ctypes.c_double), _ptr(k, ctypes.c_double),
                                    n_visible, q.shape[-1], scale, _ptr(p, ctypes.c_double))
    if rc != OK:
        raise OracleError(rc, "attention_row")
    return p


def window_sums(q_sel, k, scale: float) -> np.ndarray:
    """S[h][j] over the full key range [0, L) (Sec. 3.3). q_sel [n_sel, w, d], k [L, d]."""
    q_sel, k = _f64(q_sel), _f64(k)
    n_sel, w, d = q_sel.shape
    L = k.shape[0]
    S = np.empty((n_sel, L), dtype=np.float64)
    rc = _load().ckvo_window_sums(_ptr(q_sel, ctypes.c_double), n_sel, _ptr(k, ctypes.c_double),
                                  L, d, w, scale, _ptr(S, ctypes.c_double))
    if rc != OK:
        raise OracleError(rc, "window_sums")
    return S


def window_lse(q_sel, k, scale: float) -> np.ndarray:
    """Natural-log softmax normaliser of every window row (Eq. 2), [n_sel, w].
    q_sel [n_sel, w, d], k [L, d]; row i sees keys 0..L-w+i."""
    q_sel, k = _f64(q_sel), _f64(k)
    n_sel, w, d = q_sel.shape
    L = k.shape[0]
    out = np.empty((n_sel, w), dtype=np.float64)
    rc = _load().ckvo_window_lse(_ptr(q_sel, ctypes.c_double), n_sel, _ptr(k, ctypes.c_double),
                                 L, d, w, scale, _ptr(out, ctypes.c_double))
    if rc != OK:
        raise OracleError(rc, "window_lse")
    return out


def pool(x, kp: int, mode: int) -> np.ndarray:
    x = _f64(x)
    y = np.empty_like(x)
    rc = _load().ckvo_pool(_ptr(x, ctypes.c_double), x.shape[0], kp, mode, _ptr(y, ctypes.c_double))
    if rc != OK:
        raise OracleError(rc, "pool")
    return y


def select_tokens(a, L: int, w: int, budget: int) -> np.ndarray:
    a = _f64(a)
    out = np.empty(max(min(budget, L), 1), dtype=np.int32)
    n = _load().ckvo_select_tokens(_ptr(a, ctypes.c_double), L, w, budget, _ptr(out, ctypes.c_int32))
    if n < 0:
        raise OracleError(int(n), "select_tokens")
    return out[:n]


def gather_rows(src: np.ndarray, idx) -> np.ndarray:
    """Rows src[idx] copied byte for byte (any dtype; src [L, ...])."""
    src = np.ascontiguousarray(src)
    idx = np.ascontiguousarray(np.asarray(idx, dtype=np.int32))
    row_bytes = src[0].nbytes if src.shape[0] else 0
    dst = np.empty((idx.shape[0],) + src.shape[1:], dtype=src.dtype)
    rc = _load().ckvo_gather_rows(src.ctypes.data, row_bytes, _ptr(idx, ctypes.c_int32),
                                  idx.shape[0], dst.ctypes.data)
    if rc != OK:
        raise OracleError(rc, "gather_rows")
    return dst


def streaming_indices(L: int, budget: int, n_sink: int) -> np.ndarray:
    """StreamingLLM-style retention, which the paper's Sec. 2 describes as
    keeping the first and the last tokens of the prompt: of n_ret = min(budget,
    L) kept tokens, the first min(n_sink, n_ret) are the prompt's first tokens
    (attention sinks) and the others its most recent tokens; ascending."""
    n_ret = min(budget, L)
    n_first = min(n_sink, n_ret)
    first = np.arange(n_first)
    last = np.arange(L - (n_ret - n_first), L)
    return np.concatenate([first, last]).astype(np.int32)


def select_group(q_sel, k, w: int, scale: float, pool_mode: int, kp: int, budget: int,
                 want_pooled: bool = False):
    """One KV group: returns (scores [L-w], idx [min(B, L)], pooled [n_sel, L-w] or None)."""
    q_sel, k = _f64(q_sel), _f64(k)
    n_sel, w_, d = q_sel.shape
    assert w_ == w
    L = k.shape[0]
    scores = np.empty(L - w, dtype=np.float64)
    pooled = np.empty((n_sel, L - w), dtype=np.float64) if want_pooled else None
    idx = np.empty(min(budget, L), dtype=np.int32)
    n = _load().ckvo_select_group(
        _ptr(q_sel, ctypes.c_double), n_sel, _ptr(k, ctypes.c_double), L, d, w, scale,
        pool_mode, kp, budget, _ptr(scores, ctypes.c_double),
        _ptr(pooled, ctypes.c_double) if pooled is not None else None,
        _ptr(idx, ctypes.c_int32))
    if n < 0:
        raise OracleError(int(n), "select_group")
    return scores, idx[:n], pooled


def select_layer(q, mask, k, w: int, scale: float, pool_mode: int, kp: int, budget: int,
                 n_threads: int = 0):
    """One layer. q [H, w, d], mask [H] (nonzero = chosen), k [n_kv, L, d].

    Returns (scores [n_kv, L-w] fp64, idx [n_kv, min(B, L)] int32)."""
    q, k = _f64(q), _f64(k)
    mask = np.ascontiguousarray(np.asarray(mask, dtype=np.uint8))
    H, w_, d = q.shape
    n_kv, L, d2 = k.shape
    assert w_ == w and d2 == d and mask.shape == (H,)
    scores = np.empty((n_kv, L - w), dtype=np.float64)
    idx = np.empty((n_kv, min(budget, L)), dtype=np.int32)
    n = _load().ckvo_select_layer(
        _ptr(q, ctypes.c_double), _ptr(mask, ctypes.c_uint8), H, n_kv, _ptr(k, ctypes.c_double),
        L, d, w, scale, pool_mode, kp, budget, _ptr(scores, ctypes.c_double),
        _ptr(idx, ctypes.c_int32), n_threads)
    if n < 0:
        raise OracleError(int(n), "select_layer")
    return scores, idx


def select_layer_shared(q, mask, k, w: int, scale: float, pool_mode: int, kp: int, budget: int,
                        n_threads: int = 0):
    """The paper's layer-shared variant. q [H, w, d], mask [H], k [n_kv, L, d].

    Returns (scores [L-w] fp64, idx [min(B, L)] int32), one index set for every
    KV head of the layer."""
    q, k = _f64(q), _f64(k)
    mask = np.ascontiguousarray(np.asarray(mask, dtype=np.uint8))
    H, w_, d = q.shape
    n_kv, L, d2 = k.shape
    assert w_ == w and d2 == d and mask.shape == (H,)
    scores = np.empty(L - w, dtype=np.float64)
    idx = np.empty(min(budget, L), dtype=np.int32)
    n = _load().ckvo_select_layer_shared(
        _ptr(q, ctypes.c_double), _ptr(mask, ctypes.c_uint8), H, n_kv, _ptr(k, ctypes.c_double),
        L, d, w, scale, pool_mode, kp, budget, _ptr(scores, ctypes.c_double),
        _ptr(idx, ctypes.c_int32), n_threads)
    if n < 0:
        raise OracleError(int(n), "select_layer_shared")
    return scores, idx


def select_tokens_all(a, L: int, budget: int) -> np.ndarray:
    """Keep-window flag off: the budget best tokens of [0, L) by score a[L]
    (lower index first on ties), ascending; all L when budget >= L."""
    a = _f64(a)
    out = np.empty(min(budget, L) if budget >= 1 else 1, dtype=np.int32)
    n = _load().ckvo_select_tokens_all(_ptr(a, ctypes.c_double), L, budget, _ptr(out, ctypes.c_int32))
    if n < 0:
        raise OracleError(int(n), "select_tokens_all")
    return out[:n]


def select_group_all(q_sel, k, w: int, scale: float, pool_mode: int, kp: int, budget: int):
    """One KV group with the keep-window flag off: (scores [L], idx [min(B, L)])."""
    q_sel, k = _f64(q_sel), _f64(k)
    n_sel, w_, d = q_sel.shape
    assert w_ == w
    L = k.shape[0]
    scores = np.empty(L, dtype=np.float64)
    idx = np.empty(max(1, min(budget, L)), dtype=np.int32)
    n = _load().ckvo_select_group_all(
        _ptr(q_sel, ctypes.c_double), n_sel, _ptr(k, ctypes.c_double), L, d, w, scale,
        pool_mode, kp, budget, _ptr(scores, ctypes.c_double), _ptr(idx, ctypes.c_int32))
    if n < 0:
        raise OracleError(int(n), "select_group_all")
    return scores, idx[:n]


def select_layer_shared_all(q, mask, k, w: int, scale: float, pool_mode: int, kp: int,
                            budget: int):
    """The layer-shared selection with the keep-window flag off. q [H, w, d],
    mask [H], k [n_kv, L, d]: (scores [L], idx [min(B, L)])."""
    q, k = _f64(q), _f64(k)
    mask = np.ascontiguousarray(np.asarray(mask, dtype=np.uint8))
    H, w_, d = q.shape
    n_kv, L, d2 = k.shape
    assert w_ == w and d2 == d and mask.shape == (H,)
    scores = np.empty(L, dtype=np.float64)
    idx = np.empty(max(1, min(budget, L)), dtype=np.int32)
    n = _load().ckvo_select_layer_shared_all(
        _ptr(q, ctypes.c_double), _ptr(mask, ctypes.c_uint8), H, n_kv, _ptr(k, ctypes.c_double),
        L, d, w, scale, pool_mode, kp, budget, _ptr(scores, ctypes.c_double),
        _ptr(idx, ctypes.c_int32))
    if n < 0:
        raise OracleError(int(n), "select_layer_shared_all")
    return scores, idx[:n]


def decode_attention(q, k, v, scale: float):
    """Decode attention, one query per head. q [H, d], k/v [n_kv, n, d] -> [H, d]."""
    q, k, v = _f64(q), _f64(k), _f64(v)
    H, d = q.shape
    n_kv, n, d2 = k.shape
    assert d2 == d and v.shape == k.shape
    out = np.empty((H, d), dtype=np.float64)
    rc = _load().ckvo_decode_attention(_ptr(q, ctypes.c_double), _ptr(k, ctypes.c_double),
                                       _ptr(v, ctypes.c_double), H, n_kv, n, d, scale,
                                       _ptr(out, ctypes.c_double))
    if rc != OK:
        raise OracleError(rc, "decode_attention")
    return out


def layer_error(q_dec, k, v, k_comp, v_comp, w_o, scale: float, eps: float = 1e-6):
    """Eq. 6-8 for one layer. q_dec [T, H, d]; k/v [n_kv, L, d]; k_comp/v_comp
    [n_kv, n_c, d]; w_o [D, H*d]. Returns (e, per-step terms [T])."""
    q_dec, k, v, kc, vc, w_o = map(_f64, (q_dec, k, v, k_comp, v_comp, w_o))
    T, H, d = q_dec.shape
    n_kv, L, _ = k.shape
    n_c = kc.shape[1]
    D = w_o.shape[0]
    assert w_o.shape[1] == H * d and kc.shape == vc.shape and kc.shape[0] == n_kv
    ratio = np.empty(T, dtype=np.float64)
    e = np.empty(1, dtype=np.float64)
    rc = _load().ckvo_layer_error(_ptr(q_dec, ctypes.c_double), T, H, n_kv, d,
                                  _ptr(k, ctypes.c_double), _ptr(v, ctypes.c_double), L,
                                  _ptr(kc, ctypes.c_double), _ptr(vc, ctypes.c_double), n_c,
                                  _ptr(w_o, ctypes.c_double), D, scale, eps,
                                  _ptr(ratio, ctypes.c_double), _ptr(e, ctypes.c_double))
    if rc != OK:
        raise OracleError(rc, "layer_error")
    return float(e[0]), ratio


def normalize_errors(e):
    """Eq. 10-12: e [n_sets, n_layers] -> e_tilde [n_layers]."""
    e = _f64(np.atleast_2d(e))
    out = np.empty(e.shape[1], dtype=np.float64)
    rc = _load().ckvo_normalize_errors(_ptr(e, ctypes.c_double), e.shape[0], e.shape[1],
                                       _ptr(out, ctypes.c_double))
    if rc != OK:
        raise OracleError(rc, "normalize_errors")
    return out


def allocate_budgets(e, total: int, m: int, M: int):
    """Algorithm 1. Returns (budgets int64 [n], status) with status 0 or EBUDGET."""
    e = _f64(e)
    B = np.empty(e.shape[0], dtype=np.int64)
    rc = _load().ckvo_allocate_budgets(_ptr(e, ctypes.c_double), e.shape[0], total, m, M,
                                       _ptr(B, ctypes.c_int64))
    if rc not in (OK, EBUDGET):
        raise OracleError(rc, "allocate_budgets")
    return B, rc
