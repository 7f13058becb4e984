"""Comparison rules shared by the GPU parity tests, smoke() and the bench.

Acceptance, stated once:
  * scores: |gpu - oracle| <= 1e-3 * |oracle| + 1e-9 element-wise (fp32
    accumulation against fp64);
  * retained indices: identical window positions; over the prefix the sets
    may differ only by equal numbers of swaps, each involving a token whose
    oracle score is within 1e-5 (absolute) of the oracle's threshold score;
  * compact K/V: bit-exact copies of the input rows the GPU kept.
"""
from __future__ import annotations

import numpy as np

SCORE_RTOL = 1e-3
SCORE_ATOL = 1e-9
TIE_GAP = 1e-5


def score_errors(gpu: np.ndarray, ref: np.ndarray):
    """(ok, max relative error, count of violations)."""
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    err = np.abs(gpu - ref)
    bound = SCORE_RTOL * np.abs(ref) + SCORE_ATOL
    bad = int(np.count_nonzero(~(err <= bound)))
    rel = float(np.max(err / np.maximum(np.abs(ref), 1e-30))) if ref.size else 0.0
    return bad == 0, rel, bad


def index_swaps(gpu_idx: np.ndarray, ref_idx: np.ndarray, ref_scores: np.ndarray, L: int, w: int):
    """Check one KV head's retained set; w is the number of tokens at the end
    kept by rule (the window), 0 when every token is ranked. Returns (ok,
    swap count, message)."""
    gpu_idx = np.asarray(gpu_idx, dtype=np.int64)
    ref_idx = np.asarray(ref_idx, dtype=np.int64)
    if gpu_idx.shape != ref_idx.shape:
        return False, -1, "shape %s vs %s" % (gpu_idx.shape, ref_idx.shape)
    n = ref_idx.size
    if n >= L:
        ok = np.array_equal(gpu_idx, ref_idx)
        return ok, 0, "" if ok else "keep-all differs"
    if not np.array_equal(gpu_idx[n - w:], np.arange(L - w, L)):
        return False, -1, "window positions differ"
    g, r = gpu_idx[: n - w], ref_idx[: n - w]
    if np.any(np.diff(g) <= 0):
        return False, -1, "gpu indices not strictly ascending"
    if g.size and (g[0] < 0 or g[-1] >= L - w):
        return False, -1, "gpu index out of the prefix"
    d1 = np.setdiff1d(g, r)
    d2 = np.setdiff1d(r, g)
    if d1.size != d2.size:
        return False, -1, "swap counts differ"
    if d1.size == 0:
        return True, 0, ""
    t = np.min(ref_scores[r]) if r.size else 0.0
    gaps = np.abs(ref_scores[np.concatenate([d1, d2])] - t)
    ok = bool(np.all(gaps < TIE_GAP))
    return ok, int(d1.size), "" if ok else "swap with oracle gap %.3g" % gaps.max()


def topn_reference(scores: np.ndarray, n_keep: int) -> np.ndarray:
    """Top n_keep by (score desc, index asc), returned ascending (numpy lexsort)."""
    order = np.lexsort((np.arange(scores.size), -scores))
    return np.sort(order[:n_keep])
