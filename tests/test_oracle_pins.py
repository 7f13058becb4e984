"""Pins of the fp64 oracle against what the paper and the mathematics fix.

The paper (CompressKV, arXiv 2508.02401) prints no worked numeric example of
its token selection, so the oracle is pinned by:
  * hand-worked exact examples (rational arithmetic, derivations below);
  * closed forms (constant keys);
  * invariants (softmax rows sum to 1, window sums total w, pooling bounds,
    top-N count/order/ties);
  * library routines the definitions reduce to (scipy softmax, numpy matmul,
    torch avg/max pooling, numpy lexsort, numpy fancy indexing);
  * brute force on tiny inputs (exhaustive subset search for the top-N).
Every oracle function is covered; a plausible slip (dropped term, wrong sign
or index, transposed operand, off-by-one mask, mean vs sum, pool order)
fails at least one test here.
"""
import itertools
import json
import math
import os
from fractions import Fraction as F

import numpy as np
import pytest
import scipy.special
import torch

import oracle

LN2 = math.log(2.0)

# ---------------------------------------------------------------------------
# Hand-worked example (my own construction, exact in rationals); the values
# and their derivation are in tests/golden/hand_example.json.
# ---------------------------------------------------------------------------
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _frac(text):
    """'a/b+c/d' -> exact Fraction."""
    return sum((F(t) for t in text.split("+")), F(0))


HAND = _golden("hand_example.json")
HW_K = np.array(HAND["K"], dtype=np.float64)[:, None]
HW_Q = np.array([[[sg * LN2]] * HAND["window"] for sg in HAND["q_sign"]])  # [head, row, d]
HW_S0 = [_frac(t) for t in HAND["window_sums"]["head0"]]
HW_S1 = [_frac(t) for t in HAND["window_sums"]["head1"]]
POOLS = {"avg": oracle.POOL_AVG, "max": oracle.POOL_MAX}


def _close(x, fr, rel=1e-12):
    return abs(x - float(fr)) <= rel * abs(float(fr)) + 1e-15


def test_hand_example_window_sums_exact():
    S = oracle.window_sums(HW_Q, HW_K, 1.0)
    assert S.shape == (2, 6)
    for j in range(6):
        assert _close(S[0, j], HW_S0[j]), (j, S[0, j], HW_S0[j])
        assert _close(S[1, j], HW_S1[j]), (j, S[1, j], HW_S1[j])
    assert sum(HW_S0) == 2 and sum(HW_S1) == 2


def test_hand_example_head1_prefix_values():
    assert HW_S1[:4] == [_frac(t) for t in HAND["head1_prefix_reduced"]]


@pytest.mark.parametrize("case", HAND["selection"], ids=lambda c: c["why"][:40])
def test_hand_example_selection(case):
    mask = case["mask"]
    scores, idx, _ = oracle.select_group(HW_Q[mask], HW_K, HAND["window"], 1.0, POOLS[case["pool"]],
                                         case["kp"], case["budget"])
    assert idx.tolist() == case["idx"]
    for j in range(4):
        expect = _frac(case["scores"][j])
        assert _close(scores[j], expect), (j, scores[j], expect)


def test_hand_example_mean_then_pool_differs():
    # pinning reading R6: the mean-then-pool order would give these scores instead
    mean = [(a + b) / 2 for a, b in zip(HW_S0[:4], HW_S1[:4])]
    mtp = [max(mean[max(0, j - 1):j + 2]) for j in range(4)]
    assert mtp == [_frac(t) for t in HAND["mean_then_pool_max3"]]
    scores, _, _ = oracle.select_group(HW_Q, HW_K, 2, 1.0, oracle.POOL_MAX, 3, 4)
    assert not _close(scores[0], mtp[0], rel=1e-3)


# ---------------------------------------------------------------------------
# Keep-window flag off: the whole prompt competes for the budget.
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("case", HAND["selection_no_window"]["cases"], ids=lambda c: c["why"][:40])
def test_hand_example_selection_no_window(case):
    mask = case["mask"]
    scores, idx = oracle.select_group_all(HW_Q[mask], HW_K, HAND["window"], 1.0,
                                          POOLS[case["pool"]], case["kp"], case["budget"])
    assert idx.tolist() == case["idx"]
    assert scores.shape == (6,)
    for j in range(6):
        expect = _frac(case["scores"][j])
        assert _close(scores[j], expect), (j, scores[j], expect)


@pytest.mark.parametrize("seed", range(30))
def test_select_tokens_all_brute_force(seed):
    # every subset of size B of a tiny prompt with many tied scores: exactly
    # one of them has every kept token ranked above every dropped one (score
    # descending, then lower index), and it is the oracle's
    from itertools import combinations
    rng = np.random.default_rng(300 + seed)
    L = int(rng.integers(1, 9))
    a = rng.integers(0, 4, size=L).astype(np.float64) / 4.0
    for B in range(1, L + 2):
        idx = oracle.select_tokens_all(a, L, B).tolist()
        if B >= L:
            assert idx == list(range(L))
            continue
        good = []
        for T in combinations(range(L), B):
            drop = [u for u in range(L) if u not in T]
            if all(a[t] > a[u] or (a[t] == a[u] and t < u) for t in T for u in drop):
                good.append(list(T))
        assert len(good) == 1 and idx == good[0], (a.tolist(), B, idx, good)


def test_select_tokens_all_rejects_empty_budget():
    with pytest.raises(oracle.OracleError):
        oracle.select_tokens_all(np.ones(5), 5, 0)


@pytest.mark.parametrize("pool,kp", [("avg", 5), ("max", 7), ("max", 1)])
def test_select_group_all_agrees_with_prefix_path_away_from_the_window(pool, kp):
    # the prefix columns' scores are the same whether or not the window is
    # kept, except within the pool radius of the prefix's end (where the
    # whole-prompt pooling sees window columns instead of padding); with the
    # window tokens excluded the whole-prompt top-B is a top-(B-w) of the prefix
    rng = np.random.default_rng(kp)
    L, w, d = 90, 6, 8
    q = rng.standard_normal((2, w, d))
    k = rng.standard_normal((L, d))
    s_kw, _, _ = oracle.select_group(q, k, w, 0.3, POOLS[pool], kp, 20)
    s_all, _ = oracle.select_group_all(q, k, w, 0.3, POOLS[pool], kp, 20)
    r = kp // 2
    np.testing.assert_allclose(s_all[:L - w - r], s_kw[:L - w - r], rtol=1e-14, atol=0)
    assert not np.allclose(s_all[L - w - r:L - w], s_kw[L - w - r:], rtol=1e-6) or r == 0


def test_select_layer_shared_all_matches_group_all_for_one_group():
    # a layer of one KV group: the shared selection over its chosen heads is
    # that group's own selection
    rng = np.random.default_rng(12)
    H, w, d, L = 4, 5, 8, 70
    q = rng.standard_normal((H, w, d))
    k = rng.standard_normal((1, L, d))
    mask = np.array([1, 0, 1, 1], np.uint8)
    s_sh, i_sh = oracle.select_layer_shared_all(q, mask, k, w, 0.4, oracle.POOL_MAX, 5, 17)
    s_g, i_g = oracle.select_group_all(q[mask.astype(bool)], k[0], w, 0.4, oracle.POOL_MAX, 5, 17)
    np.testing.assert_allclose(s_sh, s_g, rtol=1e-13)
    assert i_sh.tolist() == i_g.tolist()


# ---------------------------------------------------------------------------
# Attention rows: library softmax, normalisation, scale, operand order.
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_attention_row_matches_scipy_softmax(seed):
    rng = np.random.default_rng(seed)
    d, L = 7, 23
    q = rng.standard_normal(d)
    k = rng.standard_normal((L, d)) * 2.0
    scale = 0.37
    n_vis = 17
    p = oracle.attention_row(q, k, n_vis, scale)
    ref = scipy.special.softmax(scale * (k[:n_vis] @ q))
    np.testing.assert_allclose(p, ref, rtol=1e-13, atol=1e-16)
    assert abs(p.sum() - 1.0) < 1e-13


def test_attention_row_large_logits_stable():
    q = np.array([50.0, -20.0])
    k = np.array([[10.0, 0.0], [9.0, 1.0], [-10.0, 0.0]])
    p = oracle.attention_row(q, k, 3, 1.0)
    ref = scipy.special.softmax(k @ q)
    np.testing.assert_allclose(p, ref, rtol=1e-12)


# ---------------------------------------------------------------------------
# Window sums: library route, invariants, closed form.
# ---------------------------------------------------------------------------
def _window_sums_library(q_sel, k, scale):
    """Attention matrices via numpy matmul and scipy softmax with a causal mask."""
    n_sel, w, d = q_sel.shape
    L = k.shape[0]
    out = np.zeros((n_sel, L))
    pos = np.arange(L)[None, :]
    row_pos = (L - w + np.arange(w))[:, None]
    for h in range(n_sel):
        logits = scale * (q_sel[h] @ k.T)            # [w, L]
        logits = np.where(pos <= row_pos, logits, -np.inf)
        out[h] = scipy.special.softmax(logits, axis=1).sum(axis=0)
    return out


@pytest.mark.parametrize("seed,n_sel,w,d,L", [(3, 1, 1, 4, 9), (4, 2, 3, 5, 11), (5, 3, 4, 8, 40)])
def test_window_sums_library_route(seed, n_sel, w, d, L):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((n_sel, w, d))
    k = rng.standard_normal((L, d))
    scale = 1.0 / math.sqrt(d)
    S = oracle.window_sums(q, k, scale)
    np.testing.assert_allclose(S, _window_sums_library(q, k, scale), rtol=1e-12, atol=1e-15)


@pytest.mark.parametrize("seed", [6, 7])
def test_window_sums_total_mass_is_w(seed):
    rng = np.random.default_rng(seed)
    n_sel, w, d, L = 2, 5, 6, 50
    q = rng.standard_normal((n_sel, w, d)) * 3
    k = rng.standard_normal((L, d))
    S = oracle.window_sums(q, k, 0.5)
    np.testing.assert_allclose(S.sum(axis=1), [w] * n_sel, rtol=1e-13)
    assert np.all(S[:, : L - w].sum(axis=1) <= w + 1e-12)
    assert np.all(S >= 0)
    # the last key is seen only by the last window row
    assert np.all(S[:, L - 1] <= 1 + 1e-15)


# ---------------------------------------------------------------------------
# Window-row log-sum-exp (the softmax normaliser of Eq. 2, natural log).
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("seed,n_sel,w,d,L", [(11, 1, 1, 3, 7), (12, 2, 4, 5, 19), (13, 3, 6, 8, 50)])
def test_window_lse_library_route(seed, n_sel, w, d, L):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((n_sel, w, d)) * 2
    k = rng.standard_normal((L, d))
    scale = 0.61
    lse = oracle.window_lse(q, k, scale)
    for h in range(n_sel):
        for i in range(w):
            n_vis = L - w + i + 1
            ref = scipy.special.logsumexp(scale * (k[:n_vis] @ q[h, i]))
            assert abs(lse[h, i] - ref) <= 1e-12 * max(1.0, abs(ref))


def test_window_lse_hand_example_and_softmax_identity():
    # head 0 of the hand example: exp(s) over keys 0..4 sums to 9 (row 0) and
    # over keys 0..5 to 10 (row 1), so lse = ln 9, ln 10
    lse = oracle.window_lse(HW_Q, HW_K, 1.0)
    assert abs(lse[0, 0] - math.log(9.0)) < 1e-14 and abs(lse[0, 1] - math.log(10.0)) < 1e-14
    # exp(s - lse) is the attention row, whatever the row
    rng = np.random.default_rng(14)
    q = rng.standard_normal((1, 3, 4))
    k = rng.standard_normal((12, 4))
    lse = oracle.window_lse(q, k, 0.8)
    for i in range(3):
        n_vis = 12 - 3 + i + 1
        p = oracle.attention_row(q[0, i], k, n_vis, 0.8)
        np.testing.assert_allclose(np.exp(0.8 * (k[:n_vis] @ q[0, i]) - lse[0, i]), p,
                                   rtol=1e-12, atol=1e-16)


def test_window_lse_constant_keys_closed_form():
    # every visible logit equal to c: lse = c + ln(number of visible keys)
    w, L, d = 4, 13, 3
    q = np.ones((1, w, d))
    k = np.ones((L, d)) * 0.5
    lse = oracle.window_lse(q, k, 2.0)
    for i in range(w):
        assert abs(lse[0, i] - (2.0 * 1.5 + math.log(L - w + i + 1))) < 1e-13


@pytest.mark.parametrize("w,L", [(1, 5), (3, 10), (8, 64)])
def test_window_sums_constant_keys_closed_form(w, L):
    # identical keys give uniform rows: row i spreads 1 over L-w+i+1 keys, so a
    # prefix key collects sum_i 1/(L-w+i+1); window key L-w+t collects the
    # rows i >= t.
    rng = np.random.default_rng(0)
    d = 3
    q = rng.standard_normal((1, w, d))
    k = np.tile(rng.standard_normal((1, d)), (L, 1))
    S = oracle.window_sums(q, k, 1.0)[0]
    prefix = sum(1.0 / (L - w + i + 1) for i in range(w))
    np.testing.assert_allclose(S[: L - w], prefix, rtol=1e-13)
    for t in range(w):
        expect = sum(1.0 / (L - w + i + 1) for i in range(t, w))
        assert abs(S[L - w + t] - expect) < 1e-13


def test_window_sums_scale_and_transpose_sensitivity():
    # a non-symmetric key matrix and a non-trivial scale: the library route
    # with k transposed or the scale dropped must disagree with the oracle
    rng = np.random.default_rng(11)
    q = rng.standard_normal((1, 2, 4))
    k = rng.standard_normal((9, 4))
    S = oracle.window_sums(q, k, 0.3)
    assert np.allclose(S, _window_sums_library(q, k, 0.3), rtol=1e-12)
    assert not np.allclose(S, _window_sums_library(q, k, 1.0), rtol=1e-3)


# ---------------------------------------------------------------------------
# Pooling: library routines, closed forms, bounds.
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("kp", [1, 3, 5, 7, 9])
@pytest.mark.parametrize("n", [1, 2, 6, 31])
def test_pool_matches_torch(kp, n):
    rng = np.random.default_rng(kp * 100 + n)
    x = rng.random(n)
    r = kp // 2
    xt = torch.from_numpy(x).view(1, 1, n)
    avg = torch.nn.functional.avg_pool1d(xt, kp, stride=1, padding=r, count_include_pad=True)
    mx = torch.nn.functional.max_pool1d(xt, kp, stride=1, padding=r)
    np.testing.assert_allclose(oracle.pool(x, kp, oracle.POOL_AVG), avg.view(-1).numpy(), rtol=1e-14)
    np.testing.assert_array_equal(oracle.pool(x, kp, oracle.POOL_MAX), mx.view(-1).numpy())


def test_pool_constant_closed_form():
    c, n, kp = 2.5, 12, 7
    x = np.full(n, c)
    avg = oracle.pool(x, kp, oracle.POOL_AVG)
    mx = oracle.pool(x, kp, oracle.POOL_MAX)
    r = kp // 2
    for j in range(n):
        covered = min(j, r) + min(n - 1 - j, r) + 1
        assert abs(avg[j] - c * covered / kp) < 1e-14
    np.testing.assert_array_equal(mx, x)


def test_pool_bounds_and_mass():
    rng = np.random.default_rng(5)
    x = rng.random(40)
    kp, r = 5, 2
    mx = oracle.pool(x, kp, oracle.POOL_MAX)
    assert np.all(mx >= x)
    avg = oracle.pool(x, kp, oracle.POOL_AVG)
    cover = np.array([min(j, r) + min(39 - j, r) + 1 for j in range(40)])
    assert abs(avg.sum() - (x * cover).sum() / kp) < 1e-12


def test_pool_rejects_even_kernel():
    with pytest.raises(oracle.OracleError):
        oracle.pool(np.ones(4), 4, oracle.POOL_AVG)


# ---------------------------------------------------------------------------
# Top-N: brute force, library sort, invariants.
# ---------------------------------------------------------------------------
def _brute_topn(a, k):
    """Exhaustive: the k-subset with the largest sorted score vector, ties broken
    towards the lexicographically smallest index set."""
    best = None
    for sub in itertools.combinations(range(len(a)), k):
        key = (sorted((a[j] for j in sub), reverse=True), [-j for j in sub])
        if best is None or key > best[0]:
            best = (key, sub)
    return list(best[1]) if best else []


@pytest.mark.parametrize("seed", range(12))
def test_select_tokens_brute_force(seed):
    rng = np.random.default_rng(seed)
    L, w = 10, 2
    a = rng.integers(0, 4, size=L - w).astype(float)  # many exact ties
    for budget in range(w, L + 2):
        idx = oracle.select_tokens(a, L, w, budget).tolist()
        if budget >= L:
            assert idx == list(range(L))
            continue
        k = budget - w
        assert idx == _brute_topn(list(a), k) + list(range(L - w, L))


@pytest.mark.parametrize("seed", range(5))
def test_select_tokens_library_sort_and_invariants(seed):
    rng = np.random.default_rng(100 + seed)
    L, w = 300, 7
    a = np.round(rng.random(L - w), 2)
    budget = 50
    idx = oracle.select_tokens(a, L, w, budget)
    order = np.lexsort((np.arange(L - w), -a))
    ref = np.sort(order[: budget - w])
    np.testing.assert_array_equal(idx[: budget - w], ref)
    assert len(idx) == budget
    assert np.all(np.diff(idx) > 0)
    np.testing.assert_array_equal(idx[budget - w:], np.arange(L - w, L))
    kept = idx[: budget - w]
    evicted = np.setdiff1d(np.arange(L - w), kept)
    assert a[kept].min() >= a[evicted].max()
    t = a[kept].min()
    # at the threshold value, every kept index precedes every evicted one
    tied_out = evicted[a[evicted] == t]
    if tied_out.size:
        assert kept[a[kept] == t].max() < tied_out.min()


def test_select_tokens_rejects_budget_below_window():
    with pytest.raises(oracle.OracleError) as e:
        oracle.select_tokens(np.ones(8), 10, 2, 1)
    assert e.value.code == oracle.EBUDGET


# ---------------------------------------------------------------------------
# Group and layer composition, special cases.
# ---------------------------------------------------------------------------
def test_single_head_single_row_reduces_to_softmax():
    # one head, w = 1, no pooling: the score of prefix key j is the softmax
    # probability of the last prompt position on key j
    rng = np.random.default_rng(21)
    d, L = 5, 30
    q = rng.standard_normal((1, 1, d))
    k = rng.standard_normal((L, d))
    scores, idx, _ = oracle.select_group(q, k, 1, 0.4, oracle.POOL_AVG, 1, 6)
    p = scipy.special.softmax(0.4 * (k @ q[0, 0]))
    np.testing.assert_allclose(scores, p[: L - 1], rtol=1e-13)
    top = np.sort(np.lexsort((np.arange(L - 1), -p[: L - 1]))[:5])
    np.testing.assert_array_equal(idx, list(top) + [L - 1])


def test_group_mean_is_linear_in_heads():
    # avg pooling commutes with the head mean; the group score equals the mean
    # of the single-head scores
    rng = np.random.default_rng(22)
    q = rng.standard_normal((3, 4, 6))
    k = rng.standard_normal((40, 6))
    s_all, _, pooled = oracle.select_group(q, k, 4, 0.5, oracle.POOL_AVG, 5, 10, want_pooled=True)
    singles = [oracle.select_group(q[h:h + 1], k, 4, 0.5, oracle.POOL_AVG, 5, 10)[0] for h in range(3)]
    np.testing.assert_allclose(s_all, np.mean(singles, axis=0), rtol=1e-13)
    np.testing.assert_allclose(pooled.mean(axis=0), s_all, rtol=1e-13)


def test_layer_routes_heads_to_groups():
    rng = np.random.default_rng(23)
    H, n_kv, w, d, L = 6, 2, 3, 4, 25
    q = rng.standard_normal((H, w, d))
    k = rng.standard_normal((n_kv, L, d))
    mask = np.array([0, 1, 1, 1, 0, 0], dtype=np.uint8)  # group 0: {1,2}, group 1: {3}
    scores, idx = oracle.select_layer(q, mask, k, w, 0.5, oracle.POOL_MAX, 3, 9)
    s0, i0, _ = oracle.select_group(q[[1, 2]], k[0], w, 0.5, oracle.POOL_MAX, 3, 9)
    s1, i1, _ = oracle.select_group(q[[3]], k[1], w, 0.5, oracle.POOL_MAX, 3, 9)
    np.testing.assert_array_equal(scores[0], s0)
    np.testing.assert_array_equal(scores[1], s1)
    np.testing.assert_array_equal(idx[0], i0)
    np.testing.assert_array_equal(idx[1], i1)


def test_layer_rejects_group_without_head():
    q = np.zeros((4, 2, 2))
    k = np.zeros((2, 8, 2))
    with pytest.raises(oracle.OracleError) as e:
        oracle.select_layer(q, np.array([1, 1, 0, 0], np.uint8), k, 2, 1.0, 0, 1, 4)
    assert e.value.code == oracle.EMASK


def test_planted_keys_survive():
    # keys aligned with the window queries get much larger scores and are kept
    rng = np.random.default_rng(24)
    d, L, w = 16, 200, 4
    q = rng.standard_normal((1, w, d))
    k = rng.standard_normal((L, d))
    qbar = q[0].mean(axis=0)
    planted = [0, 1, 2, 3, 90, 91, 92]
    for j in planted:
        k[j] += 6.0 * math.sqrt(d) * qbar / (qbar @ qbar)
    _, idx, _ = oracle.select_group(q, k, w, 1 / math.sqrt(d), oracle.POOL_MAX, 1, 20)
    assert set(planted) <= set(idx.tolist())


def test_gather_rows_bitwise():
    rng = np.random.default_rng(25)
    src = rng.integers(0, 65535, size=(30, 8), dtype=np.uint16)
    idx = np.array([0, 5, 7, 29], dtype=np.int32)
    np.testing.assert_array_equal(oracle.gather_rows(src, idx), src[idx])


# ---------------------------------------------------------------------------
# Algorithm 1: hand-worked examples and invariants.
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("case", _golden("algorithm1_examples.json")["cases"],
                         ids=lambda c: str(c["budgets"]))
def test_algorithm1_hand_examples(case):
    B, rc = oracle.allocate_budgets(case["e"], case["total"], case["m"], case["M"])
    assert rc == oracle.OK
    assert B.tolist() == case["budgets"]


@pytest.mark.parametrize("seed", range(40))
def test_algorithm1_invariants(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 40))
    e = rng.dirichlet(np.ones(n) * float(rng.choice([0.1, 1.0, 10.0])))
    per = int(rng.integers(32, 2048))
    total = n * per
    m, M = 32, 3 * per
    B, rc = oracle.allocate_budgets(e, total, m, M)
    assert rc == oracle.OK
    assert B.sum() == total
    assert B.min() >= m and B.max() <= M


def _algorithm1_token_by_token(e, total, m, M):
    """Algorithm 1's gap rule applied literally, one token per step: each
    missing token goes to the largest-error layer below M, each extra token
    leaves the smallest-error layer above m (equal errors: the lower layer)."""
    n = len(e)
    R = total - n * m
    B = [min(M, max(m, m + int(np.rint(x * R)))) for x in e]
    while sum(B) != total:
        short = sum(B) < total
        cand = [i for i in range(n) if (B[i] < M if short else B[i] > m)]
        if not cand:
            return B, False
        key = (lambda i: (-e[i], i)) if short else (lambda i: (e[i], i))
        j = min(cand, key=key)
        B[j] += 1 if short else -1
    return B, True


@pytest.mark.parametrize("seed", range(60))
def test_algorithm1_matches_token_by_token_rule(seed):
    # tight bounds and repeated error values force long fix-ups that cross
    # several layers, in both directions, and infeasible totals
    rng = np.random.default_rng(1000 + seed)
    n = int(rng.integers(1, 12))
    e = rng.choice([0.05, 0.1, 0.2, 0.3], size=n).astype(float)
    e = (e / e.sum()).tolist()
    m = int(rng.integers(0, 6))
    M = m + int(rng.integers(0, 9))
    total = int(rng.integers(max(0, n * m - 3), n * M + 4))
    want, ok = _algorithm1_token_by_token(e, total, m, M)
    B, rc = oracle.allocate_budgets(e, total, m, M)
    assert B.tolist() == want
    assert rc == (oracle.OK if ok else oracle.EBUDGET)


def test_algorithm1_infeasible_reports_shortfall():
    B, rc = oracle.allocate_budgets([0.5, 0.5], 1000, 32, 100)
    assert rc == oracle.EBUDGET and B.tolist() == [100, 100]
    B, rc = oracle.allocate_budgets([0.5, 0.5], 10, 32, 100)
    assert rc == oracle.EBUDGET and B.tolist() == [32, 32]


# ---------------------------------------------------------------------------
# Layer-shared selection (the paper's own variant of Sec. 3.3).
# ---------------------------------------------------------------------------
SHARED = HAND["shared"]


@pytest.mark.parametrize("case", SHARED["cases"], ids=lambda c: c["why"][:40])
def test_shared_hand_example(case):
    k = np.array(SHARED["K"], dtype=np.float64)[:, :, None]          # [n_kv, L, 1]
    q = np.full((2, SHARED["window"], 1), LN2)                        # [H, w, 1]
    scores, idx = oracle.select_layer_shared(q, [1, 1], k, SHARED["window"], 1.0,
                                             POOLS[case["pool"]], case["kp"], case["budget"])
    assert idx.tolist() == case["idx"]
    for j, t in enumerate(case["scores"]):
        assert _close(scores[j], _frac(t)), (j, scores[j], t)


def test_shared_hand_example_differs_from_each_group():
    k = np.array(SHARED["K"], dtype=np.float64)[:, :, None]
    q = np.full((1, 2, 1), LN2)
    per_group = [oracle.select_group(q, k[g], 2, 1.0, oracle.POOL_AVG, 1, 4)[1].tolist()
                 for g in range(2)]
    assert per_group == [[0, 3, 4, 5], [0, 1, 4, 5]]


def _layer_case(seed, H=8, n_kv=2, L=97, w=5, d=6):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((H, w, d)), rng.standard_normal((n_kv, L, d)), w


@pytest.mark.parametrize("seed", range(6))
def test_shared_one_group_reduces_to_group_selection(seed):
    # every chosen head in one group: the shared set is that group's selection
    q, k, w = _layer_case(seed)
    G = q.shape[0] // k.shape[0]
    g = seed % k.shape[0]
    mask = np.zeros(q.shape[0], np.uint8)
    mask[g * G: g * G + 1 + seed % G] = 1
    chosen = np.nonzero(mask)[0]
    s_sh, i_sh = oracle.select_layer_shared(q, mask, k, w, 0.4, oracle.POOL_MAX, 5, 20)
    s_g, i_g, _ = oracle.select_group(q[chosen], k[g], w, 0.4, oracle.POOL_MAX, 5, 20)
    np.testing.assert_allclose(s_sh, s_g, rtol=1e-14, atol=0)
    assert i_sh.tolist() == i_g.tolist()


@pytest.mark.parametrize("seed", range(6))
def test_shared_is_head_weighted_mean_of_group_scores(seed):
    # the mean runs over all chosen heads, so a group with more chosen heads
    # weighs more: shared = sum_g n_g * A_g / sum_g n_g
    q, k, w = _layer_case(seed + 100, H=12, n_kv=3)
    G = 4
    rng = np.random.default_rng(seed)
    mask = np.zeros(12, np.uint8)
    counts = []
    for g in range(3):
        n = int(rng.integers(1, G + 1))
        mask[g * G + rng.choice(G, n, replace=False)] = 1
        counts.append(n)
    s_sh, _ = oracle.select_layer_shared(q, mask, k, w, 0.3, oracle.POOL_AVG, 3, 30)
    s_groups, _ = oracle.select_layer(q, mask, k, w, 0.3, oracle.POOL_AVG, 3, 30)
    expect = sum(n * s_groups[g] for g, n in enumerate(counts)) / sum(counts)
    np.testing.assert_allclose(s_sh, expect, rtol=1e-12, atol=1e-15)
    # and not the plain mean of the group means (unless the counts are equal)
    if len(set(counts)) > 1:
        assert not np.allclose(s_sh, s_groups.mean(axis=0), rtol=1e-6, atol=0)


@pytest.mark.parametrize("seed", range(4))
def test_shared_library_route(seed):
    # per head: dense scipy softmax rows over the visible keys of its own
    # group, window sum, torch max pooling, then the mean over all chosen heads
    q, k, w = _layer_case(seed + 200, H=6, n_kv=3, L=64, w=4, d=5)
    mask = np.array([1, 0, 1, 1, 0, 1], np.uint8)
    G, L, scale, kp = 2, k.shape[1], 0.7, 5
    pooled = []
    for h in np.nonzero(mask)[0]:
        kg = k[h // G]
        S = np.zeros(L)
        for i in range(w):
            vis = L - w + i + 1
            S[:vis] += scipy.special.softmax(scale * (kg[:vis] @ q[h, i]))
        x = torch.from_numpy(S[:L - w])[None, None]
        pooled.append(torch.nn.functional.max_pool1d(x, kp, 1, kp // 2)[0, 0].numpy())
    expect = np.mean(pooled, axis=0)
    s_sh, idx = oracle.select_layer_shared(q, mask, k, w, scale, oracle.POOL_MAX, kp, 12)
    np.testing.assert_allclose(s_sh, expect, rtol=1e-12, atol=1e-15)
    order = np.lexsort((np.arange(L - w), -expect))[:12 - w]
    assert idx.tolist() == sorted(order.tolist()) + list(range(L - w, L))


def test_shared_rejects_empty_mask():
    q, k, w = _layer_case(7)
    with pytest.raises(oracle.OracleError):
        oracle.select_layer_shared(q, np.zeros(q.shape[0], np.uint8), k, w, 0.3,
                                   oracle.POOL_AVG, 3, 20)


# ---- StreamingLLM-style retention (Sec. 2: first and last tokens) ----------
@pytest.mark.parametrize("L,budget,n_sink", [(10, 4, 2), (10, 4, 0), (10, 4, 9), (7, 20, 4),
                                             (1, 1, 1), (1000, 128, 4), (33, 33, 3)])
def test_streaming_indices_brute_force(L, budget, n_sink):
    # membership decided token by token: a token is kept when fewer than
    # n_sink tokens precede it, or when it is among the last (kept - sinks)
    got = oracle.streaming_indices(L, budget, n_sink)
    n_ret = min(budget, L)
    kept = []
    sinks_taken = 0
    for j in range(L):
        if sinks_taken < n_sink and len(kept) < n_ret:
            kept.append(j)
            sinks_taken += 1
    n_recent = n_ret - len(kept)
    recent = list(range(L))[::-1][:n_recent][::-1]
    assert set(kept).isdisjoint(recent)
    np.testing.assert_array_equal(got, np.array(sorted(kept + recent), dtype=np.int32))


def test_streaming_indices_special_cases():
    # budget >= L keeps the whole prompt; no sinks keeps the last B tokens
    # (the window-only cache); sinks >= budget keeps the first B tokens
    np.testing.assert_array_equal(oracle.streaming_indices(9, 50, 4), np.arange(9))
    np.testing.assert_array_equal(oracle.streaming_indices(100, 8, 0), np.arange(92, 100))
    np.testing.assert_array_equal(oracle.streaming_indices(100, 8, 30), np.arange(8))
    idx = oracle.streaming_indices(5000, 256, 4)
    assert idx.dtype == np.int32 and len(idx) == 256 and np.all(np.diff(idx) > 0)
    assert list(idx[:5]) == [0, 1, 2, 3, 5000 - 252]
