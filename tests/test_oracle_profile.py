"""Pins of the oracle's compression-error profile (paper Sec. 3.4, Eq. 6-8;
Appendix B.1, Eq. 9-12): decode attention, the per-layer error of the
W_O-projected output with the full and the compressed cache, and the
normalisation over profiling sets that feeds Algorithm 1."""
import json
import os
from fractions import Fraction as F

import numpy as np
import pytest
import scipy.special

import oracle

GOLDEN = json.load(open(os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden",
                                     "error_profile.json")))


def _decode_ref(q, k, v, scale):
    """Library route: scipy softmax rows and a numpy matrix product per head."""
    H, d = q.shape
    G = H // k.shape[0]
    out = np.empty((H, d))
    for h in range(H):
        p = scipy.special.softmax(scale * (k[h // G] @ q[h]))
        out[h] = p @ v[h // G]
    return out


@pytest.mark.parametrize("seed", range(5))
def test_decode_attention_library_route(seed):
    rng = np.random.default_rng(seed)
    H, n_kv, n, d = 8, 2, 50 + seed, 16
    q, k, v = rng.standard_normal((H, d)), rng.standard_normal((n_kv, n, d)), rng.standard_normal((n_kv, n, d))
    np.testing.assert_allclose(oracle.decode_attention(q, k, v, 0.3), _decode_ref(q, k, v, 0.3),
                               rtol=1e-12, atol=1e-14)


def test_decode_attention_special_cases():
    rng = np.random.default_rng(7)
    q = rng.standard_normal((4, 8))
    v = rng.standard_normal((2, 5, 8))
    # constant keys: uniform weights, the mean of the group's values
    out = oracle.decode_attention(q, np.ones((2, 5, 8)), v, 0.5)
    np.testing.assert_allclose(out[:2], np.repeat(v[0].mean(0)[None], 2, 0), rtol=1e-13)
    np.testing.assert_allclose(out[2:], np.repeat(v[1].mean(0)[None], 2, 0), rtol=1e-13)
    # one key: its value
    out = oracle.decode_attention(q, rng.standard_normal((2, 1, 8)), v[:, :1], 0.5)
    np.testing.assert_allclose(out[3], v[1, 0], rtol=1e-15)
    # heads follow their own group: swapping the groups' caches swaps the outputs
    k = rng.standard_normal((2, 5, 8))
    a = oracle.decode_attention(q, k, v, 0.5)
    b = oracle.decode_attention(q, k[::-1].copy(), v[::-1].copy(), 0.5)
    assert not np.allclose(a, b)
    np.testing.assert_allclose(_decode_ref(q, k, v, 0.5), a, rtol=1e-12)


def test_layer_error_hand_example():
    g = GOLDEN["layer_error"]
    e, ratio = oracle.layer_error(g["q_dec"], g["k"], g["v"], g["k_comp"], g["v_comp"],
                                  g["w_o"], 1.0, g["eps"])
    term = g["ratio_num"] / (g["ratio_den"] + g["eps"])
    np.testing.assert_allclose(ratio, [term] * g["steps"], rtol=1e-15)
    assert abs(e - g["steps"] * term) < 1e-15


def _profile_case(seed, H=8, n_kv=2, L=60, n_c=12, d=8, T=5, D=24):
    rng = np.random.default_rng(seed)
    q = rng.standard_normal((T, H, d))
    k, v = rng.standard_normal((n_kv, L, d)), rng.standard_normal((n_kv, L, d))
    idx = np.sort(rng.choice(L, n_c, replace=False))
    w_o = rng.standard_normal((D, H * d)) / np.sqrt(H * d)
    return q, k, v, k[:, idx], v[:, idx], w_o


@pytest.mark.parametrize("seed", range(5))
def test_layer_error_library_route(seed):
    q, k, v, kc, vc, w_o = _profile_case(seed)
    terms = []
    for t in range(q.shape[0]):
        af = _decode_ref(q[t], k, v, 0.35).reshape(-1)
        ac = _decode_ref(q[t], kc, vc, 0.35).reshape(-1)
        terms.append(np.linalg.norm(w_o @ (ac - af)) / (np.linalg.norm(w_o @ af) + 1e-6))
    e, ratio = oracle.layer_error(q, k, v, kc, vc, w_o, 0.35)
    np.testing.assert_allclose(ratio, terms, rtol=1e-11)
    np.testing.assert_allclose(e, sum(terms), rtol=1e-11)


def test_layer_error_invariants():
    q, k, v, kc, vc, w_o = _profile_case(11)
    # the full cache "compressed" to itself has no error
    e0, _ = oracle.layer_error(q, k, v, k, v, w_o, 0.35)
    assert e0 == 0.0
    # a scaled W_O leaves every ratio unchanged up to eps
    e1, r1 = oracle.layer_error(q, k, v, kc, vc, w_o, 0.35, eps=0.0)
    e2, r2 = oracle.layer_error(q, k, v, kc, vc, 7.5 * w_o, 0.35, eps=0.0)
    np.testing.assert_allclose(r1, r2, rtol=1e-12)
    # a real compression has a positive error
    assert e1 > 0


@pytest.mark.parametrize("case", GOLDEN["normalize"], ids=lambda c: str(c["e"]))
def test_normalize_errors_hand_examples(case):
    out = oracle.normalize_errors(case["e"])
    np.testing.assert_allclose(out, [float(F(x)) for x in case["e_tilde"]], rtol=1e-15)


def test_normalize_errors_invariants():
    rng = np.random.default_rng(5)
    e = rng.random((4, 32))
    out = oracle.normalize_errors(e)
    assert abs(out.sum() - 1.0) < 1e-14 and (out > 0).all()
    # each set is normalised first, so scaling one set changes nothing
    e2 = e.copy()
    e2[2] *= 1000.0
    np.testing.assert_allclose(oracle.normalize_errors(e2), out, rtol=1e-13)
    # and it is not the normalised plain sum over sets
    assert not np.allclose(oracle.normalize_errors(e2), e2.sum(0) / e2.sum(), rtol=1e-3)
    with pytest.raises(oracle.OracleError):
        oracle.normalize_errors(np.zeros((1, 3)))
