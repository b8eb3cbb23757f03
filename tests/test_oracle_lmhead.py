"""Pins of the oracle's LM head and per-position statistics (kappa, x_hat, entropy).

kappa = max_v p(v) (Eq. app-confidence), x_hat = argmax_v p(v) (Alg. 5) and the
Shannon entropy H = -sum p ln p (Sec. 5.1, before normalisation by ln|V|) are pinned by
closed forms, bounds, special cases and a streaming re-derivation."""
import math

import numpy as np
import pytest

from oracle import confidence_stats, lmhead_confidence, lmhead_logits


def test_probabilities_sum_to_one_and_kappa_is_max_prob():
    rng = np.random.default_rng(0)
    z = rng.standard_normal((5, 3000)) * 3
    st = confidence_stats(z)
    e = np.exp(z - z.max(1, keepdims=True))
    p = e / e.sum(1, keepdims=True)
    np.testing.assert_allclose(p.sum(1), 1.0, atol=1e-12)
    np.testing.assert_allclose(st["conf"], p.max(1), rtol=1e-13)


@pytest.mark.parametrize("V", [1, 2, 7, 2048, 126464])
def test_constant_logits(V):
    st = confidence_stats(np.full((2, V), 3.25))
    np.testing.assert_allclose(st["entropy"], math.log(V), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(st["conf"], 1.0 / V, rtol=1e-12)
    assert (st["argmax"] == 0).all()


@pytest.mark.parametrize("j", [0, 1, 999])
def test_one_hot_logits(j):
    z = np.zeros((1, 1000)); z[0, j] = 1000.0
    st = confidence_stats(z)
    assert st["entropy"][0] < 1e-12
    assert st["conf"][0] == 1.0
    assert st["argmax"][0] == j
    assert st["max_logit"][0] == 1000.0


@pytest.mark.parametrize("V,k,a", [(10, 1, 2.0), (2048, 3, 5.0), (126464, 17, 9.5), (50, 49, 0.3)])
def test_two_level_closed_form(V, k, a):
    rng = np.random.default_rng(V + k)
    idx = np.sort(rng.choice(V, size=k, replace=False))
    z = np.zeros((1, V)); z[0, idx] = a
    Z = k * math.exp(a) + V - k
    st = confidence_stats(z)
    np.testing.assert_allclose(st["entropy"][0], math.log(Z) - k * a * math.exp(a) / Z, rtol=1e-11)
    np.testing.assert_allclose(st["conf"][0], math.exp(a) / Z, rtol=1e-12)
    assert st["argmax"][0] == idx[0]          # lowest id among the tied maxima


def test_argmax_ties_take_lowest_id():
    z = np.array([[1.0, 5.0, 2.0, 5.0, 5.0], [7.0, 7.0, 7.0, 7.0, 7.0], [0.0, -1.0, 0.0, 3.0, 3.0]])
    np.testing.assert_array_equal(confidence_stats(z)["argmax"], [1, 0, 3])


def test_entropy_bounds():
    rng = np.random.default_rng(1)
    for scale in (0.01, 1.0, 10.0, 100.0):
        z = rng.standard_normal((20, 500)) * scale
        st = confidence_stats(z)
        assert (st["entropy"] >= -np.log(st["conf"]) - 1e-12).all()   # min-entropy <= Shannon
        assert (st["entropy"] <= math.log(500) + 1e-12).all()
        assert (st["entropy"] >= 0).all()


def test_gaussian_logits_entropy_sanity():
    # iid N(0, 1) logits over a large vocabulary: H ~ ln V - sigma^2 / 2.
    rng = np.random.default_rng(2)
    V = 200000
    st = confidence_stats(rng.standard_normal((4, V)))
    np.testing.assert_allclose(st["entropy"], math.log(V) - 0.5, atol=0.02)


def test_streaming_identity_matches_two_pass():
    # A chunked running (m, s, t) with s = sum e^(z-m), t = sum e^(z-m)(z-m), merged in fixed
    # order, gives H = ln s - t/s and kappa = 1/s.  Derived here in scalar steps, independently
    # of the two-pass oracle.
    rng = np.random.default_rng(3)
    z = np.concatenate([rng.standard_normal(3000) * 4, [40.0], rng.standard_normal(1000)])
    m, s, t = -math.inf, 0.0, 0.0
    for c0 in range(0, z.size, 256):
        ch = z[c0:c0 + 256]
        mc = max(ch)
        sc = sum(math.exp(x - mc) for x in ch)
        tc = sum(math.exp(x - mc) * (x - mc) for x in ch)
        if mc > m:
            if m != -math.inf:
                f = math.exp(m - mc)
                t = f * (t + s * (m - mc))
                s = f * s
            m = mc
        else:
            f = math.exp(mc - m)
            tc = f * (tc + sc * (mc - m))
            sc = f * sc
        s += sc
        t += tc
    st = confidence_stats(z[None, :])
    np.testing.assert_allclose(math.log(s) - t / s, st["entropy"][0], rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(1.0 / s, st["conf"][0], rtol=1e-12)


def test_logits_orientation_and_values():
    # W rows [I_d; -I_d; 2*e_0; 0] give z = [h, -h, 2 h_0, 0]: pins z = W h (not W^T h).
    d = 6
    W = np.concatenate([np.eye(d), -np.eye(d), 2 * np.eye(d)[:1], np.zeros((3, d))])
    h = np.arange(1.0, d + 1)[None, :] * np.array([[1.0], [-0.5]])
    z = lmhead_logits(h, W)
    assert z.shape == (2, 2 * d + 4)
    np.testing.assert_array_equal(z[:, :d], h)
    np.testing.assert_array_equal(z[:, d:2 * d], -h)
    np.testing.assert_array_equal(z[:, 2 * d], 2 * h[:, 0])
    np.testing.assert_array_equal(z[:, 2 * d + 1:], 0.0)


def test_chunked_lmhead_equals_plain_definition():
    rng = np.random.default_rng(4)
    h = rng.standard_normal((37, 64)).astype(np.float32)
    W = rng.standard_normal((5000, 64)).astype(np.float32)
    a = lmhead_confidence(h, W, v_chunk=999, row_chunk=8)
    z = np.zeros((37, 5000))
    for i in range(37):                       # plain dot products, row by row
        z[i] = [float(np.dot(W[v].astype(np.float64), h[i].astype(np.float64))) for v in range(5000)]
    b = confidence_stats(z)
    np.testing.assert_array_equal(a["argmax"], b["argmax"])
    for k in ("conf", "entropy", "max_logit"):
        np.testing.assert_allclose(a[k], b[k], rtol=1e-12, atol=1e-12)
    rows = np.array([36, 0, 5])
    c = lmhead_confidence(h, W, rows=rows)
    np.testing.assert_array_equal(c["argmax"], b["argmax"][rows])
