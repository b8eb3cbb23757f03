"""Pin of the oracle's whole step, oracle.decode_step (the checker of the package smoke test
and the timed CPU baseline).

Its outputs must equal the three parts of a step (Alg. 5, one iteration) composed by hand
from implementations written separately from the oracle: the scalar attention loop of
test_oracle_attention, the two-pass statistics of explicit scalar dot products, and Alg. 5's
block commit of test_oracle_unmask.  Prefix and block lengths differ per sequence and one block
is empty, so a wiring slip (offset arrays swapped, statistics of the wrong rows, tau of the
wrong block) changes the result."""
import math

import numpy as np
import pytest

import oracle
from tests.test_oracle_attention import brute_force
from tests.test_oracle_unmask import alg5_block


def scalar_stats(h_row, w):
    """kappa, entropy (nats), first argmax and max logit of softmax(W h) by scalar loops."""
    V, d = w.shape
    z = [sum(float(w[v, k]) * float(h_row[k]) for k in range(d)) for v in range(V)]
    m = max(z)
    x_hat = z.index(m)
    e = [math.exp(x - m) for x in z]
    tot = sum(e)
    p = [x / tot for x in e]
    H = -sum(pi * math.log(pi) for pi in p if pi > 0)
    return max(p), H, x_hat, m


def small_step(seed):
    rng = np.random.default_rng(seed)
    lens, pres = [3, 0, 5, 2], [4, 2, 0, 6]
    hq, hkv, D, d, V = 4, 2, 8, 16, 40
    cu_b = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    cu_p = np.concatenate([[0], np.cumsum(pres)]).astype(np.int32)
    T, S = int(cu_b[-1]), int(cu_p[-1])
    f32 = lambda *s: rng.standard_normal(s).astype(np.float32)
    w = f32(V, d) / 4
    h = f32(T, d) * 2
    h[1] = 6 * w[7] / np.linalg.norm(w[7])      # a confident row
    masked = (rng.random(T) < 0.7).astype(np.uint8)
    masked[cu_b[2]:cu_b[3]] = 1
    tokens = np.where(masked == 1, -1, rng.integers(0, V, T)).astype(np.int32)
    tau = np.array([0.3, 0.9, 0.05, 0.99], np.float32)
    return dict(q=f32(T, hq, D), k_blk=f32(T, hkv, D), v_blk=f32(T, hkv, D), k_pre=f32(S, hkv, D),
                v_pre=f32(S, hkv, D), cu_block=cu_b, cu_prefix=cu_p, hq=hq, hkv=hkv, h=h, w=w,
                masked=masked, tokens=tokens, tau=tau)


@pytest.mark.parametrize("seed", [1, 2, 3])
def test_decode_step_equals_parts_composed_by_hand(seed):
    a = small_step(seed)
    got = oracle.decode_step(**a)
    cu_b = a["cu_block"]
    want_attn = brute_force(a["q"], a["k_blk"], a["v_blk"], a["k_pre"], a["v_pre"], cu_b,
                            a["cu_prefix"], a["hq"], a["hkv"])
    np.testing.assert_allclose(got["attn"], want_attn, rtol=1e-12, atol=1e-12)
    T = a["h"].shape[0]
    stats = [scalar_stats(a["h"][i], a["w"]) for i in range(T)]
    np.testing.assert_allclose(got["conf"], [s[0] for s in stats], rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(got["entropy"], [s[1] for s in stats], rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(got["argmax"], [s[2] for s in stats])
    np.testing.assert_allclose(got["max_logit"], [s[3] for s in stats], rtol=1e-12, atol=1e-12)
    commits = 0
    for b in range(len(cu_b) - 1):
        sl = slice(cu_b[b], cu_b[b + 1])
        conf = [stats[i][0] for i in range(cu_b[b], cu_b[b + 1])]
        A, x, m, res = alg5_block(conf, a["masked"][sl].tolist(),
                                  got["argmax"][sl].tolist(), a["tokens"][sl].tolist(),
                                  a["tau"][b])
        un = np.zeros(cu_b[b + 1] - cu_b[b], np.uint8)
        un[A] = 1
        np.testing.assert_array_equal(got["unmask"][sl], un)
        np.testing.assert_array_equal(got["tokens"][sl], x)
        np.testing.assert_array_equal(got["masked"][sl], m)
        assert got["n_commit"][b] == len(A) and got["resolved"][b] == res
        commits += len(A)
    assert commits > 0


def test_decode_step_wiring_slip_is_caught():
    # the same step with the offset arrays swapped must not pass for the real one
    a = small_step(4)
    good = oracle.decode_step(**a)
    bad = dict(a, cu_block=a["cu_prefix"], cu_prefix=a["cu_block"])
    try:
        swapped = oracle.decode_step(**bad)
    except (IndexError, ValueError):
        return
    assert not np.allclose(swapped["attn"], good["attn"])
