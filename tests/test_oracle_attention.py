"""Pins of the oracle's block attention (bidirectional, prefix KV cache, GQA).

Pinned against a scalar brute-force loop on tiny ragged shapes, and against closed
forms that a dropped term, a wrong head mapping, a wrong scale or a mixed-up
sequence offset would break."""
import math

import numpy as np
import pytest

from oracle import block_attention


def brute_force(q, k_blk, v_blk, k_pre, v_pre, cu_block, cu_prefix, hq, hkv, bonus=None):
    """Scalar loops.  bonus[(b, j)] adds a constant to the score of key j of sequence b."""
    T, _, D = q.shape
    group = hq // hkv
    out = np.zeros((T, hq, D))
    for b in range(len(cu_block) - 1):
        keys = [("p", j) for j in range(cu_prefix[b], cu_prefix[b + 1])] + \
               [("b", j) for j in range(cu_block[b], cu_block[b + 1])]
        for i in range(cu_block[b], cu_block[b + 1]):
            for h in range(hq):
                g = h // group
                scores = []
                for jj, (seg, j) in enumerate(keys):
                    kv = k_pre[j, g] if seg == "p" else k_blk[j, g]
                    s = sum(float(q[i, h, d]) * float(kv[d]) for d in range(D)) / math.sqrt(D)
                    if bonus is not None:
                        s += bonus.get((b, jj), 0.0)
                    scores.append(s)
                mx = max(scores)
                ws = [math.exp(s - mx) for s in scores]
                tot = sum(ws)
                for d in range(D):
                    acc = 0.0
                    for (seg, j), wgt in zip(keys, ws):
                        vv = v_pre[j, g] if seg == "p" else v_blk[j, g]
                        acc += wgt * float(vv[d])
                    out[i, h, d] = acc / tot
    return out


def rand_case(rng, B, hq, hkv, D, max_len=5, max_pre=5, min_len=0):
    lens = rng.integers(min_len, max_len + 1, B)
    pres = rng.integers(0, max_pre + 1, B)
    lens[0] = max(lens[0], 1)
    cu_b = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    cu_p = np.concatenate([[0], np.cumsum(pres)]).astype(np.int32)
    T, S = int(cu_b[-1]), int(cu_p[-1])
    return dict(q=rng.standard_normal((T, hq, D)), k_blk=rng.standard_normal((T, hkv, D)),
                v_blk=rng.standard_normal((T, hkv, D)), k_pre=rng.standard_normal((S, hkv, D)),
                v_pre=rng.standard_normal((S, hkv, D)), cu_block=cu_b, cu_prefix=cu_p,
                hq=hq, hkv=hkv)


@pytest.mark.parametrize("hq,hkv", [(1, 1), (2, 1), (4, 2), (4, 4), (4, 1)])
def test_matches_brute_force(hq, hkv):
    rng = np.random.default_rng(hq * 10 + hkv)
    for _ in range(3):
        c = rand_case(rng, B=int(rng.integers(1, 4)), hq=hq, hkv=hkv, D=int(rng.choice([4, 8])))
        np.testing.assert_allclose(block_attention(**c), brute_force(**c), rtol=1e-12, atol=1e-12)


def test_single_key_returns_its_value():
    rng = np.random.default_rng(0)
    c = rand_case(rng, B=1, hq=2, hkv=2, D=8, max_len=1, max_pre=0, min_len=1)
    c["cu_prefix"] = np.array([0, 0], np.int32)
    c["k_pre"] = c["k_pre"][:0]
    c["v_pre"] = c["v_pre"][:0]
    o = block_attention(**c)
    np.testing.assert_allclose(o[0], c["v_blk"][0], rtol=0, atol=1e-15)


def test_zero_query_gives_mean_of_values():
    rng = np.random.default_rng(1)
    c = rand_case(rng, B=2, hq=2, hkv=1, D=8, max_len=4, max_pre=3, min_len=1)
    c["q"][:] = 0.0
    o = block_attention(**c)
    for b in range(2):
        vals = np.concatenate([c["v_pre"][c["cu_prefix"][b]:c["cu_prefix"][b + 1], 0],
                               c["v_blk"][c["cu_block"][b]:c["cu_block"][b + 1], 0]])
        for i in range(c["cu_block"][b], c["cu_block"][b + 1]):
            np.testing.assert_allclose(o[i, 0], vals.mean(axis=0), atol=1e-14)
            np.testing.assert_allclose(o[i, 1], vals.mean(axis=0), atol=1e-14)


def test_gqa_head_mapping_is_contiguous_groups():
    # Each key/value head g carries constant values c_g: query head h must return c_{h // 4}.
    rng = np.random.default_rng(2)
    c = rand_case(rng, B=2, hq=8, hkv=2, D=4, max_len=3, max_pre=3, min_len=1)
    for g in range(2):
        c["v_pre"][:, g, :] = 10.0 * (g + 1)
        c["v_blk"][:, g, :] = 10.0 * (g + 1)
    o = block_attention(**c)
    for h in range(8):
        np.testing.assert_allclose(o[:, h, :], 10.0 * (h // 4 + 1), atol=1e-12)


def test_two_keys_closed_form_pins_scale():
    # q.k1 - q.k2 = delta  =>  O = sigmoid(delta / sqrt(D)) v1 + (1 - sigmoid) v2.
    D = 16
    q = np.zeros((1, 1, D)); q[0, 0, 0] = 3.0
    k1 = np.zeros(D); k1[0] = 1.0          # q.k1 = 3
    k2 = np.zeros(D); k2[0] = -0.5         # q.k2 = -1.5
    v1 = np.arange(D, dtype=float); v2 = -np.ones(D)
    o = block_attention(q, k1[None, None], v1[None, None], k2[None, None], v2[None, None],
                        np.array([0, 1]), np.array([0, 1]), 1, 1)
    s = 1.0 / (1.0 + math.exp(-(4.5 / math.sqrt(D))))
    np.testing.assert_allclose(o[0, 0], s * v1 + (1 - s) * v2, rtol=1e-13)


def test_key_order_and_segment_split_do_not_matter():
    # The prefix and the block form one unordered key set.
    rng = np.random.default_rng(4)
    D, hq = 8, 2
    n_keys = 7
    K = rng.standard_normal((n_keys, 1, D)); Vv = rng.standard_normal((n_keys, 1, D))
    q = rng.standard_normal((3, hq, D))
    # split A: prefix = keys 0..3, block keys = 4..6 ; split B: permuted, prefix = 4 keys
    perm = rng.permutation(n_keys)
    oA = block_attention(q, K[4:7], Vv[4:7], K[:4], Vv[:4], np.array([0, 3]), np.array([0, 4]), hq, 1)
    Kp, Vp = K[perm], Vv[perm]
    # block keys must still be 3 rows (one per query row); put any 3 of the permuted keys there
    oB = block_attention(q, Kp[:3], Vp[:3], Kp[3:], Vp[3:], np.array([0, 3]), np.array([0, 4]), hq, 1)
    np.testing.assert_allclose(oA, oB, rtol=1e-12, atol=1e-13)


def test_sequences_do_not_mix():
    rng = np.random.default_rng(5)
    c = rand_case(rng, B=3, hq=2, hkv=2, D=4, max_len=4, max_pre=4, min_len=1)
    for b in range(3):
        c["v_pre"][c["cu_prefix"][b]:c["cu_prefix"][b + 1]] = float(b + 1)
        c["v_blk"][c["cu_block"][b]:c["cu_block"][b + 1]] = float(b + 1)
    o = block_attention(**c)
    for b in range(3):
        np.testing.assert_allclose(o[c["cu_block"][b]:c["cu_block"][b + 1]], float(b + 1), atol=1e-13)


def test_prefix_keys_participate():
    # A prefix key with a dominant score drives the output to its value.
    D = 8
    q = np.ones((2, 1, D))
    k_blk = np.zeros((2, 1, D)); v_blk = np.zeros((2, 1, D))
    k_pre = np.zeros((3, 1, D)); v_pre = np.zeros((3, 1, D))
    k_pre[1] = 20.0; v_pre[1] = 7.0
    o = block_attention(q, k_blk, v_blk, k_pre, v_pre, np.array([0, 2]), np.array([0, 3]), 1, 1)
    np.testing.assert_allclose(o, 7.0, rtol=1e-12)


def test_duplicate_key_equals_ln2_bonus():
    # Duplicating one (k, v) pair equals one copy whose score is raised by ln 2.
    rng = np.random.default_rng(6)
    c = rand_case(rng, B=1, hq=1, hkv=1, D=4, max_len=3, max_pre=3, min_len=2)
    P = int(c["cu_prefix"][-1])
    if P == 0:
        c["k_pre"] = rng.standard_normal((1, 1, 4)); c["v_pre"] = rng.standard_normal((1, 1, 4))
        c["cu_prefix"] = np.array([0, 1], np.int32); P = 1
    dup = dict(c)
    dup["k_pre"] = np.concatenate([c["k_pre"], c["k_pre"][:1]])
    dup["v_pre"] = np.concatenate([c["v_pre"], c["v_pre"][:1]])
    dup["cu_prefix"] = np.array([0, P + 1], np.int32)
    o_dup = block_attention(**dup)
    o_bonus = brute_force(**c, bonus={(0, 0): math.log(2.0)})
    np.testing.assert_allclose(o_dup, o_bonus, rtol=1e-12, atol=1e-13)


def test_empty_block_leaves_no_rows():
    rng = np.random.default_rng(7)
    c = rand_case(rng, B=3, hq=2, hkv=1, D=4, max_len=3, max_pre=2, min_len=0)
    c2 = dict(c)
    o = block_attention(**c)
    assert o.shape[0] == int(c["cu_block"][-1])
    np.testing.assert_allclose(o, brute_force(**c2), atol=1e-12)
