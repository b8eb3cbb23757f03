"""Pins of the oracle's next-row functions: the top-1/top-2 gap and the LPS features
(Sec. 5.2, Alg. 5), the union accept rule (Alg. 5), the top-m budget commit (Eq.
prelim-update), the LBS post-pass (Sec. 5.1, Alg. 5) and dual-cache attention (Sec. 6.3).

Each is pinned by hand-derived cases (tests/golden/*.txt, each citing its rule), closed forms,
brute force against a second implementation written separately from the paper's steps, and
invariants."""
import itertools
import math
import os

import numpy as np
import pytest

from oracle import (block_attention, confidence_stats, lbs_select, lps_features,
                    unmask_select, unmask_select_lps, unmask_select_topm)

GOLDEN_DIR = os.path.join(os.path.dirname(__file__), "golden")


def _ints(s):
    s = s.strip()
    return [] if s == "-" else [int(x) for x in s.split()]


def _floats(s):
    s = s.strip()
    return [] if s == "-" else [float(x) for x in s.split()]


def _rows(name):
    for line in open(os.path.join(GOLDEN_DIR, name)):
        line = line.strip()
        if line and not line.startswith("#"):
            lhs, rhs = line.split("||")
            yield [x.strip() for x in lhs.split("|")], [x.strip() for x in rhs.split("|")]


# --------------------------------------------------------------------------------------
# top-1 / top-2 gap
# --------------------------------------------------------------------------------------

def test_gap_constant_logits_is_zero():
    st = confidence_stats(np.full((2, 1000), 3.25))
    np.testing.assert_array_equal(st["top2_gap"], 0.0)


def test_gap_one_hot_is_one():
    z = np.zeros((1, 5000))
    z[0, 7] = 1000.0
    assert abs(confidence_stats(z)["top2_gap"][0] - 1.0) < 1e-12


def test_gap_three_level_closed_form():
    V, a, b = 10, 3.0, 1.5
    z = np.zeros((1, V))
    z[0, 4], z[0, 8] = a, b
    Z = math.exp(a) + math.exp(b) + (V - 2)
    assert abs(confidence_stats(z)["top2_gap"][0] - (math.exp(a) - math.exp(b)) / Z) < 1e-14


@pytest.mark.parametrize("k", [2, 3, 7])
def test_gap_shared_maximum_is_zero(k):
    z = np.zeros((1, 50))
    z[0, 10:10 + k] = 4.0
    assert confidence_stats(z)["top2_gap"][0] == 0.0


def test_gap_single_entry_vocabulary():
    st = confidence_stats(np.array([[0.3]]))
    assert st["top2_gap"][0] == 1.0 and st["conf"][0] == 1.0


def test_gap_streaming_form_by_scalar_scan():
    """Delta = (1 - exp(z2 - m)) / s with m, z2 the two largest logits found by a scalar
    left-to-right scan and s = sum exp(z - m): the form the kernels reduce to."""
    rng = np.random.default_rng(11)
    for V in (2, 3, 17, 500):
        z = rng.normal(0, 2, (20, V))
        z[3, 1] = z[3, 0]                                     # a shared maximum
        st = confidence_stats(z)
        for r in range(z.shape[0]):
            m1, m2 = -math.inf, -math.inf
            for x in z[r]:
                if x > m1:
                    m1, m2 = x, m1
                elif x > m2:
                    m2 = x
            s = sum(math.exp(x - m1) for x in z[r])
            assert abs(st["top2_gap"][r] - (1.0 - math.exp(m2 - m1)) / s) < 1e-12


def test_gap_bounds_and_permutation():
    rng = np.random.default_rng(12)
    z = rng.normal(0, 3, (30, 257))
    st = confidence_stats(z)
    assert (st["top2_gap"] >= 0).all() and (st["top2_gap"] <= st["conf"] + 1e-15).all()
    perm = rng.permutation(z.shape[1])
    np.testing.assert_allclose(confidence_stats(z[:, perm])["top2_gap"], st["top2_gap"],
                               rtol=0, atol=1e-14)


# --------------------------------------------------------------------------------------
# LPS features
# --------------------------------------------------------------------------------------

def test_lps_features_hand_derived():
    # two blocks: rows 0..3 (masked 1 0 1 1) and rows 4..5 (masked 0 0); V = 4
    conf = np.array([0.9, 0.5, 0.3, 0.2, 1.0, 0.6])
    ent = np.array([math.log(2), 0.0, math.log(4), 1.0, 0.0, 0.5])
    gap = np.array([0.85, 0.1, 0.0, 0.05, 1.0, 0.3])
    masked = np.array([1, 0, 1, 1, 0, 0], np.uint8)
    r = lps_features(conf, ent, gap, masked, np.array([0, 4, 6]), vocab=4)
    np.testing.assert_allclose(r["mask_ratio"], [0.75, 0.0])
    np.testing.assert_allclose(r["pos"], [0.0, 0.25, 0.5, 0.75, 0.0, 0.5])
    np.testing.assert_allclose(r["feat"][0], [0.9, 0.5, 0.85, 0.75])
    np.testing.assert_allclose(r["feat"][2], [0.3, 1.0, 0.0, 0.75])
    np.testing.assert_allclose(r["feat"][5], [0.6, 0.5 / math.log(4), 0.3, 0.0])


def _golden_positions():
    from fractions import Fraction
    cases = []
    for lhs, rhs in _rows("lps_position_examples.txt"):
        cases.append((lhs[0], _ints(lhs[1]), [Fraction(x) for x in rhs[0].split()]))
    return cases


def test_lps_positions_printed_formula_golden():
    # all hand-derived blocks as one ragged batch, placed at unrelated packed offsets
    cases = _golden_positions()
    lens = [len(c[1]) for c in cases]
    cu = np.concatenate([[0], np.cumsum(lens)])
    seq_pos = np.concatenate([c[1] for c in cases]).astype(np.int32)
    T = int(cu[-1])
    z = np.zeros(T)
    r = lps_features(z, z, z, np.ones(T, np.uint8), cu, vocab=10, seq_pos=seq_pos)
    for b, (name, _, want) in enumerate(cases):
        got = r["pos"][cu[b]:cu[b + 1]]
        np.testing.assert_allclose(got, [float(x) for x in want], rtol=0, atol=1e-15,
                                   err_msg=name)


def test_lps_positions_contiguous_blocks_equal_rank_form():
    # a contiguous block's sequence positions differ from its packed rows by a constant, so the
    # printed formula and the rank form agree there
    rng = np.random.default_rng(14)
    lens = [0, 1, 7, 32, 5]
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    seq_pos = np.concatenate([np.arange(n) + rng.integers(0, 400) for n in lens]).astype(np.int32)
    x = rng.random(T)
    masked = (rng.random(T) < 0.5).astype(np.uint8)
    a = lps_features(x, x, x, masked, cu, vocab=50, seq_pos=seq_pos)
    b = lps_features(x, x, x, masked, cu, vocab=50)
    np.testing.assert_array_equal(a["pos"], b["pos"])
    np.testing.assert_array_equal(a["feat"], b["feat"])


def test_lps_positions_on_lbs_blocks():
    # blocks chosen by the LBS post-pass with g_max = 5: each position's value is its distance
    # from the block's first position over the block size, and a block with a gap reaches past 1
    rng = np.random.default_rng(15)
    n, L = 6, 64
    masked = (rng.random((n, L)) < 0.8).astype(np.uint8)
    p_phi = rng.random((n, L)).astype(np.float32)
    x_hat = rng.integers(0, 9, (n, L)).astype(np.int32)
    sel = lbs_select(masked, p_phi, x_hat, eos_id=8, l_min=2, l_b=8, g_max=5)
    rows = [np.nonzero(sel["block"][s])[0] for s in range(n)]
    lens = [len(x) for x in rows]
    cu = np.concatenate([[0], np.cumsum(lens)])
    seq_pos = np.concatenate(rows).astype(np.int32)
    T = int(cu[-1])
    z = np.zeros(T)
    r = lps_features(z, z, z, np.ones(T, np.uint8), cu, vocab=10, seq_pos=seq_pos)
    some_gap = False
    for s in range(n):
        got = r["pos"][cu[s]:cu[s + 1]]
        if lens[s]:
            assert got[0] == 0.0
            np.testing.assert_allclose(got * lens[s], rows[s] - rows[s][0], rtol=0, atol=1e-12)
            some_gap |= bool((np.diff(rows[s]) > 1).any())
    assert some_gap and r["pos"].max() > 1.0


def test_lps_features_ranges_random():
    rng = np.random.default_rng(13)
    lens = rng.integers(0, 30, 9)
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    masked = (rng.random(T) < 0.4).astype(np.uint8)
    r = lps_features(rng.random(T), rng.random(T) * 5, rng.random(T), masked, cu, vocab=1000)
    assert ((r["pos"] >= 0) & (r["pos"] < 1)).all()
    for b in range(len(lens)):
        sl = slice(cu[b], cu[b + 1])
        if lens[b]:
            assert r["mask_ratio"][b] == masked[sl].sum() / lens[b]
            np.testing.assert_array_equal(r["feat"][sl, 3], r["mask_ratio"][b])
            np.testing.assert_allclose(r["pos"][sl] * lens[b], np.arange(lens[b]))


# --------------------------------------------------------------------------------------
# union accept rule
# --------------------------------------------------------------------------------------

UNION = list(_rows("union_accept_examples.txt"))


@pytest.mark.parametrize("case", UNION, ids=[c[0][0] for c in UNION])
def test_union_golden(case):
    (name, tau, tau_psi, conf, p_psi, masked, argmax, tokens), (unmask, tok_out, nc, res) = case
    n = len(_floats(conf))
    r = unmask_select_lps(np.array(_floats(conf), np.float32), np.array(_ints(argmax), np.int32),
                          np.array(_ints(masked), np.uint8), np.array(_ints(tokens), np.int32),
                          np.array([float(tau)], np.float32), np.array([0, n]),
                          np.array(_floats(p_psi), np.float32), np.float32(float(tau_psi)))
    np.testing.assert_array_equal(r["unmask"], _ints(unmask))
    np.testing.assert_array_equal(r["tokens"], _ints(tok_out))
    assert int(r["n_commit"][0]) == int(nc) and int(r["resolved"][0]) == int(res)


def union_block(conf, p_psi, masked, tau, tau_psi):
    """Alg. 5's accept set for one block, as boolean arrays in float32."""
    conf = np.asarray(conf, np.float32)
    p_psi = np.asarray(p_psi, np.float32)
    mk = np.asarray(masked).astype(bool)
    acc = mk & ((conf >= np.float32(tau)) | (p_psi > np.float32(tau_psi)))
    if not acc.any() and mk.any():
        c = np.where(mk, conf, np.float32(-1))
        acc = np.zeros_like(mk)
        acc[int(np.argmax(c))] = True                        # first maximal index
    return acc


@pytest.mark.parametrize("n", [1, 2, 3])
def test_union_exhaustive(n):
    tau, tau_psi = np.float32(0.9), np.float32(0.95)
    kappas = np.array([0.1, 0.5, 0.9, 1.0], np.float32)
    psis = np.array([0.2, 0.95, 0.99], np.float32)
    argmax = np.arange(50, 50 + n, dtype=np.int32)
    for bits in itertools.product([0, 1], repeat=n):
        masked = np.array(bits, np.uint8)
        tokens = np.where(masked == 1, -1, 3).astype(np.int32)
        for conf in itertools.product(kappas, repeat=n):
            for psi in itertools.product(psis, repeat=n):
                r = unmask_select_lps(np.array(conf), argmax, masked, tokens, [tau],
                                      np.array([0, n]), np.array(psi), tau_psi)
                acc = union_block(conf, psi, masked, tau, tau_psi)
                np.testing.assert_array_equal(r["unmask"].astype(bool), acc)
                np.testing.assert_array_equal(r["tokens"], np.where(acc, argmax, tokens))
                assert r["resolved"][0] == int(not (masked.astype(bool) & ~acc).any())


def test_union_reduces_to_threshold_rule_and_covers_it():
    rng = np.random.default_rng(14)
    lens = rng.integers(0, 25, 12)
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    conf = rng.random(T).astype(np.float32)
    masked = (rng.random(T) < 0.6).astype(np.uint8)
    argmax = rng.integers(0, 99, T).astype(np.int32)
    tokens = np.where(masked == 1, -1, 7).astype(np.int32)
    tau = rng.choice(np.array([0.7, 0.9], np.float32), len(lens))
    base = unmask_select(conf, argmax, masked, tokens, tau, cu)
    low = unmask_select_lps(conf, argmax, masked, tokens, tau, cu,
                            rng.random(T).astype(np.float32) * 0.5, np.float32(0.5))
    for k in base:
        np.testing.assert_array_equal(low[k], base[k])
    allin = unmask_select_lps(conf, argmax, masked, tokens, tau, cu,
                              np.ones(T, np.float32), np.float32(0.5))
    np.testing.assert_array_equal(allin["unmask"], masked)   # every masked row commits
    np.testing.assert_array_equal(allin["resolved"], 1)


# --------------------------------------------------------------------------------------
# top-m budget commit
# --------------------------------------------------------------------------------------

TOPM = list(_rows("topm_examples.txt"))


@pytest.mark.parametrize("case", TOPM, ids=[c[0][0] for c in TOPM])
def test_topm_golden(case):
    (name, tau, m, conf, masked, argmax, tokens), (unmask, tok_out, nc, res) = case
    n = len(_floats(conf))
    r = unmask_select_topm(np.array(_floats(conf), np.float32), np.array(_ints(argmax), np.int32),
                           np.array(_ints(masked), np.uint8), np.array(_ints(tokens), np.int32),
                           np.array([float(tau)], np.float32), np.array([0, n]), int(m))
    np.testing.assert_array_equal(r["unmask"], _ints(unmask))
    np.testing.assert_array_equal(r["tokens"], _ints(tok_out))
    assert int(r["n_commit"][0]) == int(nc) and int(r["resolved"][0]) == int(res)


def topm_block(conf, masked, tau, m):
    """Eq. prelim-update by rank counting: masked row i is in Top-m when fewer than m masked
    rows rank above it (larger conf, or equal conf and a lower row)."""
    conf = np.asarray(conf, np.float32)
    n = len(conf)
    mk = np.asarray(masked).astype(bool)
    acc = np.zeros(n, bool)
    for i in range(n):
        if not mk[i]:
            continue
        above = sum(1 for j in range(n) if mk[j] and (conf[j] > conf[i] or (conf[j] == conf[i] and j < i)))
        acc[i] = conf[i] >= np.float32(tau) or above < m
    if not acc.any() and mk.any():
        best = max(range(n), key=lambda i: (mk[i], conf[i], -i))
        acc[best] = True
    return acc


@pytest.mark.parametrize("n", [1, 2, 3, 4])
def test_topm_exhaustive(n):
    kappas = np.array([0.1, 0.5, 0.9, 1.0], np.float32)
    argmax = np.arange(20, 20 + n, dtype=np.int32)
    for m in range(0, n + 2):
        for tau in (np.float32(0.9), np.float32(2.0)):
            for bits in itertools.product([0, 1], repeat=n):
                masked = np.array(bits, np.uint8)
                tokens = np.where(masked == 1, -1, 3).astype(np.int32)
                for conf in itertools.product(kappas, repeat=n):
                    r = unmask_select_topm(np.array(conf), argmax, masked, tokens, [tau],
                                           np.array([0, n]), m)
                    acc = topm_block(conf, masked, tau, m)
                    np.testing.assert_array_equal(r["unmask"].astype(bool), acc)
                    np.testing.assert_array_equal(r["tokens"], np.where(acc, argmax, tokens))


def test_topm_zero_is_threshold_rule():
    rng = np.random.default_rng(15)
    lens = rng.integers(0, 25, 12)
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    conf = rng.random(T).astype(np.float32)
    masked = (rng.random(T) < 0.6).astype(np.uint8)
    argmax = rng.integers(0, 99, T).astype(np.int32)
    tokens = np.where(masked == 1, -1, 7).astype(np.int32)
    tau = rng.choice(np.array([0.7, 0.9], np.float32), len(lens))
    base = unmask_select(conf, argmax, masked, tokens, tau, cu)
    r = unmask_select_topm(conf, argmax, masked, tokens, tau, cu, 0)
    for k in base:
        np.testing.assert_array_equal(r[k], base[k])
    r = unmask_select_topm(conf, argmax, masked, tokens, np.full(len(lens), 2.0, np.float32), cu, 3)
    for b in range(len(lens)):
        sl = slice(cu[b], cu[b + 1])
        assert r["n_commit"][b] == min(3, int(masked[sl].sum()))


# --------------------------------------------------------------------------------------
# LBS post-pass
# --------------------------------------------------------------------------------------

LBS = list(_rows("lbs_examples.txt"))


@pytest.mark.parametrize("case", LBS, ids=[c[0][0] for c in LBS])
def test_lbs_golden(case):
    (name, l_min, l_b, g_max, eos, masked, p_phi, x_hat), (block,) = case
    r = lbs_select(np.array([_ints(masked)], np.uint8), np.array([_floats(p_phi)], np.float32),
                   np.array([_ints(x_hat)], np.int32), int(eos), int(l_min), int(l_b), int(g_max))
    np.testing.assert_array_equal(r["block"][0], _ints(block))
    sel = np.nonzero(_ints(block))[0]
    assert r["size"][0] == sel.size and r["first"][0] == (sel[0] if sel.size else -1)


def lbs_vectorised(masked, p_phi, x_hat, eos, l_min, l_b, g_max):
    """The same post-pass with array operations: positions of M, a boolean candidate mask,
    and the max-gap cut found from the first difference of candidate positions above g_max."""
    M = np.flatnonzero(masked)
    if M.size <= l_min:
        return M
    cand = M[(np.asarray(p_phi, np.float32)[M] > np.float32(0.5)) & (x_hat[M] != eos)]
    if cand.size:
        big = np.flatnonzero(np.diff(cand) > g_max)
        cand = cand[:big[0] + 1] if big.size else cand
    return cand if cand.size >= l_min else M[:l_b]


def test_lbs_random_windows_against_vectorised():
    rng = np.random.default_rng(16)
    for _ in range(400):
        L = int(rng.integers(1, 70))
        masked = (rng.random((3, L)) < rng.random()).astype(np.uint8)
        p_phi = rng.choice(np.array([0.1, 0.5, 0.6, 0.95], np.float32), (3, L))
        x_hat = rng.integers(0, 6, (3, L)).astype(np.int32)
        l_min, l_b, g_max = int(rng.integers(0, 8)), int(rng.integers(1, 40)), int(rng.integers(1, 6))
        r = lbs_select(masked, p_phi, x_hat, 5, l_min, l_b, g_max)
        for s in range(3):
            exp = lbs_vectorised(masked[s], p_phi[s], x_hat[s], 5, l_min, l_b, g_max)
            np.testing.assert_array_equal(np.flatnonzero(r["block"][s]), exp)
            assert not (r["block"][s] & (1 - masked[s])).any()   # the block holds masked rows


# --------------------------------------------------------------------------------------
# dual-cache attention
# --------------------------------------------------------------------------------------

def _attn_case(rng, lens, plens, slens, hq, hkv, D):
    T, S, U = sum(lens), sum(plens), sum(slens)
    cu = lambda x: np.concatenate([[0], np.cumsum(x)]).astype(np.int32)
    return dict(q=rng.normal(size=(T, hq, D)), k_blk=rng.normal(size=(T, hkv, D)),
                v_blk=rng.normal(size=(T, hkv, D)), k_pre=rng.normal(size=(S, hkv, D)),
                v_pre=rng.normal(size=(S, hkv, D)), k_suf=rng.normal(size=(U, hkv, D)),
                v_suf=rng.normal(size=(U, hkv, D)), cu_block=cu(lens), cu_prefix=cu(plens),
                cu_suffix=cu(slens))


def test_dual_cache_brute_force():
    rng = np.random.default_rng(17)
    c = _attn_case(rng, [3, 0, 2], [2, 4, 1], [1, 3, 4], 4, 2, 5)
    out = block_attention(c["q"], c["k_blk"], c["v_blk"], c["k_pre"], c["v_pre"], c["cu_block"],
                          c["cu_prefix"], 4, 2, k_suf=c["k_suf"], v_suf=c["v_suf"],
                          cu_suffix=c["cu_suffix"])
    for b in range(3):
        for i in range(c["cu_block"][b], c["cu_block"][b + 1]):
            for h in range(4):
                g = h // 2
                keys, vals = [], []
                for lo, hi, K, Vv in ((c["cu_prefix"][b], c["cu_prefix"][b + 1], c["k_pre"], c["v_pre"]),
                                      (c["cu_block"][b], c["cu_block"][b + 1], c["k_blk"], c["v_blk"]),
                                      (c["cu_suffix"][b], c["cu_suffix"][b + 1], c["k_suf"], c["v_suf"])):
                    for j in range(lo, hi):
                        keys.append(K[j, g])
                        vals.append(Vv[j, g])
                sc = [sum(c["q"][i, h, d] * k[d] for d in range(5)) / math.sqrt(5) for k in keys]
                mx = max(sc)
                w = [math.exp(x - mx) for x in sc]
                tot = sum(w)
                ref = [sum(w[j] * vals[j][d] for j in range(len(w))) / tot for d in range(5)]
                np.testing.assert_allclose(out[i, h], ref, rtol=1e-12, atol=1e-12)


def test_dual_cache_empty_suffix_and_key_set():
    rng = np.random.default_rng(18)
    c = _attn_case(rng, [4, 3], [5, 2], [0, 0], 2, 1, 8)
    base = block_attention(c["q"], c["k_blk"], c["v_blk"], c["k_pre"], c["v_pre"], c["cu_block"],
                           c["cu_prefix"], 2, 1)
    dual = block_attention(c["q"], c["k_blk"], c["v_blk"], c["k_pre"], c["v_pre"], c["cu_block"],
                           c["cu_prefix"], 2, 1, k_suf=c["k_suf"], v_suf=c["v_suf"],
                           cu_suffix=c["cu_suffix"])
    np.testing.assert_array_equal(dual, base)
    # the suffix rows moved into the prefix give the same output: keys form a set
    c = _attn_case(rng, [4, 3], [5, 2], [3, 6], 2, 1, 8)
    dual = block_attention(c["q"], c["k_blk"], c["v_blk"], c["k_pre"], c["v_pre"], c["cu_block"],
                           c["cu_prefix"], 2, 1, k_suf=c["k_suf"], v_suf=c["v_suf"],
                           cu_suffix=c["cu_suffix"])
    kp, vp, cp = [], [], [0]
    for b in range(2):
        for src_k, src_v, cu in ((c["k_pre"], c["v_pre"], c["cu_prefix"]), (c["k_suf"], c["v_suf"], c["cu_suffix"])):
            kp.append(src_k[cu[b]:cu[b + 1]])
            vp.append(src_v[cu[b]:cu[b + 1]])
        cp.append(cp[-1] + (c["cu_prefix"][b + 1] - c["cu_prefix"][b]) + (c["cu_suffix"][b + 1] - c["cu_suffix"][b]))
    merged = block_attention(c["q"], c["k_blk"], c["v_blk"], np.concatenate(kp), np.concatenate(vp),
                             c["cu_block"], np.array(cp), 2, 1)
    np.testing.assert_allclose(dual, merged, rtol=1e-12, atol=1e-13)
