"""Pins of the oracle's unmask rule (threshold commit + anti-stall fallback).

Pinned against hand-derived cases (tests/golden/unmask_examples.txt, each following
Eq. prelim-update and Alg. 5), against a second scalar implementation written from
Alg. 5's accept / fallback / commit steps, and against invariants of the rule."""
import itertools
import os

import numpy as np
import pytest

from oracle import unmask_select

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "unmask_examples.txt")


def _ints(s):
    s = s.strip()
    return [] if s == "-" else [int(x) for x in s.split()]


def _floats(s):
    s = s.strip()
    return [] if s == "-" else [float(x) for x in s.split()]


def load_golden():
    cases = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        lhs, rhs = line.split("||")
        name, tau, conf, masked, argmax, tokens = [x.strip() for x in lhs.split("|")]
        unmask, tok_out, n_commit, resolved = [x.strip() for x in rhs.split("|")]
        cases.append(dict(
            name=name, tau=np.float32(float(tau)),
            conf=np.array(_floats(conf), dtype=np.float32),
            masked=np.array(_ints(masked), dtype=np.uint8),
            argmax=np.array(_ints(argmax), dtype=np.int32),
            tokens=np.array(_ints(tokens), dtype=np.int32),
            unmask=np.array(_ints(unmask), dtype=np.uint8),
            tok_out=np.array(_ints(tok_out), dtype=np.int32),
            n_commit=int(n_commit), resolved=int(resolved)))
    return cases


GOLDEN_CASES = load_golden()


@pytest.mark.parametrize("c", GOLDEN_CASES, ids=[c["name"] for c in GOLDEN_CASES])
def test_golden_single_block(c):
    n = c["conf"].size
    r = unmask_select(c["conf"], c["argmax"], c["masked"], c["tokens"], [c["tau"]],
                      np.array([0, n], np.int32))
    np.testing.assert_array_equal(r["unmask"], c["unmask"])
    np.testing.assert_array_equal(r["tokens"], c["tok_out"])
    np.testing.assert_array_equal(r["masked"], c["masked"] & ~c["unmask"].astype(bool))
    assert int(r["n_commit"][0]) == c["n_commit"]
    assert int(r["resolved"][0]) == c["resolved"]


def test_golden_as_one_ragged_batch():
    cs = GOLDEN_CASES
    lens = [c["conf"].size for c in cs]
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    cat = lambda k, dt: np.concatenate([c[k] for c in cs]).astype(dt)
    r = unmask_select(cat("conf", np.float32), cat("argmax", np.int32), cat("masked", np.uint8),
                      cat("tokens", np.int32), np.array([c["tau"] for c in cs], np.float32), cu)
    np.testing.assert_array_equal(r["unmask"], cat("unmask", np.uint8))
    np.testing.assert_array_equal(r["tokens"], cat("tok_out", np.int32))
    np.testing.assert_array_equal(r["n_commit"], [c["n_commit"] for c in cs])
    np.testing.assert_array_equal(r["resolved"], [c["resolved"] for c in cs])


def alg5_block(conf, masked, argmax, tokens, tau):
    """Alg. 5's accept / fallback / commit for one block, as plain scalar steps.

    conf is compared as given (float32 inputs widen exactly); tau as the exact widening of its
    float32 value."""
    n = len(conf)
    tau = float(np.float32(tau))
    conf = [float(c) for c in conf]
    A = [i for i in range(n) if masked[i] == 1 and conf[i] >= tau]
    if len(A) == 0:
        best = -1
        for i in range(n):
            if masked[i] == 1 and (best < 0 or conf[i] > conf[best]):
                best = i
        A = [best] if best >= 0 else []
    x = list(tokens)
    m = list(masked)
    for i in A:
        x[i] = argmax[i]
        m[i] = 0
    return A, x, m, int(all(v == 0 for v in m))


LEVELS = np.array([0.1, 0.5, 0.9, 0.95, 1.0], dtype=np.float32)


@pytest.mark.parametrize("n", [1, 2, 3, 4, 5, 6])
def test_exhaustive_small_blocks(n):
    # every mask pattern of n positions x every confidence vector over LEVELS (exact ties and
    # kappa == tau included); all confidence vectors of one mask pattern go through the oracle
    # as one ragged batch of blocks
    tau = np.float32(0.9)
    confs = np.array(list(itertools.product(LEVELS, repeat=n)), np.float32)
    C = confs.shape[0]
    argmax = np.arange(100, 100 + n, dtype=np.int32)
    cu = (np.arange(C + 1) * n).astype(np.int32)
    conf_rows = [[float(c) for c in row] for row in confs]
    for mask_bits in itertools.product([0, 1], repeat=n):
        masked = np.array(mask_bits, np.uint8)
        tokens = np.where(masked == 1, -1, np.arange(n)).astype(np.int32)
        r = unmask_select(confs.ravel(), np.tile(argmax, C), np.tile(masked, C),
                          np.tile(tokens, C), np.full(C, tau, np.float32), cu)
        exp_unmask = np.zeros((C, n), np.uint8)
        exp_tokens = np.empty((C, n), np.int32)
        exp_masked = np.empty((C, n), np.uint8)
        exp_commit = np.empty(C, np.int32)
        exp_res = np.empty(C, np.uint8)
        ml, al, tl = list(mask_bits), argmax.tolist(), tokens.tolist()
        for c in range(C):
            A, x, m, res = alg5_block(conf_rows[c], ml, al, tl, tau)
            exp_unmask[c, A] = 1
            exp_tokens[c] = x
            exp_masked[c] = m
            exp_commit[c] = len(A)
            exp_res[c] = res
        np.testing.assert_array_equal(r["unmask"].reshape(C, n), exp_unmask)
        np.testing.assert_array_equal(r["tokens"].reshape(C, n), exp_tokens)
        np.testing.assert_array_equal(r["masked"].reshape(C, n), exp_masked)
        np.testing.assert_array_equal(r["n_commit"], exp_commit)
        np.testing.assert_array_equal(r["resolved"], exp_res)


@pytest.mark.parametrize("n", [5, 6])
def test_sampled_blocks_other_tau(n):
    # tau = 0.5 sits on a level too; sampled, with random argmax ids and unmasked tokens
    rng = np.random.default_rng(n)
    tau = np.float32(0.5)
    for _ in range(1500):
        masked = (rng.random(n) < 0.6).astype(np.uint8)
        conf = LEVELS[rng.integers(0, LEVELS.size, n)]
        argmax = rng.integers(0, 50, n).astype(np.int32)
        tokens = np.where(masked == 1, -1, rng.integers(0, 50, n)).astype(np.int32)
        r = unmask_select(conf, argmax, masked, tokens, [tau], np.array([0, n], np.int32))
        A, x, m, res = alg5_block(conf, masked, argmax, tokens, tau)
        assert sorted(np.nonzero(r["unmask"])[0].tolist()) == sorted(A)
        np.testing.assert_array_equal(r["tokens"], x)
        assert r["resolved"][0] == res


def test_invariants_random_ragged():
    rng = np.random.default_rng(3)
    for _ in range(50):
        B = int(rng.integers(1, 8))
        lens = rng.integers(0, 40, B)
        cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        T = int(cu[-1])
        conf = rng.random(T).astype(np.float32)
        masked = (rng.random(T) < 0.5).astype(np.uint8)
        argmax = rng.integers(0, 1000, T).astype(np.int32)
        tokens = np.where(masked == 1, -1, rng.integers(0, 1000, T)).astype(np.int32)
        tau = rng.choice(np.array([0.7, 0.8, 0.9], np.float32), B)
        r = unmask_select(conf, argmax, masked, tokens, tau, cu)
        for b in range(B):
            sl = slice(cu[b], cu[b + 1])
            mk = masked[sl].astype(bool)
            un = r["unmask"][sl].astype(bool)
            assert not (un & ~mk).any()                       # A is a subset of the masked rows
            assert (un.sum() >= 1) == mk.any()                # progress iff something is masked
            passing = mk & (conf[sl] >= tau[b])
            if passing.any():
                np.testing.assert_array_equal(un, passing)    # A is the >= tau set when non-empty
            else:
                assert un.sum() == (1 if mk.any() else 0)
            np.testing.assert_array_equal(r["tokens"][sl][un], argmax[sl][un])
            np.testing.assert_array_equal(r["tokens"][sl][~un], tokens[sl][~un])
            assert r["n_commit"][b] == un.sum()
            assert r["resolved"][b] == int(not r["masked"][sl].any())
