"""The seeded generator: determinism, structure of the drawn step, and the properties
the easy/hard construction promises (checked with the oracle on the tiny workload)."""
import numpy as np
import pytest

import oracle
from workloads import CONFIGS, custom_config, make_step, f32_to_bf16_bits, bf16_bits_to_f32
from tests._cases import as_f32, enforce_margins


def test_bf16_rounding_is_rne():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, 1.0 + 2 ** -9, -2.5, 3.0e-3], np.float32)
    r = bf16_bits_to_f32(f32_to_bf16_bits(x))
    # 1 + 2^-8 is a tie -> even (1.0); 1 + 3*2^-8 is a tie -> even (1 + 2^-6)
    np.testing.assert_array_equal(r[:4], np.array([1.0, 1.0, 1.0 + 2 ** -6, 1.0], np.float32))
    assert r[4] == -2.5
    assert abs(r[5] - 3.0e-3) <= 3.0e-3 * 2 ** -8


def test_deterministic():
    a, b = make_step("tiny_f32_b1"), make_step("tiny_f32_b1")
    for k in ("q", "k_blk", "v_blk", "k_pre", "v_pre", "w", "h", "masked", "tokens", "tau", "easy"):
        np.testing.assert_array_equal(getattr(a, k), getattr(b, k))
    c = make_step("tiny_f32_b1", seed=5)
    assert not np.array_equal(a.h, c.h)


def test_structure_ragged_custom():
    cfg = custom_config(batch=5, block_len=("uniform", 0, 40), prefix_len=("uniform", 0, 30),
                        mask=("fraction", 0.2, 1.0), taus=(0.7, 0.8, 0.9), vocab=777, hidden=96,
                        hq=6, hkv=2, head_dim=64, run_max=5)
    c = make_step(cfg)
    assert c.cu_block[0] == 0 and (np.diff(c.cu_block) == c.block_lens).all()
    assert c.q.shape == (c.T, 6, 64) and c.k_pre.shape == (c.S, 2, 64)
    assert c.w.shape == (777, 96) and c.h.shape == (c.T, 96) and c.w.dtype == np.uint16
    assert ((c.tokens == -1) == c.masked.astype(bool)).all()
    for b in range(5):
        n = int(c.block_lens[b])
        k = int(c.masked[c.cu_block[b]:c.cu_block[b + 1]].sum())
        assert n == 0 or 0.2 * n - 1 <= k <= n
    assert set(np.unique(c.tau)) <= {np.float32(0.7), np.float32(0.8), np.float32(0.9)}


def test_runs_alternate_and_are_bounded():
    c = make_step(custom_config(block_len=("fixed", 400), run_max=6))
    e = c.easy.astype(int)
    runs = np.diff(np.flatnonzero(np.diff(np.concatenate([[-1], e, [-1]])) != 0))
    assert (runs[:-1] >= 2).all() and (runs <= 6).all()


def test_easy_rows_point_at_target_and_hard_rows_are_flat():
    c = enforce_margins(make_step("tiny_f32_b1"))
    st = oracle.lmhead_confidence(as_f32(c.h, c.dtype), as_f32(c.w, c.dtype))
    np.testing.assert_array_equal(st["argmax"][c.easy], c.target[c.easy])
    assert (st["conf"][c.easy] > 0.99).all() and (st["entropy"][c.easy] < 0.05).all()
    assert (st["conf"][~c.easy] < 0.1).all()
    assert (st["entropy"][~c.easy] > np.log(2048) - 2).all()


def test_named_workloads_have_stated_shapes():
    c = CONFIGS
    assert (c["llada8b_b1"].hidden, c["llada8b_b1"].vocab) == (4096, 126464)
    assert (c["dream7b_b64"].hq, c["dream7b_b64"].hkv, c["dream7b_b64"].vocab) == (28, 4, 152064)
    assert c["llada8b_b1"].hq * c["llada8b_b1"].head_dim == c["llada8b_b1"].hidden
    assert c["dream7b_b64"].hq * c["dream7b_b64"].head_dim == c["dream7b_b64"].hidden
