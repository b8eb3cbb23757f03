"""GPU parity of the HIP path against the fp64 oracle, through the C ABI.

Bars (written here, enforced below):
  * argmax token ids, unmask flags, committed tokens, mask flags, n_commit, resolved:
    bit-exact (inputs carry away-from-tie margins, see oracle/margins.py);
  * kappa and raw entropy (nats): within 1e-3 absolute;
  * max logit within ARGMAX_GAP / 4 and ln kappa within 1e-3 (the margins suffice);
  * attention output: bf16 within rtol 2e-2 / atol 2e-2, fp32 within 1e-4.
"""
import math
import os
import sys

import numpy as np
import pytest
import torch

import oracle
from oracle import margins
from paper_2609_16450_amd import (EB_BF16, Ragged, eb_block_attn, eb_decode_step,
                                  eb_lmhead_confidence, eb_unmask_select)
from paper_2609_16450_amd.device_case import DeviceStep
from tests._cases import as_f32, enforce_margins
from workloads import CONFIGS, custom_config, make_step, f32_to_bf16_bits, bf16_bits_to_f32

pytestmark = pytest.mark.gpu

ATTN_TOL_BF16 = dict(rtol=2e-2, atol=2e-2)
ATTN_TOL_F32 = dict(rtol=1e-4, atol=1e-4)
STAT_ATOL = 1e-3


def say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def attn_out_f32(t: torch.Tensor) -> np.ndarray:
    return t.float().cpu().numpy()


def check_stats(gpu_conf, gpu_ent, gpu_arg, gpu_ml, ref, rows=None):
    sel = slice(None) if rows is None else rows
    np.testing.assert_array_equal(gpu_arg[sel], ref["argmax"])
    np.testing.assert_allclose(gpu_conf[sel], ref["conf"], rtol=0, atol=STAT_ATOL)
    np.testing.assert_allclose(gpu_ent[sel], ref["entropy"], rtol=0, atol=STAT_ATOL)
    assert np.max(np.abs(gpu_ml[sel] - ref["max_logit"])) < margins.ARGMAX_GAP / 4
    assert np.max(np.abs(np.log(gpu_conf[sel]) - np.log(ref["conf"]))) < 1e-3


# ----------------------------------------------------------------------------------------
# LM head + statistics, small shapes spanning several tiles and ragged tails
# ----------------------------------------------------------------------------------------
LM_CASES = [
    # (n_rows, hidden, vocab, dtype)
    (1, 64, 1000, "bf16"),
    (5, 256, 2048 + 77, "bf16"),
    (32, 320, 3000, "bf16"),
    (33, 128, 1537, "bf16"),
    (64, 192, 4099, "bf16"),
    (65, 256, 2500, "bf16"),
    (200, 512, 5000, "bf16"),
    # large-batch kernel: several row tiles, vocabulary bands with a partial last band
    (600, 192, 9000, "bf16"),
    (300, 128, 1100, "bf16"),
    # more tiles than persistent workgroups: several tiles per workgroup, the next tile's first
    # stages issued in the previous tile's tail (hidden of exactly 4 stages; 6 stages, so the
    # ring position of a tile's first stage moves), or not (hidden of 2 stages)
    (300, 128, 70000, "bf16"),
    (1100, 192, 100000, "bf16"),
    (700, 64, 40000, "bf16"),
    # streaming kernel: 16 waves with 1..3 row tiles each, 8 waves with 7 or 8, partial h chunks;
    # two row tiles per wave with one, two and four position tiles (100003: a partial last slice)
    (32, 256, 126464, "bf16"),
    (5, 4160, 100003, "bf16"),
    (20, 64, 100000, "bf16"),
    (64, 128, 126464, "bf16"),
    (17, 128, 152064, "bf16"),
    (48, 192, 152064, "bf16"),
    (8, 64, 200000, "bf16"),
    (2, 64, 262144, "bf16"),
    (40, 1600, 9000, "bf16"),
    (3, 4160, 20000, "bf16"),
    # extremes: a one- and a two-entry vocabulary (both kernels), a hidden size of 8192
    (4, 64, 1, "bf16"),
    (70, 64, 1, "bf16"),
    (3, 64, 2, "bf16"),
    (16, 8192, 3000, "bf16"),
    (130, 8192, 2000, "bf16"),
    (32, 256, 2048, "f32"),
    (7, 100, 999, "f32"),
]


@pytest.mark.parametrize("n_rows,hidden,vocab,dt", LM_CASES)
def test_lmhead_small(n_rows, hidden, vocab, dt):
    say(f"lmhead n_rows={n_rows} hidden={hidden} vocab={vocab} dtype={dt}")
    cfg = custom_config(seed=11 + n_rows, block_len=("fixed", n_rows), hidden=hidden, vocab=vocab,
                        dtype=dt, hq=1, hkv=1, head_dim=64, prefix_len=("fixed", 0))
    case = enforce_margins(make_step(cfg))
    ref = oracle.lmhead_confidence(as_f32(case.h, dt), as_f32(case.w, dt))
    ds = DeviceStep(case)
    eb_lmhead_confidence(ds.h, ds.w, ds.conf, ds.entropy, ds.argmax, ds.max_logit)
    torch.cuda.synchronize()
    check_stats(ds.conf.cpu().numpy(), ds.entropy.cpu().numpy(), ds.argmax.cpu().numpy(),
                ds.max_logit.cpu().numpy(), ref)


# Duplicates of the winning W row.  The large-batch kernel holds vocabulary row 16 tm + 4 r + q
# of a wave's 128 rows in register r of lane group q, so ids 130 / 134 share a lane and differ
# in the register chain, 130 / 146 share a chain and differ in the block, 129 / 130 sit in
# different lanes of one column, and 2999 lies in the last, partial vocabulary tile.
TIE_CASES = [
    (40, (130, 2999)),          # streaming kernel (at most 64 positions)
    (300, (146, 134, 130, 2999)),  # tile kernel: lowest in the same lane, other chain / block
    (300, (146, 134, 129, 2999)),  # tile kernel: lowest in another lane of the column
    (300, (2999,)),             # tile kernel: the winner in the partial last tile only
]


@pytest.mark.parametrize("n,dups", TIE_CASES)
def test_lmhead_vocab_ties_take_lowest_id(n, dups):
    # Duplicate rows of W give bit-identical logits (same accumulation order, no split over the
    # hidden dimension), so the lowest duplicated id must win.
    say(f"lmhead ties n={n} dups={dups}")
    rng = np.random.default_rng(5)
    d, V = 256, 3000
    h = torch.from_numpy(rng.standard_normal((n, d)).astype(np.float32)).to(torch.bfloat16).cuda()
    w = torch.from_numpy((rng.standard_normal((V, d)) / 16).astype(np.float32)).to(torch.bfloat16)
    # make row 2900 the clear winner for every position, then copy it to the duplicate ids
    w[2900] = (h.float().cpu().mean(0) * 4).to(torch.bfloat16)
    for i in dups:
        w[i] = w[2900]
    w = w.cuda()
    conf = torch.empty(n, device="cuda")
    ent = torch.empty(n, device="cuda")
    am = torch.empty(n, dtype=torch.int32, device="cuda")
    eb_lmhead_confidence(h, w, conf, ent, am)
    torch.cuda.synchronize()
    z = h.float().cpu().double().numpy() @ w.float().cpu().double().numpy().T
    m = z.max(1)
    winners = [np.flatnonzero(z[i] == m[i])[0] for i in range(n)]
    np.testing.assert_array_equal(am.cpu().numpy(), winners)
    assert (am.cpu().numpy() == min(min(dups), 2900)).sum() > 0


# ----------------------------------------------------------------------------------------
# block attention, small ragged shapes
# ----------------------------------------------------------------------------------------
ATTN_CASES = [
    # batch, hq, hkv, D, block_len spec, prefix_len spec, dtype
    (1, 4, 4, 64, ("fixed", 32), ("fixed", 96), "f32"),
    (3, 4, 2, 64, ("uniform", 0, 20), ("uniform", 0, 70), "f32"),
    (1, 2, 2, 128, ("fixed", 1), ("fixed", 0), "bf16"),
    (4, 8, 2, 128, ("uniform", 0, 40), ("uniform", 0, 200), "bf16"),
    (3, 6, 6, 64, ("uniform", 1, 70), ("uniform", 60, 130), "bf16"),
    (2, 28, 4, 128, ("uniform", 10, 60), ("fixed", 300), "bf16"),
    (5, 4, 1, 128, ("choice", (0, 1, 63, 64, 65, 129)), ("choice", (0, 1, 63, 64, 65)), "bf16"),
    # small steps (<= 64 block rows, <= 256 query rows per sequence and K/V head) take the
    # 16-row kernel that also runs inside the LM-head launch of a step
    (1, 32, 32, 128, ("fixed", 32), ("fixed", 512), "bf16"),    # batch-1 LLaDA shape, 9 ranges
    (1, 32, 8, 128, ("fixed", 64), ("fixed", 200), "bf16"),     # 256 query rows: all 16 waves
    (4, 8, 2, 64, ("uniform", 0, 16), ("uniform", 0, 150), "bf16"),  # D = 64, empty blocks
    (3, 4, 4, 128, ("choice", (1, 5, 17)), ("choice", (0, 1, 63)), "bf16"),  # one range: no split
    (2, 28, 4, 128, ("fixed", 32), ("fixed", 700), "bf16"),     # G = 7: 224 rows, 14 waves
    (8, 16, 2, 64, ("fixed", 8), ("uniform", 300, 1100), "bf16"),  # G = 8, many key ranges
]


@pytest.mark.parametrize("batch,hq,hkv,D,bl,pl,dt", ATTN_CASES)
def test_block_attn_small(batch, hq, hkv, D, bl, pl, dt):
    say(f"attn batch={batch} hq={hq} hkv={hkv} D={D} bl={bl} pl={pl} dtype={dt}")
    cfg = custom_config(seed=100 + batch * hq, batch=batch, hq=hq, hkv=hkv, head_dim=D,
                        block_len=bl, prefix_len=pl, hidden=64, vocab=64, dtype=dt)
    case = make_step(cfg)
    if case.T == 0:
        pytest.skip("all blocks empty")
    f = {k: as_f32(getattr(case, k), dt) for k in ("q", "k_blk", "v_blk", "k_pre", "v_pre")}
    ref = oracle.block_attention(**f, cu_block=case.cu_block, cu_prefix=case.cu_prefix,
                                 hq=hq, hkv=hkv)
    ds = DeviceStep(case)
    eb_block_attn(ds.ragged, ds.q, ds.k_blk, ds.v_blk, ds.k_pre, ds.v_pre, ds.attn_out)
    torch.cuda.synchronize()
    tol = ATTN_TOL_BF16 if dt == "bf16" else ATTN_TOL_F32
    np.testing.assert_allclose(attn_out_f32(ds.attn_out), ref, **tol)


# head dimension 128, not small: the register-staged kernel the library keeps for K/V segments
# too long for 32-bit buffer offsets, selected here by EB_ATTN_STAGED
STAGED_CASES = [c for c in ATTN_CASES if c[3] == 128 and c[6] == "bf16"]


@pytest.mark.parametrize("batch,hq,hkv,D,bl,pl,dt", STAGED_CASES)
def test_block_attn_register_staged_form(batch, hq, hkv, D, bl, pl, dt, monkeypatch):
    monkeypatch.setenv("EB_ATTN_STAGED", "1")
    test_block_attn_small(batch, hq, hkv, D, bl, pl, dt)


@pytest.mark.parametrize("staged", [False, True])
@pytest.mark.parametrize("split", [False, True])
def test_block_attn_scores_growing_along_the_keys(split, staged, monkeypatch):
    if staged:
        monkeypatch.setenv("EB_ATTN_STAGED", "1")
    # Keys scaled up along each sequence, so the running maximum of a row keeps moving by more
    # than the kernel's rescale slack (2^8) from tile to tile; with split the key ranges are
    # merged from partials (batch 1: the split plan cuts the keys to fill the chip).
    # batch 16 x 4 K/V heads x 7 row tiles: two key ranges of ~8 tiles per workgroup;
    # batch 2: one or two tiles per range
    batch, hq, hkv = (2, 8, 2) if split else (16, 28, 4)
    say(f"attn growing scores split={split}")
    cfg = custom_config(seed=4242 + batch, batch=batch, hq=hq, hkv=hkv, head_dim=128,
                        block_len=("fixed", 128), prefix_len=("uniform", 500, 900),
                        hidden=64, vocab=64, dtype="bf16")
    case = make_step(cfg)
    for b in range(case.batch):
        p0, p1 = case.cu_prefix[b], case.cu_prefix[b + 1]
        ramp = (1.0 + 9.0 * np.arange(p1 - p0) / max(1, p1 - p0)).astype(np.float32)
        k = bf16_bits_to_f32(case.k_pre[p0:p1]) * ramp[:, None, None]
        case.k_pre[p0:p1] = f32_to_bf16_bits(k)
        b0, b1 = case.cu_block[b], case.cu_block[b + 1]
        case.k_blk[b0:b1] = f32_to_bf16_bits(bf16_bits_to_f32(case.k_blk[b0:b1]) * 10.0)
    f = {k: as_f32(getattr(case, k), "bf16") for k in ("q", "k_blk", "v_blk", "k_pre", "v_pre")}
    ref = oracle.block_attention(**f, cu_block=case.cu_block, cu_prefix=case.cu_prefix,
                                 hq=hq, hkv=hkv)
    ds = DeviceStep(case)
    eb_block_attn(ds.ragged, ds.q, ds.k_blk, ds.v_blk, ds.k_pre, ds.v_pre, ds.attn_out)
    torch.cuda.synchronize()
    np.testing.assert_allclose(attn_out_f32(ds.attn_out), ref, **ATTN_TOL_BF16)


# ----------------------------------------------------------------------------------------
# unmask: constructed confidences (exact ties, kappa == tau, empty and length-1 blocks)
# ----------------------------------------------------------------------------------------
def _run_unmask(lens, conf, masked, argmax, tokens, tau):
    r = Ragged.from_lengths(lens, [0] * len(lens))
    T, B = r.total_block, r.batch
    d = lambda x, dt: torch.from_numpy(np.asarray(x, dtype=dt)).cuda()
    c, a, t = d(conf, np.float32), d(argmax, np.int32), d(tau, np.float32)
    m, tk = d(masked, np.uint8), d(tokens, np.int32)
    un = torch.full((T,), 7, dtype=torch.uint8, device="cuda")
    nc = torch.full((B,), -5, dtype=torch.int32, device="cuda")
    rs = torch.full((B,), 9, dtype=torch.uint8, device="cuda")
    eb_unmask_select(r, c, a, t, m, tk, un, nc, rs)
    torch.cuda.synchronize()
    return dict(unmask=un.cpu().numpy(), tokens=tk.cpu().numpy(), masked=m.cpu().numpy(),
                n_commit=nc.cpu().numpy(), resolved=rs.cpu().numpy())


def _compare_unmask(lens, conf, masked, argmax, tokens, tau):
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    ref = oracle.unmask_select(conf, argmax, masked, tokens, tau, cu)
    got = _run_unmask(lens, conf, masked, argmax, tokens, tau)
    for k in ("unmask", "tokens", "masked", "n_commit", "resolved"):
        np.testing.assert_array_equal(got[k], ref[k], err_msg=k)


def test_unmask_constructed_edge_cases():
    say("unmask edge cases")
    rng = np.random.default_rng(0)
    levels = np.array([0.1, 0.5, 0.9, 0.95, 1.0], np.float32)
    lens = [0, 1, 1, 2, 5, 6, 0, 33, 256, 257, 700, 3]
    T = sum(lens)
    conf = levels[rng.integers(0, levels.size, T)]
    masked = (rng.random(T) < 0.6).astype(np.uint8)
    # block 1: single masked row below tau; block 2: single unmasked row
    conf[0], masked[0] = 0.1, 1
    masked[1] = 0
    # block 3: two masked rows with equal conf below tau -> lower wins
    conf[2:4], masked[2:4] = 0.5, 1
    # block 4: every row masked and exactly at tau
    conf[4:9], masked[4:9] = 0.9, 1
    argmax = rng.integers(0, 1000, T).astype(np.int32)
    tokens = np.where(masked == 1, -1, rng.integers(0, 1000, T)).astype(np.int32)
    tau = np.full(len(lens), 0.9, np.float32)
    tau[5] = 1.0
    _compare_unmask(lens, conf, masked, argmax, tokens, tau)


def test_unmask_random_ragged_with_ties():
    say("unmask random")
    rng = np.random.default_rng(1)
    for it in range(20):
        B = int(rng.integers(1, 70))
        lens = rng.integers(0, 300, B).tolist()
        T = sum(lens)
        # coarse grid of confidences gives many exact ties
        conf = (rng.integers(0, 20, T) / 20.0).astype(np.float32)
        masked = (rng.random(T) < rng.random()).astype(np.uint8)
        argmax = rng.integers(0, 152064, T).astype(np.int32)
        tokens = np.where(masked == 1, -1, rng.integers(0, 152064, T)).astype(np.int32)
        tau = rng.choice(np.array([0.7, 0.8, 0.9, 0.95], np.float32), B)
        _compare_unmask(lens, conf, masked, argmax, tokens, tau)


# ----------------------------------------------------------------------------------------
# whole step on the named workloads, in the launch configuration the benchmark times
# ----------------------------------------------------------------------------------------
POSITION_TILE = 256   # block positions per position tile of the large-batch LM-head kernel


def _sample_blocks(case, k=3):
    """Blocks checked element by element on a large workload: the first and the longest block,
    the last non-empty one (its rows fall in the last, partial position tile), every block with
    a row among the first 256 block positions (so that one whole position tile is checked row by
    row), and random ones up to k beyond those."""
    lens = case.block_lens
    nonempty = np.flatnonzero(lens > 0)
    if nonempty.size <= k:
        return nonempty.tolist()
    rng = np.random.default_rng(case.cfg.seed + 77)
    pick = {int(nonempty[0]), int(nonempty[np.argmax(lens[nonempty])]), int(nonempty[-1])}
    pick |= {int(b) for b in nonempty if case.cu_block[b] < POSITION_TILE}
    want = len(pick) + 1
    while len(pick) < max(k, want):
        pick.add(int(rng.choice(nonempty)))
    return sorted(pick)


@pytest.mark.parametrize("name", list(CONFIGS))
def test_decode_step_workload(name):
    _check_workload(name, None)


# the two small workloads also on further seeds (other block contents, masks and runs)
@pytest.mark.parametrize("name,seed", [(n, s) for n in ("tiny_f32_b1", "llada8b_b1")
                                       for s in (1, 2, 3)])
def test_decode_step_workload_other_seeds(name, seed):
    _check_workload(name, seed)


def _check_workload(name, seed):
    say(f"decode_step workload={name} seed={seed}")
    case = make_step(name, seed)
    full = case.T <= 64
    blocks = list(range(case.batch)) if full else _sample_blocks(case)
    enforce_margins(case, blocks)
    dt = case.dtype
    ds = DeviceStep(case)
    eb_decode_step(ds.buffers)
    torch.cuda.synchronize()
    say(f"  gpu done; oracle over blocks {blocks}")

    rows = np.concatenate([np.arange(case.cu_block[b], case.cu_block[b + 1]) for b in blocks])
    if not full:
        assert set(range(min(POSITION_TILE, case.T))) <= set(rows.tolist())
        assert case.T - 1 in set(rows.tolist())
    conf = ds.conf.cpu().numpy()
    ent = ds.entropy.cpu().numpy()
    am = ds.argmax.cpu().numpy()
    ml = ds.max_logit.cpu().numpy()
    ref = oracle.lmhead_confidence(as_f32(case.h, dt), as_f32(case.w, dt), rows=rows)
    check_stats(conf, ent, am, ml, ref, rows)

    # unmask on the checked blocks, from the oracle's own statistics
    sub_lens = [int(case.block_lens[b]) for b in blocks]
    sub_cu = np.concatenate([[0], np.cumsum(sub_lens)]).astype(np.int32)
    uref = oracle.unmask_select(ref["conf"], ref["argmax"], case.masked[rows], case.tokens[rows],
                                case.tau[blocks], sub_cu)
    np.testing.assert_array_equal(ds.unmask.cpu().numpy()[rows], uref["unmask"])
    np.testing.assert_array_equal(ds.tokens.cpu().numpy()[rows], uref["tokens"])
    np.testing.assert_array_equal(ds.masked.cpu().numpy()[rows], uref["masked"])
    np.testing.assert_array_equal(ds.n_commit.cpu().numpy()[blocks], uref["n_commit"])
    np.testing.assert_array_equal(ds.resolved.cpu().numpy()[blocks], uref["resolved"])

    # attention on the checked sequences
    sub_pl = [int(case.prefix_lens[b]) for b in blocks]
    prow = np.concatenate([np.arange(case.cu_prefix[b], case.cu_prefix[b + 1]) for b in blocks])
    f = lambda a: as_f32(a, dt)
    aref = oracle.block_attention(f(case.q[rows]), f(case.k_blk[rows]), f(case.v_blk[rows]),
                                  f(case.k_pre[prow]), f(case.v_pre[prow]), sub_cu,
                                  np.concatenate([[0], np.cumsum(sub_pl)]).astype(np.int32),
                                  case.cfg.hq, case.cfg.hkv)
    tol = ATTN_TOL_BF16 if dt == "bf16" else ATTN_TOL_F32
    np.testing.assert_allclose(attn_out_f32(ds.attn_out)[rows], aref, **tol)

    # properties over every row and block
    V = case.cfg.vocab
    assert (am >= 0).all() and (am < V).all()
    assert (conf > 0).all() and (conf <= 1.0).all()
    assert (ent >= -1e-4).all() and (ent <= math.log(V) + 1e-3).all()
    assert (ent >= -np.log(conf) - 1e-3).all()
    un = ds.unmask.cpu().numpy().astype(bool)
    m0 = case.masked.astype(bool)
    assert not (un & ~m0).any()
    np.testing.assert_array_equal(ds.tokens.cpu().numpy()[un], am[un])
    nc = ds.n_commit.cpu().numpy()
    for b in range(case.batch):
        sl = slice(case.cu_block[b], case.cu_block[b + 1])
        assert nc[b] == un[sl].sum()
        assert (nc[b] >= 1) == m0[sl].any()


@pytest.mark.parametrize("name", ["llada8b_b16", "dream7b_b64"])
def test_decode_step_is_deterministic(name):
    say(f"determinism {name}")
    case = make_step(name)
    ds = DeviceStep(case)
    outs = []
    for _ in range(2):
        ds.reset_state()
        eb_decode_step(ds.buffers)
        torch.cuda.synchronize()
        outs.append([t.clone() for t in (ds.attn_out, ds.conf, ds.entropy, ds.argmax, ds.max_logit,
                                         ds.tokens, ds.masked, ds.unmask, ds.n_commit, ds.resolved)])
    for a, b in zip(*outs):
        assert torch.equal(a.view(torch.uint8) if a.dtype == torch.bfloat16 else a,
                           b.view(torch.uint8) if b.dtype == torch.bfloat16 else b)


# The step composes its kernels differently from the separate entry points (one epilogue launch
# merges the attention key splits, reduces the LM-head partials and runs the unmask step), with
# the same arithmetic, so every output must match them bit for bit.
FUSE_CASES = [
    # fused epilogue, attention key split merged there
    ("llada8b_b1", None),
    # fused, ragged blocks (some empty), GQA, large-batch LM kernel
    ("ragged", dict(seed=31, batch=5, hq=8, hkv=2, head_dim=128, hidden=256, vocab=5000,
                    block_len=("uniform", 0, 40), prefix_len=("uniform", 0, 300))),
    # too many partials for one workgroup per block: separate kernels
    ("long_block", dict(seed=32, batch=1, hq=2, hkv=2, head_dim=64, hidden=64, vocab=60000,
                        block_len=("fixed", 300), prefix_len=("fixed", 64))),
    # small steps: the attention runs inside the LM-head launch (key split merged in the
    # epilogue, or no split at all)
    ("hosted_gqa_d64", dict(seed=34, batch=4, hq=8, hkv=2, head_dim=64, hidden=256, vocab=7000,
                            block_len=("uniform", 0, 16), prefix_len=("uniform", 0, 150))),
    ("hosted_no_split", dict(seed=35, batch=2, hq=4, hkv=4, head_dim=128, hidden=128,
                             vocab=3000, block_len=("fixed", 20), prefix_len=("fixed", 10))),
    ("hosted_256_rows", dict(seed=36, batch=1, hq=16, hkv=4, head_dim=128, hidden=512,
                             vocab=20000, block_len=("fixed", 64), prefix_len=("fixed", 333))),
    # small attention, but an 8-wave LM-head launch: the attention runs on its own
    ("small_attn_8wave_lm", dict(seed=37, batch=1, hq=4, hkv=4, head_dim=128, hidden=64,
                                 vocab=262144, block_len=("fixed", 16), prefix_len=("fixed", 100))),
    # fp32 path
    ("f32", dict(seed=33, batch=3, hq=4, hkv=2, head_dim=64, hidden=128, vocab=999,
                 block_len=("uniform", 1, 20), prefix_len=("uniform", 0, 50), dtype="f32")),
]


@pytest.mark.parametrize("name,spec", FUSE_CASES, ids=[c[0] for c in FUSE_CASES])
def test_decode_step_matches_separate_entry_points(name, spec):
    say(f"decode_step vs separate entry points: {name}")
    case = make_step(name if spec is None else custom_config(name, **spec))
    a = DeviceStep(case)
    eb_decode_step(a.buffers)
    b = DeviceStep(case)
    eb_block_attn(b.ragged, b.q, b.k_blk, b.v_blk, b.k_pre, b.v_pre, b.attn_out)
    eb_lmhead_confidence(b.h, b.w, b.conf, b.entropy, b.argmax, b.max_logit)
    eb_unmask_select(b.ragged, b.conf, b.argmax, b.tau, b.masked, b.tokens, b.unmask, b.n_commit,
                     b.resolved)
    torch.cuda.synchronize()
    for field in ("attn_out", "conf", "entropy", "argmax", "max_logit", "tokens", "masked",
                  "unmask", "n_commit", "resolved"):
        x, y = getattr(a, field), getattr(b, field)
        if x.dtype == torch.bfloat16:
            x, y = x.view(torch.int16), y.view(torch.int16)
        assert torch.equal(x, y), field


@pytest.mark.parametrize("dt", ["bf16", "f32"])
def test_decode_step_all_blocks_empty(dt):
    # T = 0: no attention rows and no LM-head rows; the epilogue still settles every block
    # (nothing to commit, nothing masked left).
    say(f"decode_step with every block empty ({dt})")
    case = make_step(custom_config("empty", seed=41, batch=3, hq=4, hkv=2, head_dim=64, hidden=128,
                                   vocab=1000, block_len=("fixed", 0),
                                   prefix_len=("uniform", 0, 40), dtype=dt))
    assert case.T == 0
    ds = DeviceStep(case)
    ds.n_commit.fill_(-7)
    ds.resolved.fill_(9)
    eb_decode_step(ds.buffers)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(ds.n_commit.cpu().numpy(), [0, 0, 0])
    np.testing.assert_array_equal(ds.resolved.cpu().numpy(), [1, 1, 1])


_STEP_FIELDS = ("attn_out", "conf", "entropy", "argmax", "max_logit", "tokens", "masked", "unmask",
                "n_commit", "resolved")


@pytest.mark.parametrize("name,spec", [
    ("llada8b_b1", None),  # attention inside the LM-head launch, fused epilogue
    ("ragged", dict(seed=31, batch=5, hq=8, hkv=2, head_dim=128, hidden=256, vocab=5000,
                    block_len=("uniform", 0, 40), prefix_len=("uniform", 0, 300))),
], ids=["llada8b_b1", "ragged"])
def test_decode_step_hip_graph_replays(name, spec):
    # The step allocates nothing and records no memset, so it can be captured in a HIP graph.
    # Each replay, with eager steps and host synchronisations between replays, must equal an
    # eager step on the same inputs bit for bit.
    say(f"decode_step captured in a HIP graph: {name}")
    case = make_step(name if spec is None else custom_config(name, **spec))
    g_in, e_in = DeviceStep(case), DeviceStep(case)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        eb_decode_step(g_in.buffers)  # warm-up outside the capture
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    g_in.reset_state()
    torch.cuda.synchronize()
    with torch.cuda.graph(graph):
        eb_decode_step(g_in.buffers)
    torch.cuda.synchronize()
    for rep in range(3):
        g_in.reset_state()
        e_in.reset_state()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        eb_decode_step(e_in.buffers)
        torch.cuda.synchronize()
        for field in _STEP_FIELDS:
            x, y = getattr(g_in, field), getattr(e_in, field)
            if x.dtype == torch.bfloat16:
                x, y = x.view(torch.int16), y.view(torch.int16)
            assert torch.equal(x, y), (rep, field)


def _random_step_spec(i):
    # Seeded shapes around the dispatch boundaries of the step: total block rows near 64 (the
    # small-step attention and the streaming LM head), query rows per K/V head near 256, both
    # head dimensions, GQA groups 1-8, empty blocks, vocabularies for 16- and 8-wave streaming.
    r = np.random.default_rng(9000 + i)
    hq, hkv = [(4, 4), (8, 2), (16, 4), (28, 4), (32, 32), (12, 3), (32, 4)][r.integers(7)]
    batch = int(r.integers(1, 5))
    hi = int(r.choice([8, 16, 24, 40, 70]))
    return dict(seed=700 + i, batch=batch, hq=hq, hkv=hkv, head_dim=int(r.choice([64, 128])),
                hidden=int(r.choice([64, 128, 256])),
                vocab=int(r.choice([2000, 9000, 33000, 200000, 250000])),
                block_len=("uniform", 0, hi), prefix_len=("uniform", 0, int(r.integers(1, 700))))


@pytest.mark.parametrize("i", range(40))
def test_decode_step_random_shapes(i):
    spec = _random_step_spec(i)
    say(f"decode_step random shape {i}: {spec}")
    case = enforce_margins(make_step(custom_config(f"random{i}", **spec)))
    a = DeviceStep(case)
    eb_decode_step(a.buffers)
    b = DeviceStep(case)
    eb_block_attn(b.ragged, b.q, b.k_blk, b.v_blk, b.k_pre, b.v_pre, b.attn_out)
    eb_lmhead_confidence(b.h, b.w, b.conf, b.entropy, b.argmax, b.max_logit)
    eb_unmask_select(b.ragged, b.conf, b.argmax, b.tau, b.masked, b.tokens, b.unmask, b.n_commit,
                     b.resolved)
    torch.cuda.synchronize()
    for field in _STEP_FIELDS:
        x, y = getattr(a, field), getattr(b, field)
        if x.dtype == torch.bfloat16:
            x, y = x.view(torch.int16), y.view(torch.int16)
        assert torch.equal(x, y), field
    if case.T:
        f = {k: as_f32(getattr(case, k), "bf16") for k in ("q", "k_blk", "v_blk", "k_pre", "v_pre")}
        ref = oracle.block_attention(**f, cu_block=case.cu_block, cu_prefix=case.cu_prefix,
                                     hq=spec["hq"], hkv=spec["hkv"])
        np.testing.assert_allclose(attn_out_f32(a.attn_out), ref, **ATTN_TOL_BF16)
        ref = oracle.lmhead_confidence(as_f32(case.h, "bf16"), as_f32(case.w, "bf16"))
        check_stats(a.conf.cpu().numpy(), a.entropy.cpu().numpy(), a.argmax.cpu().numpy(),
                    a.max_logit.cpu().numpy(), ref)


class _DebugChecks:
    """EB_DEBUG_CHECKS=1 for the duration of a with-block."""

    def __enter__(self):
        self.old = os.environ.get("EB_DEBUG_CHECKS")
        os.environ["EB_DEBUG_CHECKS"] = "1"

    def __exit__(self, *exc):
        if self.old is None:
            os.environ.pop("EB_DEBUG_CHECKS", None)
        else:
            os.environ["EB_DEBUG_CHECKS"] = self.old


def test_debug_checks_reject_bad_device_arrays():
    # With EB_DEBUG_CHECKS set, entry points check the device offset arrays and tau against the
    # contract on the host and launch nothing when they break it.  Every bad array below keeps
    # all row indices inside [0, T), so no kernel could read out of bounds even unchecked.
    say("debug checks of the device-array contract")
    from paper_2609_16450_amd import EbError
    T, B = 32, 2
    dev = lambda x, dt: torch.tensor(x, dtype=dt, device="cuda")
    conf = dev(np.linspace(0.1, 0.95, T), torch.float32)
    argmax = dev(np.arange(T), torch.int32)
    masked = torch.ones(T, dtype=torch.uint8, device="cuda")
    tokens = torch.full((T,), -1, dtype=torch.int32, device="cuda")
    unmask = torch.empty(T, dtype=torch.uint8, device="cuda")
    n_commit = torch.empty(B, dtype=torch.int32, device="cuda")
    resolved = torch.empty(B, dtype=torch.uint8, device="cuda")
    tau = dev([0.9, 0.9], torch.float32)
    zero = dev([0, 0, 0], torch.int32)
    rag = lambda cu: Ragged(B, T, 20, 0, 0, dev(cu, torch.int32), zero)
    run = lambda r, t: eb_unmask_select(r, conf, argmax, t, masked, tokens, unmask, n_commit,
                                        resolved)
    with _DebugChecks():
        run(rag([0, 20, 32]), tau)  # a valid call passes the checks
        torch.cuda.synchronize()
        for cu, what in (([0, 20, 12], "decreases"), ([0, 16, 30], "host total"),
                         ([2, 16, 32], "expected 0"), ([0, 10, 32], "host maximum")):
            with pytest.raises(EbError) as err:
                run(rag(cu), tau)
            assert "EB_ERR_INVALID" in str(err.value) and what in str(err.value), err.value
        with pytest.raises(EbError) as err:
            run(rag([0, 20, 32]), dev([0.0, 0.9], torch.float32))
        assert "tau[0]" in str(err.value)
        # attention: a prefix offset array that does not end at the host total
        r = Ragged(1, 8, 8, 40, 40, dev([0, 8], torch.int32), dev([0, 39], torch.int32))
        x = torch.zeros(8, 4, 64, dtype=torch.bfloat16, device="cuda")
        kv = torch.zeros(40, 4, 64, dtype=torch.bfloat16, device="cuda")
        with pytest.raises(EbError) as err:
            eb_block_attn(r, x, x, x, kv, kv, torch.empty_like(x))
        assert "cu_prefix" in str(err.value)
    torch.cuda.synchronize()
