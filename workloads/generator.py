"""Seeded synthetic inputs for one denoising step over ragged active blocks.

This module draws inputs only.  It holds none of the step's arithmetic
(no attention, no logits, no softmax statistics, no unmask rule); both the
fp64 oracle and the HIP path consume what it returns.

The paper's workloads (generation length 512, base block 32, threshold 0.9,
LLaDA-8B / Dream-7B backbones; Sec. 6 and App. F) cannot be reproduced here:
no weights, routers or benchmark items exist.  A step is therefore emulated:

* Block hidden states come in contiguous runs of "easy" and "hard" positions
  (the staircase entropy pattern of Sec. 4, Fig. 2).  An easy position of
  target token t has h = 8 * u_t + n with u_t = 16 * W_t / ||W_t||_2 and
  n ~ N(0, I_d); a hard position has h = n.  Easy rows are near one-hot
  (kappa ~ 1, H ~ 0), hard rows near uniform.
* Block lengths may differ per sequence (variable-length blocks chosen by the
  learnable block selector, Sec. 5.1).
* Q, K, V of one attention layer and the cached prefix K/V are N(0, 1).
* W ~ N(0, 1/d) in the nn.Linear layout [V, d].

Draw order (frozen; VERSION names it).  The sequential generator
default_rng(seed) draws: block lengths -> prefix lengths -> masks ->
thresholds -> unmasked token ids -> easy/hard labels -> targets -> later
redraws of h rows.  The large normal arrays (Q, K_blk, V_blk, K_pre, V_pre,
W, h noise) each come from their own counter-keyed streams
default_rng([seed, stream, chunk]), filled in parallel.
"""
from __future__ import annotations

import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import Optional, Sequence

import numpy as np

VERSION = "eb-workload-1"


# --------------------------------------------------------------------------
# storage helpers (input decoding only)
# --------------------------------------------------------------------------

def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round finite float32 values to bfloat16 (round-to-nearest-even); return raw bits as uint16."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    b = x.view(np.uint32)
    r = (b >> np.uint32(16)) & np.uint32(1)
    r += np.uint32(0x7FFF)
    r += b                      # finite inputs: b + 0x8000 stays below 2**32
    r >>= np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(u: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bit patterns to float32 exactly."""
    u = np.ascontiguousarray(u, dtype=np.uint16)
    return (u.astype(np.uint32) << np.uint32(16)).view(np.float32)


def to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    """fp32/fp64 values -> storage form: float32 for 'f32', bf16 bits (uint16) for 'bf16'."""
    x32 = np.asarray(x, dtype=np.float32)
    if dtype == "f32":
        return np.ascontiguousarray(x32)
    if dtype == "bf16":
        return f32_to_bf16_bits(x32)
    raise ValueError(f"unknown dtype {dtype!r}")


def widen_f64(x: np.ndarray, dtype: str) -> np.ndarray:
    """Storage form -> exact float64 values."""
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        return bf16_bits_to_f32(x).astype(np.float64)
    raise ValueError(f"unknown dtype {dtype!r}")


# --------------------------------------------------------------------------
# configurations
# --------------------------------------------------------------------------

@dataclass(frozen=True)
class StepConfig:
    """Shape and distribution of one synthetic denoising step.

    block_len: ("fixed", n) | ("choice", (n0, n1, ...)) | ("uniform", lo, hi)  (inclusive)
    prefix_len: same forms as block_len
    run_max: easy/hard runs have integer lengths uniform on [2, run_max];
             None means one fair-coin label per whole block.
    mask: ("bernoulli", p) each position masked with prob p;
          ("fraction", lo, hi) per sequence f ~ U[lo, hi], exactly round(f*len) masked.
    taus: thresholds; one value = fixed, several = uniform choice per sequence.
    """
    name: str
    seed: int
    batch: int
    hq: int
    hkv: int
    head_dim: int
    hidden: int
    vocab: int
    block_len: tuple
    prefix_len: tuple
    run_max: Optional[int]
    mask: tuple
    taus: tuple
    dtype: str
    description: str = ""


CONFIGS = {
    c.name: c for c in [
        StepConfig(
            name="tiny_f32_b1", seed=1001, batch=1, hq=4, hkv=4, head_dim=64,
            hidden=256, vocab=2048, block_len=("fixed", 32), prefix_len=("fixed", 96),
            run_max=8, mask=("bernoulli", 0.5), taus=(0.9,), dtype="f32",
            description="tiny fp32 step: 4x64 heads, d=256, V=2048, prefix 96, block 32"),
        StepConfig(
            name="llada8b_b1", seed=1002, batch=1, hq=32, hkv=32, head_dim=128,
            hidden=4096, vocab=126464, block_len=("fixed", 32), prefix_len=("fixed", 512),
            run_max=16, mask=("bernoulli", 0.5), taus=(0.9,), dtype="bf16",
            description="LLaDA-8B-shaped step, batch 1: 32x128 heads, V=126464, prefix 512, block 32"),
        StepConfig(
            name="llada8b_b16", seed=1003, batch=16, hq=32, hkv=32, head_dim=128,
            hidden=4096, vocab=126464, block_len=("fixed", 64), prefix_len=("fixed", 1024),
            run_max=16, mask=("fraction", 0.2, 1.0), taus=(0.9,), dtype="bf16",
            description="LLaDA-8B-shaped step, batch 16: prefix 1024, block 64, masked fraction U[0.2,1]"),
        StepConfig(
            name="llada8b_ragged_b32", seed=1004, batch=32, hq=32, hkv=32, head_dim=128,
            hidden=4096, vocab=126464, block_len=("choice", tuple(range(8, 129, 8))),
            prefix_len=("fixed", 2048), run_max=None, mask=("bernoulli", 0.5),
            taus=(0.7, 0.8, 0.9), dtype="bf16",
            description="LLaDA-8B-shaped ragged step, batch 32: prefix 2048, blocks {8..128 step 8}, "
                        "homogeneous blocks, tau in {0.7,0.8,0.9}"),
        StepConfig(
            name="dream7b_b64", seed=1005, batch=64, hq=28, hkv=4, head_dim=128,
            hidden=3584, vocab=152064, block_len=("uniform", 16, 256), prefix_len=("fixed", 4096),
            run_max=32, mask=("bernoulli", 0.5), taus=(0.9,), dtype="bf16",
            description="Dream-7B-shaped GQA step, batch 64: 28/4x128 heads, V=152064, prefix 4096, "
                        "blocks U[16,256]"),
    ]
}


# --------------------------------------------------------------------------
# the case object
# --------------------------------------------------------------------------

@dataclass
class StepCase:
    cfg: StepConfig
    block_lens: np.ndarray      # [B] int32
    prefix_lens: np.ndarray     # [B] int32
    cu_block: np.ndarray        # [B+1] int32
    cu_prefix: np.ndarray       # [B+1] int32
    masked: np.ndarray          # [T] uint8 (1 = position still [MASK])
    tokens: np.ndarray          # [T] int32 (-1 at masked positions)
    tau: np.ndarray             # [B] float32
    q: np.ndarray               # [T, hq, D]   storage dtype
    k_blk: np.ndarray           # [T, hkv, D]
    v_blk: np.ndarray           # [T, hkv, D]
    k_pre: np.ndarray           # [S, hkv, D]
    v_pre: np.ndarray           # [S, hkv, D]
    w: np.ndarray               # [V, d]
    h: np.ndarray               # [T, d]
    easy: np.ndarray            # [T] bool
    target: np.ndarray          # [T] int32 (token the easy rows point at; -1 for hard rows)
    rng: np.random.Generator = field(repr=False)
    redraws: int = 0

    @property
    def dtype(self) -> str:
        return self.cfg.dtype

    @property
    def T(self) -> int:
        return int(self.cu_block[-1])

    @property
    def S(self) -> int:
        return int(self.cu_prefix[-1])

    @property
    def batch(self) -> int:
        return int(self.cfg.batch)

    def redraw_h_rows(self, rows: Sequence[int]) -> None:
        """Redraw the N(0, I) noise of the given rows (ascending order), keeping labels/targets."""
        rows = np.unique(np.asarray(rows, dtype=np.int64))
        if rows.size == 0:
            return
        d = self.cfg.hidden
        noise = self.rng.standard_normal((rows.size, d), dtype=np.float32)
        self.h[rows] = _hidden_rows(noise, self.easy[rows], self.target[rows], self.w, self.dtype)
        self.redraws += int(rows.size)


# --------------------------------------------------------------------------
# drawing
# --------------------------------------------------------------------------

def _draw_lens(rng: np.random.Generator, spec: tuple, n: int) -> np.ndarray:
    kind = spec[0]
    if kind == "fixed":
        return np.full(n, int(spec[1]), dtype=np.int32)
    if kind == "choice":
        vals = np.asarray(spec[1], dtype=np.int32)
        return vals[rng.integers(0, vals.size, size=n)].astype(np.int32)
    if kind == "uniform":
        return rng.integers(int(spec[1]), int(spec[2]) + 1, size=n).astype(np.int32)
    raise ValueError(f"unknown length spec {spec!r}")


def _cu(lens: np.ndarray) -> np.ndarray:
    cu = np.zeros(lens.size + 1, dtype=np.int64)
    np.cumsum(lens, out=cu[1:])
    if cu[-1] > np.iinfo(np.int32).max:
        raise ValueError("ragged total exceeds int32")
    return cu.astype(np.int32)


_CHUNK = 1 << 22          # elements per independent normal stream chunk
_STREAM = {"q": 1, "k_blk": 2, "v_blk": 3, "k_pre": 4, "v_pre": 5, "w": 6, "h_noise": 7,
           "k_suf": 8, "v_suf": 9}


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def _normal_stream(seed: int, stream: str, shape, scale: float, dtype: str) -> np.ndarray:
    """N(0, scale^2) array in storage form.

    Chunk c (of _CHUNK flat elements) is drawn from default_rng([seed, stream_id, c]), so the
    values do not depend on how many threads fill them.
    """
    n = int(np.prod(shape, dtype=np.int64))
    out = np.empty(n, dtype=np.float32 if dtype == "f32" else np.uint16)
    sid = _STREAM[stream]

    def fill(c: int) -> None:
        lo, hi = c * _CHUNK, min(n, (c + 1) * _CHUNK)
        g = np.random.default_rng([seed, sid, c])
        x = g.standard_normal(hi - lo, dtype=np.float32)
        if scale != 1.0:
            x *= np.float32(scale)
        out[lo:hi] = to_storage(x, dtype)

    nchunks = (n + _CHUNK - 1) // _CHUNK
    if nchunks <= 1:
        for c in range(nchunks):
            fill(c)
    else:
        with ThreadPoolExecutor(_threads()) as ex:
            list(ex.map(fill, range(nchunks)))
    return out.reshape(shape)


def _unit_rows_scaled(w_store: np.ndarray, rows: np.ndarray, dtype: str) -> np.ndarray:
    """16 * W_t / ||W_t||_2 for the given rows of the rounded W, in float64."""
    wt = widen_f64(w_store[rows], dtype)
    nrm = np.sqrt(np.sum(wt * wt, axis=1, keepdims=True))
    nrm[nrm == 0] = 1.0
    return 16.0 * wt / nrm


def _hidden_rows(noise: np.ndarray, easy: np.ndarray, target: np.ndarray,
                 w_store: np.ndarray, dtype: str) -> np.ndarray:
    h = noise.astype(np.float64)
    idx = np.nonzero(easy)[0]
    chunk = 4096
    for s in range(0, idx.size, chunk):
        sel = idx[s:s + chunk]
        h[sel] += 8.0 * _unit_rows_scaled(w_store, target[sel], dtype)
    return to_storage(h.astype(np.float32), dtype)


def make_step(cfg: StepConfig | str, seed: Optional[int] = None) -> StepCase:
    """Draw one synthetic step for `cfg` (a StepConfig or a name in CONFIGS)."""
    if isinstance(cfg, str):
        cfg = CONFIGS[cfg]
    if cfg.hq % cfg.hkv:
        raise ValueError("hq must be a multiple of hkv")
    seed_used = int(cfg.seed if seed is None else seed)
    rng = np.random.default_rng(seed_used)
    B = cfg.batch

    # 1. lengths
    block_lens = _draw_lens(rng, cfg.block_len, B)
    prefix_lens = _draw_lens(rng, cfg.prefix_len, B)
    cu_block, cu_prefix = _cu(block_lens), _cu(prefix_lens)
    T, S = int(cu_block[-1]), int(cu_prefix[-1])

    # 2. masks
    kind = cfg.mask[0]
    if kind == "bernoulli":
        masked = (rng.random(T) < float(cfg.mask[1])).astype(np.uint8)
    elif kind == "fraction":
        masked = np.zeros(T, dtype=np.uint8)
        lo, hi = float(cfg.mask[1]), float(cfg.mask[2])
        for b in range(B):
            n = int(block_lens[b])
            f = rng.uniform(lo, hi)
            k = int(round(f * n))
            pick = rng.choice(n, size=k, replace=False) if k > 0 else np.zeros(0, np.int64)
            masked[cu_block[b] + pick] = 1
    else:
        raise ValueError(f"unknown mask spec {cfg.mask!r}")

    # 3. thresholds
    taus = np.asarray(cfg.taus, dtype=np.float32)
    if taus.size == 1:
        tau = np.full(B, taus[0], dtype=np.float32)
    else:
        tau = taus[rng.integers(0, taus.size, size=B)].astype(np.float32)

    # 4. token ids already committed at unmasked positions
    tokens = rng.integers(0, cfg.vocab, size=T).astype(np.int32)
    tokens[masked.astype(bool)] = -1

    # 5. attention operands (independent seeded streams)
    D, hq, hkv = cfg.head_dim, cfg.hq, cfg.hkv
    q = _normal_stream(seed_used, "q", (T, hq, D), 1.0, cfg.dtype)
    k_blk = _normal_stream(seed_used, "k_blk", (T, hkv, D), 1.0, cfg.dtype)
    v_blk = _normal_stream(seed_used, "v_blk", (T, hkv, D), 1.0, cfg.dtype)
    k_pre = _normal_stream(seed_used, "k_pre", (S, hkv, D), 1.0, cfg.dtype)
    v_pre = _normal_stream(seed_used, "v_pre", (S, hkv, D), 1.0, cfg.dtype)

    # 6. LM-head weight W ~ N(0, 1/d), nn.Linear layout [V, d]
    V, d = cfg.vocab, cfg.hidden
    w = _normal_stream(seed_used, "w", (V, d), float(1.0 / np.sqrt(d)), cfg.dtype)

    # 7. easy/hard labels (runs alternate, starting from a fair coin)
    easy = np.zeros(T, dtype=bool)
    for b in range(B):
        n = int(block_lens[b])
        base = int(cu_block[b])
        label = bool(rng.integers(0, 2))
        if cfg.run_max is None:
            easy[base:base + n] = label
            continue
        pos = 0
        while pos < n:
            run = int(rng.integers(2, cfg.run_max + 1))
            easy[base + pos: base + min(n, pos + run)] = label
            pos += run
            label = not label

    # 8. targets
    target = rng.integers(0, V, size=T).astype(np.int32)
    target[~easy] = -1

    # 9. hidden states
    noise = _normal_stream(seed_used, "h_noise", (T, d), 1.0, "f32")
    h = _hidden_rows(noise, easy, target, w, cfg.dtype)

    return StepCase(cfg=cfg, block_lens=block_lens, prefix_lens=prefix_lens,
                    cu_block=cu_block, cu_prefix=cu_prefix, masked=masked, tokens=tokens,
                    tau=tau, q=q, k_blk=k_blk, v_blk=v_blk, k_pre=k_pre, v_pre=v_pre,
                    w=w, h=h, easy=easy, target=target, rng=rng)


def custom_config(name: str = "custom", *, seed: int = 7, batch: int = 1, hq: int = 4, hkv: int = 4,
                  head_dim: int = 64, hidden: int = 256, vocab: int = 2048,
                  block_len: tuple = ("fixed", 32), prefix_len: tuple = ("fixed", 96),
                  run_max: Optional[int] = 8, mask: tuple = ("bernoulli", 0.5),
                  taus: tuple = (0.9,), dtype: str = "bf16") -> StepConfig:
    """A StepConfig for test shapes that are not one of the named workloads."""
    return StepConfig(name=name, seed=seed, batch=batch, hq=hq, hkv=hkv, head_dim=head_dim,
                      hidden=hidden, vocab=vocab, block_len=block_len, prefix_len=prefix_len,
                      run_max=run_max, mask=mask, taus=taus, dtype=dtype)


# --------------------------------------------------------------------------------------------
# Router-score stand-ins.  The LBS and LPS routers are trained networks (absent here); the
# post-passes that consume their outputs take the scores as inputs.  These draws are uniform on
# [0, 1) in float32 from their own counter-keyed streams, so they never shift the step's draws.
# --------------------------------------------------------------------------------------------
def router_scores(seed: int, stream: str, shape) -> np.ndarray:
    """Seeded float32 scores on [0, 1), e.g. stream "p_psi" (one per block row) or "p_phi"."""
    key = sum(ord(c) * 131 ** i for i, c in enumerate(stream)) % (2 ** 31)
    rng = np.random.default_rng([seed, 7, key])
    return rng.random(shape, dtype=np.float32)


def suffix_segment(seed: int, suffix_lens, hkv: int, head_dim: int, dtype: str):
    """Seeded cached-suffix keys/values (the context right of the block, for dual-cache
    attention): N(0, 1) entries in the storage dtype from their own streams.  Returns
    (cu_suffix int32 [B+1], k_suf, v_suf [U, hkv, head_dim])."""
    lens = np.asarray(suffix_lens, dtype=np.int64)
    cu = _cu(lens)
    U = int(cu[-1])
    k = _normal_stream(seed, "k_suf", (U, hkv, head_dim), 1.0, dtype)
    v = _normal_stream(seed, "v_suf", (U, hkv, head_dim), 1.0, dtype)
    return cu, k, v


def lbs_window(seed: int, n_seq: int, window: int, vocab: int, eos_id: int):
    """Seeded inputs of the LBS post-pass over a generation window: per sequence a decoding
    progress f ~ U[0, 1] (positions left of f * window mostly committed, masked fraction 0.9
    to the right), router probabilities p_phi from router_scores, and predicted tokens that are
    uniform ids except an EOS tail (from a per-sequence start in the last 40% of the window),
    where the predictions concentrate on EOS at the end of the response (App. H)."""
    rng = np.random.default_rng([seed, 11])
    masked = np.zeros((n_seq, window), dtype=np.uint8)
    x_hat = rng.integers(0, vocab, (n_seq, window)).astype(np.int32)
    x_hat[x_hat == eos_id] = (eos_id + 1) % vocab
    pos = np.arange(window)
    for s in range(n_seq):
        f = rng.random()
        left = rng.random(window) < 0.05
        right = rng.random(window) < 0.9
        masked[s] = np.where(pos < int(f * window), left, right).astype(np.uint8)
        tail = int(window * (0.6 + 0.4 * rng.random()))
        x_hat[s, tail:] = eos_id
    p_phi = router_scores(seed, "p_phi", (n_seq, window))
    return masked, p_phi, x_hat
