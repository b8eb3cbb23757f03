"""Plain fp64 CPU oracle for one Early-Bird denoising step.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and
the benchmark's CPU-baseline leg may import or call this module; the HIP
product path never does, and shares no code with it.

Everything here is the plain definition of what a denoising step computes,
written with numpy float64 and no blocking, fusion or streaming beyond what
the definitions state:

* block attention  - bidirectional softmax attention of the active block's
  queries over the cached prefix keys and the block's own keys (Sec. 3 and
  App. B: the mask predictor is a bidirectional Transformer; Sec. 6.3: prefix
  KV cache to the left of the leftmost selected position);
* LM head          - logits z = W h for every block position (Alg. 5, the
  softmax of the backbone output);
* confidence stats - kappa = max_v p(v) (Eq. app-confidence), greedy token
  x_hat = argmax_v p(v) (Alg. 5), Shannon entropy H = -sum p ln p in nats,
  whose normalised form H / ln|V| is the LBS router input (Sec. 5.1);
* unmask           - the threshold commit rule kappa >= tau (Eq. prelim-update,
  union accept rule of Alg. 5 without the router term) with the anti-stall
  fallback that commits the single most confident masked position when no
  masked position passes (Sec. 5.2, Alg. 5), then commit x_i <- x_hat_i.

Readings where the paper is silent: ties in the vocabulary argmax go to the
lowest token id; ties in the fallback argmax go to the lowest packed block
position; 0 ln 0 = 0; tau is compared as the exact fp64 widening of its fp32
value; every block position is scored, masked-ness only enters the unmask rule;
K/V arrive after any positional encoding; the key/value head of query head h is
h // (hq / hkv).
"""
from __future__ import annotations

import numpy as np

__all__ = ["block_attention", "lmhead_logits", "confidence_stats", "lmhead_confidence",
           "unmask_select", "decode_step"]


def _f64(x) -> np.ndarray:
    return np.asarray(x).astype(np.float64, copy=False)


# --------------------------------------------------------------------------
# block attention
# --------------------------------------------------------------------------

def block_attention(q, k_blk, v_blk, k_pre, v_pre, cu_block, cu_prefix, hq: int, hkv: int,
                    scale: float | None = None) -> np.ndarray:
    """O[i, h] = sum_j softmax_j(q_i,h . k_j / sqrt(D)) v_j over the keys j of sequence b.

    The keys of sequence b are its cached prefix rows cu_prefix[b]:cu_prefix[b+1] followed by
    its block rows cu_block[b]:cu_block[b+1] (bidirectional: no causal mask and no masking by
    [MASK] state).  Query head h reads key/value head h // (hq // hkv).

    q [T, hq, D]; k_blk, v_blk [T, hkv, D]; k_pre, v_pre [S, hkv, D]  ->  O [T, hq, D] float64.
    """
    q, k_blk, v_blk, k_pre, v_pre = map(_f64, (q, k_blk, v_blk, k_pre, v_pre))
    T, _, D = q.shape
    if scale is None:
        scale = 1.0 / np.sqrt(D)
    group = hq // hkv
    out = np.zeros((T, hq, D), dtype=np.float64)
    B = len(cu_block) - 1
    for b in range(B):
        b0, b1 = int(cu_block[b]), int(cu_block[b + 1])
        p0, p1 = int(cu_prefix[b]), int(cu_prefix[b + 1])
        if b1 == b0:
            continue
        for h in range(hq):
            g = h // group
            keys = np.concatenate([k_pre[p0:p1, g, :], k_blk[b0:b1, g, :]], axis=0)
            vals = np.concatenate([v_pre[p0:p1, g, :], v_blk[b0:b1, g, :]], axis=0)
            s = (q[b0:b1, h, :] @ keys.T) * scale                  # [len, nkeys]
            s = s - s.max(axis=1, keepdims=True)
            p = np.exp(s)
            p /= p.sum(axis=1, keepdims=True)
            out[b0:b1, h, :] = p @ vals
    return out


# --------------------------------------------------------------------------
# LM head and per-position statistics
# --------------------------------------------------------------------------

def lmhead_logits(h, w) -> np.ndarray:
    """z[i, v] = sum_k W[v, k] h[i, k]  (W in the [V, d] nn.Linear layout)."""
    return _f64(h) @ _f64(w).T


def confidence_stats(z) -> dict:
    """Two-pass statistics of each row of logits z [n, V].

    m = max z; x_hat = lowest v with z_v = m; p = exp(z - m) / sum exp(z - m);
    kappa = max_v p_v; H = -sum_{p_v > 0} p_v ln p_v (nats).
    """
    z = _f64(z)
    m = z.max(axis=1)
    x_hat = np.argmax(z, axis=1).astype(np.int32)        # first maximal index
    e = np.exp(z - m[:, None])
    p = e / e.sum(axis=1, keepdims=True)
    kappa = p.max(axis=1)
    with np.errstate(divide="ignore", invalid="ignore"):
        plogp = np.where(p > 0, p * np.log(np.where(p > 0, p, 1.0)), 0.0)
    H = -plogp.sum(axis=1)
    return {"conf": kappa, "entropy": H, "argmax": x_hat, "max_logit": m}


def lmhead_confidence(h, w, rows=None, v_chunk: int = 16384, row_chunk: int = 256) -> dict:
    """Statistics of z = W h for the given rows of h (all rows if rows is None).

    Logits are formed in fp64 chunk by chunk over the vocabulary (to bound the fp64 copy of W)
    and reduced per row with confidence_stats on the complete row.
    """
    h = np.asarray(h)
    idx = np.arange(h.shape[0]) if rows is None else np.asarray(rows, dtype=np.int64)
    V = w.shape[0]
    res = {"conf": np.empty(idx.size), "entropy": np.empty(idx.size),
           "argmax": np.empty(idx.size, dtype=np.int32), "max_logit": np.empty(idx.size)}
    for r0 in range(0, idx.size, row_chunk):
        sel = idx[r0:r0 + row_chunk]
        hs = _f64(h[sel])
        z = np.empty((sel.size, V), dtype=np.float64)
        for v0 in range(0, V, v_chunk):
            z[:, v0:v0 + v_chunk] = hs @ _f64(w[v0:v0 + v_chunk]).T
        st = confidence_stats(z)
        for k in res:
            res[k][r0:r0 + sel.size] = st[k]
    return res


# --------------------------------------------------------------------------
# threshold unmask with anti-stall fallback
# --------------------------------------------------------------------------

def unmask_select(conf, argmax, masked, tokens, tau, cu_block) -> dict:
    """Per block b (rows cu_block[b]:cu_block[b+1]):

    A_b = {i masked : conf_i >= tau_b}; if A_b is empty and some i is masked,
    A_b = {lowest i among the masked rows of maximal conf}.  For i in A_b:
    tokens_i <- argmax_i, masked_i <- 0, unmask_i <- 1.  n_commit_b = |A_b|;
    resolved_b = 1 iff no masked row is left in the block.
    """
    conf = _f64(conf)
    tau = np.asarray(tau, dtype=np.float32).astype(np.float64)
    masked_out = np.array(masked, dtype=np.uint8, copy=True)
    tokens_out = np.array(tokens, dtype=np.int32, copy=True)
    unmask = np.zeros(len(masked_out), dtype=np.uint8)
    B = len(cu_block) - 1
    n_commit = np.zeros(B, dtype=np.int32)
    resolved = np.zeros(B, dtype=np.uint8)
    for b in range(B):
        rows = range(int(cu_block[b]), int(cu_block[b + 1]))
        m_rows = [i for i in rows if masked_out[i]]
        accept = [i for i in m_rows if conf[i] >= tau[b]]
        if not accept and m_rows:
            best = max(conf[i] for i in m_rows)
            accept = [min(i for i in m_rows if conf[i] == best)]
        for i in accept:
            tokens_out[i] = argmax[i]
            masked_out[i] = 0
            unmask[i] = 1
        n_commit[b] = len(accept)
        resolved[b] = 1 if not any(masked_out[i] for i in rows) else 0
    return {"unmask": unmask, "tokens": tokens_out, "masked": masked_out,
            "n_commit": n_commit, "resolved": resolved}


# --------------------------------------------------------------------------
# one whole step
# --------------------------------------------------------------------------

def decode_step(q, k_blk, v_blk, k_pre, v_pre, cu_block, cu_prefix, hq, hkv, h, w,
                masked, tokens, tau) -> dict:
    """Attention output, per-position statistics of the LM head, and the unmask result."""
    out = {"attn": block_attention(q, k_blk, v_blk, k_pre, v_pre, cu_block, cu_prefix, hq, hkv)}
    st = lmhead_confidence(h, w)
    out.update(st)
    out.update(unmask_select(st["conf"], st["argmax"], masked, tokens, tau, cu_block))
    return out
