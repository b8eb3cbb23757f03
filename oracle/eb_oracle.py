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
  masked position passes (Sec. 5.2, Alg. 5), then commit x_i <- x_hat_i;
* LPS features     - the top-1/top-2 probability gap Delta, the normalised
  entropy H / ln|V|, the block-wise mask ratio rho and the intra-block position
  (i - b) / |B| (Sec. 5.2, Alg. 5), and the union accept rule
  kappa >= tau or p_psi > tau_psi with a caller-supplied router score p_psi;
* top-m commit     - the budgeted form of Eq. prelim-update: the threshold set
  together with the m most confident masked positions of the block;
* LBS post-pass    - candidate positions p_phi > 0.5 that do not predict EOS,
  the max-gap filter, the min-tokens fallback to the first L_B masked positions
  and the size fallback |M| <= L_min (Sec. 5.1, Alg. 5), with a caller-supplied
  router score p_phi;
* dual cache       - attention whose keys also include a cached suffix segment
  right of the block (Sec. 6.3, Tab. 6).

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
           "unmask_select", "decode_step", "lps_features", "unmask_select_lps",
           "unmask_select_topm", "lbs_select"]


def _f64(x) -> np.ndarray:
    return np.asarray(x).astype(np.float64, copy=False)


# --------------------------------------------------------------------------
# block attention
# --------------------------------------------------------------------------

def block_attention(q, k_blk, v_blk, k_pre, v_pre, cu_block, cu_prefix, hq: int, hkv: int,
                    scale: float | None = None, k_suf=None, v_suf=None,
                    cu_suffix=None) -> np.ndarray:
    """O[i, h] = sum_j softmax_j(q_i,h . k_j / sqrt(D)) v_j over the keys j of sequence b.

    The keys of sequence b are its cached prefix rows cu_prefix[b]:cu_prefix[b+1], its block
    rows cu_block[b]:cu_block[b+1] and, with a dual cache (Sec. 6.3), its cached suffix rows
    cu_suffix[b]:cu_suffix[b+1] (bidirectional: no causal mask and no masking by [MASK]
    state).  Query head h reads key/value head h // (hq // hkv).

    q [T, hq, D]; k_blk, v_blk [T, hkv, D]; k_pre, v_pre [S, hkv, D]; k_suf, v_suf [U, hkv, D]
    ->  O [T, hq, D] float64.
    """
    q, k_blk, v_blk, k_pre, v_pre = map(_f64, (q, k_blk, v_blk, k_pre, v_pre))
    dual = cu_suffix is not None
    if dual:
        k_suf, v_suf = _f64(k_suf), _f64(v_suf)
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
            kp = [k_pre[p0:p1, g, :], k_blk[b0:b1, g, :]]
            vp = [v_pre[p0:p1, g, :], v_blk[b0:b1, g, :]]
            if dual:
                u0, u1 = int(cu_suffix[b]), int(cu_suffix[b + 1])
                kp.append(k_suf[u0:u1, g, :])
                vp.append(v_suf[u0:u1, g, :])
            keys = np.concatenate(kp, axis=0)
            vals = np.concatenate(vp, axis=0)
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
    kappa = max_v p_v; H = -sum_{p_v > 0} p_v ln p_v (nats); top2_gap = p_(1) - p_(2), the
    largest minus the second largest probability counted with multiplicity (0 when the
    maximum is shared; p_(2) = 0 when V = 1), the LPS gap feature Delta (Sec. 5.2).
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
    if p.shape[1] >= 2:
        two = np.partition(p, p.shape[1] - 2, axis=1)[:, -2:]   # two largest, ascending
        gap = two[:, 1] - two[:, 0]
    else:
        gap = p[:, 0].copy()
    return {"conf": kappa, "entropy": H, "argmax": x_hat, "max_logit": m, "top2_gap": gap}


def lmhead_confidence(h, w, rows=None, v_chunk: int = 16384, row_chunk: int = 256) -> dict:
    """Statistics of z = W h for the given rows of h (all rows if rows is None).

    Logits are formed in fp64 chunk by chunk over the vocabulary (to bound the fp64 copy of W)
    and reduced per row with confidence_stats on the complete row.
    """
    h = np.asarray(h)
    idx = np.arange(h.shape[0]) if rows is None else np.asarray(rows, dtype=np.int64)
    V = w.shape[0]
    res = {"conf": np.empty(idx.size), "entropy": np.empty(idx.size),
           "argmax": np.empty(idx.size, dtype=np.int32), "max_logit": np.empty(idx.size),
           "top2_gap": np.empty(idx.size)}
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
# LPS features and the union accept rule
# --------------------------------------------------------------------------

def lps_features(conf, entropy, top2_gap, masked, cu_block, vocab: int, seq_pos=None) -> dict:
    """LPS router inputs of every block row (Sec. 5.2, Alg. 5).

    feat[i] = (kappa_i, H_i / ln|V|, Delta_i, rho_b) for row i of block b, where rho_b is the
    fraction of the block's rows still masked before this step's commit.  Empty blocks have
    rho = 0.

    pos[i] is the normalised intra-block position (i - b) / |B| of Sec. 5.2 and Alg. 5, with b
    the block's left boundary and |B| its size (len_b rows):
      * seq_pos given (the sequence position of every packed row, ascending within a block):
        pos[i] = (seq_pos[i] - seq_pos[b0]) / len_b with b0 the block's first row, i.e. the
        printed formula on sequence positions; for a block with gaps this exceeds 1 towards
        its right end;
      * seq_pos None: pos[i] = (i - b0) / len_b, the row's rank within the packed block, which
        is the printed formula when the block is contiguous and stays in [0, 1) otherwise.
    """
    conf, entropy, top2_gap = _f64(conf), _f64(entropy), _f64(top2_gap)
    T = len(conf)
    B = len(cu_block) - 1
    feat = np.zeros((T, 4), dtype=np.float64)
    pos = np.zeros(T, dtype=np.float64)
    rho = np.zeros(B, dtype=np.float64)
    lnv = np.log(float(vocab))
    for b in range(B):
        b0, b1 = int(cu_block[b]), int(cu_block[b + 1])
        n = b1 - b0
        if n == 0:
            continue
        rho[b] = sum(1 for i in range(b0, b1) if masked[i]) / n
        left = int(seq_pos[b0]) if seq_pos is not None else b0
        for i in range(b0, b1):
            feat[i] = (conf[i], entropy[i] / lnv, top2_gap[i], rho[b])
            where = int(seq_pos[i]) if seq_pos is not None else i
            pos[i] = (where - left) / n
    return {"feat": feat, "pos": pos, "mask_ratio": rho}


def _commit(accept_rows, argmax, masked_out, tokens_out, unmask):
    for i in accept_rows:
        tokens_out[i] = argmax[i]
        masked_out[i] = 0
        unmask[i] = 1


def unmask_select_lps(conf, argmax, masked, tokens, tau, cu_block, p_psi, tau_psi) -> dict:
    """Union accept rule of Alg. 5 per block b:

    A_b = {i masked : conf_i >= tau_b or p_psi_i > tau_psi}; if A_b is empty and some i is
    masked, A_b = {lowest i among the masked rows of maximal conf} (anti-stall fallback); then
    commit as in unmask_select.  p_psi (the router's commit probability) and tau_psi are fp32
    inputs compared as their exact fp64 widenings.
    """
    conf = _f64(conf)
    tau = np.asarray(tau, dtype=np.float32).astype(np.float64)
    p_psi = np.asarray(p_psi, dtype=np.float32).astype(np.float64)
    tau_psi = float(np.float32(tau_psi))
    masked_out = np.array(masked, dtype=np.uint8, copy=True)
    tokens_out = np.array(tokens, dtype=np.int32, copy=True)
    unmask = np.zeros(len(masked_out), dtype=np.uint8)
    B = len(cu_block) - 1
    n_commit = np.zeros(B, dtype=np.int32)
    resolved = np.zeros(B, dtype=np.uint8)
    for b in range(B):
        rows = range(int(cu_block[b]), int(cu_block[b + 1]))
        m_rows = [i for i in rows if masked_out[i]]
        accept = [i for i in m_rows if conf[i] >= tau[b] or p_psi[i] > tau_psi]
        if not accept and m_rows:
            best = max(conf[i] for i in m_rows)
            accept = [min(i for i in m_rows if conf[i] == best)]
        _commit(accept, argmax, masked_out, tokens_out, unmask)
        n_commit[b] = len(accept)
        resolved[b] = 1 if not any(masked_out[i] for i in rows) else 0
    return {"unmask": unmask, "tokens": tokens_out, "masked": masked_out,
            "n_commit": n_commit, "resolved": resolved}


# --------------------------------------------------------------------------
# top-m budget commit
# --------------------------------------------------------------------------

def unmask_select_topm(conf, argmax, masked, tokens, tau, cu_block, m: int) -> dict:
    """Budgeted block update of Eq. prelim-update per block b:

    A_b = {i masked : conf_i >= tau_b} united with Top-m_b, the m masked rows of largest conf
    (equal conf: lower row first; all masked rows if fewer than m).  With m = 0 this is the
    threshold rule, and then the anti-stall fallback of unmask_select applies.
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
        ranked = sorted(m_rows, key=lambda i: (-conf[i], i))
        top = set(ranked[:max(0, m)])
        accept = sorted(set(i for i in m_rows if conf[i] >= tau[b]) | top)
        if not accept and m_rows:
            best = max(conf[i] for i in m_rows)
            accept = [min(i for i in m_rows if conf[i] == best)]
        _commit(accept, argmax, masked_out, tokens_out, unmask)
        n_commit[b] = len(accept)
        resolved[b] = 1 if not any(masked_out[i] for i in rows) else 0
    return {"unmask": unmask, "tokens": tokens_out, "masked": masked_out,
            "n_commit": n_commit, "resolved": resolved}


# --------------------------------------------------------------------------
# LBS block selection post-pass
# --------------------------------------------------------------------------

def lbs_select(masked, p_phi, x_hat, eos_id: int, l_min: int, l_b: int, g_max: int) -> dict:
    """Block selection of the LBS router's post-pass (Sec. 5.1; Alg. 5) for each sequence.

    Inputs cover the generation window: masked, p_phi (the router's inclusion probability, an
    fp32 input compared with 0.5 exactly) and x_hat, each [n_seq, L].  For one sequence, with M
    its masked positions in ascending order:
      * a sequence with at most l_min masked positions takes all of them as its block;
      * otherwise the block is grown from the left over the masked positions the router
        includes (p_phi > 0.5) and whose predicted token is not eos_id; it stops before the
        first such position lying more than g_max positions after the last one taken, so
        positions past a wide gap never join;
      * a block grown this way with fewer than l_min positions is replaced by the l_b lowest
        positions of M.
    Returns the block as a 0/1 mask [n_seq, L] (u8), its size and its first position (-1 when
    empty).
    """
    masked = np.asarray(masked)
    p_phi = np.asarray(p_phi, dtype=np.float32).astype(np.float64)
    x_hat = np.asarray(x_hat)
    n, L = masked.shape
    block = np.zeros((n, L), dtype=np.uint8)
    size = np.zeros(n, dtype=np.int32)
    first = np.full(n, -1, dtype=np.int32)
    for s in range(n):
        M = [i for i in range(L) if masked[s, i]]
        if len(M) <= l_min:
            sel = M
        else:
            C = [i for i in M if p_phi[s, i] > 0.5 and int(x_hat[s, i]) != eos_id]
            sel = []
            for i in C:
                if sel and i - sel[-1] > g_max:
                    break
                sel.append(i)
            if len(sel) < l_min:
                sel = M[:l_b]
        for i in sel:
            block[s, i] = 1
        size[s] = len(sel)
        first[s] = sel[0] if sel else -1
    return {"block": block, "size": size, "first": first}


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
