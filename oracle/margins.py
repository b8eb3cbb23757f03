"""Away-from-tie margins for exact comparisons (test infrastructure only).

A GPU path that accumulates logits in fp32 may differ from the fp64 oracle by
~1e-5 in a logit.  Integer decisions (the vocabulary argmax, kappa >= tau, the
fallback argmax over kappa) are compared bit-exactly only on inputs whose fp64
values sit clear of every decision boundary:

  (i)   argmax margin   top-1 minus top-2 logit >= ARGMAX_GAP for every checked row;
  (ii)  threshold margin |kappa - tau_b| >= TAU_GAP for every checked masked row;
  (iii) fallback margin in a block where no masked row passes tau, ln kappa of the
        best masked row minus that of the runner-up >= FALLBACK_GAP.

find_violations() names the offending rows; the caller redraws their noise.
"""
from __future__ import annotations

import numpy as np

ARGMAX_GAP = 4e-3
TAU_GAP = 1e-3
FALLBACK_GAP = 4e-3


def _row_logit_stats(h, w, rows, v_chunk=16384, row_chunk=256):
    rows = np.asarray(rows, dtype=np.int64)
    V = w.shape[0]
    top1 = np.empty(rows.size)
    top2 = np.empty(rows.size)
    lnkappa = np.empty(rows.size)
    for r0 in range(0, rows.size, row_chunk):
        sel = rows[r0:r0 + row_chunk]
        hs = np.asarray(h[sel]).astype(np.float64)
        z = np.empty((sel.size, V))
        for v0 in range(0, V, v_chunk):
            z[:, v0:v0 + v_chunk] = hs @ np.asarray(w[v0:v0 + v_chunk]).astype(np.float64).T
        part = -np.partition(-z, 1, axis=1)[:, :2] if V > 1 else np.concatenate([z, z - np.inf], 1)
        m = part[:, 0]
        top1[r0:r0 + sel.size] = m
        top2[r0:r0 + sel.size] = part[:, 1]
        lnkappa[r0:r0 + sel.size] = -np.log(np.exp(z - m[:, None]).sum(axis=1))
    return top1, top2, lnkappa


def find_violations(h, w, cu_block, masked, tau, blocks=None) -> np.ndarray:
    """Rows (global indices) of the given blocks (all if None) that break a margin."""
    B = len(cu_block) - 1
    blocks = range(B) if blocks is None else blocks
    bad = []
    for b in blocks:
        r0, r1 = int(cu_block[b]), int(cu_block[b + 1])
        if r1 == r0:
            continue
        rows = np.arange(r0, r1)
        top1, top2, lnk = _row_logit_stats(h, w, rows)
        bad.extend(rows[(top1 - top2) < ARGMAX_GAP].tolist())
        mk = np.asarray(masked[r0:r1]).astype(bool)
        t = float(np.float32(tau[b]))
        kappa = np.exp(lnk)
        bad.extend(rows[mk & (np.abs(kappa - t) < TAU_GAP)].tolist())
        if mk.any() and not (mk & (kappa >= t)).any():
            cand = np.sort(lnk[mk])[::-1]
            if cand.size >= 2 and cand[0] - cand[1] < FALLBACK_GAP:
                mrows = rows[mk]
                order = np.argsort(-lnk[mk], kind="stable")
                bad.extend(mrows[order[:2]].tolist())
    return np.unique(np.asarray(bad, dtype=np.int64))
