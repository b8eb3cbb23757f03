"""Test-side helpers: seeded cases with away-from-tie margins enforced on the checked rows."""
from __future__ import annotations

import numpy as np

from oracle import margins
from workloads import make_step, widen_f64, bf16_bits_to_f32


def as_f32(x: np.ndarray, dtype: str) -> np.ndarray:
    """Exact float32 view of storage values (bf16 bits widen exactly)."""
    return bf16_bits_to_f32(x) if dtype == "bf16" else np.asarray(x, np.float32)


def enforce_margins(case, blocks=None, max_rounds=30):
    """Redraw the hidden-state noise of rows breaking a margin until none does (checked blocks only)."""
    w32 = as_f32(case.w, case.dtype)
    for _ in range(max_rounds):
        bad = margins.find_violations(as_f32(case.h, case.dtype), w32, case.cu_block,
                                      case.masked, case.tau, blocks)
        if bad.size == 0:
            return case
        case.redraw_h_rows(bad)
    raise RuntimeError("margins not reached after redraws")


def prepared(cfg, seed=None, blocks=None):
    return enforce_margins(make_step(cfg, seed), blocks)


def oracle_args(case, rows_of=None):
    """Exact float32 copies of the step's float inputs, for the fp64 oracle."""
    dt = case.dtype
    return dict(q=as_f32(case.q, dt), k_blk=as_f32(case.k_blk, dt), v_blk=as_f32(case.v_blk, dt),
                k_pre=as_f32(case.k_pre, dt), v_pre=as_f32(case.v_pre, dt),
                h=as_f32(case.h, dt), w=as_f32(case.w, dt))
