"""ctypes binding of libeb.so (include/eb.h), same entry-point names.

Argument marshalling only: torch tensors supply device memory and the current HIP stream;
every step of the computation runs in the library's kernels.  Shapes of the tensors are
checked here against the host-side sizes before a call, because the library cannot see the
extent of a device allocation.  If libeb.so has not been built, loading raises.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libeb.so")

EB_F32, EB_BF16 = 0, 1
EB_OK, EB_ERR_INVALID, EB_ERR_UNSUPPORTED, EB_ERR_WORKSPACE, EB_ERR_HIP = 0, 1, 2, 3, 4

_P = ctypes.c_void_p


class eb_ragged(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("total_block", ctypes.c_int32),
                ("max_block", ctypes.c_int32), ("total_prefix", ctypes.c_int32),
                ("max_prefix", ctypes.c_int32), ("cu_block", _P), ("cu_prefix", _P)]


class eb_suffix(ctypes.Structure):
    _fields_ = [("total_suffix", ctypes.c_int32), ("max_suffix", ctypes.c_int32),
                ("cu_suffix", _P)]


class eb_step_trace(ctypes.Structure):
    _fields_ = [("attn_begin", _P), ("attn_end", _P), ("lmhead_begin", _P), ("lmhead_end", _P),
                ("select_begin", _P), ("select_end", _P)]


class eb_step_desc(ctypes.Structure):
    _fields_ = [("dtype", ctypes.c_int), ("ragged", eb_ragged),
                ("hq", ctypes.c_int32), ("hkv", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("attn_scale", ctypes.c_float),
                ("q", _P), ("k_blk", _P), ("v_blk", _P), ("k_pre", _P), ("v_pre", _P),
                ("attn_out", _P),
                ("hidden", ctypes.c_int32), ("vocab", ctypes.c_int32),
                ("h", _P), ("w", _P), ("conf", _P), ("entropy_nats", _P), ("argmax", _P),
                ("max_logit", _P),
                ("tau", _P), ("masked", _P), ("tokens", _P), ("unmask", _P),
                ("n_commit", _P), ("resolved", _P), ("trace", ctypes.POINTER(eb_step_trace))]


EXPORTS = {
    "eb_block_attn_workspace": (ctypes.c_size_t, [ctypes.c_int, ctypes.POINTER(eb_ragged),
                                                  ctypes.c_int, ctypes.c_int, ctypes.c_int]),
    "eb_block_attn": (ctypes.c_int, [ctypes.c_int, ctypes.POINTER(eb_ragged), ctypes.c_int,
                                     ctypes.c_int, ctypes.c_int, ctypes.c_float, _P, _P, _P, _P,
                                     _P, _P, _P, ctypes.c_size_t, _P]),
    "eb_block_attn_dual_workspace": (ctypes.c_size_t, [ctypes.c_int, ctypes.POINTER(eb_ragged),
                                                       ctypes.POINTER(eb_suffix), ctypes.c_int,
                                                       ctypes.c_int, ctypes.c_int]),
    "eb_block_attn_dual": (ctypes.c_int, [ctypes.c_int, ctypes.POINTER(eb_ragged),
                                          ctypes.POINTER(eb_suffix), ctypes.c_int, ctypes.c_int,
                                          ctypes.c_int, ctypes.c_float, _P, _P, _P, _P, _P, _P,
                                          _P, _P, _P, ctypes.c_size_t, _P]),
    "eb_lmhead_workspace": (ctypes.c_size_t, [ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                              ctypes.c_int]),
    "eb_lmhead_confidence": (ctypes.c_int, [ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                            ctypes.c_int, _P, _P, _P, _P, _P, _P, _P,
                                            ctypes.c_size_t, _P]),
    "eb_unmask_select": (ctypes.c_int, [ctypes.POINTER(eb_ragged), _P, _P, _P, _P, _P, _P, _P,
                                        _P, _P]),
    "eb_lmhead_features_workspace": (ctypes.c_size_t, [ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                                       ctypes.c_int]),
    "eb_lmhead_features": (ctypes.c_int, [ctypes.c_int, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                          _P, _P, _P, _P, _P, _P, _P, _P, ctypes.c_size_t, _P]),
    "eb_lps_features": (ctypes.c_int, [ctypes.POINTER(eb_ragged), ctypes.c_int, _P, _P, _P, _P,
                                       _P, _P, _P, _P, _P]),
    "eb_unmask_select_lps": (ctypes.c_int, [ctypes.POINTER(eb_ragged), _P, _P, _P, _P,
                                            ctypes.c_float, _P, _P, _P, _P, _P, _P]),
    "eb_unmask_select_topm": (ctypes.c_int, [ctypes.POINTER(eb_ragged), _P, _P, _P,
                                             ctypes.c_int32, _P, _P, _P, _P, _P, _P]),
    "eb_lbs_select": (ctypes.c_int, [ctypes.c_int32, ctypes.c_int32, _P, _P, _P, ctypes.c_int32,
                                     ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, _P, _P, _P,
                                     _P]),
    "eb_decode_step_workspace": (ctypes.c_size_t, [ctypes.POINTER(eb_step_desc)]),
    "eb_decode_step": (ctypes.c_int, [ctypes.POINTER(eb_step_desc), _P, ctypes.c_size_t, _P]),
    "eb_decode_step_noalloc": (ctypes.c_int, [ctypes.POINTER(eb_step_desc), _P]),
    "eb_decode_step_attn_in_lmhead": (ctypes.c_int32, [ctypes.POINTER(eb_step_desc)]),
    "eb_probe_mfma_bf16": (ctypes.c_int, [_P, ctypes.c_int32, ctypes.c_int32, _P]),
    "eb_probe_mfma_bf16_flops": (ctypes.c_double, [ctypes.c_int32, ctypes.c_int32]),
    "eb_status_string": (ctypes.c_char_p, [ctypes.c_int]),
    "eb_last_error": (ctypes.c_char_p, []),
    "eb_version": (ctypes.c_char_p, []),
}

_lib = None


def lib_path() -> str:
    return _LIB_PATH


def load() -> ctypes.CDLL:
    """Load libeb.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with "
                               "`python -m paper_2609_16450_amd.build`")
        lib = ctypes.CDLL(_LIB_PATH)
        for name, (res, args) in EXPORTS.items():
            fn = getattr(lib, name)
            fn.restype = res
            fn.argtypes = args
        _lib = lib
    return _lib


class EbError(RuntimeError):
    def __init__(self, status: int, where: str):
        lib = load()
        self.status = status
        msg = lib.eb_last_error().decode()
        super().__init__(f"{where}: {lib.eb_status_string(status).decode()}: {msg}")


def _check(status: int, where: str) -> None:
    if status != EB_OK:
        raise EbError(status, where)


def eb_status_string(status: int) -> str:
    return load().eb_status_string(status).decode()


def eb_last_error() -> str:
    return load().eb_last_error().decode()


def eb_version() -> str:
    return load().eb_version().decode()


# --------------------------------------------------------------------------------------
# marshalling helpers
# --------------------------------------------------------------------------------------

def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return EB_BF16
    if t.dtype == torch.float32:
        return EB_F32
    raise ValueError(f"unsupported dtype {t.dtype} (bfloat16 or float32)")


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _dev(t: torch.Tensor, name: str, dtype=None, shape=None) -> None:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be a device tensor (got {t.device})")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype} (got {t.dtype})")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")


def _stream(stream) -> int:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, torch.cuda.Stream):
        return stream.cuda_stream
    return int(stream)


@dataclass
class Ragged:
    """Host sizes plus device offset arrays of a ragged batch (see eb_ragged in eb.h)."""
    batch: int
    total_block: int
    max_block: int
    total_prefix: int
    max_prefix: int
    cu_block: torch.Tensor   # int32 [batch+1] on the device
    cu_prefix: torch.Tensor  # int32 [batch+1] on the device

    @staticmethod
    def from_lengths(block_lens, prefix_lens, device="cuda") -> "Ragged":
        bl = [int(x) for x in block_lens]
        pl = [int(x) for x in prefix_lens]
        if len(bl) != len(pl) or not bl or min(bl + pl) < 0:
            raise ValueError("need equally long, non-empty, non-negative length lists")
        cb = [0]
        for x in bl:
            cb.append(cb[-1] + x)
        cp = [0]
        for x in pl:
            cp.append(cp[-1] + x)
        return Ragged(len(bl), cb[-1], max(bl), cp[-1], max(pl),
                      torch.tensor(cb, dtype=torch.int32, device=device),
                      torch.tensor(cp, dtype=torch.int32, device=device))

    def c(self) -> eb_ragged:
        _dev(self.cu_block, "cu_block", torch.int32, (self.batch + 1,))
        _dev(self.cu_prefix, "cu_prefix", torch.int32, (self.batch + 1,))
        return eb_ragged(self.batch, self.total_block, self.max_block, self.total_prefix,
                         self.max_prefix, self.cu_block.data_ptr(), self.cu_prefix.data_ptr())


def _torch_stream(stream):
    if stream is None:
        return torch.cuda.current_stream()
    if isinstance(stream, torch.cuda.Stream):
        return stream
    return torch.cuda.ExternalStream(int(stream))


def _workspace(nbytes: int, ws: Optional[torch.Tensor], device, stream) -> tuple:
    """(pointer, bytes) of the caller's workspace, or of a temporary one.  A temporary is
    allocated on the stream the kernels run on, so that torch's caching allocator, once the
    tensor is dropped here, hands its memory only to later work of that same stream."""
    if nbytes == 0:
        return (None if ws is None else ws.data_ptr()), (0 if ws is None else ws.numel())
    if ws is None:
        with torch.cuda.stream(_torch_stream(stream)):
            ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
    _dev(ws, "ws", torch.uint8)
    return ws.data_ptr(), ws.numel()


# --------------------------------------------------------------------------------------
# entry points
# --------------------------------------------------------------------------------------

def eb_block_attn_workspace(dtype: int, r: Ragged, hq: int, hkv: int, head_dim: int) -> int:
    rc = r.c()
    return int(load().eb_block_attn_workspace(dtype, ctypes.byref(rc), hq, hkv, head_dim))


def eb_block_attn(r: Ragged, q, k_blk, v_blk, k_pre, v_pre, out, scale: Optional[float] = None,
                  ws: Optional[torch.Tensor] = None, stream=None) -> None:
    """out[T, hq, D] <- block attention of q over the prefix and block keys (eb.h)."""
    dt = _dtype_code(q)
    T, hq, D = q.shape
    hkv = k_blk.shape[1]
    _dev(q, "q", q.dtype, (r.total_block, hq, D))
    _dev(k_blk, "k_blk", q.dtype, (r.total_block, hkv, D))
    _dev(v_blk, "v_blk", q.dtype, (r.total_block, hkv, D))
    _dev(k_pre, "k_pre", q.dtype, (r.total_prefix, hkv, D))
    _dev(v_pre, "v_pre", q.dtype, (r.total_prefix, hkv, D))
    _dev(out, "out", q.dtype, (r.total_block, hq, D))
    scale = 0.0 if scale is None else float(scale)    # 0: the library's 1/sqrt(D)
    rc = r.c()
    lib = load()
    need = int(lib.eb_block_attn_workspace(dt, ctypes.byref(rc), hq, hkv, D))
    wp, wn = _workspace(need, ws, q.device, stream)
    _check(lib.eb_block_attn(dt, ctypes.byref(rc), hq, hkv, D, scale, q.data_ptr(),
                             k_blk.data_ptr(), v_blk.data_ptr(), k_pre.data_ptr(),
                             v_pre.data_ptr(), out.data_ptr(), wp, wn, _stream(stream)),
           "eb_block_attn")


def eb_block_attn_dual(r: Ragged, cu_suffix: torch.Tensor, max_suffix: int, q, k_blk, v_blk,
                       k_pre, v_pre, k_suf, v_suf, out, scale: Optional[float] = None,
                       ws: Optional[torch.Tensor] = None, stream=None) -> None:
    """out <- block attention over the prefix, block and cached suffix keys (eb.h)."""
    dt = _dtype_code(q)
    T, hq, D = q.shape
    hkv = k_blk.shape[1]
    U = k_suf.shape[0]
    _dev(q, "q", q.dtype, (r.total_block, hq, D))
    _dev(k_blk, "k_blk", q.dtype, (r.total_block, hkv, D))
    _dev(v_blk, "v_blk", q.dtype, (r.total_block, hkv, D))
    _dev(k_pre, "k_pre", q.dtype, (r.total_prefix, hkv, D))
    _dev(v_pre, "v_pre", q.dtype, (r.total_prefix, hkv, D))
    _dev(k_suf, "k_suf", q.dtype, (U, hkv, D))
    _dev(v_suf, "v_suf", q.dtype, (U, hkv, D))
    _dev(out, "out", q.dtype, (r.total_block, hq, D))
    _dev(cu_suffix, "cu_suffix", torch.int32, (r.batch + 1,))
    scale = 0.0 if scale is None else float(scale)    # 0: the library's 1/sqrt(D)
    rc = r.c()
    sc = eb_suffix(U, int(max_suffix), cu_suffix.data_ptr())
    lib = load()
    need = int(lib.eb_block_attn_dual_workspace(dt, ctypes.byref(rc), ctypes.byref(sc), hq, hkv, D))
    wp, wn = _workspace(need, ws, q.device, stream)
    _check(lib.eb_block_attn_dual(dt, ctypes.byref(rc), ctypes.byref(sc), hq, hkv, D, scale,
                                  q.data_ptr(), k_blk.data_ptr(), v_blk.data_ptr(),
                                  k_pre.data_ptr(), v_pre.data_ptr(), k_suf.data_ptr(),
                                  v_suf.data_ptr(), out.data_ptr(), wp, wn, _stream(stream)),
           "eb_block_attn_dual")


def eb_lmhead_workspace(dtype: int, n_rows: int, hidden: int, vocab: int) -> int:
    return int(load().eb_lmhead_workspace(dtype, n_rows, hidden, vocab))


def eb_lmhead_confidence(h, w, conf, entropy_nats, argmax, max_logit=None,
                         ws: Optional[torch.Tensor] = None, stream=None) -> None:
    """conf / entropy_nats / argmax / max_logit [n_rows] of softmax(W h) per row (eb.h)."""
    dt = _dtype_code(h)
    n_rows, hidden = h.shape
    vocab = w.shape[0]
    _dev(h, "h", h.dtype, (n_rows, hidden))
    _dev(w, "w", h.dtype, (vocab, hidden))
    _dev(conf, "conf", torch.float32, (n_rows,))
    _dev(entropy_nats, "entropy_nats", torch.float32, (n_rows,))
    _dev(argmax, "argmax", torch.int32, (n_rows,))
    if max_logit is not None:
        _dev(max_logit, "max_logit", torch.float32, (n_rows,))
    lib = load()
    need = int(lib.eb_lmhead_workspace(dt, n_rows, hidden, vocab))
    wp, wn = _workspace(need, ws, h.device, stream)
    _check(lib.eb_lmhead_confidence(dt, n_rows, hidden, vocab, h.data_ptr(), w.data_ptr(),
                                    conf.data_ptr(), entropy_nats.data_ptr(), argmax.data_ptr(),
                                    _ptr(max_logit), wp, wn, _stream(stream)),
           "eb_lmhead_confidence")


def eb_unmask_select(r: Ragged, conf, argmax, tau, masked, tokens, unmask, n_commit, resolved,
                     stream=None) -> None:
    """Threshold commit with the anti-stall fallback inside each block (eb.h)."""
    T, B = r.total_block, r.batch
    _dev(conf, "conf", torch.float32, (T,))
    _dev(argmax, "argmax", torch.int32, (T,))
    _dev(tau, "tau", torch.float32, (B,))
    _dev(masked, "masked", torch.uint8, (T,))
    _dev(tokens, "tokens", torch.int32, (T,))
    _dev(unmask, "unmask", torch.uint8, (T,))
    _dev(n_commit, "n_commit", torch.int32, (B,))
    _dev(resolved, "resolved", torch.uint8, (B,))
    rc = r.c()
    _check(load().eb_unmask_select(ctypes.byref(rc), conf.data_ptr(), argmax.data_ptr(),
                                   tau.data_ptr(), masked.data_ptr(), tokens.data_ptr(),
                                   unmask.data_ptr(), n_commit.data_ptr(), resolved.data_ptr(),
                                   _stream(stream)),
           "eb_unmask_select")


def eb_lmhead_features_workspace(dtype: int, n_rows: int, hidden: int, vocab: int) -> int:
    return int(load().eb_lmhead_features_workspace(dtype, n_rows, hidden, vocab))


def eb_lmhead_features(h, w, conf, entropy_nats, argmax, top2_gap, max_logit=None,
                       ws: Optional[torch.Tensor] = None, stream=None) -> None:
    """eb_lmhead_confidence plus the top-1/top-2 probability gap per row (eb.h)."""
    dt = _dtype_code(h)
    n_rows, hidden = h.shape
    vocab = w.shape[0]
    _dev(h, "h", h.dtype, (n_rows, hidden))
    _dev(w, "w", h.dtype, (vocab, hidden))
    for name, t, dtype in (("conf", conf, torch.float32), ("entropy_nats", entropy_nats, torch.float32),
                           ("argmax", argmax, torch.int32), ("top2_gap", top2_gap, torch.float32)):
        _dev(t, name, dtype, (n_rows,))
    if max_logit is not None:
        _dev(max_logit, "max_logit", torch.float32, (n_rows,))
    lib = load()
    need = int(lib.eb_lmhead_features_workspace(dt, n_rows, hidden, vocab))
    wp, wn = _workspace(need, ws, h.device, stream)
    _check(lib.eb_lmhead_features(dt, n_rows, hidden, vocab, h.data_ptr(), w.data_ptr(),
                                  conf.data_ptr(), entropy_nats.data_ptr(), argmax.data_ptr(),
                                  _ptr(max_logit), top2_gap.data_ptr(), wp, wn, _stream(stream)),
           "eb_lmhead_features")


def eb_lps_features(r: Ragged, vocab: int, conf, entropy_nats, top2_gap, masked, feat, pos,
                    mask_ratio=None, seq_pos=None, stream=None) -> None:
    """LPS router inputs feat [T, 4] and intra-block positions pos [T] (eb.h); with seq_pos
    [T] int32 (sequence position of every packed row) pos is (i - b) / |B| on sequence
    positions, without it the row's rank in its block over the block size."""
    T, B = r.total_block, r.batch
    for name, t in (("conf", conf), ("entropy_nats", entropy_nats), ("top2_gap", top2_gap),
                    ("pos", pos)):
        _dev(t, name, torch.float32, (T,))
    _dev(masked, "masked", torch.uint8, (T,))
    if seq_pos is not None:
        _dev(seq_pos, "seq_pos", torch.int32, (T,))
    _dev(feat, "feat", torch.float32, (T, 4))
    if mask_ratio is not None:
        _dev(mask_ratio, "mask_ratio", torch.float32, (B,))
    rc = r.c()
    _check(load().eb_lps_features(ctypes.byref(rc), int(vocab), conf.data_ptr(),
                                  entropy_nats.data_ptr(), top2_gap.data_ptr(), masked.data_ptr(),
                                  _ptr(seq_pos), feat.data_ptr(), pos.data_ptr(), _ptr(mask_ratio),
                                  _stream(stream)),
           "eb_lps_features")


def _unmask_tensors(r: Ragged, conf, argmax, tau, masked, tokens, unmask, n_commit, resolved):
    T, B = r.total_block, r.batch
    _dev(conf, "conf", torch.float32, (T,))
    _dev(argmax, "argmax", torch.int32, (T,))
    _dev(tau, "tau", torch.float32, (B,))
    _dev(masked, "masked", torch.uint8, (T,))
    _dev(tokens, "tokens", torch.int32, (T,))
    _dev(unmask, "unmask", torch.uint8, (T,))
    _dev(n_commit, "n_commit", torch.int32, (B,))
    _dev(resolved, "resolved", torch.uint8, (B,))


def eb_unmask_select_lps(r: Ragged, conf, argmax, tau, p_psi, tau_psi: float, masked, tokens,
                         unmask, n_commit, resolved, stream=None) -> None:
    """Union accept rule conf >= tau or p_psi > tau_psi, with the anti-stall fallback (eb.h)."""
    _unmask_tensors(r, conf, argmax, tau, masked, tokens, unmask, n_commit, resolved)
    _dev(p_psi, "p_psi", torch.float32, (r.total_block,))
    rc = r.c()
    _check(load().eb_unmask_select_lps(ctypes.byref(rc), conf.data_ptr(), argmax.data_ptr(),
                                       tau.data_ptr(), p_psi.data_ptr(), float(tau_psi),
                                       masked.data_ptr(), tokens.data_ptr(), unmask.data_ptr(),
                                       n_commit.data_ptr(), resolved.data_ptr(), _stream(stream)),
           "eb_unmask_select_lps")


def eb_unmask_select_topm(r: Ragged, conf, argmax, tau, m: int, masked, tokens, unmask,
                          n_commit, resolved, stream=None) -> None:
    """Threshold set united with the m most confident masked rows of each block (eb.h)."""
    _unmask_tensors(r, conf, argmax, tau, masked, tokens, unmask, n_commit, resolved)
    rc = r.c()
    _check(load().eb_unmask_select_topm(ctypes.byref(rc), conf.data_ptr(), argmax.data_ptr(),
                                        tau.data_ptr(), int(m), masked.data_ptr(),
                                        tokens.data_ptr(), unmask.data_ptr(), n_commit.data_ptr(),
                                        resolved.data_ptr(), _stream(stream)),
           "eb_unmask_select_topm")


def eb_lbs_select(masked, p_phi, x_hat, eos_id: int, l_min: int, l_b: int, g_max: int, block,
                  size, first, stream=None) -> None:
    """LBS active-block post-pass over [n_seq, window] windows (eb.h)."""
    n, L = masked.shape
    _dev(masked, "masked", torch.uint8, (n, L))
    _dev(p_phi, "p_phi", torch.float32, (n, L))
    _dev(x_hat, "x_hat", torch.int32, (n, L))
    _dev(block, "block", torch.uint8, (n, L))
    _dev(size, "size", torch.int32, (n,))
    _dev(first, "first", torch.int32, (n,))
    _check(load().eb_lbs_select(n, L, masked.data_ptr(), p_phi.data_ptr(), x_hat.data_ptr(),
                                int(eos_id), int(l_min), int(l_b), int(g_max), block.data_ptr(),
                                size.data_ptr(), first.data_ptr(), _stream(stream)),
           "eb_lbs_select")


class StepBuffers:
    """All tensors of one eb_decode_step call, checked once; build(), then call repeatedly."""

    def __init__(self, r: Ragged, q, k_blk, v_blk, k_pre, v_pre, attn_out, h, w, conf,
                 entropy_nats, argmax, tau, masked, tokens, unmask, n_commit, resolved,
                 max_logit=None, attn_scale: Optional[float] = None,
                 ws: Optional[torch.Tensor] = None):
        dt = _dtype_code(q)
        T, B = r.total_block, r.batch
        hq, D = q.shape[1], q.shape[2]
        hkv = k_blk.shape[1]
        hidden, vocab = h.shape[1], w.shape[0]
        for name, t, shape in [("q", q, (T, hq, D)), ("k_blk", k_blk, (T, hkv, D)),
                               ("v_blk", v_blk, (T, hkv, D)), ("k_pre", k_pre, (r.total_prefix, hkv, D)),
                               ("v_pre", v_pre, (r.total_prefix, hkv, D)),
                               ("attn_out", attn_out, (T, hq, D)), ("h", h, (T, hidden)),
                               ("w", w, (vocab, hidden))]:
            _dev(t, name, q.dtype, shape)
        for name, t, dtype, shape in [("conf", conf, torch.float32, (T,)),
                                      ("entropy_nats", entropy_nats, torch.float32, (T,)),
                                      ("argmax", argmax, torch.int32, (T,)),
                                      ("tau", tau, torch.float32, (B,)),
                                      ("masked", masked, torch.uint8, (T,)),
                                      ("tokens", tokens, torch.int32, (T,)),
                                      ("unmask", unmask, torch.uint8, (T,)),
                                      ("n_commit", n_commit, torch.int32, (B,)),
                                      ("resolved", resolved, torch.uint8, (B,))]:
            _dev(t, name, dtype, shape)
        if max_logit is not None:
            _dev(max_logit, "max_logit", torch.float32, (T,))
        self._keep = (r, q, k_blk, v_blk, k_pre, v_pre, attn_out, h, w, conf, entropy_nats,
                      argmax, tau, masked, tokens, unmask, n_commit, resolved, max_logit)
        self.desc = eb_step_desc(
            dt, r.c(), hq, hkv, D, 0.0 if attn_scale is None else float(attn_scale),
            q.data_ptr(), k_blk.data_ptr(), v_blk.data_ptr(), k_pre.data_ptr(), v_pre.data_ptr(),
            attn_out.data_ptr(), hidden, vocab, h.data_ptr(), w.data_ptr(), conf.data_ptr(),
            entropy_nats.data_ptr(), argmax.data_ptr(), _ptr(max_logit), tau.data_ptr(),
            masked.data_ptr(), tokens.data_ptr(), unmask.data_ptr(), n_commit.data_ptr(),
            resolved.data_ptr())
        need = int(load().eb_decode_step_workspace(ctypes.byref(self.desc)))
        if ws is None and need:
            ws = torch.empty(need, dtype=torch.uint8, device=q.device)
        if ws is not None:
            _dev(ws, "ws", torch.uint8)
        self.ws = ws
        self.ws_bytes = 0 if ws is None else ws.numel()


def eb_decode_step_workspace(buffers: StepBuffers) -> int:
    return int(load().eb_decode_step_workspace(ctypes.byref(buffers.desc)))


def eb_decode_step_attn_in_lmhead(buffers: StepBuffers) -> bool:
    """Whether eb_decode_step runs the attention inside the LM-head launch for these buffers."""
    return bool(load().eb_decode_step_attn_in_lmhead(ctypes.byref(buffers.desc)))


def eb_probe_mfma_bf16(out: torch.Tensor, groups: int, iters: int, stream=None) -> float:
    """Launch the register-only bf16 MFMA loop (eb.h, measurement aid) into `out` (float32,
    at least groups * 256 elements); returns the launch's flop count."""
    _dev(out, "out", torch.float32)
    if out.numel() < groups * 256:
        raise ValueError(f"out holds {out.numel()} floats, the probe writes {groups * 256}")
    lib = load()
    _check(lib.eb_probe_mfma_bf16(out.data_ptr(), groups, iters, _stream(stream)),
           "eb_probe_mfma_bf16")
    return float(lib.eb_probe_mfma_bf16_flops(groups, iters))


def eb_decode_step(buffers: StepBuffers, stream=None, trace: Optional[eb_step_trace] = None) -> None:
    """One whole denoising step on one stream (eb.h).  `trace` optionally names hipEvents
    (as integer handles) to record around the step's kernels."""
    buffers.desc.trace = ctypes.pointer(trace) if trace is not None else None
    _check(load().eb_decode_step(ctypes.byref(buffers.desc), _ptr(buffers.ws), buffers.ws_bytes,
                                 _stream(stream)),
           "eb_decode_step")


EB_NOALLOC_SCRATCH_BYTES = 128 << 20   # the library's per-device scratch (eb.h)


def eb_decode_step_noalloc(buffers: StepBuffers, stream=None,
                           trace: Optional[eb_step_trace] = None) -> None:
    """The same step with the library's own per-device scratch instead of buffers.ws (eb.h):
    no device memory is allocated by the call; calls on one device must not overlap."""
    buffers.desc.trace = ctypes.pointer(trace) if trace is not None else None
    _check(load().eb_decode_step_noalloc(ctypes.byref(buffers.desc), _stream(stream)),
           "eb_decode_step_noalloc")
