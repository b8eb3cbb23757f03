"""The C ABI library loads, exports every function include/eb.h declares, and rejects bad
arguments on the host (no GPU work is launched by any of these calls)."""
import ctypes
import os
import re

import pytest

from paper_2609_16450_amd import binding as B

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "eb.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"\b(eb_[a-z0-9_]+)\s*\(", text)
    return sorted(set(names))


def test_header_declares_the_step_entry_points():
    names = declared_functions()
    for n in ("eb_block_attn", "eb_lmhead_confidence", "eb_unmask_select", "eb_decode_step"):
        assert n in names


def test_library_exports_every_declared_function():
    lib = B.load()
    for n in declared_functions():
        assert hasattr(lib, n), n
    assert set(declared_functions()) == set(B.EXPORTS)


def _ragged(batch=1, T=4, maxb=4, S=0, maxp=0, cu_b=0x1000, cu_p=0x2000):
    return B.eb_ragged(batch, T, maxb, S, maxp, cu_b, cu_p)


def test_invalid_arguments_are_rejected_before_launch():
    lib = B.load()
    r = _ragged(batch=0)
    assert lib.eb_unmask_select(ctypes.byref(r), *([None] * 9)) == B.EB_ERR_INVALID
    assert "batch" in B.eb_last_error()
    r = _ragged()
    # NULL outputs
    assert lib.eb_unmask_select(ctypes.byref(r), *([None] * 9)) == B.EB_ERR_INVALID
    # hq not a multiple of hkv
    assert lib.eb_block_attn(B.EB_BF16, ctypes.byref(r), 6, 4, 128, 0.1, *([0x100] * 6), None, 0,
                             None) == B.EB_ERR_INVALID
    # head_dim 96 is valid but unimplemented
    assert lib.eb_block_attn(B.EB_BF16, ctypes.byref(r), 4, 4, 96, 0.1, *([0x100] * 6), None, 0,
                             None) == B.EB_ERR_UNSUPPORTED
    # misaligned bf16 pointer
    assert lib.eb_block_attn(B.EB_BF16, ctypes.byref(r), 4, 4, 128, 0.1, 0x101, *([0x100] * 5),
                             None, 0, None) == B.EB_ERR_INVALID
    # negative or non-finite scale (0 selects 1/sqrt(head_dim))
    assert lib.eb_block_attn(B.EB_BF16, ctypes.byref(r), 4, 4, 128, -0.5, *([0x100] * 6), None, 0,
                             None) == B.EB_ERR_INVALID
    assert lib.eb_block_attn(B.EB_BF16, ctypes.byref(r), 4, 4, 128, float("inf"), *([0x100] * 6),
                             None, 0, None) == B.EB_ERR_INVALID
    # unknown dtype
    assert lib.eb_lmhead_confidence(7, 4, 64, 100, *([0x100] * 5), None, None, 0, None) == \
        B.EB_ERR_INVALID
    # bf16 hidden not a multiple of 64
    assert lib.eb_lmhead_confidence(B.EB_BF16, 4, 96, 100, *([0x100] * 5), None, None, 0, None) \
        == B.EB_ERR_UNSUPPORTED
    # short workspace
    need = lib.eb_lmhead_workspace(B.EB_BF16, 4, 64, 1000)
    assert need > 0
    assert lib.eb_lmhead_confidence(B.EB_BF16, 4, 64, 1000, *([0x100] * 5), None, 0x100, need - 1,
                                    None) == B.EB_ERR_WORKSPACE
    assert "workspace" in B.eb_last_error()


def test_next_row_entry_points_reject_bad_arguments():
    lib = B.load()
    r = _ragged()
    # the gap output is required
    assert lib.eb_lmhead_features(B.EB_BF16, 4, 64, 1000, *([0x100] * 5), None, None, 0x100,
                                  1 << 20, None) == B.EB_ERR_INVALID
    assert "top2_gap" in B.eb_last_error()
    # short workspace: the gap path needs more than the plain one
    plain = lib.eb_lmhead_workspace(B.EB_BF16, 4, 64, 1000)
    need = lib.eb_lmhead_features_workspace(B.EB_BF16, 4, 64, 1000)
    assert need > plain
    assert lib.eb_lmhead_features(B.EB_BF16, 4, 64, 1000, *([0x100] * 5), None, 0x100, 0x100,
                                  need - 1, None) == B.EB_ERR_WORKSPACE
    # vocab must allow ln(vocab) > 0; feat must be 16-byte aligned
    assert lib.eb_lps_features(ctypes.byref(r), 1, *([0x100] * 4), None, 0x100, 0x100, None,
                               None) == B.EB_ERR_INVALID
    assert lib.eb_lps_features(ctypes.byref(r), 100, *([0x100] * 4), 0x100, 0x104, 0x100, None,
                               None) == B.EB_ERR_INVALID
    # router score required; budget must not be negative
    assert lib.eb_unmask_select_lps(ctypes.byref(r), 0x100, 0x100, 0x100, None, 0.9,
                                    *([0x100] * 5), None) == B.EB_ERR_INVALID
    assert lib.eb_unmask_select_topm(ctypes.byref(r), 0x100, 0x100, 0x100, -1, *([0x100] * 5),
                                     None) == B.EB_ERR_INVALID
    assert "m must be" in B.eb_last_error()
    # LBS post-pass: g_max >= 1, outputs required
    assert lib.eb_lbs_select(2, 16, *([0x100] * 3), 1, 2, 32, 0, *([0x100] * 3), None) == \
        B.EB_ERR_INVALID
    assert lib.eb_lbs_select(2, 16, *([0x100] * 3), 1, 2, 32, 5, 0x100, None, 0x100, None) == \
        B.EB_ERR_INVALID
    # dual cache: descriptor required, suffix pointers required when it has rows
    assert lib.eb_block_attn_dual(B.EB_BF16, ctypes.byref(r), None, 4, 4, 128, 0.1,
                                  *([0x100] * 8), None, 0, None) == B.EB_ERR_INVALID
    sfx = B.eb_suffix(10, 10, 0x3000)
    assert lib.eb_block_attn_dual(B.EB_BF16, ctypes.byref(r), ctypes.byref(sfx), 4, 4, 128, 0.1,
                                  *([0x100] * 5), None, None, 0x100, None, 0, None) == \
        B.EB_ERR_INVALID


def test_workspace_queries():
    lib = B.load()
    assert lib.eb_lmhead_workspace(B.EB_BF16, 0, 4096, 126464) == 0
    small = lib.eb_lmhead_workspace(B.EB_BF16, 32, 4096, 126464)
    big = lib.eb_lmhead_workspace(B.EB_BF16, 64, 4096, 126464)
    assert small > 0 and big >= 2 * small - 256 and small % 256 == 0
    r = _ragged()
    assert lib.eb_block_attn_workspace(B.EB_BF16, ctypes.byref(r), 4, 4, 128) == 0


def test_status_strings():
    assert B.eb_status_string(0) == "EB_OK"
    assert B.eb_status_string(3) == "EB_ERR_WORKSPACE"
    assert "gfx950" in B.eb_version()


def test_attention_in_lmhead_query():
    # Host-only query: which decode steps run the attention inside the LM-head launch.
    lib = B.load()

    def desc(dtype, batch, total, max_block, hq, hkv, head_dim, vocab):
        d = B.eb_step_desc()
        d.dtype = dtype
        d.ragged = B.eb_ragged(batch, total, max_block, 512 * batch, 512, 0x1000, 0x2000)
        d.hq, d.hkv, d.head_dim, d.hidden, d.vocab = hq, hkv, head_dim, 4096, vocab
        return ctypes.byref(d)

    q = lib.eb_decode_step_attn_in_lmhead
    assert q(None) == 0
    assert q(desc(B.EB_BF16, 1, 32, 32, 32, 32, 128, 126464)) == 1   # batch-1 LLaDA shape
    assert q(desc(B.EB_BF16, 1, 64, 64, 16, 4, 64, 20000)) == 1      # 256 query rows per head
    assert q(desc(B.EB_BF16, 1, 65, 65, 4, 4, 128, 20000)) == 0      # more than 64 block rows
    assert q(desc(B.EB_BF16, 1, 40, 40, 28, 4, 128, 20000)) == 0     # 280 query rows per head
    assert q(desc(B.EB_BF16, 1, 16, 16, 4, 4, 128, 262144)) == 0     # 8-wave LM-head launch
    assert q(desc(B.EB_F32, 1, 32, 32, 4, 4, 64, 2048)) == 0          # fp32 path
    assert q(desc(B.EB_BF16, 2, 0, 0, 4, 4, 128, 2048)) == 0          # no block rows


def test_mfma_probe_rejects_bad_arguments():
    lib = B.load()
    dummy = 0x1000  # never dereferenced: every call below is rejected on the host
    assert lib.eb_probe_mfma_bf16(None, 1, 1, None) == B.EB_ERR_INVALID
    assert lib.eb_probe_mfma_bf16(dummy, 0, 1, None) == B.EB_ERR_INVALID
    assert lib.eb_probe_mfma_bf16(dummy, 65537, 1, None) == B.EB_ERR_INVALID
    assert lib.eb_probe_mfma_bf16(dummy, 1, 0, None) == B.EB_ERR_INVALID
    assert lib.eb_probe_mfma_bf16(dummy, 1, (1 << 20) + 1, None) == B.EB_ERR_INVALID
    assert lib.eb_probe_mfma_bf16_flops(0, 1) == 0.0
    # 8 chains x 4 waves x 2*32*32*16 flops per MFMA
    assert lib.eb_probe_mfma_bf16_flops(3, 5) == 3 * 5 * 8 * 4 * 2 * 32 * 32 * 16


def test_noalloc_step_rejects_oversized_steps_on_the_host():
    # eb_decode_step_noalloc: a step whose workspace exceeds the library's scratch is refused
    # before anything touches the device
    lib = B.load()
    assert lib.eb_decode_step_noalloc(None, None) == B.EB_ERR_INVALID
    d = B.eb_step_desc()
    d.dtype = B.EB_BF16
    d.ragged = B.eb_ragged(64, 20000, 400, 64 * 4096, 4096, 0x1000, 0x2000)
    d.hq, d.hkv, d.head_dim, d.hidden, d.vocab = 28, 4, 128, 3584, 152064
    need = lib.eb_decode_step_workspace(ctypes.byref(d))
    assert need > B.EB_NOALLOC_SCRATCH_BYTES
    assert lib.eb_decode_step_noalloc(ctypes.byref(d), None) == B.EB_ERR_WORKSPACE
    assert "scratch" in B.eb_last_error()
