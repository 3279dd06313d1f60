"""The C-ABI library loads and exports every entry point the header
declares; its host-only paths (sizes, validation, error strings) behave as
documented. Nothing here launches GPU work."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "attn_abft.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    names = re.findall(r"^[A-Za-z_][\w\s\*]*?\b(\w+)\s*\(", text, flags=re.M)
    return sorted({n for n in names if n not in ("if", "defined")})


def test_header_declares_the_boundary():
    names = _declared_functions()
    for want in ("attn_abft_forward", "attn_abft_backward", "encode_checksums",
                 "verify_and_correct", "attn_abft_workspace_bytes", "attn_abft_report_bytes",
                 "attn_abft_report_init", "attn_abft_workspace_offsets", "attn_abft_strerror",
                 "attn_abft_unsafe_probability", "attn_abft_optimize_frequencies",
                 "attn_abft_sections_for_step"):
        assert want in names


def test_library_exports_every_declared_symbol():
    from paper_2410_11720_amd import abft
    lib = ctypes.CDLL(abft.LIB_PATH)
    for name in _declared_functions():
        assert hasattr(lib, name), name


def test_struct_sizes_match_header_layout():
    from paper_2410_11720_amd import abft
    assert ctypes.sizeof(abft.Config) == 13 * 4
    assert ctypes.sizeof(abft.Fault) == 28
    assert ctypes.sizeof(abft.Event) == 40
    assert ctypes.sizeof(abft.FreqOp) == 32 and ctypes.sizeof(abft.FreqSection) == 16
    assert abft.attn_abft_report_bytes(0) == abft.REPORT_HEADER
    assert abft.attn_abft_report_bytes(10) == abft.REPORT_HEADER + 400


def test_workspace_sizes_and_validation():
    from paper_2410_11720_amd import abft
    cfg = abft.LayerConfig(8, 1024, 768, 12, causal=True)
    n = abft.attn_abft_workspace_bytes(cfg)
    S2 = 8 * 12 * 1024 * 1024 * 2
    assert 3 * S2 < n < 3 * S2 + 200 * 2 ** 20
    q, a, l = abft.attn_abft_workspace_offsets(cfg)
    assert q == 0 and a >= 8 * 1024 * 3 * 768 * 2 and l >= a + S2
    bad = [abft.LayerConfig(1, 100, 64, 1, block_rows=128),      # R does not divide seq
           abft.LayerConfig(1, 128, 96, 1),                      # head_dim 96
           abft.LayerConfig(1, 128, 64, 3),                      # hidden % heads
           abft.LayerConfig(1, 128, 64, 1, block_rows=96),       # R not a power of two
           abft.LayerConfig(1, 128, 64, 1, block_rows=16),       # R too small for bf16
           abft.LayerConfig(0, 128, 64, 1)]
    for c in bad:
        with pytest.raises(abft.AbftError):
            abft.attn_abft_workspace_bytes(c)
    assert abft.attn_abft_workspace_bytes(abft.LayerConfig(1, 128, 64, 1, dtype="f32",
                                                           block_rows=16)) > 0


def test_entry_points_reject_bad_arguments_before_any_launch():
    from paper_2410_11720_amd import abft
    lib = ctypes.CDLL(abft.LIB_PATH)
    lib.attn_abft_forward.restype = ctypes.c_int
    cfg = abft.LayerConfig(1, 128, 64, 1).to_c()
    st = lib.attn_abft_forward(ctypes.byref(cfg), None, None, None, None, None,
                               ctypes.c_size_t(0), None, 0, None, None)
    assert st == -1
    bad = abft.LayerConfig(1, 128, 96, 1).to_c()
    st = lib.attn_abft_forward(ctypes.byref(bad), None, None, None, None, None,
                               ctypes.c_size_t(0), None, 0, None, None)
    assert st == -2
    lib.encode_checksums.restype = ctypes.c_int
    st = lib.encode_checksums(None, 0, ctypes.c_int64(1), ctypes.c_int64(4), ctypes.c_int64(4),
                              ctypes.c_int64(4), ctypes.c_int64(0), 2, 2, None, None, None)
    assert st == -1
    assert abft.strerror(-4) == "workspace too small"
    assert abft.strerror(0) == "ok"
