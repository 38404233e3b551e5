"""The C-ABI library loads, exports every symbol that include/qlinear.h
declares, and rejects bad arguments before touching the GPU (no GPU needed)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "qlinear.h")
LIB = os.path.join(ROOT, "paper_2608_30877_amd", "libqlinear.so")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[A-Za-z_][A-Za-z0-9_]*\**\s+\**([a-z][a-z0-9_]*)\s*\(",
                       src, flags=re.M)
    return sorted(set(names))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(LIB):
        pytest.fail(f"{LIB} not built (run python paper_2608_30877_amd/build.py)")
    return ctypes.CDLL(LIB)


def test_header_declares_the_boundary():
    names = declared_functions()
    for need in ["qlinear_pack", "qlinear_forward", "qlayer_stack_forward", "qlinear_dequant",
                 "qlinear_forward_ex", "qlinear_workspace_bytes", "qlinear_status_string",
                 "qlayer_stack_workspace_bytes", "qlinear_rmsnorm",
                 "qlayer_stack_workspace_offsets", "qlinear_attention",
                 "qlayer_stack_forward_attn", "qlinear_attention_varlen",
                 "qlayer_stack_forward_streamed", "qlayer_stack_slot_bytes",
                 "qlinear_tile_codes", "qlinear_untile_codes"]:
        assert need in names, need


def test_library_exports_every_declared_symbol(lib):
    for name in declared_functions():
        assert hasattr(lib, name), f"libqlinear.so does not export {name}"


def test_forward_path_allocates_nothing():
    """The forward entry points call no allocator, free, or synchronisation
    and keep no workspace map (source check of the C ABI file)."""
    src = open(os.path.join(ROOT, "paper_2608_30877_amd", "csrc", "ql_api.hip")).read()
    for banned in ("hipMalloc", "hipFree", "hipStreamSynchronize", "hipDeviceSynchronize",
                   "std::map", "std::mutex"):
        assert banned not in src, banned


def test_status_strings(lib):
    f = lib.qlinear_status_string
    f.restype = ctypes.c_char_p
    f.argtypes = [ctypes.c_int]
    assert f(0) == b"ok"
    for code in range(1, 8):
        assert f(code) and f(code) != b"unknown status"
    assert f(99) == b"unknown status"


def _fwd(lib):
    f = lib.qlinear_forward
    vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    f.argtypes = [vp, vp, vp, vp, i64, i64, i64, i32, vp]
    f.restype = ctypes.c_int
    return f


def test_argument_errors_without_launch(lib):
    f = _fwd(lib)
    p = ctypes.c_void_p(4096)          # never dereferenced: validation fails first
    assert f(None, p, p, p, 4, 4, 128, 128, None) == 1           # null pointer
    assert f(p, p, p, p, 0, 4, 128, 128, None) == 1              # M <= 0
    assert f(p, p, p, p, 4, 4, 100, 128, None) == 1              # K % 128
    assert f(p, p, p, p, 4, 4, 128, 64, None) == 2               # group != 128
    odd = ctypes.c_void_p(4096 + 8)
    assert f(odd, p, p, p, 4, 4, 128, 128, None) == 3            # misaligned x


def test_forward_ex_errors_without_launch(lib):
    f = lib.qlinear_forward_ex
    vp, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    f.argtypes = [vp, i64, vp, vp, vp, i64, i64, i64, i64, i32, i32, vp, sz, vp]
    f.restype = ctypes.c_int
    p = ctypes.c_void_p(4096)
    # unknown epilogue
    assert f(p, 128, p, p, p, 64, 64, 64, 128, 128, 7, p, 1 << 20, None) == 2
    # ldx smaller than K
    assert f(p, 64, p, p, p, 64, 64, 64, 128, 128, 0, p, 1 << 20, None) == 1
    # a workspace that is given must be large enough and 256-byte aligned
    # (without one the MFMA kernel reads x as stored)
    assert f(p, 128, p, p, p, 64, 64, 64, 128, 128, 0, p, 16, None) == 6
    assert f(p, 128, p, p, p, 64, 64, 64, 128, 128, 0, ctypes.c_void_p(4096 + 16),
             1 << 20, None) == 3
    ws = lib.qlinear_workspace_bytes
    ws.argtypes = [i64, i64, i32]
    ws.restype = sz
    assert ws(16, 4096, 128) == 0                     # small-M path uses none
    assert ws(16, 49152, 128) == 0                    # largest K it serves
    assert ws(16, 49280, 128) > 0                     # beyond: MFMA path
    assert ws(2048, 12288, 128) >= 2048 * 12288 * 2   # permuted activation copy
    assert ws(4, 100, 128) == 0                        # invalid shape -> 0


def test_stack_errors_without_launch(lib):
    f = lib.qlayer_stack_forward
    vp, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    f.argtypes = [vp, i32, vp, i64, i64, i64, i32, ctypes.c_float, vp, sz, vp]
    f.restype = ctypes.c_int
    p = ctypes.c_void_p(4096)
    assert f(None, 1, p, 8, 256, 512, 128, 1e-5, p, 1 << 30, None) == 1
    assert f(p, 1, p, 8, 200, 512, 128, 1e-5, p, 1 << 30, None) == 1      # d % 128
    assert f(p, 1, p, 8, 256, 512, 128, 1e-5, p, 16, None) == 6           # workspace


def test_attention_errors_without_launch(lib):
    f = lib.qlinear_attention
    vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    f.argtypes = [vp, i64, vp, i64, i64, i64, i32, i32, i32, vp]
    f.restype = ctypes.c_int
    q, o = ctypes.c_void_p(1 << 20), ctypes.c_void_p(1 << 30)   # never dereferenced
    assert f(None, 768, o, 256, 128, 256, 2, 64, 8, None) == 1      # null pointer
    assert f(q, 768, o, 256, 0, 256, 2, 64, 8, None) == 1           # M <= 0
    assert f(q, 768, o, 256, 128, 256, 2, 100, 8, None) == 1        # M % seq_len
    assert f(q, 768, o, 256, 128, 256, 2, 64, 0, None) == 1         # window 0
    assert f(q, 768, o, 256, 128, 256, 2, 0, 8, None) == 1          # seq_len 0
    assert f(q, 768, o, 256, 128, 384, 2, 64, 8, None) == 2         # head dim 192
    assert f(q, 700, o, 256, 128, 256, 2, 64, 8, None) == 1         # ldqkv < 3d
    assert f(q, 772, o, 256, 128, 256, 2, 64, 8, None) == 3         # row stride not 16 B
    assert f(ctypes.c_void_p((1 << 20) + 8), 768, o, 256, 128, 256, 2, 64, 8, None) == 3
    # out overlapping qkv
    assert f(q, 768, ctypes.c_void_p((1 << 20) + 4096), 256, 128, 256, 2, 64, 8, None) == 1


def test_stack_attention_errors_without_launch(lib):
    class Cfg(ctypes.Structure):
        _fields_ = [("heads", ctypes.c_int32), ("seq_len", ctypes.c_int32),
                    ("window", ctypes.c_int32)]

    f = lib.qlayer_stack_forward_attn
    vp, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    f.argtypes = [vp, i32, vp, i64, i64, i64, i32, ctypes.c_float, vp, vp, sz, vp, vp]
    f.restype = ctypes.c_int
    p = ctypes.c_void_p(4096)
    cfg = lambda *a: ctypes.byref(Cfg(*a))
    assert f(p, 1, p, 64, 256, 512, 128, 1e-5, cfg(3, 64, 8), p, 1 << 30, None, None) == 2
    assert f(p, 1, p, 64, 256, 512, 128, 1e-5, cfg(2, 48, 8), p, 1 << 30, None, None) == 1
    assert f(p, 1, p, 64, 256, 512, 128, 1e-5, cfg(2, 64, -1), p, 1 << 30, None, None) == 1
    assert f(p, 1, p, 64, 256, 512, 128, 1e-5, cfg(2, 64, 8), p, 16, None, None) == 6


def test_attention_varlen_errors_without_launch(lib):
    f = lib.qlinear_attention_varlen
    vp, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    f.argtypes = [vp, i64, vp, i64, i64, i64, i32, vp, i32, i32, i32, vp]
    f.restype = ctypes.c_int
    q, o, cu = ctypes.c_void_p(1 << 20), ctypes.c_void_p(1 << 30), ctypes.c_void_p(1 << 12)
    assert f(q, 768, o, 256, 100, 256, 2, None, 3, 64, 8, None) == 1     # no offsets
    assert f(q, 768, o, 256, 100, 256, 2, cu, 0, 64, 8, None) == 1       # no sequences
    assert f(q, 768, o, 256, 100, 256, 2, cu, 3, 0, 8, None) == 1        # max length 0
    assert f(q, 768, o, 256, 100, 256, 2, ctypes.c_void_p((1 << 12) + 2), 3, 64, 8, None) == 3
    assert f(q, 768, o, 256, 100, 384, 2, cu, 3, 64, 8, None) == 2       # head dim 192


def test_streamed_stack_errors_without_launch(lib):
    f = lib.qlayer_stack_forward_streamed
    vp, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    f.argtypes = [vp, i32, vp, i64, i64, i64, i32, ctypes.c_float, vp, vp, sz, vp, sz, vp, vp]
    f.restype = ctypes.c_int
    sb = lib.qlayer_stack_slot_bytes
    sb.argtypes = [i64, i64, i32]
    sb.restype = sz
    slot = sb(256, 1024, 128)
    # codes + scales of qkv, out, up, down, each 256-byte aligned
    assert slot == (3 * 256 * 128 + 3 * 256 * 2 * 2 + 256 * 128 + 256 * 2 * 2 +
                    1024 * 128 + 1024 * 2 * 2 + 256 * 512 + 256 * 8 * 2)
    assert sb(256, 1000, 128) == 0
    p, s1, s2 = ctypes.c_void_p(4096), ctypes.c_void_p(1 << 12), ctypes.c_void_p(1 << 13)
    big = 1 << 30
    # the copy stream must differ from the compute stream
    assert f(p, 1, p, 8, 256, 1024, 128, 1e-5, None, p, big, p, big, s1, s1) == 1
    # no slots
    assert f(p, 1, p, 8, 256, 1024, 128, 1e-5, None, p, big, None, big, s1, s2) == 1
    # slots smaller than two blocks
    assert f(p, 1, p, 8, 256, 1024, 128, 1e-5, None, p, big, p, 2 * slot - 1, s1, s2) == 6
    # slots not 256-byte aligned
    assert f(p, 1, p, 8, 256, 1024, 128, 1e-5, None, p, big, ctypes.c_void_p(4096 + 16), big,
             s1, s2) == 3


def test_tiled_layout_definition_matches_header_formula():
    """tests/layout_ref.tile_np against the header's byte formula, byte by byte."""
    import numpy as np
    from tests.layout_ref import tile_np, untile_np
    N, K = 48, 384
    qw = np.random.default_rng(5).integers(0, 256, (N, K // 2), dtype=np.uint8)
    t = tile_np(qw)
    G = K // 128
    for n in range(N):
        for kb in range(K // 2):
            j, hh, i = kb // 64, (kb % 64) // 16, kb % 16
            assert t[16 * (64 * ((n // 16) * G + j) + 16 * hh + n % 16) + i] == qw[n, kb]
    assert np.array_equal(untile_np(t, N, K), qw)


def test_tile_codes_errors_without_launch(lib):
    vp, i64 = ctypes.c_void_p, ctypes.c_int64
    a, b = ctypes.c_void_p(1 << 20), ctypes.c_void_p(1 << 30)   # never dereferenced
    for name in ("qlinear_tile_codes", "qlinear_untile_codes"):
        f = getattr(lib, name)
        f.argtypes = [vp, vp, i64, i64, vp]
        f.restype = ctypes.c_int
        assert f(None, b, 16, 128, None) == 1                          # null pointer
        assert f(a, b, 24, 128, None) == 1                             # N % 16
        assert f(a, b, 16, 100, None) == 1                             # K % 128
        assert f(a, b, 0, 128, None) == 1                              # N <= 0
        assert f(ctypes.c_void_p((1 << 20) + 8), b, 16, 128, None) == 3
        assert f(a, ctypes.c_void_p((1 << 20) + 512), 16, 128, None) == 1   # overlap


def test_tiled_flag_errors_without_launch(lib):
    f = lib.qlinear_forward_ex
    vp, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    f.argtypes = [vp, i64, vp, vp, vp, i64, i64, i64, i64, i32, i32, vp, sz, vp]
    f.restype = ctypes.c_int
    p = ctypes.c_void_p(4096)
    assert f(p, 128, p, p, p, 24, 8, 24, 128, 128, 0x100, None, 0, None) == 1   # tiled, N % 16
    assert f(p, 128, p, p, p, 64, 8, 64, 128, 128, 0x200, None, 0, None) == 2   # unknown flag
    assert f(p, 128, p, p, p, 64, 8, 64, 128, 128, 0x103, None, 0, None) == 2   # unknown epilogue


def test_stack_layout_errors_without_launch(lib):
    class QMat(ctypes.Structure):
        _fields_ = [("qweight", ctypes.c_void_p), ("scales", ctypes.c_void_p),
                    ("layout", ctypes.c_int32)]

    class Layer(ctypes.Structure):
        _fields_ = [(n, QMat) for n in ("qkv", "out", "up", "down")]

    f = lib.qlayer_stack_forward
    vp, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    f.argtypes = [vp, i32, vp, i64, i64, i64, i32, ctypes.c_float, vp, sz, vp]
    f.restype = ctypes.c_int
    p = ctypes.c_void_p(4096)
    L = Layer()
    for n in ("qkv", "out", "up", "down"):
        m = getattr(L, n)
        m.qweight, m.scales, m.layout = 1 << 20, 1 << 21, 0
    L.up.layout = 2                                       # neither ROWS nor TILED
    assert f(ctypes.byref(L), 1, p, 8, 256, 512, 128, 1e-5, p, 1 << 30, None) == 2
    L.up.layout = 1
    L.out.qweight = (1 << 20) + 8                         # misaligned codes
    assert f(ctypes.byref(L), 1, p, 8, 256, 512, 128, 1e-5, p, 1 << 30, None) == 3
