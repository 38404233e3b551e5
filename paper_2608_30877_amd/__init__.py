"""Python binding of libqlinear (int4-weight linear projections on gfx950).

Argument marshalling only: every step of the path runs in the HIP kernels of
``libqlinear.so`` behind the C ABI declared in ``include/qlinear.h``; torch
supplies device memory and streams.  There is no CPU fallback: importing
this package without the built library raises.

bf16 tensors may be passed as ``torch.bfloat16`` or as their 16-bit patterns
(``torch.int16`` / ``torch.uint16``); fp16 scales likewise.
"""
from __future__ import annotations

import ctypes
import os

import torch

__all__ = [
    "LIB_PATH", "QLError", "lib", "GROUP", "EPI_NONE", "EPI_GELU", "EPI_RESID_F32",
    "pack", "dequant", "forward", "forward_ex", "workspace_bytes", "rmsnorm",
    "stack_workspace_bytes", "stack_workspace_offsets", "stack_forward",
    "stack_forward_timed", "make_layers", "attention", "attention_varlen",
    "stack_slot_bytes", "stack_forward_streamed", "stack_forward_noalloc",
    "stack_scratch_capacity", "LAYOUT_ROWS", "LAYOUT_TILED", "EPI_WEIGHTS_TILED",
    "tile_codes", "untile_codes",
]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libqlinear.so")
GROUP = 128
EPI_NONE, EPI_GELU, EPI_RESID_F32 = 0, 1, 2
EPI_WEIGHTS_TILED = 0x100          # flag: qweight in LAYOUT_TILED (forward_ex)
LAYOUT_ROWS, LAYOUT_TILED = 0, 1   # ql_layout


class QLError(RuntimeError):
    def __init__(self, code: int, where: str):
        self.code = code
        super().__init__(f"{where}: status {code} ({_status_string(code)})")


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            f"{LIB_PATH} is missing: build it with `python paper_2608_30877_amd/build.py` "
            "(there is no CPU fallback)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    sig = {
        "qlinear_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "qlinear_pack": (ctypes.c_int, [vp, vp, vp, i64, i64, i32, vp, vp]),
        "qlinear_dequant": (ctypes.c_int, [vp, vp, vp, i64, i64, i32, vp]),
        "qlinear_tile_codes": (ctypes.c_int, [vp, vp, i64, i64, vp]),
        "qlinear_untile_codes": (ctypes.c_int, [vp, vp, i64, i64, vp]),
        "qlinear_forward": (ctypes.c_int, [vp, vp, vp, vp, i64, i64, i64, i32, vp]),
        "qlinear_workspace_bytes": (sz, [i64, i64, i32]),
        "qlinear_forward_ex": (ctypes.c_int, [vp, i64, vp, vp, vp, i64, i64, i64, i64, i32,
                                              i32, vp, sz, vp]),
        "qlayer_stack_workspace_bytes": (sz, [i64, i64, i64, i32]),
        "qlayer_stack_workspace_offsets": (None, [i64, i64, i64, i32,
                                                  ctypes.POINTER(sz), ctypes.POINTER(sz)]),
        "qlayer_stack_forward": (ctypes.c_int, [vp, i32, vp, i64, i64, i64, i32,
                                                ctypes.c_float, vp, sz, vp]),
        "qlayer_stack_forward_timed": (ctypes.c_int, [vp, i32, vp, i64, i64, i64, i32,
                                                      ctypes.c_float, vp, sz, vp, vp]),
        "qlinear_rmsnorm": (ctypes.c_int, [vp, vp, i64, i64, ctypes.c_float, vp]),
        "qlayer_stack_slot_bytes": (sz, [i64, i64, i32]),
        "qlayer_stack_forward_streamed": (ctypes.c_int, [vp, i32, vp, i64, i64, i64, i32,
                                                         ctypes.c_float, vp, vp, sz, vp, sz, vp,
                                                         vp]),
        "qlayer_stack_forward_noalloc": (ctypes.c_int, [vp, i32, vp, i64, i64, i64, i32,
                                                        ctypes.c_float, vp]),
        "qlayer_stack_scratch_capacity": (sz, []),
        "qlinear_attention": (ctypes.c_int, [vp, i64, vp, i64, i64, i64, i32, i32, i32, vp]),
        "qlinear_attention_varlen": (ctypes.c_int, [vp, i64, vp, i64, i64, i64, i32, vp, i32,
                                                    i32, i32, vp]),
        "qlayer_stack_forward_attn": (ctypes.c_int, [vp, i32, vp, i64, i64, i64, i32,
                                                     ctypes.c_float, vp, vp, sz, vp, vp]),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    return L


lib = _load()


def _status_string(code: int) -> str:
    return lib.qlinear_status_string(int(code)).decode()


def _check(code: int, where: str):
    if code != 0:
        raise QLError(code, where)


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _need(t: torch.Tensor, name: str, dtypes, ndim=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be on a CUDA (HIP) device")
    if t.dtype not in dtypes:
        raise TypeError(f"{name}: dtype {t.dtype} not in {dtypes}")
    if ndim is not None and t.dim() != ndim:
        raise ValueError(f"{name} must be {ndim}-D")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous (row-major)")


_BITS16 = (torch.bfloat16, torch.int16, torch.uint16, torch.float16)


class _AttnCfg(ctypes.Structure):
    _fields_ = [("heads", ctypes.c_int32), ("seq_len", ctypes.c_int32),
                ("window", ctypes.c_int32), ("n_seqs", ctypes.c_int32),
                ("cu_seqlens", ctypes.c_void_p)]


def _attn_cfg(attn):
    """None, (heads, seq_len, window) or (heads, cu_seqlens, max_seq_len,
    window) with cu_seqlens a CUDA int32 tensor -> pointer to a
    ql_attention_cfg (or None)."""
    if attn is None:
        return None
    if len(attn) == 3:
        heads, seq_len, window = (int(v) for v in attn)
        return ctypes.pointer(_AttnCfg(heads, seq_len, window, 0, None))
    heads, cu, max_len, window = attn
    _need(cu, "cu_seqlens", (torch.int32,), 1)
    return ctypes.pointer(_AttnCfg(int(heads), int(max_len), int(window), cu.numel() - 1,
                                   cu.data_ptr()))


class _QMat(ctypes.Structure):
    _fields_ = [("qweight", ctypes.c_void_p), ("scales", ctypes.c_void_p),
                ("layout", ctypes.c_int32)]


class _QLayer(ctypes.Structure):
    _fields_ = [(n, _QMat) for n in ("qkv", "out", "up", "down")]


# ---------------------------------------------------------------------------

def pack(w: torch.Tensor, group: int = GROUP, stream=None, check: bool = True,
         status: torch.Tensor | None = None):
    """fp32 W [N, K] -> (qweight uint8 [N, K/2], scales int16 bits [N, K/g]).
    Without `status`, synchronises and raises QLError on QL_ERR_RANGE (when
    check=True).  With a caller's zeroed int32 device `status`, nothing is
    synchronised and the kernel writes QL_ERR_RANGE into it on a range error."""
    _need(w, "w", (torch.float32,), 2)
    w = w.contiguous()
    N, K = w.shape
    qw = torch.empty((N, K // 2), dtype=torch.uint8, device=w.device)
    sc = torch.empty((N, K // group), dtype=torch.int16, device=w.device)
    own = status is None
    if own:
        status = torch.zeros(1, dtype=torch.int32, device=w.device)
    _check(lib.qlinear_pack(_ptr(w), _ptr(qw), _ptr(sc), N, K, group, _ptr(status),
                            _stream(stream)), "qlinear_pack")
    if own and check:
        code = int(status.item())
        _check(code, "qlinear_pack (device status)")
    return qw, sc


def tile_codes(qweight: torch.Tensor, stream=None) -> torch.Tensor:
    """Row-major codes uint8 [N, K/2] -> the same bytes in LAYOUT_TILED order
    (returned as a [N, K/2] uint8 tensor whose rows are not weight rows)."""
    _need(qweight, "qweight", (torch.uint8,), 2)
    N, H = qweight.shape
    out = torch.empty_like(qweight, memory_format=torch.contiguous_format)
    _check(lib.qlinear_tile_codes(_ptr(qweight.contiguous()), _ptr(out), N, 2 * H,
                                  _stream(stream)), "qlinear_tile_codes")
    return out


def untile_codes(tiled: torch.Tensor, stream=None) -> torch.Tensor:
    """Inverse of tile_codes: LAYOUT_TILED bytes [N, K/2] -> row-major codes."""
    _need(tiled, "tiled", (torch.uint8,), 2)
    N, H = tiled.shape
    out = torch.empty_like(tiled, memory_format=torch.contiguous_format)
    _check(lib.qlinear_untile_codes(_ptr(tiled.contiguous()), _ptr(out), N, 2 * H,
                                    _stream(stream)), "qlinear_untile_codes")
    return out


def dequant(qweight: torch.Tensor, scales: torch.Tensor, group: int = GROUP, stream=None):
    _need(qweight, "qweight", (torch.uint8,), 2)
    _need(scales, "scales", _BITS16, 2)
    N, H = qweight.shape
    w = torch.empty((N, 2 * H), dtype=torch.float32, device=qweight.device)
    _check(lib.qlinear_dequant(_ptr(qweight.contiguous()), _ptr(scales.contiguous()), _ptr(w),
                               N, 2 * H, group, _stream(stream)), "qlinear_dequant")
    return w


def forward(x: torch.Tensor, qweight: torch.Tensor, scales: torch.Tensor,
            out: torch.Tensor | None = None, group: int = GROUP, stream=None):
    """out [M, N] bf16 = x [M, K] (bf16) @ dequant(qweight, scales)^T."""
    _need(x, "x", _BITS16, 2)
    _need(qweight, "qweight", (torch.uint8,), 2)
    _need(scales, "scales", _BITS16, 2)
    M, K = x.shape
    N = qweight.shape[0]
    if out is None:
        out = torch.empty((M, N), dtype=torch.bfloat16, device=x.device)
    _need(out, "out", _BITS16, 2)
    _check(lib.qlinear_forward(_ptr(x), _ptr(qweight), _ptr(scales), _ptr(out),
                               M, N, K, group, _stream(stream)), "qlinear_forward")
    return out


def workspace_bytes(M: int, K: int, group: int = GROUP) -> int:
    return int(lib.qlinear_workspace_bytes(M, K, group))


def forward_ex(x, qweight, scales, out, epilogue: int = EPI_NONE, workspace=None,
               M=None, N=None, K=None, ldx=None, ldo=None, group: int = GROUP, stream=None,
               x_ptr=None, tiled: bool = False):
    """Strided / fused-epilogue forward with an optional caller workspace
    (uint8 tensor; None runs the MFMA kernel on x as stored).  x may be a
    strided 2-D view (row stride ldx); out is bf16 for NONE/GELU and fp32
    (updated in place) for RESID_F32.  tiled: qweight holds LAYOUT_TILED
    codes (tile_codes)."""
    if tiled:
        epilogue |= EPI_WEIGHTS_TILED
    M = x.shape[0] if M is None else M
    K = x.shape[1] if K is None else K
    N = qweight.shape[0] if N is None else N
    ldx = x.stride(0) if ldx is None else ldx
    ldo = out.stride(0) if ldo is None else ldo
    xp = ctypes.c_void_p(x.data_ptr()) if x_ptr is None else ctypes.c_void_p(x_ptr)
    ws_ptr = None if workspace is None else ctypes.c_void_p(workspace.data_ptr())
    ws_n = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _check(lib.qlinear_forward_ex(xp, ldx, _ptr(qweight), _ptr(scales), _ptr(out), ldo,
                                  M, N, K, group, epilogue, ws_ptr, ws_n, _stream(stream)),
           "qlinear_forward_ex")
    return out


def rmsnorm(h: torch.Tensor, eps: float = 1e-5, stream=None):
    _need(h, "h", (torch.float32,), 2)
    M, d = h.shape
    a = torch.empty((M, d), dtype=torch.bfloat16, device=h.device)
    _check(lib.qlinear_rmsnorm(_ptr(h.contiguous()), _ptr(a), M, d, eps, _stream(stream)),
           "qlinear_rmsnorm")
    return a


def attention(qkv: torch.Tensor, heads: int, seq_len: int, window: int,
              out: torch.Tensor | None = None, stream=None):
    """Causal sliding-window attention over a [Q | K | V] bf16 buffer
    qkv [M, >= 3d] (row stride qkv.stride(0)), d = 128 * heads; returns
    out [M, d] bf16 (or writes the caller's `out`, row stride out.stride(0))."""
    if not isinstance(qkv, torch.Tensor) or not qkv.is_cuda or qkv.dtype not in _BITS16 \
            or qkv.dim() != 2 or qkv.stride(1) != 1:
        raise ValueError("qkv must be a 2-D CUDA bf16 tensor with unit column stride")
    M = qkv.shape[0]
    d = 128 * int(heads)
    if out is None:
        out = torch.empty((M, d), dtype=torch.bfloat16, device=qkv.device)
    if not isinstance(out, torch.Tensor) or not out.is_cuda or out.dtype not in _BITS16 \
            or out.dim() != 2 or out.stride(1) != 1:
        raise ValueError("out must be a 2-D CUDA bf16 tensor with unit column stride")
    _check(lib.qlinear_attention(_ptr(qkv), qkv.stride(0), _ptr(out), out.stride(0), M, d,
                                 int(heads), int(seq_len), int(window), _stream(stream)),
           "qlinear_attention")
    return out


def attention_varlen(qkv: torch.Tensor, heads: int, cu_seqlens: torch.Tensor,
                     max_seq_len: int, window: int, out: torch.Tensor | None = None,
                     stream=None):
    """attention() over a ragged batch: sequence s is rows cu_seqlens[s] ..
    cu_seqlens[s+1]-1 (cu_seqlens: CUDA int32 [n_seqs + 1])."""
    if not isinstance(qkv, torch.Tensor) or not qkv.is_cuda or qkv.dtype not in _BITS16 \
            or qkv.dim() != 2 or qkv.stride(1) != 1:
        raise ValueError("qkv must be a 2-D CUDA bf16 tensor with unit column stride")
    _need(cu_seqlens, "cu_seqlens", (torch.int32,), 1)
    M = qkv.shape[0]
    d = 128 * int(heads)
    if out is None:
        out = torch.empty((M, d), dtype=torch.bfloat16, device=qkv.device)
    if not isinstance(out, torch.Tensor) or not out.is_cuda or out.dtype not in _BITS16 \
            or out.dim() != 2 or out.stride(1) != 1:
        raise ValueError("out must be a 2-D CUDA bf16 tensor with unit column stride")
    _check(lib.qlinear_attention_varlen(_ptr(qkv), qkv.stride(0), _ptr(out), out.stride(0), M, d,
                                        int(heads), _ptr(cu_seqlens), cu_seqlens.numel() - 1,
                                        int(max_seq_len), int(window), _stream(stream)),
           "qlinear_attention_varlen")
    return out


def stack_workspace_bytes(M: int, d: int, d_ff: int, group: int = GROUP) -> int:
    return int(lib.qlayer_stack_workspace_bytes(M, d, d_ff, group))


def stack_workspace_offsets(M: int, d: int, d_ff: int, group: int = GROUP):
    q, u = ctypes.c_size_t(), ctypes.c_size_t()
    lib.qlayer_stack_workspace_offsets(M, d, d_ff, group, ctypes.byref(q), ctypes.byref(u))
    return int(q.value), int(u.value)


def make_layers(layers):
    """layers: list of dicts {"qkv": (qw, sc), "out": ..., "up": ..., "down": ...}
    of device tensors, each entry optionally (qw, sc, layout) with layout
    LAYOUT_ROWS (default) or LAYOUT_TILED -> ctypes array for stack_forward
    (keep the tensors alive)."""
    arr = (_QLayer * len(layers))()
    for i, L in enumerate(layers):
        for name in ("qkv", "out", "up", "down"):
            q, s, *rest = L[name]
            m = getattr(arr[i], name)
            m.qweight = q.data_ptr()
            m.scales = s.data_ptr()
            m.layout = rest[0] if rest else LAYOUT_ROWS
    return arr


def stack_forward(layers_arr, h: torch.Tensor, d_ff: int, workspace: torch.Tensor,
                  n_layers: int | None = None, eps: float = 1e-5, group: int = GROUP,
                  stream=None, attn=None):
    """Run the linear stack in place on the fp32 residual h [M, d].  attn =
    (heads, seq_len, window) runs sliding-window attention between the QKV
    and out projections over uniform sequences, (heads, cu_seqlens,
    max_seq_len, window) over a ragged batch; None runs the width-1
    stand-in."""
    _need(h, "h", (torch.float32,), 2)
    M, d = h.shape
    n = len(layers_arr) if n_layers is None else n_layers
    ws_n = workspace.numel() * workspace.element_size()
    if attn is None:
        rc = lib.qlayer_stack_forward(ctypes.cast(layers_arr, ctypes.c_void_p), n, _ptr(h), M, d,
                                      d_ff, group, eps, _ptr(workspace), ws_n, _stream(stream))
        _check(rc, "qlayer_stack_forward")
    else:
        rc = lib.qlayer_stack_forward_attn(ctypes.cast(layers_arr, ctypes.c_void_p), n, _ptr(h),
                                           M, d, d_ff, group, eps, _attn_cfg(attn),
                                           _ptr(workspace), ws_n, None, _stream(stream))
        _check(rc, "qlayer_stack_forward_attn")
    return h


def stack_forward_timed(layers_arr, h: torch.Tensor, d_ff: int, workspace: torch.Tensor,
                        events, n_layers: int | None = None, eps: float = 1e-5,
                        group: int = GROUP, stream=None, attn=None):
    """stack_forward with events: a list of 8 * n_layers torch.cuda.Event
    (enable_timing=True) recorded around each projection launch."""
    _need(h, "h", (torch.float32,), 2)
    M, d = h.shape
    n = len(layers_arr) if n_layers is None else n_layers
    if len(events) != 8 * n:
        raise ValueError("need 8 events per block")
    st = torch.cuda.current_stream() if stream is None else stream
    for e in events:                      # materialise the handles
        if e.cuda_event == 0:
            e.record(st)
    ev_arr = (ctypes.c_void_p * len(events))(*[e.cuda_event for e in events])
    ws_n = workspace.numel() * workspace.element_size()
    if attn is None:
        rc = lib.qlayer_stack_forward_timed(ctypes.cast(layers_arr, ctypes.c_void_p), n, _ptr(h),
                                            M, d, d_ff, group, eps, _ptr(workspace), ws_n,
                                            ctypes.cast(ev_arr, ctypes.c_void_p), _stream(st))
        _check(rc, "qlayer_stack_forward_timed")
    else:
        rc = lib.qlayer_stack_forward_attn(ctypes.cast(layers_arr, ctypes.c_void_p), n, _ptr(h),
                                           M, d, d_ff, group, eps, _attn_cfg(attn),
                                           _ptr(workspace), ws_n,
                                           ctypes.cast(ev_arr, ctypes.c_void_p), _stream(st))
        _check(rc, "qlayer_stack_forward_attn")
    return h


def stack_forward_noalloc(layers_arr, h: torch.Tensor, d_ff: int, n_layers: int | None = None,
                          eps: float = 1e-5, group: int = GROUP, stream=None):
    """stack_forward with the workspace in the library's fixed device scratch
    (no caller buffer, no allocation; calls overlapping on one GPU race)."""
    _need(h, "h", (torch.float32,), 2)
    M, d = h.shape
    n = len(layers_arr) if n_layers is None else n_layers
    rc = lib.qlayer_stack_forward_noalloc(ctypes.cast(layers_arr, ctypes.c_void_p), n, _ptr(h),
                                          M, d, d_ff, group, eps, _stream(stream))
    _check(rc, "qlayer_stack_forward_noalloc")
    return h


def stack_scratch_capacity() -> int:
    return int(lib.qlayer_stack_scratch_capacity())


def stack_slot_bytes(d: int, d_ff: int, group: int = GROUP) -> int:
    return int(lib.qlayer_stack_slot_bytes(d, d_ff, group))


def stack_forward_streamed(host_layers_arr, h: torch.Tensor, d_ff: int, workspace: torch.Tensor,
                           slots: torch.Tensor, copy_stream, n_layers: int | None = None,
                           eps: float = 1e-5, group: int = GROUP, stream=None, attn=None):
    """stack_forward with the packed weights in page-locked host memory
    (make_layers over pinned CPU tensors), copied block by block into the two
    device slots of `slots` (uint8 CUDA tensor of 2 * stack_slot_bytes) on
    `copy_stream` while the previous block computes on `stream`.  Keep the
    host tensors and slots alive until `stream` has finished."""
    _need(h, "h", (torch.float32,), 2)
    M, d = h.shape
    n = len(host_layers_arr) if n_layers is None else n_layers
    ws_n = workspace.numel() * workspace.element_size()
    sl_n = slots.numel() * slots.element_size()
    rc = lib.qlayer_stack_forward_streamed(ctypes.cast(host_layers_arr, ctypes.c_void_p), n,
                                           _ptr(h), M, d, d_ff, group, eps, _attn_cfg(attn),
                                           _ptr(workspace), ws_n, _ptr(slots), sl_n,
                                           _stream(stream), _stream(copy_stream))
    _check(rc, "qlayer_stack_forward_streamed")
    return h

