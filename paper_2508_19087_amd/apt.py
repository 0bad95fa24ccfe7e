"""Python binding of libapt.so (include/apt.h): argument marshalling only.

Every function named ``apt_*`` calls the C entry point of the same name with
plain integers and device pointers.  The torch helpers below (``pack``,
``gemm``, ...) only allocate outputs with torch and pass ``data_ptr()`` and the
current HIP stream; every step of the computation runs in the library's
kernels.  Importing this module fails loudly when the library is not built.
"""
from __future__ import annotations

import ctypes
import os
import re
from dataclasses import dataclass

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libapt.so")
HEADER_PATH = os.path.join(os.path.dirname(_HERE), "include", "apt.h")

APT_OK = 0
APT_ERR_INVALID_ARG = 1
APT_ERR_UNSUPPORTED = 2
APT_ERR_HIP = 3
APT_ERR_WORKSPACE = 4

APT_ROUTE_AUTO = 0
APT_ROUTE_XOR = 1
APT_ROUTE_PM1_MFMA = 2
APT_ROUTE_INT8_MFMA = 3
APT_ROUTE_FP4_MFMA = 4
APT_ROUTE_FP6_MFMA = 5
APT_ROUTE_FP8_MFMA = 6
APT_ACT_CODES = 1
APT_ACT_FP16 = 2
APT_DECODE_MAX_M = 8
ROUTE_NAMES = {APT_ROUTE_XOR: "xor_popcount", APT_ROUTE_PM1_MFMA: "pm1_planes_mfma",
               APT_ROUTE_INT8_MFMA: "reassembled_int8_mfma", APT_ROUTE_FP4_MFMA: "reassembled_fp4_mfma",
               APT_ROUTE_FP6_MFMA: "reassembled_fp6_mfma", APT_ROUTE_FP8_MFMA: "reassembled_fp8_mfma"}


class apt_config_t(ctypes.Structure):
    _fields_ = [("route", ctypes.c_int32), ("bm", ctypes.c_int32), ("bn", ctypes.c_int32),
                ("bk", ctypes.c_int32), ("waves_m", ctypes.c_int32), ("waves_n", ctypes.c_int32),
                ("grid", ctypes.c_int32), ("lds_stages", ctypes.c_int32), ("mt", ctypes.c_int32),
                ("split_n", ctypes.c_int32), ("tail_bm", ctypes.c_int32), ("tail_bn", ctypes.c_int32),
                ("tail_grid", ctypes.c_int32), ("reserved", ctypes.c_int32 * 3)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_ if f != "reserved"}

    @classmethod
    def make(cls, route, bm=0, bn=0, bk=0, waves_m=0, waves_n=0, grid=0, lds_stages=0, mt=0,
             split_n=0, tail_bm=0, tail_bn=0, tail_grid=0):
        c = cls()
        c.route, c.bm, c.bn, c.bk = route, bm, bn, bk
        c.waves_m, c.waves_n, c.grid, c.lds_stages, c.mt = waves_m, waves_n, grid, lds_stages, mt
        c.split_n, c.tail_bm, c.tail_bn, c.tail_grid = split_n, tail_bm, tail_bn, tail_grid
        return c


class AptError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        self.hip_error = apt_last_hip_error() if status == APT_ERR_HIP else 0
        extra = ", hipError_t %d" % self.hip_error if status == APT_ERR_HIP else ""
        super().__init__("%s: %s (status %d%s)" % (where, status_string(status), status, extra))


_vp = ctypes.c_void_p
_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libapt.so is not built (run __graft_entry__.build() or "
                              "python paper_2508_19087_amd/build.py): %s" % LIB_PATH)
        # torch's HIP runtime must be loaded first: the library's libamdhip64
        # dependency then binds to the runtime that owns torch's device memory
        # and streams, not to a second copy of it.
        import torch  # noqa: F401
        L = ctypes.CDLL(LIB_PATH)
        L.apt_packed_bytes.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int]
        L.apt_packed_bytes.restype = ctypes.c_size_t
        for name in ("apt_pack_weights", "apt_quantize_pack_activations"):
            f = getattr(L, name)
            f.argtypes = [_vp, ctypes.c_int, ctypes.c_int, ctypes.c_int, _vp, _vp, _vp]
            f.restype = ctypes.c_int
        L.apt_quantize_pack_activations_fp16.argtypes = [_vp, ctypes.c_int, ctypes.c_int,
                                                         ctypes.c_int, _vp, _vp, _vp, _vp]
        L.apt_quantize_pack_activations_fp16.restype = ctypes.c_int
        L.apt_select_config.argtypes = [ctypes.c_int] * 5 + [ctypes.POINTER(apt_config_t)]
        L.apt_select_config.restype = ctypes.c_int
        L.apt_gemm_workspace_bytes.argtypes = [ctypes.c_int] * 5 + [ctypes.POINTER(apt_config_t)]
        L.apt_gemm_workspace_bytes.restype = ctypes.c_size_t
        L.apt_gemm.argtypes = ([ctypes.c_int] * 5 + [_vp] * 8 + [ctypes.POINTER(apt_config_t)] +
                               [_vp, ctypes.c_size_t, _vp])
        L.apt_gemm.restype = ctypes.c_int
        L.apt_gemm_noalloc.argtypes = ([ctypes.c_int] * 5 + [_vp] * 8 +
                                       [ctypes.POINTER(apt_config_t), _vp])
        L.apt_gemm_noalloc.restype = ctypes.c_int
        L.apt_gemm_affine.argtypes = ([ctypes.c_int] * 5 + [_vp] * 10 +
                                      [ctypes.POINTER(apt_config_t)] + [_vp, ctypes.c_size_t, _vp])
        L.apt_gemm_affine.restype = ctypes.c_int
        L.apt_gemm_decode.argtypes = ([ctypes.c_int] * 5 + [_vp, ctypes.c_int] + [_vp] * 6 +
                                      [ctypes.POINTER(apt_config_t), _vp])
        L.apt_gemm_decode.restype = ctypes.c_int
        L.apt_gemm_act_workspace_bytes.argtypes = [ctypes.c_int] * 6 + [ctypes.POINTER(apt_config_t)]
        L.apt_gemm_act_workspace_bytes.restype = ctypes.c_size_t
        L.apt_gemm_act.argtypes = ([ctypes.c_int] * 5 + [_vp, ctypes.c_int] + [_vp] * 7 +
                                   [ctypes.POINTER(apt_config_t), _vp, ctypes.c_size_t, _vp])
        L.apt_gemm_act.restype = ctypes.c_int
        L.apt_search_workspace_bytes.argtypes = [ctypes.c_int] * 5
        L.apt_search_workspace_bytes.restype = ctypes.c_size_t
        L.apt_search_config.argtypes = ([ctypes.c_int] * 5 + [_vp] * 6 + [ctypes.c_size_t, _vp,
                                        ctypes.POINTER(apt_config_t), ctypes.POINTER(ctypes.c_float)])
        L.apt_search_config.restype = ctypes.c_int
        L.apt_config_table_clear.argtypes = []
        L.apt_config_table_clear.restype = None
        L.apt_config_table_size.argtypes = []
        L.apt_config_table_size.restype = ctypes.c_int
        L.apt_last_hip_error.argtypes = []
        L.apt_last_hip_error.restype = ctypes.c_int
        L.apt_status_string.argtypes = [ctypes.c_int]
        L.apt_status_string.restype = ctypes.c_char_p
        _lib = L
    return _lib


def header_functions() -> list:
    """Names of the functions include/apt.h declares."""
    text = open(HEADER_PATH).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(apt_[a-z0-9_]+)\s*\(", text)))


# ---- C entry points, same names -------------------------------------------------

def apt_packed_bytes(rows: int, K: int, bits: int) -> int:
    return int(lib().apt_packed_bytes(rows, K, bits))


def apt_pack_weights(w_codes, N, K, p, w_packed, w_rowsum, stream) -> int:
    return lib().apt_pack_weights(w_codes, N, K, p, w_packed, w_rowsum, stream)


def apt_quantize_pack_activations(a_codes, M, K, q, a_packed, a_rowsum, stream) -> int:
    return lib().apt_quantize_pack_activations(a_codes, M, K, q, a_packed, a_rowsum, stream)


def apt_quantize_pack_activations_fp16(a_fp16, M, K, q, a_packed, a_rowsum, a_scale,
                                       stream) -> int:
    return lib().apt_quantize_pack_activations_fp16(a_fp16, M, K, q, a_packed, a_rowsum, a_scale,
                                                    stream)


def apt_select_config(M, N, K, p, q):
    """(status, apt_config_t)."""
    c = apt_config_t()
    st = lib().apt_select_config(M, N, K, p, q, ctypes.byref(c))
    return st, c


def apt_gemm_workspace_bytes(M, N, K, p, q, cfg=None) -> int:
    return int(lib().apt_gemm_workspace_bytes(M, N, K, p, q, ctypes.byref(cfg) if cfg else None))


def apt_gemm(M, N, K, p, q, a_packed, w_packed, a_rowsum, w_rowsum, c_int32, a_scale, w_scale,
             c_fp16, cfg, workspace, workspace_bytes, stream) -> int:
    return lib().apt_gemm(M, N, K, p, q, a_packed, w_packed, a_rowsum, w_rowsum, c_int32,
                          a_scale, w_scale, c_fp16, ctypes.byref(cfg) if cfg is not None else None,
                          workspace, workspace_bytes, stream)


def apt_gemm_noalloc(M, N, K, p, q, a_packed, w_packed, a_rowsum, w_rowsum, c_int32, a_scale,
                     w_scale, c_fp16, cfg, stream) -> int:
    return lib().apt_gemm_noalloc(M, N, K, p, q, a_packed, w_packed, a_rowsum, w_rowsum, c_int32,
                                  a_scale, w_scale, c_fp16,
                                  ctypes.byref(cfg) if cfg is not None else None, stream)


def apt_gemm_affine(M, N, K, p, q, a_packed, w_packed, a_rowsum, w_rowsum, a_scale, a_zero,
                    w_scale, w_zero, c_fp16, c_int32, cfg, workspace, workspace_bytes,
                    stream) -> int:
    return lib().apt_gemm_affine(M, N, K, p, q, a_packed, w_packed, a_rowsum, w_rowsum, a_scale,
                                 a_zero, w_scale, w_zero, c_fp16, c_int32,
                                 ctypes.byref(cfg) if cfg is not None else None, workspace,
                                 workspace_bytes, stream)


def apt_gemm_decode(M, N, K, p, q, a_src, a_kind, w_packed, c_int32, a_scale, w_scale, c_fp16,
                    a_scale_out, cfg, stream) -> int:
    return lib().apt_gemm_decode(M, N, K, p, q, a_src, a_kind, w_packed, c_int32, a_scale,
                                 w_scale, c_fp16, a_scale_out,
                                 ctypes.byref(cfg) if cfg is not None else None, stream)


def apt_gemm_act_workspace_bytes(M, N, K, p, q, a_kind, cfg=None) -> int:
    return int(lib().apt_gemm_act_workspace_bytes(M, N, K, p, q, a_kind,
                                                  ctypes.byref(cfg) if cfg else None))


def apt_gemm_act(M, N, K, p, q, a_src, a_kind, w_packed, w_rowsum, c_int32, a_scale, w_scale,
                 c_fp16, a_scale_out, cfg, workspace, workspace_bytes, stream) -> int:
    return lib().apt_gemm_act(M, N, K, p, q, a_src, a_kind, w_packed, w_rowsum, c_int32, a_scale,
                              w_scale, c_fp16, a_scale_out,
                              ctypes.byref(cfg) if cfg is not None else None, workspace,
                              workspace_bytes, stream)


def apt_search_workspace_bytes(M, N, K, p, q) -> int:
    return int(lib().apt_search_workspace_bytes(M, N, K, p, q))


def apt_search_config(M, N, K, p, q, a_packed, w_packed, a_rowsum, w_rowsum, c_int32, workspace,
                      workspace_bytes, stream):
    """(status, apt_config_t, microseconds per call)."""
    c = apt_config_t()
    us = ctypes.c_float(0.0)
    st = lib().apt_search_config(M, N, K, p, q, a_packed, w_packed, a_rowsum, w_rowsum, c_int32,
                                 workspace, workspace_bytes, stream, ctypes.byref(c),
                                 ctypes.byref(us))
    return st, c, float(us.value)


def apt_config_table_clear() -> None:
    lib().apt_config_table_clear()


def apt_config_table_size() -> int:
    return int(lib().apt_config_table_size())


def apt_last_hip_error() -> int:
    return int(lib().apt_last_hip_error())


def status_string(status: int) -> str:
    return lib().apt_status_string(status).decode()


def check(status: int, where: str):
    if status != APT_OK:
        raise AptError(status, where)


# ---- torch helpers (allocation + pointers only) -------------------------------

def _torch():
    import torch
    return torch


def _stream_ptr(stream=None):
    torch = _torch()
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def _on_stream(stream):
    """Context in which torch allocations belong to `stream` (the stream the
    library's kernels use): the caching allocator then does not hand a block
    to other work while those kernels may still use it."""
    import contextlib
    torch = _torch()
    if stream is None:
        return contextlib.nullcontext()
    return torch.cuda.stream(stream)


def _ptr(t):
    return None if t is None else t.data_ptr()


@dataclass
class Packed:
    """A packed bit-plane operand on the device: uint8 buffer + int32 row sums."""
    data: "object"
    rowsum: "object"
    rows: int
    K: int
    bits: int


def pack(codes, bits: int, activations: bool = False, stream=None) -> Packed:
    """Packs int8 codes [rows][K] (a CUDA tensor) into bit-planes on the device."""
    torch = _torch()
    assert codes.is_cuda and codes.dtype == torch.int8 and codes.dim() == 2
    codes = codes.contiguous()
    rows, K = codes.shape
    nbytes = apt_packed_bytes(rows, K, bits)
    if nbytes == 0:
        raise AptError(APT_ERR_INVALID_ARG, "apt_packed_bytes")
    with _on_stream(stream):
        buf = torch.empty(nbytes, dtype=torch.uint8, device=codes.device)
        rs = torch.empty(rows, dtype=torch.int32, device=codes.device)
    fn = apt_quantize_pack_activations if activations else apt_pack_weights
    check(fn(codes.data_ptr(), rows, K, bits, buf.data_ptr(), rs.data_ptr(), _stream_ptr(stream)),
          fn.__name__)
    return Packed(buf, rs, rows, K, bits)


def quantize_pack(x, bits: int, stream=None):
    """Quantizes fp16 activations x [M][K] (a CUDA tensor) per row to bipolar
    codes and packs them on the device.  Returns (Packed, fp16 scales [M])."""
    torch = _torch()
    assert x.is_cuda and x.dtype == torch.float16 and x.dim() == 2
    x = x.contiguous()
    rows, K = x.shape
    nbytes = apt_packed_bytes(rows, K, bits)
    if nbytes == 0:
        raise AptError(APT_ERR_INVALID_ARG, "apt_packed_bytes")
    with _on_stream(stream):
        buf = torch.empty(nbytes, dtype=torch.uint8, device=x.device)
        rs = torch.empty(rows, dtype=torch.int32, device=x.device)
        scale = torch.empty(rows, dtype=torch.float16, device=x.device)
    check(apt_quantize_pack_activations_fp16(x.data_ptr(), rows, K, bits, buf.data_ptr(),
                                             rs.data_ptr(), scale.data_ptr(), _stream_ptr(stream)),
          "apt_quantize_pack_activations_fp16")
    return Packed(buf, rs, rows, K, bits), scale


def gemm(a: Packed, w: Packed, out_int32: bool = True, a_scale=None, w_scale=None,
         out_fp16: bool = False, cfg: apt_config_t | None = None, stream=None, workspace=None):
    """C = A W^T on packed operands.  Returns (c_int32 or None, c_fp16 or None).
    A workspace of apt_gemm_workspace_bytes is allocated with torch unless one
    is passed."""
    torch = _torch()
    assert a.K == w.K
    M, N, K = a.rows, w.rows, a.K
    dev = a.data.device
    ws_bytes = apt_gemm_workspace_bytes(M, N, K, w.bits, a.bits, cfg)
    with _on_stream(stream):
        c32 = torch.empty((M, N), dtype=torch.int32, device=dev) if out_int32 else None
        c16 = torch.empty((M, N), dtype=torch.float16, device=dev) if out_fp16 else None
        if workspace is None and ws_bytes > 0:
            workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    ws_ptr = workspace.data_ptr() if workspace is not None else None
    ws_len = workspace.numel() * workspace.element_size() if workspace is not None else 0
    check(apt_gemm(M, N, K, w.bits, a.bits, a.data.data_ptr(), w.data.data_ptr(),
                   _ptr(a.rowsum), _ptr(w.rowsum), _ptr(c32), _ptr(a_scale), _ptr(w_scale),
                   _ptr(c16), cfg, ws_ptr, ws_len, _stream_ptr(stream)), "apt_gemm")
    return c32, c16


def gemm_decode(x, q: int, w: Packed, out_int32: bool = True, a_scale=None, w_scale=None,
                out_fp16: bool = False, cfg: apt_config_t | None = None, stream=None):
    """Decode GEMM on unpacked activations x [M][K] (M <= 8, a CUDA tensor):
    int8 q-bit codes, or fp16 values quantized per row inside the kernel.
    Returns (c_int32 or None, c_fp16 or None, scales): the fp16 row scales the
    kernel computed for fp16 x, else None."""
    torch = _torch()
    assert x.is_cuda and x.dim() == 2 and x.dtype in (torch.int8, torch.float16)
    x = x.contiguous()
    M, K = x.shape
    assert K == w.K
    N = w.rows
    fp16_src = x.dtype == torch.float16
    dev = x.device
    with _on_stream(stream):
        c32 = torch.empty((M, N), dtype=torch.int32, device=dev) if out_int32 else None
        c16 = torch.empty((M, N), dtype=torch.float16, device=dev) if out_fp16 else None
        scale = torch.empty(M, dtype=torch.float16, device=dev) if fp16_src else None
    check(apt_gemm_decode(M, N, K, w.bits, q, x.data_ptr(),
                          APT_ACT_FP16 if fp16_src else APT_ACT_CODES, w.data.data_ptr(),
                          _ptr(c32), _ptr(a_scale), _ptr(w_scale), _ptr(c16), _ptr(scale), cfg,
                          _stream_ptr(stream)), "apt_gemm_decode")
    return c32, c16, scale


def gemm_act(x, q: int, w: Packed, out_int32: bool = True, a_scale=None, w_scale=None,
             out_fp16: bool = False, cfg: apt_config_t | None = None, stream=None,
             workspace=None):
    """C = A W^T for unpacked activations x [M][K] (a CUDA tensor: int8 q-bit
    codes, or fp16 values quantized per row inside the call), any M.  Returns
    (c_int32 or None, c_fp16 or None, scales): the fp16 row scales for fp16 x,
    else None.  A workspace of apt_gemm_act_workspace_bytes is allocated with
    torch unless one is passed."""
    torch = _torch()
    assert x.is_cuda and x.dim() == 2 and x.dtype in (torch.int8, torch.float16)
    x = x.contiguous()
    M, K = x.shape
    assert K == w.K
    N = w.rows
    kind = APT_ACT_FP16 if x.dtype == torch.float16 else APT_ACT_CODES
    dev = x.device
    ws_bytes = apt_gemm_act_workspace_bytes(M, N, K, w.bits, q, kind, cfg)
    with _on_stream(stream):
        c32 = torch.empty((M, N), dtype=torch.int32, device=dev) if out_int32 else None
        c16 = torch.empty((M, N), dtype=torch.float16, device=dev) if out_fp16 else None
        scale = torch.empty(M, dtype=torch.float16, device=dev) if kind == APT_ACT_FP16 else None
        if workspace is None and ws_bytes > 0:
            workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    ws_ptr = workspace.data_ptr() if workspace is not None else None
    ws_len = workspace.numel() * workspace.element_size() if workspace is not None else 0
    check(apt_gemm_act(M, N, K, w.bits, q, x.data_ptr(), kind, w.data.data_ptr(), _ptr(w.rowsum),
                       _ptr(c32), _ptr(a_scale), _ptr(w_scale), _ptr(c16), _ptr(scale), cfg,
                       ws_ptr, ws_len, _stream_ptr(stream)), "apt_gemm_act")
    return c32, c16, scale


def gemm_affine(a: Packed, w: Packed, a_scale, a_zero, w_scale, w_zero, out_int32: bool = False,
                cfg: apt_config_t | None = None, stream=None, workspace=None):
    """fp16 product of two zero-point quantizers in bipolar form (scales and
    zeros are fp16 CUDA tensors [M] / [N]).  Returns (c_fp16, c_int32 or None)."""
    torch = _torch()
    assert a.K == w.K
    M, N, K = a.rows, w.rows, a.K
    dev = a.data.device
    ws_bytes = apt_gemm_workspace_bytes(M, N, K, w.bits, a.bits, cfg)
    with _on_stream(stream):
        c16 = torch.empty((M, N), dtype=torch.float16, device=dev)
        c32 = torch.empty((M, N), dtype=torch.int32, device=dev) if out_int32 else None
        if workspace is None and ws_bytes > 0:
            workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=dev)
    ws_ptr = workspace.data_ptr() if workspace is not None else None
    ws_len = workspace.numel() * workspace.element_size() if workspace is not None else 0
    check(apt_gemm_affine(M, N, K, w.bits, a.bits, a.data.data_ptr(), w.data.data_ptr(),
                          _ptr(a.rowsum), _ptr(w.rowsum), _ptr(a_scale), _ptr(a_zero),
                          _ptr(w_scale), _ptr(w_zero), _ptr(c16), _ptr(c32), cfg, ws_ptr, ws_len,
                          _stream_ptr(stream)), "apt_gemm_affine")
    return c16, c32


def search_config(a: Packed, w: Packed, stream=None):
    """Runs the search module on packed operands (device tensors); returns
    (best apt_config_t, microseconds per call).  The result is recorded in the
    library's table for this (M, N, K, p, q)."""
    torch = _torch()
    assert a.K == w.K
    M, N, K = a.rows, w.rows, a.K
    dev = a.data.device
    ws_bytes = apt_search_workspace_bytes(M, N, K, w.bits, a.bits)
    with _on_stream(stream):
        c32 = torch.empty((M, N), dtype=torch.int32, device=dev)
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev) if ws_bytes > 0 else None
    st, c, us = apt_search_config(M, N, K, w.bits, a.bits, a.data.data_ptr(), w.data.data_ptr(),
                                  a.rowsum.data_ptr(), w.rowsum.data_ptr(), c32.data_ptr(),
                                  ws.data_ptr() if ws is not None else None, ws_bytes,
                                  _stream_ptr(stream))
    check(st, "apt_search_config")
    return c, us


def select_config(M, N, K, p, q) -> apt_config_t:
    st, c = apt_select_config(M, N, K, p, q)
    check(st, "apt_select_config")
    return c
