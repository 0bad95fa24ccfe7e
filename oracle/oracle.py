"""CPU oracle for the WpAq bipolar-INT GEMM (APT-LLM, arXiv 2508.19087).

TEST INFRASTRUCTURE ONLY: imported by ``tests/``, ``__graft_entry__.smoke()``
and the ``cpu_baseline`` leg of ``bench.py``; nothing in the GPU package
imports it, and it imports nothing from the GPU package.

The integer parts live in ``apt_oracle.c`` (plain loops, int64 accumulation);
this module wraps them with ctypes and adds the fp16 scale epilogue, which is
evaluated exactly in float64 and rounded to fp16 by numpy (round to nearest
even).  Exactness: |C| < 2^31 and each fp16 scale carries 11 significant bits,
so C * s_a * s_w needs at most 31 + 11 + 11 = 53 bits and is exact in float64.
It also holds the zero-point epilogue of two linear quantizers in bipolar form
(``dequant_matmul``, the definition; ``affine_epilogue``, the expanded form
from the integer GEMM and the row sums) and the per-token fp16 activation
quantizer (``quantize_fp16``).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "apt_oracle.c")
_LIB = os.path.join(_HERE, "libapt_oracle.so")

_i8p = ctypes.POINTER(ctypes.c_int8)
_u8p = ctypes.POINTER(ctypes.c_uint8)
_i32p = ctypes.POINTER(ctypes.c_int32)
_u32p = ctypes.POINTER(ctypes.c_uint32)


def build(force: bool = False) -> str:
    """Compiles ``apt_oracle.c`` into ``libapt_oracle.so`` with gcc."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-Wall", "-Wextra", _SRC, "-o", tmp])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        L.apt_oracle_convert.argtypes = [_i8p, ctypes.c_int64, ctypes.c_int, _u8p]
        L.apt_oracle_decode.argtypes = [_u8p, ctypes.c_int64, ctypes.c_int, _i32p]
        L.apt_oracle_matmul.argtypes = [_i32p, _i32p, ctypes.c_int, ctypes.c_int, ctypes.c_int, _i32p]
        L.apt_oracle_matmul.restype = ctypes.c_int64
        L.apt_oracle_matmul_entries.argtypes = [_i32p, _i32p, ctypes.c_int, _i32p, _i32p,
                                                ctypes.c_int64, _i32p]
        L.apt_oracle_matmul_entries.restype = ctypes.c_int64
        L.apt_oracle_rowsum.argtypes = [_i32p, ctypes.c_int, ctypes.c_int, _i32p]
        L.apt_oracle_pack.argtypes = [_u8p, ctypes.c_int, ctypes.c_int, ctypes.c_int, _u32p]
        L.apt_oracle_unpack.argtypes = [_u32p, ctypes.c_int, ctypes.c_int, ctypes.c_int, _u8p]
        L.apt_oracle_unpack.restype = ctypes.c_int64
        L.apt_oracle_num_threads.restype = ctypes.c_int
        _lib = L
    return _lib


def _ptr(a: np.ndarray, t):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(t)


def num_threads() -> int:
    return int(lib().apt_oracle_num_threads())


def convert(codes: np.ndarray, bits: int) -> np.ndarray:
    """Signed b-bit codes (int8) -> bipolar words u (uint8), Sec. III-A."""
    x = np.ascontiguousarray(codes, dtype=np.int8)
    u = np.empty(x.shape, dtype=np.uint8)
    if lib().apt_oracle_convert(_ptr(x, _i8p), x.size, bits, _ptr(u, _u8p)) != 0:
        raise ValueError("bits must be in [1, 8]")
    return u


def decode(u: np.ndarray, bits: int) -> np.ndarray:
    """Bipolar words -> decimal values (int32), Sec. III-A value equation."""
    u = np.ascontiguousarray(u, dtype=np.uint8)
    v = np.empty(u.shape, dtype=np.int32)
    if lib().apt_oracle_decode(_ptr(u, _u8p), u.size, bits, _ptr(v, _i32p)) != 0:
        raise ValueError("bits must be in [1, 8]")
    return v


def values(codes: np.ndarray, bits: int) -> np.ndarray:
    """Decimal bipolar values of signed codes: decode(convert(codes))."""
    return decode(convert(codes, bits), bits)


def matmul(va: np.ndarray, vw: np.ndarray) -> np.ndarray:
    """C = va @ vw.T with int64 accumulation; raises if an entry leaves int32."""
    va = np.ascontiguousarray(va, dtype=np.int32)
    vw = np.ascontiguousarray(vw, dtype=np.int32)
    M, K = va.shape
    N, K2 = vw.shape
    assert K == K2
    C = np.empty((M, N), dtype=np.int32)
    ov = lib().apt_oracle_matmul(_ptr(va, _i32p), _ptr(vw, _i32p), M, N, K, _ptr(C, _i32p))
    if ov:
        raise OverflowError("%d entries exceed int32" % ov)
    return C


def matmul_entries(va: np.ndarray, vw: np.ndarray, m_idx, n_idx) -> np.ndarray:
    """C[m_idx[t], n_idx[t]] for each t, from the decoded values."""
    va = np.ascontiguousarray(va, dtype=np.int32)
    vw = np.ascontiguousarray(vw, dtype=np.int32)
    mi = np.ascontiguousarray(m_idx, dtype=np.int32)
    ni = np.ascontiguousarray(n_idx, dtype=np.int32)
    assert mi.shape == ni.shape and va.shape[1] == vw.shape[1]
    out = np.empty(mi.shape, dtype=np.int32)
    ov = lib().apt_oracle_matmul_entries(_ptr(va, _i32p), _ptr(vw, _i32p), va.shape[1],
                                         _ptr(mi, _i32p), _ptr(ni, _i32p), mi.size,
                                         _ptr(out, _i32p))
    if ov:
        raise OverflowError("%d entries exceed int32" % ov)
    return out


def rowsum(v: np.ndarray) -> np.ndarray:
    v = np.ascontiguousarray(v, dtype=np.int32)
    R, K = v.shape
    out = np.empty(R, dtype=np.int32)
    lib().apt_oracle_rowsum(_ptr(v, _i32p), R, K, _ptr(out, _i32p))
    return out


def packed_words(rows: int, K: int, bits: int) -> int:
    return (rows + 7) // 8 * 8 * ((K + 127) // 128) * bits * 4


def pack(u: np.ndarray, bits: int) -> np.ndarray:
    """Reference packed buffer (uint32 words) of bipolar words u [R][K]."""
    u = np.ascontiguousarray(u, dtype=np.uint8)
    R, K = u.shape
    out = np.empty(packed_words(R, K, bits), dtype=np.uint32)
    if lib().apt_oracle_pack(_ptr(u, _u8p), R, K, bits, _ptr(out, _u32p)) != 0:
        raise ValueError("bad arguments")
    return out


def unpack(words: np.ndarray, R: int, K: int, bits: int):
    """(u [R][K], number of non-zero padding elements) from a packed buffer."""
    w = np.ascontiguousarray(words, dtype=np.uint32)
    assert w.size == packed_words(R, K, bits)
    u = np.empty((R, K), dtype=np.uint8)
    stray = lib().apt_oracle_unpack(_ptr(w, _u32p), R, K, bits, _ptr(u, _u8p))
    if stray < 0:
        raise ValueError("bad arguments")
    return u, int(stray)


def gemm(a_codes: np.ndarray, w_codes: np.ndarray, p: int, q: int) -> np.ndarray:
    """Exact C = A W^T (int32) for signed q-bit activation and p-bit weight codes."""
    return matmul(values(a_codes, q), values(w_codes, p))


def epilogue(C: np.ndarray, a_scale: np.ndarray, w_scale: np.ndarray):
    """(E, H): the exact float64 product C[m,n] * a_scale[m] * w_scale[n] and its
    fp16 rounding (nearest even).  Scales are numpy float16 arrays."""
    sa = np.asarray(a_scale, dtype=np.float16).astype(np.float64)
    sw = np.asarray(w_scale, dtype=np.float16).astype(np.float64)
    E = np.asarray(C, dtype=np.int64).astype(np.float64) * sa[:, None] * sw[None, :]
    with np.errstate(over="ignore"):
        H = E.astype(np.float16)
    return E, H


FP16_REL_TOL = 1e-3
FP16_ABS_TOL = 2.0 ** -25


def fp16_close(g: np.ndarray, E: np.ndarray) -> np.ndarray:
    """Element-wise acceptance of a GPU fp16 result g against the exact value E:
    |g - E| <= 1e-3 |E|, or |g - E| <= 2^-25 for values near zero."""
    g = np.asarray(g, dtype=np.float16).astype(np.float64)
    d = np.abs(g - E)
    return (d <= FP16_REL_TOL * np.abs(E)) | (d <= FP16_ABS_TOL)


def quantize_fp16(x: np.ndarray, q: int):
    """Per-token quantization of fp16 activations to q-bit bipolar-INT codes.

    The paper quantizes activations linearly and rewrites the signed-INT
    quantizer in bipolar form (Sec. III-A: value 2x + 1, scale s/2); it does
    not fix the rounding.  This follows the reading used throughout this
    repository: the bipolar scale of row m is
        s_m = fp16(absmax_k |x[m,k]| / (2^q - 1))      (fp32 divide, RNE)
    so the largest magnitude lands on the outermost odd level, and each
    element goes to the odd level 2 floor(t / 2) + 1 of t = x / s_m (fp32
    divide), clamped to +-(2^q - 1): the nearest odd integer, ties upward.
    A row whose scale is 0 gets t = 0 (level +1; its values dequantize to 0).
    Returns (signed codes int8 [M][K] with value 2 code + 1, scales fp16 [M]).
    Inputs must be finite.
    """
    x32 = np.asarray(x, dtype=np.float16).astype(np.float32)
    levels = np.float32((1 << q) - 1)
    absmax = np.max(np.abs(x32), axis=1) if x32.shape[1] else np.zeros(x32.shape[0], np.float32)
    s16 = (absmax / levels).astype(np.float16)
    s = s16.astype(np.float32)[:, None]
    with np.errstate(divide="ignore", invalid="ignore"):
        t = np.where(s > 0, x32 / np.where(s > 0, s, np.float32(1)), np.float32(0)).astype(np.float32)
    v = np.float32(2) * np.floor(t / np.float32(2)) + np.float32(1)
    v = np.clip(v, -levels, levels)
    codes = ((v - 1) / 2).astype(np.int64).astype(np.int8)
    return codes, s16


# ---- linear quantizers with a zero-point (Sec. III-A) ---------------------------
#
# A linear quantizer stores X = s * x + z for a signed code x.  Sec. III-A
# rewrites it in bipolar form: with the bipolar value x' = 2x + 1,
#     X = (s / 2) * x' + (z - s / 2),
# i.e. bipolar scale s' = s / 2 and bipolar zero z' = z - s / 2.  With a
# per-token (s'_a, z'_a) for the activations and a per-channel (s'_w, z'_w)
# for the weights, the product of the dequantized operands is
#     Y[m,n] = sum_k (s'_a[m] a'[m,k] + z'_a[m]) (s'_w[n] w'[n,k] + z'_w[n]).

def dequant_matmul(a_codes: np.ndarray, w_codes: np.ndarray, p: int, q: int, a_scale, a_zero,
                   w_scale, w_zero) -> np.ndarray:
    """The definition: dequantize both operands from their bipolar values and
    bipolar (scale, zero) and multiply them in float64."""
    sa = np.asarray(a_scale, dtype=np.float16).astype(np.float64)[:, None]
    za = np.asarray(a_zero, dtype=np.float16).astype(np.float64)[:, None]
    sw = np.asarray(w_scale, dtype=np.float16).astype(np.float64)[:, None]
    zw = np.asarray(w_zero, dtype=np.float16).astype(np.float64)[:, None]
    A = sa * values(a_codes, q).astype(np.float64) + za
    W = sw * values(w_codes, p).astype(np.float64) + zw
    return A @ W.T


def affine_epilogue(C: np.ndarray, a_rowsum: np.ndarray, w_rowsum: np.ndarray, K: int, a_scale,
                    a_zero, w_scale, w_zero):
    """(E, T): the expanded form of the same product from the integer GEMM and
    the bipolar row sums R_a[m] = sum_k a'[m,k], R_w[n] = sum_k w'[n,k]:
        E = s'_a s'_w C + s'_a z'_w R_a + z'_a s'_w R_w + K z'_a z'_w,
    each term exact in float64 (at most 31 + 11 + 11 significant bits), and
    T = the sum of the terms' magnitudes, which bounds the rounding error of a
    float32 evaluation."""
    sa = np.asarray(a_scale, dtype=np.float16).astype(np.float64)[:, None]
    za = np.asarray(a_zero, dtype=np.float16).astype(np.float64)[:, None]
    sw = np.asarray(w_scale, dtype=np.float16).astype(np.float64)[None, :]
    zw = np.asarray(w_zero, dtype=np.float16).astype(np.float64)[None, :]
    Cd = np.asarray(C, dtype=np.int64).astype(np.float64)
    Ra = np.asarray(a_rowsum, dtype=np.int64).astype(np.float64)[:, None]
    Rw = np.asarray(w_rowsum, dtype=np.int64).astype(np.float64)[None, :]
    terms = (sa * sw * Cd, sa * zw * Ra, za * sw * Rw, float(K) * za * zw)
    E = terms[0] + terms[1] + terms[2] + terms[3]
    T = np.abs(terms[0]) + np.abs(terms[1]) + np.abs(terms[2]) + np.abs(terms[3])
    return E, T


# A float32 evaluation of the four terms (two roundings per product, three
# per sum, one per int32 -> float32 conversion) is off by at most about
# 6 * 2^-24 * T; the fp16 result adds half an ulp (2^-11 relative, 2^-25 in
# the subnormal range).  The tolerance leaves a margin over both.
AFFINE_T_TOL = 2.0 ** -20


def fp16_affine_close(g: np.ndarray, E: np.ndarray, T: np.ndarray) -> np.ndarray:
    """Element-wise acceptance of a GPU fp16 result g of the affine epilogue:
    |g - E| <= 1e-3 |E| + 2^-20 T + 2^-25."""
    g = np.asarray(g, dtype=np.float16).astype(np.float64)
    d = np.abs(g - E)
    return d <= FP16_REL_TOL * np.abs(E) + AFFINE_T_TOL * T + FP16_ABS_TOL
