"""CPU fp64 oracle for bifurcated decode attention -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. The GPU library never imports, links or
calls anything here, and nothing here imports the GPU library.

Two independent evaluations of the same quantity:

* :func:`attention` / :func:`attention_rows` (C, ``oracle.c``): standard
  multi-group attention over per-sample explicitly replicated KV (Section 3.3,
  Eq. 1-2), fp64, two-pass max-subtracted softmax, sequential sums.
* :func:`bifurcated.bifurcated_attention` (numpy): the bifurcated formulation
  of Section 4.2 (Eq. 3 for the logits, joint softmax over the concatenated
  context and decode logits, Eq. 4 for the output), fp64.

Their agreement to ~1e-12 is the paper's exactness claim (Section 4.2,
Appendix E.1), checked in ``tests/test_oracle_pins.py``.

Caches may hold 8-bit codes (``kv="fp8_e4m3"`` or ``kv="int8"``, arrays of
uint8 bit patterns) or 4-bit codes (``kv="int4"``, two per byte: uint8
arrays whose last axis is d/2, element 2u in the low nibble of byte u and
element 2u+1 in the high nibble) with per-group fp32 ``k_scale`` /
``v_scale`` [g]: the key of a row is ``k_scale[gam]`` times the code's value
(the FAQ on attention quantization; the reading is spelled out in
``oracle.c``).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

_ERRORS = {-1: "invalid dimensions or row index", -4: "out of memory",
           -6: "decode length outside [0, m_d_max]"}

#: Cache element types: name -> (code of oracle.c, numpy dtype of the stored
#: bits, elements per stored item).
KV_TYPES = {"bf16": (0, np.uint16, 1), "fp8_e4m3": (1, np.uint8, 1), "int8": (2, np.uint8, 1),
            "int4": (3, np.uint8, 2)}


def build(force: bool = False) -> str:
    """Compile oracle.c with gcc (IEEE fp64: no fast-math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11",
                               "-Wall", "-Werror", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        lib = ctypes.CDLL(build())
        u16 = ctypes.POINTER(ctypes.c_uint16)
        i32 = ctypes.POINTER(ctypes.c_int32)
        f64 = ctypes.POINTER(ctypes.c_double)
        f32 = ctypes.POINTER(ctypes.c_float)
        vp = ctypes.c_void_p
        ci = ctypes.c_int
        lib.oracle_attention_kv_fp64.argtypes = [ci, ci, ci, ci, ci, ci, ci, ctypes.c_double, ci,
                                                 u16, vp, vp, vp, vp, i32, f32, f32, f64, ci]
        lib.oracle_attention_kv_fp64.restype = ci
        lib.oracle_attention_kv_rows_fp64.argtypes = [ci, ci, ci, ci, ci, ci, ci, ctypes.c_double,
                                                      ci, u16, vp, vp, vp, vp, i32, f32, f32, ci,
                                                      i32, i32, i32, f64, ci]
        lib.oracle_attention_kv_rows_fp64.restype = ci
        lib.oracle_code_value.argtypes = [ci, ci]
        lib.oracle_code_value.restype = ctypes.c_double
        lib.oracle_max_threads.restype = ci
        _lib = lib
    return _lib


def _ptr(a, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _prep(q, Kc, Vc, Kd, Vd, lens, kv="bf16", k_scale=None, v_scale=None):
    """q is [b, h, d] (one new token per sample) or [b, h, n, d] (n new tokens)."""
    if kv not in KV_TYPES:
        raise ValueError(f"unknown cache type {kv!r}")
    code, dt, per = KV_TYPES[kv]
    q = np.ascontiguousarray(q, dtype=np.uint16)
    caches = []
    for x in (Kc, Vc, Kd, Vd):
        x = np.ascontiguousarray(x)
        if x.dtype.itemsize != np.dtype(dt).itemsize or x.dtype.kind not in "ui":
            raise ValueError(f"{kv} caches are {np.dtype(dt).itemsize}-byte bit patterns")
        caches.append(x.view(dt))
    Kc, Vc, Kd, Vd = caches
    lens = np.ascontiguousarray(lens, dtype=np.int32)
    if q.ndim == 3:
        b, h, d = q.shape
        n = 1
    else:
        b, h, n, d = q.shape
    g, m_c, d2 = Kc.shape
    b2, g2, m_d_max, d3 = Kd.shape
    if not (d == d2 * per == d3 * per and b == b2 and g == g2 and Vc.shape == Kc.shape
            and Vd.shape == Kd.shape and lens.shape == (b,)):
        raise ValueError("inconsistent shapes")
    scales = []
    for sc in (k_scale, v_scale):
        if sc is not None:
            sc = np.ascontiguousarray(sc, dtype=np.float32)
            if sc.shape != (g,):
                raise ValueError("scales must be [g]")
        scales.append(sc)
    return (q, Kc, Vc, Kd, Vd, lens), (b, h, g, d, m_c, m_d_max, n), code, scales


def _vp(a):
    return ctypes.c_void_p(a.ctypes.data)


def _fp(a):
    return None if a is None else _ptr(a, ctypes.c_float)


def default_scale(d: int) -> float:
    """Softmax scale 1/sqrt(d); the paper omits it (Appendix E.3 leaves the
    softmax out), this is the standard choice for scaled dot-product."""
    return 1.0 / np.sqrt(float(d))


def attention(q, Kc, Vc, Kd, Vd, lens, scale=None, nthreads=0, kv="bf16", k_scale=None,
              v_scale=None):
    """Full fp64 output, shaped like q: [b, h, d] or [b, h, n, d] (q is bf16
    bit patterns, uint16; caches bf16 bits or 8-bit codes as ``kv`` says).
    With n tokens per sample, token r sees the first max(0, len_i - n + r + 1)
    decode rows."""
    arrs, (b, h, g, d, m_c, m_d_max, n), code, (ks, vs) = _prep(q, Kc, Vc, Kd, Vd, lens, kv,
                                                               k_scale, v_scale)
    scale = default_scale(d) if scale is None else float(scale)
    out = np.empty(arrs[0].shape, dtype=np.float64)
    q, Kc, Vc, Kd, Vd, lens = arrs
    rc = _load().oracle_attention_kv_fp64(b, h, g, d, m_c, m_d_max, n, scale, code,
                                          _ptr(q, ctypes.c_uint16), _vp(Kc), _vp(Vc), _vp(Kd),
                                          _vp(Vd), _ptr(lens, ctypes.c_int32), _fp(ks), _fp(vs),
                                          _ptr(out, ctypes.c_double), int(nthreads))
    if rc:
        raise ValueError(f"oracle: {_ERRORS.get(rc, rc)}")
    return out


def attention_rows(q, Kc, Vc, Kd, Vd, lens, rows_i, rows_j, scale=None, nthreads=0, rows_t=None,
                   kv="bf16", k_scale=None, v_scale=None):
    """fp64 output rows (sample rows_i[r], head rows_j[r], token rows_t[r]
    (default 0)) -> [nrows, d]."""
    arrs, (b, h, g, d, m_c, m_d_max, n), code, (ks, vs) = _prep(q, Kc, Vc, Kd, Vd, lens, kv,
                                                               k_scale, v_scale)
    scale = default_scale(d) if scale is None else float(scale)
    ri = np.ascontiguousarray(rows_i, dtype=np.int32)
    rj = np.ascontiguousarray(rows_j, dtype=np.int32)
    rt = np.zeros_like(ri) if rows_t is None else np.ascontiguousarray(rows_t, dtype=np.int32)
    if ri.shape != rj.shape or rt.shape != ri.shape or ri.ndim != 1:
        raise ValueError("rows_i, rows_j and rows_t must be 1-D and equally long")
    out = np.empty((ri.size, d), dtype=np.float64)
    q, Kc, Vc, Kd, Vd, lens = arrs
    rc = _load().oracle_attention_kv_rows_fp64(b, h, g, d, m_c, m_d_max, n, scale, code,
                                               _ptr(q, ctypes.c_uint16), _vp(Kc), _vp(Vc),
                                               _vp(Kd), _vp(Vd), _ptr(lens, ctypes.c_int32),
                                               _fp(ks), _fp(vs), int(ri.size),
                                               _ptr(ri, ctypes.c_int32), _ptr(rj, ctypes.c_int32),
                                               _ptr(rt, ctypes.c_int32),
                                               _ptr(out, ctypes.c_double), int(nthreads))
    if rc:
        raise ValueError(f"oracle: {_ERRORS.get(rc, rc)}")
    return out


def code_value(kv: str, code: int) -> float:
    """The C oracle's decoded value of one cache code (unscaled)."""
    return float(_load().oracle_code_value(KV_TYPES[kv][0], int(code)))


def max_threads() -> int:
    return int(_load().oracle_max_threads())


def widen_bf16(bits) -> np.ndarray:
    """bf16 bit patterns (uint16) -> exact fp64 values."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def widen_codes(codes, kv: str) -> np.ndarray:
    """Cache codes -> exact unscaled fp64 values (numpy; independent of
    oracle.c's decoder). fp8 e4m3 follows the OCP definition: bias 7,
    exponent 0 subnormal, S.1111.111 NaN, no infinities. int4 unpacks the
    last axis (d/2 bytes -> d values, low nibble first), each nibble two's
    complement."""
    if kv == "bf16":
        return widen_bf16(codes)
    c = np.asarray(codes).view(np.uint8)
    if kv == "int8":
        return c.view(np.int8).astype(np.float64)
    if kv == "int4":
        nib = np.stack([c & 15, c >> 4], axis=-1).astype(np.int64)  # [..., d/2, 2]
        vals = np.where(nib >= 8, nib - 16, nib).astype(np.float64)
        return vals.reshape(c.shape[:-1] + (2 * c.shape[-1],))
    if kv != "fp8_e4m3":
        raise ValueError(f"unknown cache type {kv!r}")
    e = ((c >> 3) & 15).astype(np.int64)
    m = (c & 7).astype(np.float64)
    mag = np.where(e == 0, m / 8.0 * 2.0 ** -6, (1.0 + m / 8.0) * np.exp2(e - 7.0))
    mag = np.where((e == 15) & (m == 7), np.nan, mag)
    return np.where(c >= 128, -mag, mag)
