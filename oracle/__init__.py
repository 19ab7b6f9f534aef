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
        ci = ctypes.c_int
        lib.oracle_attention_fp64.argtypes = [ci, ci, ci, ci, ci, ci, ci, ctypes.c_double,
                                              u16, u16, u16, u16, u16, i32, f64, ci]
        lib.oracle_attention_fp64.restype = ci
        lib.oracle_attention_rows_fp64.argtypes = [ci, ci, ci, ci, ci, ci, ci, ctypes.c_double,
                                                   u16, u16, u16, u16, u16, i32, ci, i32, i32,
                                                   i32, f64, ci]
        lib.oracle_attention_rows_fp64.restype = ci
        lib.oracle_max_threads.restype = ci
        _lib = lib
    return _lib


def _ptr(a, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _prep(q, Kc, Vc, Kd, Vd, lens):
    """q is [b, h, d] (one new token per sample) or [b, h, n, d] (n new tokens)."""
    q, Kc, Vc, Kd, Vd = (np.ascontiguousarray(x, dtype=np.uint16) for x in (q, Kc, Vc, Kd, Vd))
    lens = np.ascontiguousarray(lens, dtype=np.int32)
    if q.ndim == 3:
        b, h, d = q.shape
        n = 1
    else:
        b, h, n, d = q.shape
    g, m_c, d2 = Kc.shape
    b2, g2, m_d_max, d3 = Kd.shape
    if not (d == d2 == d3 and b == b2 and g == g2 and Vc.shape == Kc.shape
            and Vd.shape == Kd.shape and lens.shape == (b,)):
        raise ValueError("inconsistent shapes")
    return (q, Kc, Vc, Kd, Vd, lens), (b, h, g, d, m_c, m_d_max, n)


def default_scale(d: int) -> float:
    """Softmax scale 1/sqrt(d); the paper omits it (Appendix E.3 leaves the
    softmax out), this is the standard choice for scaled dot-product."""
    return 1.0 / np.sqrt(float(d))


def attention(q, Kc, Vc, Kd, Vd, lens, scale=None, nthreads=0):
    """Full fp64 output, shaped like q: [b, h, d] or [b, h, n, d] (inputs are
    bf16 bit patterns, uint16). With n tokens per sample, token r sees the
    first max(0, len_i - n + r + 1) decode rows."""
    arrs, (b, h, g, d, m_c, m_d_max, n) = _prep(q, Kc, Vc, Kd, Vd, lens)
    scale = default_scale(d) if scale is None else float(scale)
    out = np.empty(arrs[0].shape, dtype=np.float64)
    q, Kc, Vc, Kd, Vd, lens = arrs
    rc = _load().oracle_attention_fp64(b, h, g, d, m_c, m_d_max, n, scale,
                                       _ptr(q, ctypes.c_uint16), _ptr(Kc, ctypes.c_uint16),
                                       _ptr(Vc, ctypes.c_uint16), _ptr(Kd, ctypes.c_uint16),
                                       _ptr(Vd, ctypes.c_uint16), _ptr(lens, ctypes.c_int32),
                                       _ptr(out, ctypes.c_double), int(nthreads))
    if rc:
        raise ValueError(f"oracle: {_ERRORS.get(rc, rc)}")
    return out


def attention_rows(q, Kc, Vc, Kd, Vd, lens, rows_i, rows_j, scale=None, nthreads=0, rows_t=None):
    """fp64 output rows (sample rows_i[r], head rows_j[r], token rows_t[r]
    (default 0)) -> [nrows, d]."""
    arrs, (b, h, g, d, m_c, m_d_max, n) = _prep(q, Kc, Vc, Kd, Vd, lens)
    scale = default_scale(d) if scale is None else float(scale)
    ri = np.ascontiguousarray(rows_i, dtype=np.int32)
    rj = np.ascontiguousarray(rows_j, dtype=np.int32)
    rt = np.zeros_like(ri) if rows_t is None else np.ascontiguousarray(rows_t, dtype=np.int32)
    if ri.shape != rj.shape or rt.shape != ri.shape or ri.ndim != 1:
        raise ValueError("rows_i, rows_j and rows_t must be 1-D and equally long")
    out = np.empty((ri.size, d), dtype=np.float64)
    q, Kc, Vc, Kd, Vd, lens = arrs
    rc = _load().oracle_attention_rows_fp64(b, h, g, d, m_c, m_d_max, n, scale,
                                            _ptr(q, ctypes.c_uint16), _ptr(Kc, ctypes.c_uint16),
                                            _ptr(Vc, ctypes.c_uint16), _ptr(Kd, ctypes.c_uint16),
                                            _ptr(Vd, ctypes.c_uint16), _ptr(lens, ctypes.c_int32),
                                            int(ri.size), _ptr(ri, ctypes.c_int32),
                                            _ptr(rj, ctypes.c_int32), _ptr(rt, ctypes.c_int32),
                                            _ptr(out, ctypes.c_double), int(nthreads))
    if rc:
        raise ValueError(f"oracle: {_ERRORS.get(rc, rc)}")
    return out


def max_threads() -> int:
    return int(_load().oracle_max_threads())


def widen_bf16(bits) -> np.ndarray:
    """bf16 bit patterns (uint16) -> exact fp64 values."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)
