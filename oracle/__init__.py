"""The oracle: plain CPU reference implementations used to check the HIP path.

TEST INFRASTRUCTURE ONLY.  Only the test suite, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import it; the product package never
does, and nothing here imports the product package.

* ``attn_fwd_f64`` / ``attn_fwd_rows_f64``: the fp64 two-pass-softmax attention
  forward of ``attn_oracle.c`` (Section 2.3, Eq. "eq:fa", with GQA and an
  optional top-left causal mask), called through ctypes on numpy arrays of
  bf16 bit patterns (uint16).
* ``attn_bwd_f64``, ``attn_row_stats_f64``, ``attn_bwd_dq_rows_f64``,
  ``attn_bwd_dkdv_rows_f64``: the fp64 attention backward of
  ``attn_bwd_oracle.c`` (Section 2.3, Eq. "eq:ba") and the row statistics
  (log-sum-exp, D) it is written in terms of.
* ``mapping``: the CPU enumeration of the four WG -> (b, hq, m) mappings.

``build()`` compiles ``liboracle.so`` with gcc (no HIP involved).
"""

from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

from . import mapping  # noqa: F401  (re-exported)

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "attn_oracle.c")
_BWD_SRC = os.path.join(_HERE, "attn_bwd_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

_lib = None


def build(src: str = _SRC, out: str = _LIB, extra_flags=(), bwd_src: str = _BWD_SRC) -> str:
    """Compile the C oracle (forward and backward sources) into one shared library."""
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", "-Wall", "-Werror",
           *extra_flags, src, bwd_src, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


def load(path: str = _LIB):
    """Load (building first only if nothing is built) and type the library."""
    global _lib
    if path == _LIB and _lib is not None:
        return _lib
    if not os.path.exists(path):
        build(out=path)
    lib = ctypes.CDLL(path)
    u16p = ctypes.POINTER(ctypes.c_uint16)
    f64p = ctypes.POINTER(ctypes.c_double)
    i64p = ctypes.POINTER(ctypes.c_int64)
    ci = ctypes.c_int
    lib.oracle_attn_fwd_f64.argtypes = [u16p, u16p, u16p, f64p, ci, ci, ci, ci, ci, ci, ci,
                                        ctypes.c_float, ci]
    lib.oracle_attn_fwd_f64.restype = ci
    lib.oracle_attn_fwd_rows_f64.argtypes = [u16p, u16p, u16p, i64p, ctypes.c_int64, f64p,
                                             ci, ci, ci, ci, ci, ci, ci, ctypes.c_float, ci]
    lib.oracle_attn_fwd_rows_f64.restype = ci
    lib.oracle_max_threads.argtypes = []
    lib.oracle_max_threads.restype = ci
    i64 = ctypes.c_int64
    cf = ctypes.c_float
    lib.oracle_attn_bwd_f64.argtypes = [u16p, u16p, u16p, u16p, f64p, f64p, f64p,
                                        ci, ci, ci, ci, ci, ci, ci, cf, ci]
    lib.oracle_attn_bwd_f64.restype = ci
    lib.oracle_attn_row_stats_f64.argtypes = [u16p, u16p, u16p, u16p, i64p, i64, f64p, f64p,
                                              ci, ci, ci, ci, ci, ci, ci, cf, ci]
    lib.oracle_attn_row_stats_f64.restype = ci
    lib.oracle_attn_bwd_dq_rows_f64.argtypes = [u16p, u16p, u16p, u16p, i64p, i64, f64p,
                                                ci, ci, ci, ci, ci, ci, ci, cf, ci]
    lib.oracle_attn_bwd_dq_rows_f64.restype = ci
    lib.oracle_attn_bwd_dkdv_rows_f64.argtypes = [u16p, u16p, u16p, u16p, f64p, f64p, i64p, i64,
                                                  f64p, f64p, ci, ci, ci, ci, ci, ci, ci, cf, ci]
    lib.oracle_attn_bwd_dkdv_rows_f64.restype = ci
    if path == _LIB:
        _lib = lib
    return lib


def _as_u16(a: np.ndarray) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype != np.uint16:
        raise TypeError("oracle inputs are bf16 bit patterns (uint16), got %s" % a.dtype)
    return a


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def attn_fwd_f64(q: np.ndarray, k: np.ndarray, v: np.ndarray, causal: bool, scale: float,
                 nthreads: int = 0, lib=None) -> np.ndarray:
    """O[B,Hq,Sq,d] in fp64 from bf16 bits q[B,Hq,Sq,d], k/v[B,Hkv,Skv,d]."""
    lib = lib or load()
    q, k, v = _as_u16(q), _as_u16(k), _as_u16(v)
    B, Hq, Sq, d = q.shape
    Bk, Hkv, Skv, dk = k.shape
    if v.shape != k.shape or Bk != B or dk != d:
        raise ValueError("shape mismatch")
    o = np.empty((B, Hq, Sq, d), dtype=np.float64)
    rc = lib.oracle_attn_fwd_f64(_ptr(q, ctypes.c_uint16), _ptr(k, ctypes.c_uint16),
                                 _ptr(v, ctypes.c_uint16), _ptr(o, ctypes.c_double),
                                 B, Hq, Hkv, Sq, Skv, d, int(bool(causal)),
                                 ctypes.c_float(scale), int(nthreads))
    if rc != 0:
        raise RuntimeError("oracle_attn_fwd_f64 failed with %d" % rc)
    return o


def attn_fwd_rows_f64(q: np.ndarray, k: np.ndarray, v: np.ndarray, rows: np.ndarray,
                      causal: bool, scale: float, nthreads: int = 0, lib=None) -> np.ndarray:
    """O rows [n, d] for rows[n] = (b, hq, i); exactly the rows of the full O."""
    lib = lib or load()
    q, k, v = _as_u16(q), _as_u16(k), _as_u16(v)
    rows = np.ascontiguousarray(rows, dtype=np.int64).reshape(-1, 3)
    B, Hq, Sq, d = q.shape
    _, Hkv, Skv, _ = k.shape
    o = np.empty((rows.shape[0], d), dtype=np.float64)
    rc = lib.oracle_attn_fwd_rows_f64(_ptr(q, ctypes.c_uint16), _ptr(k, ctypes.c_uint16),
                                      _ptr(v, ctypes.c_uint16), _ptr(rows, ctypes.c_int64),
                                      rows.shape[0], _ptr(o, ctypes.c_double),
                                      B, Hq, Hkv, Sq, Skv, d, int(bool(causal)),
                                      ctypes.c_float(scale), int(nthreads))
    if rc != 0:
        raise RuntimeError("oracle_attn_fwd_rows_f64 failed with %d" % rc)
    return o


def max_threads(lib=None) -> int:
    return int((lib or load()).oracle_max_threads())


def _shapes(q, k, v, dout):
    B, Hq, Sq, d = q.shape
    Bk, Hkv, Skv, dk = k.shape
    if v.shape != k.shape or Bk != B or dk != d or (dout is not None and dout.shape != q.shape):
        raise ValueError("shape mismatch")
    return B, Hq, Hkv, Sq, Skv, d


def attn_bwd_f64(q, k, v, dout, causal: bool, scale: float, nthreads: int = 0, lib=None):
    """(dQ, dK, dV) in fp64 from bf16 bits q/dout[B,Hq,Sq,d], k/v[B,Hkv,Skv,d]."""
    lib = lib or load()
    q, k, v, dout = (_as_u16(t) for t in (q, k, v, dout))
    B, Hq, Hkv, Sq, Skv, d = _shapes(q, k, v, dout)
    dq = np.empty((B, Hq, Sq, d), dtype=np.float64)
    dk = np.empty((B, Hkv, Skv, d), dtype=np.float64)
    dv = np.empty((B, Hkv, Skv, d), dtype=np.float64)
    u16, f64 = ctypes.c_uint16, ctypes.c_double
    rc = lib.oracle_attn_bwd_f64(_ptr(q, u16), _ptr(k, u16), _ptr(v, u16), _ptr(dout, u16),
                                 _ptr(dq, f64), _ptr(dk, f64), _ptr(dv, f64),
                                 B, Hq, Hkv, Sq, Skv, d, int(bool(causal)), ctypes.c_float(scale),
                                 int(nthreads))
    if rc != 0:
        raise RuntimeError("oracle_attn_bwd_f64 failed with %d" % rc)
    return dq, dk, dv


def attn_row_stats_f64(q, k, v, dout, rows, causal: bool, scale: float, nthreads: int = 0,
                       lib=None):
    """(lse[n], D[n]) of rows[n] = (b, hq, i); D is None when dout is None."""
    lib = lib or load()
    q, k, v = (_as_u16(t) for t in (q, k, v))
    dout = None if dout is None else _as_u16(dout)
    B, Hq, Hkv, Sq, Skv, d = _shapes(q, k, v, dout)
    rows = np.ascontiguousarray(rows, dtype=np.int64).reshape(-1, 3)
    lse = np.empty(rows.shape[0], dtype=np.float64)
    D = None if dout is None else np.empty(rows.shape[0], dtype=np.float64)
    u16, f64 = ctypes.c_uint16, ctypes.c_double
    rc = lib.oracle_attn_row_stats_f64(
        _ptr(q, u16), _ptr(k, u16), _ptr(v, u16), None if dout is None else _ptr(dout, u16),
        _ptr(rows, ctypes.c_int64), rows.shape[0], _ptr(lse, f64),
        None if D is None else _ptr(D, f64), B, Hq, Hkv, Sq, Skv, d, int(bool(causal)),
        ctypes.c_float(scale), int(nthreads))
    if rc != 0:
        raise RuntimeError("oracle_attn_row_stats_f64 failed with %d" % rc)
    return lse, D


def all_rows(B: int, H: int, S: int) -> np.ndarray:
    """Every (b, h, i) in row-major order."""
    b, h, i = np.meshgrid(np.arange(B), np.arange(H), np.arange(S), indexing="ij")
    return np.stack([b.ravel(), h.ravel(), i.ravel()], axis=1).astype(np.int64)


def attn_bwd_dq_rows_f64(q, k, v, dout, rows, causal: bool, scale: float, nthreads: int = 0,
                         lib=None):
    """dQ rows [n, d] of rows[n] = (b, hq, i): exact rows of the full dQ."""
    lib = lib or load()
    q, k, v, dout = (_as_u16(t) for t in (q, k, v, dout))
    B, Hq, Hkv, Sq, Skv, d = _shapes(q, k, v, dout)
    rows = np.ascontiguousarray(rows, dtype=np.int64).reshape(-1, 3)
    out = np.empty((rows.shape[0], d), dtype=np.float64)
    u16, f64 = ctypes.c_uint16, ctypes.c_double
    rc = lib.oracle_attn_bwd_dq_rows_f64(_ptr(q, u16), _ptr(k, u16), _ptr(v, u16),
                                         _ptr(dout, u16), _ptr(rows, ctypes.c_int64),
                                         rows.shape[0], _ptr(out, f64), B, Hq, Hkv, Sq, Skv, d,
                                         int(bool(causal)), ctypes.c_float(scale), int(nthreads))
    if rc != 0:
        raise RuntimeError("oracle_attn_bwd_dq_rows_f64 failed with %d" % rc)
    return out


def attn_bwd_dkdv_rows_f64(q, k, v, dout, rows, causal: bool, scale: float, nthreads: int = 0,
                           lib=None, stats=None):
    """(dK rows, dV rows) [n, d] of rows[n] = (b, g, j).

    Needs lse and D of every query row; they are computed here by the oracle
    (or passed as ``stats`` = (lse, D) arrays of shape [B, Hq, Sq])."""
    lib = lib or load()
    q, k, v, dout = (_as_u16(t) for t in (q, k, v, dout))
    B, Hq, Hkv, Sq, Skv, d = _shapes(q, k, v, dout)
    if stats is None:
        lse, D = attn_row_stats_f64(q, k, v, dout, all_rows(B, Hq, Sq), causal, scale,
                                    nthreads, lib)
    else:
        lse, D = stats
    lse = np.ascontiguousarray(lse, dtype=np.float64).reshape(-1)
    D = np.ascontiguousarray(D, dtype=np.float64).reshape(-1)
    rows = np.ascontiguousarray(rows, dtype=np.int64).reshape(-1, 3)
    dk = np.empty((rows.shape[0], d), dtype=np.float64)
    dv = np.empty((rows.shape[0], d), dtype=np.float64)
    u16, f64 = ctypes.c_uint16, ctypes.c_double
    rc = lib.oracle_attn_bwd_dkdv_rows_f64(_ptr(q, u16), _ptr(k, u16), _ptr(v, u16),
                                           _ptr(dout, u16), _ptr(lse, f64), _ptr(D, f64),
                                           _ptr(rows, ctypes.c_int64), rows.shape[0],
                                           _ptr(dk, f64), _ptr(dv, f64), B, Hq, Hkv, Sq, Skv, d,
                                           int(bool(causal)), ctypes.c_float(scale),
                                           int(nthreads))
    if rc != 0:
        raise RuntimeError("oracle_attn_bwd_dkdv_rows_f64 failed with %d" % rc)
    return dk, dv
