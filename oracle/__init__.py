"""The oracle: plain CPU reference implementations used to check the HIP path.

TEST INFRASTRUCTURE ONLY.  Only the test suite, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import it; the product package never
does, and nothing here imports the product package.

* ``attn_fwd_f64`` / ``attn_fwd_rows_f64``: the fp64 two-pass-softmax attention
  forward of ``attn_oracle.c`` (Section 2.3, Eq. "eq:fa", with GQA and an
  optional top-left causal mask), called through ctypes on numpy arrays of
  bf16 bit patterns (uint16).
* ``mapping``: the CPU enumeration of the three WG -> (b, hq, m) mappings.

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
_LIB = os.path.join(_HERE, "liboracle.so")

_lib = None


def build(src: str = _SRC, out: str = _LIB, extra_flags=()) -> str:
    """Compile the C oracle into a shared library (gcc, OpenMP, -O2)."""
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c99", "-Wall", "-Werror",
           *extra_flags, src, "-o", out + ".tmp", "-lm"]
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
