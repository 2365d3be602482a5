"""Ember CPU oracle: test infrastructure only.

A plain, slow, float64 C implementation of one step of Algorithm 1 ("Ember",
Token Geometry, Section 2) and its ctypes binding.  Only the tests, the smoke
check and the benchmark's CPU-baseline leg may import it; the product library
never does, and the two share no code.  Arrays are numpy: fp32 data as
``float32``, bf16 data as its raw ``uint16`` bit patterns.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ember_oracle.c")
_LIB = os.path.join(_HERE, "libember_oracle.so")

F32 = 0
BF16 = 1
OK = 0
BAD_ARG = -1
BAD_INDEX = -6

_lib = None


def build() -> str:
    """Compile the oracle with gcc (no fast-math, no FMA contraction)."""
    cmd = ["gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp",
           "-fPIC", "-shared", _SRC, "-o", _LIB + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(_LIB + ".tmp", _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB):
        build()
    lib = ctypes.CDLL(_LIB)
    vp, i64, f32, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_float, ctypes.c_int
    lib.ember_oracle_step.argtypes = [vp, i32, i64, vp, i32, i64, vp, i64,
                                      vp, vp, i64, i64, i64, f32, f32, f32, i32, vp, i64, i32]
    lib.ember_oracle_step.restype = i32
    lib.ember_oracle_bf16_to_f64.argtypes = [ctypes.c_uint16]
    lib.ember_oracle_bf16_to_f64.restype = ctypes.c_double
    lib.ember_oracle_f64_to_bf16.argtypes = [ctypes.c_double]
    lib.ember_oracle_f64_to_bf16.restype = ctypes.c_uint16
    lib.ember_oracle_state_bytes.argtypes = [i64, i64]
    lib.ember_oracle_state_bytes.restype = i64
    lib.ember_oracle_coalesce.argtypes = [vp, i64, vp, i32, i64, i64, i64, vp, vp, i32, i64, vp]
    lib.ember_oracle_coalesce.restype = i32
    lib.ember_oracle_lmhead_grad.argtypes = [vp, i64, vp, i64, i64, i64, i64, vp, i32, i64]
    lib.ember_oracle_lmhead_grad.restype = i32
    lib.ember_oracle_set_threads.argtypes = [i32]
    lib.ember_oracle_set_threads.restype = i32
    _lib = lib
    return lib


def _dtype_code(a: np.ndarray) -> int:
    if a.dtype == np.float32:
        return F32
    if a.dtype == np.uint16:
        return BF16
    raise TypeError(f"oracle arrays are float32 or uint16 (bf16 bits), got {a.dtype}")


def _ld(a: np.ndarray) -> int:
    if a.ndim != 2 or a.strides[1] != a.itemsize or a.strides[0] % a.itemsize:
        raise ValueError("2-D arrays with unit column stride expected")
    return a.strides[0] // a.itemsize


def step(W: np.ndarray, G: np.ndarray, r: np.ndarray, c: np.ndarray | None, t: int,
         lr: float = 1e-3, beta2: float = 0.999, eps: float = 1e-8,
         maximize: bool = False, idx: np.ndarray | None = None,
         w_rows: np.ndarray | None = None, row_only: bool = False) -> int:
    """One Ember step, in place on W, r and c.  Returns the oracle's status.

    ``idx`` (int64) selects the sparse-row form: G then holds ``len(idx)``
    rows, row k being the gradient of W's row ``idx[k]``.  ``w_rows``
    (strictly increasing int64) restricts which rows of W are written; the
    state is always updated in full.  ``row_only`` selects row-only Ember
    (c is then unused and may be None).
    """
    lib = _load()
    V, D = W.shape
    if r.dtype != np.float32 or r.shape != (V,) or not r.flags.c_contiguous:
        raise ValueError("r must be contiguous float32[V]")
    if c is None:
        if not row_only:
            raise ValueError("c is required unless row_only")
        c_ptr = None
    else:
        if c.dtype != np.float32 or c.shape != (D,) or not c.flags.c_contiguous:
            raise ValueError("c must be contiguous float32[D]")
        c_ptr = c.ctypes.data
    if idx is None:
        if G.shape != (V, D):
            raise ValueError("dense G must have W's shape")
        idx_ptr, n_idx = None, 0
    else:
        idx = np.ascontiguousarray(idx, dtype=np.int64)
        if G.shape != (idx.shape[0], D):
            raise ValueError("sparse G must be [len(idx), D]")
        idx_ptr, n_idx = idx.ctypes.data, idx.shape[0]
    if w_rows is None:
        wr_ptr, n_wr = None, 0
    else:
        w_rows = np.ascontiguousarray(w_rows, dtype=np.int64)
        wr_ptr, n_wr = w_rows.ctypes.data, w_rows.shape[0]
    g_ptr = G.ctypes.data if G.size else None
    g_ld = _ld(G) if G.shape[0] > 0 else D
    return lib.ember_oracle_step(W.ctypes.data, _dtype_code(W), _ld(W),
                                 g_ptr, _dtype_code(G), g_ld, idx_ptr, n_idx,
                                 r.ctypes.data, c_ptr, V, D, int(t),
                                 float(lr), float(beta2), float(eps), int(bool(maximize)),
                                 wr_ptr, n_wr, int(bool(row_only)))


def coalesce(tok: np.ndarray, U: np.ndarray, V: int, out_dtype=None):
    """Distinct token ids (ascending) and the float64 sum of their per-position
    gradient rows in ascending position order, rounded once to ``out_dtype``
    (``np.float32`` or ``np.uint16`` for bf16 bits; default: U's).  Returns
    (status, idx int64[n], G [n, D])."""
    lib = _load()
    tok = np.ascontiguousarray(tok, dtype=np.int64)
    P = tok.shape[0]
    if U.ndim != 2 or U.shape[0] != P:
        raise ValueError("U must be [len(tok), D]")
    D = U.shape[1]
    out_dtype = U.dtype if out_dtype is None else np.dtype(out_dtype)
    idx = np.zeros(max(P, 1), np.int64)
    G = np.zeros((max(P, 1), D), out_dtype)
    n = ctypes.c_int64(-1)
    u_ptr = U.ctypes.data if U.size else None
    st = lib.ember_oracle_coalesce(tok.ctypes.data if P else None, P, u_ptr, _dtype_code(U),
                                   _ld(U) if P else D, int(V), D, idx.ctypes.data, G.ctypes.data,
                                   _dtype_code(G), _ld(G), ctypes.byref(n))
    if st != OK:
        return st, None, None
    return st, idx[:n.value].copy(), G[:n.value].copy()


def lmhead_grad(dY: np.ndarray, H: np.ndarray, out_dtype=np.uint16) -> np.ndarray:
    """LM-head weight gradient G = dY^T H (appendix "The LM Head Factorizes
    Like the Embedding Table"): dY [T, V] and H [T, D] as bf16 bits (uint16),
    summed exactly in float64 in ascending token order and rounded once to
    ``out_dtype`` (``np.uint16`` for bf16 bits, or ``np.float32``)."""
    lib = _load()
    if dY.dtype != np.uint16 or H.dtype != np.uint16:
        raise TypeError("dY and H are bf16 bit arrays (uint16)")
    if dY.ndim != 2 or H.ndim != 2 or dY.shape[0] != H.shape[0]:
        raise ValueError("dY must be [T, V] and H [T, D]")
    T, V = dY.shape
    D = H.shape[1]
    G = np.zeros((V, D), np.dtype(out_dtype))
    st = lib.ember_oracle_lmhead_grad(dY.ctypes.data if T else None, _ld(dY) if T else V,
                                      H.ctypes.data if T else None, _ld(H) if T else D, T, V, D,
                                      G.ctypes.data, _dtype_code(G), D)
    if st != OK:
        raise ValueError("bad arguments for the LM-head gradient")
    return G


def set_threads(n: int = 0) -> int:
    """Threads the oracle's row and column loops use (0: leave as is); returns
    the count in effect.  Results are the same bits for every count."""
    return _load().ember_oracle_set_threads(int(n))


def bf16_to_f64(bits: int) -> float:
    return _load().ember_oracle_bf16_to_f64(int(bits))


def f64_to_bf16(x: float) -> int:
    return _load().ember_oracle_f64_to_bf16(float(x))


def state_bytes(V: int, D: int) -> int:
    return _load().ember_oracle_state_bytes(int(V), int(D))
