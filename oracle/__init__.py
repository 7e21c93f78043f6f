"""fp64 CPU oracle of the MonarchAttention forward pass.

TEST INFRASTRUCTURE ONLY.  The test suite, the smoke check and the
benchmark's CPU-baseline leg are the only users.  The HIP product path never
imports, links or calls anything here, and nothing here touches the HIP path.

Two independent formulations:

* ``monarch_oracle.c`` (loaded through ctypes): the state form (alpha_R, c_R,
  alpha_L, c_L, Y) of the paper's Implementation paragraph, OpenMP over the
  independent (head, block) units.  This is the one the GPU is compared with.
* ``naive.py``: the factors L and R materialised, straight from eqs. R_update,
  L_update, beta_r, beta_l and monarch_multiply.  Small N only.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "monarch_oracle.c")
_LIB = os.path.join(_HERE, "libmonarch_oracle.so")

_lib = None


def build(force: bool = True) -> str:
    """Compile the C oracle with gcc (-O2, OpenMP); returns the library path."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        cmd = ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", _SRC, "-o", tmp, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        i64, i32, dp = ctypes.c_int64, ctypes.c_int32, ctypes.POINTER(ctypes.c_double)
        lib.ma_oracle_fwd_f64.argtypes = [dp, dp, dp, dp, i64, i64, i64, i64, i64, i64, i32, i32]
        lib.ma_oracle_fwd_f64.restype = ctypes.c_int
        lib.ma_oracle_dense_attn_f64.argtypes = [dp, dp, dp, dp, i64, i64, i64,
                                                 ctypes.POINTER(ctypes.c_int64), i64, i32]
        lib.ma_oracle_dense_attn_f64.restype = ctypes.c_int
        lib.ma_oracle_max_threads.restype = ctypes.c_int
        lib.ma_oracle_fwd_obj_f64.argtypes = [dp, dp, dp, dp, dp, i64, i64, i64, i64, i64, i64, i32, i32]
        lib.ma_oracle_fwd_obj_f64.restype = ctypes.c_int
        lib.ma_oracle_fwd_varlen_f64.argtypes = [dp, dp, dp, dp, ctypes.POINTER(ctypes.c_int64),
                                                 i64, i64, i64, i64, i64, i64, i32, i32]
        lib.ma_oracle_fwd_varlen_f64.restype = ctypes.c_int
        lib.ma_oracle_fwd_prepad_f64.argtypes = [dp, dp, dp, dp, ctypes.POINTER(ctypes.c_int64),
                                                 i64, i64, i64, i64, i64, i64, i32, i32]
        lib.ma_oracle_fwd_prepad_f64.restype = ctypes.c_int
        _lib = lib
    return _lib


def _dptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def monarch_attention(q, k, v, m: int, b: int, T: int, threads: int = 0) -> np.ndarray:
    """O for all heads.  q, k, v: float64 [B, H, N, d] (any dtype-rounded values)."""
    q = np.ascontiguousarray(q, dtype=np.float64)
    k = np.ascontiguousarray(k, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    B, H, N, d = q.shape
    out = np.empty_like(q)
    rc = _load().ma_oracle_fwd_f64(_dptr(q), _dptr(k), _dptr(v), _dptr(out),
                                   B, H, N, d, m, b, T, threads)
    if rc != 0:
        raise ValueError(f"oracle rejected the arguments (code {rc})")
    return out


def monarch_attention_objective(q, k, v, m: int, b: int, T: int, threads: int = 0):
    """(O, f): O as monarch_attention, and f[B, H, T], the objective f(M^(t); Q, K)
    of Sec. 3 after every step t, in its separable form (on all m*b rows of the
    padded problem when N < m*b)."""
    q = np.ascontiguousarray(q, dtype=np.float64)
    k = np.ascontiguousarray(k, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    B, H, N, d = q.shape
    out = np.empty_like(q)
    obj = np.empty((B, H, T))
    rc = _load().ma_oracle_fwd_obj_f64(_dptr(q), _dptr(k), _dptr(v), _dptr(out), _dptr(obj),
                                       B, H, N, d, m, b, T, threads)
    if rc != 0:
        raise ValueError(f"oracle rejected the arguments (code {rc})")
    return out, obj


def monarch_attention_varlen(q, k, v, lens, m: int, b: int, T: int, threads: int = 0) -> np.ndarray:
    """O for a batch of post-padded sequences: q, k, v float64 [B, H, N, d],
    lens[B] real rows per batch element (0..N); rows >= lens[beta] of O are
    zero.  Whole key blocks of padding get R = 0 and no L weight."""
    q = np.ascontiguousarray(q, dtype=np.float64)
    k = np.ascontiguousarray(k, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    B, H, N, d = q.shape
    lens = np.ascontiguousarray(lens, dtype=np.int64)
    if lens.shape != (B,):
        raise ValueError("lens must hold one length per batch element")
    out = np.empty_like(q)
    rc = _load().ma_oracle_fwd_varlen_f64(_dptr(q), _dptr(k), _dptr(v), _dptr(out),
                                          lens.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)),
                                          B, H, N, d, m, b, T, threads)
    if rc != 0:
        raise ValueError(f"oracle rejected the arguments (code {rc})")
    return out


def monarch_attention_prepad(q, k, v, m: int, b: int, T: int, lens=None, threads: int = 0) -> np.ndarray:
    """O for pre-padded sequences (Appendix "Padding and Masking", its last
    sentence: the padding rows come first).  q, k, v float64 [B, H, N, d].
    lens None: all N rows are real, pre-padded to m*b.  lens[B]: batch
    element beta's real rows are its LAST lens[beta] rows (a left-padded
    batch), pre-padded to m*b; its other rows of O are zero."""
    q = np.ascontiguousarray(q, dtype=np.float64)
    k = np.ascontiguousarray(k, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    B, H, N, d = q.shape
    lp = None
    if lens is not None:
        lens = np.ascontiguousarray(lens, dtype=np.int64)
        if lens.shape != (B,):
            raise ValueError("lens must hold one length per batch element")
        lp = lens.ctypes.data_as(ctypes.POINTER(ctypes.c_int64))
    out = np.empty_like(q)
    rc = _load().ma_oracle_fwd_prepad_f64(_dptr(q), _dptr(k), _dptr(v), _dptr(out), lp,
                                          B, H, N, d, m, b, T, threads)
    if rc != 0:
        raise ValueError(f"oracle rejected the arguments (code {rc})")
    return out


def dense_attention_rows(q, k, v, rows=None, threads: int = 0) -> np.ndarray:
    """Exact softmax(Q K^T / sqrt(d)) V on selected query rows: [B, H, len(rows), d]."""
    q = np.ascontiguousarray(q, dtype=np.float64)
    k = np.ascontiguousarray(k, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    B, H, N, d = q.shape
    if rows is None:
        rows = np.arange(N, dtype=np.int64)
    rows = np.ascontiguousarray(rows, dtype=np.int64)
    out = np.empty((B, H, len(rows), d))
    rc = _load().ma_oracle_dense_attn_f64(
        _dptr(q), _dptr(k), _dptr(v), _dptr(out), B * H, N, d,
        rows.ctypes.data_as(ctypes.POINTER(ctypes.c_int64)), len(rows), threads)
    if rc != 0:
        raise ValueError(f"dense attention rejected the arguments (code {rc})")
    return out


def max_threads() -> int:
    return int(_load().ma_oracle_max_threads())


def macs_per_head(N: int, m: int, b: int, d: int, T: int) -> int:
    """Multiply-adds of one head: T (2 N b d + 2 N m d) + N b d.

    Each R half-step does two b x b x d products per (k) block (beta_R and
    alpha_L: 2 N b d), each L half-step two m x m x d products per (j) block
    (beta_L and alpha_R: 2 N m d); the Monarch product adds Y (N b d) and O
    (N m d), the latter replacing the alpha_R product of the last step.
    """
    return T * (2 * N * b * d + 2 * N * m * d) + N * b * d


def rel_frobenius(x, ref) -> float:
    x = np.asarray(x, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.linalg.norm((x - ref).ravel()) / np.linalg.norm(ref.ravel()))
