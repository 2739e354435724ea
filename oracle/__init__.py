"""fp64 CPU oracle for scaled-dot-product attention forward.

TEST INFRASTRUCTURE.  Only the test suite, the smoke check and the bench's
CPU-baseline leg may import this package.  The product path (the HIP library
and its binding) never imports or calls it, and it imports nothing from the
product: inputs arrive as bfloat16 bit arrays from the seeded generator.

The arithmetic lives in ``attn_oracle.c``: the plain softmax-attention
definition, row by row, in double precision (bottom-right causal alignment,
grouped-query head map h -> h // (Hq/Hkv), LSE as a natural log).  The MLA
decode and GEMM references below reduce to that code or to a float64 matmul;
the Mamba-2 SSD chunk functions are in ``oracle.ssd`` (numpy, float64).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

from . import build as _build

_lib = None
_i64 = ctypes.c_int64
_ptr = ctypes.c_void_p


def load(path: str | None = None):
    """Load (building first if absent) the oracle library; returns the handle."""
    global _lib
    if path is None and _lib is not None:
        return _lib
    lib_path = path or _build.LIB
    if not os.path.exists(lib_path):
        _build.build()
    lib = ctypes.CDLL(lib_path)
    lib.oracle_attn_fwd.restype = ctypes.c_int
    lib.oracle_attn_fwd.argtypes = [_ptr, _ptr, _ptr, _ptr, _ptr, _i64, _i64, _i64, _i64,
                                    _i64, _i64, ctypes.c_int, ctypes.c_double, ctypes.c_int]
    lib.oracle_attn_rows.restype = ctypes.c_int
    lib.oracle_attn_rows.argtypes = [_ptr, _ptr, _ptr, _i64, _i64, _i64, _i64, _i64, _i64,
                                     ctypes.c_int, ctypes.c_double, _ptr, _i64, _ptr, _ptr,
                                     ctypes.c_int]
    if path is None:
        _lib = lib
    return lib


def default_threads() -> int:
    """Host threads for the oracle: the cores this process may run on,
    capped at 16 threads."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


class OracleError(RuntimeError):
    pass


def _bits(a) -> np.ndarray:
    a = np.ascontiguousarray(a)
    if a.dtype != np.uint16 or a.ndim != 4:
        raise TypeError("oracle inputs are 4-D bfloat16 bit arrays (numpy.uint16, BHSD)")
    return a


def _shape(q, k, v):
    B, Hq, Sq, D = q.shape
    Bk, Hkv, Sk, Dk = k.shape
    if (Bk, Dk) != (B, D) or v.shape != k.shape:
        raise OracleError(f"inconsistent shapes q{q.shape} k{k.shape} v{v.shape}")
    return B, Hq, Hkv, Sq, Sk, D


def attn_fwd(q, k, v, causal: bool, scale: float, nthreads: int | None = None, lib=None):
    """Every output row: returns (O [B,Hq,Sq,D], LSE [B,Hq,Sq]) as float64."""
    q, k, v = _bits(q), _bits(k), _bits(v)
    B, Hq, Hkv, Sq, Sk, D = _shape(q, k, v)
    o = np.empty((B, Hq, Sq, D), dtype=np.float64)
    lse = np.empty((B, Hq, Sq), dtype=np.float64)
    lib = lib or load()
    rc = lib.oracle_attn_fwd(q.ctypes.data, k.ctypes.data, v.ctypes.data, o.ctypes.data,
                             lse.ctypes.data, B, Hq, Hkv, Sq, Sk, D, int(bool(causal)),
                             float(scale), nthreads or default_threads())
    if rc:
        raise OracleError(f"oracle_attn_fwd returned {rc}")
    return o, lse


def attn_rows(q, k, v, causal: bool, scale: float, rows, nthreads: int | None = None, lib=None):
    """Selected rows ``rows`` = [(b, h, i), ...]: returns (O [n,D], LSE [n])."""
    q, k, v = _bits(q), _bits(k), _bits(v)
    B, Hq, Hkv, Sq, Sk, D = _shape(q, k, v)
    idx = np.ascontiguousarray(np.asarray(rows, dtype=np.int64).reshape(-1, 3))
    n = idx.shape[0]
    o = np.empty((n, D), dtype=np.float64)
    lse = np.empty((n,), dtype=np.float64)
    lib = lib or load()
    rc = lib.oracle_attn_rows(q.ctypes.data, k.ctypes.data, v.ctypes.data, B, Hq, Hkv, Sq, Sk,
                              D, int(bool(causal)), float(scale), idx.ctypes.data, n,
                              o.ctypes.data, lse.ctypes.data, nthreads or default_threads())
    if rc:
        raise OracleError(f"oracle_attn_rows returned {rc}")
    return o, lse


# ---------------------------------------------------------------------------
# MLA decode (the paper's appendix listing "Implementation of FlashMLA with
# TileLang"): for batch b and query head h, with latent head
# hk = h // (H / Hkv),
#   s_t = scale * (q[b,h] . kv[b,t,hk] + q_pe[b,h] . k_pe[b,t,hk])
#   O[b,h] = sum_t softmax(s)_t kv[b,t,hk],   LSE[b,h] = ln sum_t exp(s_t)
# over all Skv cache positions (a decode step sees the whole cache).  This is
# the attention definition above with one query row per head, key
# [kv | k_pe] (Dl + Dr wide) and value kv.  The reduction below passes the
# key as the value too, so both share one width, and drops the Dr output
# columns that the k_pe part of that value adds.

def _mla_bits(q, q_pe, kv, k_pe):
    arrs = [np.ascontiguousarray(a) for a in (q, q_pe, kv, k_pe)]
    for a, nd in zip(arrs, (3, 3, 4, 4)):
        if a.dtype != np.uint16 or a.ndim != nd:
            raise TypeError("MLA oracle inputs are bfloat16 bit arrays: q, q_pe [B,H,D], "
                            "kv, k_pe [B,Skv,Hkv,D]")
    q, q_pe, kv, k_pe = arrs
    B, H, Dl = q.shape
    Skv, Hkv = kv.shape[1], kv.shape[2]
    Dr = q_pe.shape[2]
    if (q_pe.shape[:2] != (B, H) or kv.shape != (B, Skv, Hkv, Dl)
            or k_pe.shape != (B, Skv, Hkv, Dr) or H % Hkv):
        raise OracleError(f"inconsistent MLA shapes q{q.shape} q_pe{q_pe.shape} "
                          f"kv{kv.shape} k_pe{k_pe.shape}")
    qf = np.concatenate([q, q_pe], axis=2)[:, :, None, :]                   # [B,H,1,Dl+Dr]
    kf = np.ascontiguousarray(np.concatenate([kv, k_pe], axis=3).transpose(0, 2, 1, 3))
    return qf, kf, Dl                                                       # kf [B,Hkv,Skv,Dl+Dr]


def mla_decode(q, q_pe, kv, k_pe, scale: float, nthreads: int | None = None, lib=None):
    """Every (b, h): returns (O [B,H,Dl], LSE [B,H]) as float64."""
    qf, kf, Dl = _mla_bits(q, q_pe, kv, k_pe)
    o, lse = attn_fwd(qf, kf, kf, False, scale, nthreads=nthreads, lib=lib)
    return np.ascontiguousarray(o[:, :, 0, :Dl]), np.ascontiguousarray(lse[:, :, 0])


def mla_rows(q, q_pe, kv, k_pe, scale: float, rows, nthreads: int | None = None, lib=None):
    """Selected heads ``rows`` = [(b, h), ...]: returns (O [n,Dl], LSE [n])."""
    qf, kf, Dl = _mla_bits(q, q_pe, kv, k_pe)
    idx = [(int(b), int(h), 0) for b, h in rows]
    o, lse = attn_rows(qf, kf, kf, False, scale, idx, nthreads=nthreads, lib=lib)
    return np.ascontiguousarray(o[:, :Dl]), lse


# ---------------------------------------------------------------------------
# Matrix multiplication (the paper's Matmul listing): C = A B for row-major
# A [M, K] and B [K, N] given as bfloat16 bits.  The definition, in float64:
# the inputs widen exactly and numpy's matmul forms the products and sums.
# ``gemm_abs`` is sum_k |a_ik| |b_kj|, the scale the GPU tolerance is stated
# against.

def _widen(bits):
    b = np.ascontiguousarray(bits)
    if b.dtype != np.uint16 or b.ndim != 2:
        raise TypeError("GEMM oracle inputs are 2-D bfloat16 bit arrays (numpy.uint16)")
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)


def gemm(a, b, rows=None):
    """C = A B in float64 (all rows, or only the rows listed in ``rows``)."""
    A, B = _widen(a), _widen(b)
    if A.shape[1] != B.shape[0]:
        raise OracleError(f"inconsistent GEMM shapes a{A.shape} b{B.shape}")
    if rows is not None:
        A = A[np.asarray(rows, dtype=np.int64)]
    return A @ B


def gemm_abs(a, b, rows=None):
    """sum_k |a_ik| |b_kj| in float64, for the same rows as ``gemm``."""
    A, B = np.abs(_widen(a)), np.abs(_widen(b))
    if rows is not None:
        A = A[np.asarray(rows, dtype=np.int64)]
    return A @ B
