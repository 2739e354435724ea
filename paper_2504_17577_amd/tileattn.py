"""Python binding of libtileattn: the C entry points declared in
include/tileattn.h, under the same names, with torch tensors marshalled to
device pointers.  Every step of attention runs in the HIP library; this module
only checks dtypes/devices, allocates outputs with torch and passes pointers
and torch's current stream.  If the library is not built, every call raises.
"""
from __future__ import annotations

import ctypes
import math
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libtileattn.so")

TA_OK = 0
STATUS = {
    0: "TA_OK", 1: "TA_ERR_NULL_POINTER", 2: "TA_ERR_INVALID_SHAPE", 3: "TA_ERR_UNSUPPORTED",
    4: "TA_ERR_MISALIGNED", 5: "TA_ERR_INVALID_SCALE", 6: "TA_ERR_ALIASING", 7: "TA_ERR_LAUNCH",
}

_lib = None


class TileAttnError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


def lib():
    """The loaded libtileattn.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"HIP library not built: {LIB_PATH} is missing "
                           "(run __graft_entry__.build() or python -m paper_2504_17577_amd.build)")
    L = ctypes.CDLL(LIB_PATH)
    p, i = ctypes.c_void_p, ctypes.c_int
    L.attn_fwd.restype = i
    L.attn_fwd.argtypes = [p, p, p, p, p, i, i, i, i, i, i, i, ctypes.c_float, p]
    L.ta_schedule.restype = i
    L.ta_schedule.argtypes = [i, i, i, i, i, ctypes.POINTER(i), ctypes.POINTER(i)]
    L.ta_tile_shape.restype = i
    L.ta_tile_shape.argtypes = [i, ctypes.POINTER(i), ctypes.POINTER(i)]
    L.ta_status_string.restype = ctypes.c_char_p
    L.ta_status_string.argtypes = [i]
    L.ta_version.restype = i
    L.ta_version.argtypes = []
    _lib = L
    return L


def ta_status_string(status: int) -> str:
    return lib().ta_status_string(status).decode()


def ta_version() -> int:
    return lib().ta_version()


def ta_tile_shape(D: int):
    bm, bn = ctypes.c_int(), ctypes.c_int()
    rc = lib().ta_tile_shape(D, ctypes.byref(bm), ctypes.byref(bn))
    if rc != TA_OK:
        raise TileAttnError(rc, ta_status_string(rc))
    return bm.value, bn.value


def ta_schedule(Sq: int, Sk: int, D: int, causal: bool, q_tile: int):
    """(n_kv_tiles, first_masked) the kernel uses for one query tile."""
    n, fm = ctypes.c_int(), ctypes.c_int()
    rc = lib().ta_schedule(Sq, Sk, D, int(bool(causal)), q_tile, ctypes.byref(n), ctypes.byref(fm))
    if rc != TA_OK:
        raise TileAttnError(rc, ta_status_string(rc))
    return n.value, fm.value


def attn_fwd_raw(Q, K, V, O, LSE, B, Hq, Hkv, Sq, Sk, D, causal, scale, stream) -> int:
    """The C call with integer pointers; returns the status code."""
    return lib().attn_fwd(Q, K, V, O, LSE, B, Hq, Hkv, Sq, Sk, D, int(causal), float(scale), stream)


def attn_fwd(q, k, v, causal: bool = False, scale: float | None = None, out=None, lse=None,
             stream=None):
    """O, LSE = attention forward of bf16 BHSD tensors q [B,Hq,Sq,D] and
    k, v [B,Hkv,Sk,D] on the GPU.  Returns fp32 O [B,Hq,Sq,D] and
    LSE [B,Hq,Sq].  ``scale`` defaults to 1/sqrt(D).  The launch is
    asynchronous on ``stream`` (default: torch's current stream)."""
    import torch

    for name, t in (("q", q), ("k", k), ("v", v)):
        if t.dtype != torch.bfloat16 or not t.is_cuda or t.dim() != 4 or not t.is_contiguous():
            raise TypeError(f"{name} must be a contiguous 4-D bfloat16 GPU tensor (BHSD)")
    B, Hq, Sq, D = q.shape
    Bk, Hkv, Sk, Dk = k.shape
    if (Bk, Dk) != (B, D) or tuple(v.shape) != tuple(k.shape):
        raise TileAttnError(2, f"inconsistent shapes q{tuple(q.shape)} k{tuple(k.shape)} "
                               f"v{tuple(v.shape)}")
    if scale is None:
        scale = 1.0 / math.sqrt(D)
    if out is None:
        out = torch.empty((B, Hq, Sq, D), dtype=torch.float32, device=q.device)
    if lse is None:
        lse = torch.empty((B, Hq, Sq), dtype=torch.float32, device=q.device)
    for name, t, shape in (("out", out, (B, Hq, Sq, D)), ("lse", lse, (B, Hq, Sq))):
        if t.dtype != torch.float32 or tuple(t.shape) != shape or not t.is_contiguous():
            raise TypeError(f"{name} must be a contiguous float32 tensor of shape {shape}")
    if stream is None:
        stream = torch.cuda.current_stream(q.device)
    rc = attn_fwd_raw(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), lse.data_ptr(),
                      B, Hq, Hkv, Sq, Sk, D, causal, scale, stream.cuda_stream)
    if rc != TA_OK:
        raise TileAttnError(rc, ta_status_string(rc))
    return out, lse
