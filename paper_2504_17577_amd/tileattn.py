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
    8: "TA_ERR_WORKSPACE", 9: "TA_ERR_SCRATCH",
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
    L.attn_fwd_bf16out.restype = i
    L.attn_fwd_bf16out.argtypes = [p, p, p, p, p, i, i, i, i, i, i, i, ctypes.c_float, p]
    L.attn_fwd_split.restype = i
    L.attn_fwd_split.argtypes = [p, p, p, p, i, p, i, i, i, i, i, i, i, ctypes.c_float, i, p,
                                 ctypes.c_size_t, p]
    L.attn_fwd_split_noalloc.restype = i
    L.attn_fwd_split_noalloc.argtypes = [p, p, p, p, i, p, i, i, i, i, i, i, i, ctypes.c_float,
                                         i, p]
    L.ta_split_workspace_bytes.restype = i
    L.ta_split_workspace_bytes.argtypes = [i, i, i, i, i, ctypes.POINTER(ctypes.c_size_t)]
    L.ta_split_heuristic.restype = i
    L.ta_split_heuristic.argtypes = [i, i, i, i, i, i, i, ctypes.POINTER(i)]
    L.mla_decode.restype = i
    L.mla_decode.argtypes = [p, p, p, p, p, p, i, i, i, i, i, i, ctypes.c_float, i, p,
                             ctypes.c_size_t, p]
    L.mla_workspace_bytes.restype = i
    L.mla_workspace_bytes.argtypes = [i, i, i, ctypes.POINTER(ctypes.c_size_t)]
    L.mla_split_heuristic.restype = i
    L.mla_split_heuristic.argtypes = [i, i, i, i, ctypes.POINTER(i)]
    L.gemm_bf16.restype = i
    L.gemm_bf16.argtypes = [p, p, p, i, i, i, i, p]
    L.gemv_bf16_split.restype = i
    L.gemv_bf16_split.argtypes = [p, p, p, i, i, i, i, p, ctypes.c_size_t, p]
    L.gemv_split_workspace_bytes.restype = i
    L.gemv_split_workspace_bytes.argtypes = [i, i, ctypes.POINTER(ctypes.c_size_t)]
    L.gemv_split_heuristic.restype = i
    L.gemv_split_heuristic.argtypes = [i, i, ctypes.POINTER(i)]
    L.ssd_chunk_state.restype = i
    L.ssd_chunk_state.argtypes = [p, p, p, p, p] + [i] * 7 + [p]
    L.ssd_state_passing.restype = i
    L.ssd_state_passing.argtypes = [p, p, p, p, p] + [i] * 6 + [p]
    L.ssd_bmm_chunk.restype = i
    L.ssd_bmm_chunk.argtypes = [p, p, p] + [i] * 5 + [p]
    L.ssd_chunk_scan.restype = i
    L.ssd_chunk_scan.argtypes = [p] * 8 + [i] * 7 + [p]
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


def ta_split_workspace_bytes(B: int, Hq: int, Sq: int, D: int, num_splits: int) -> int:
    n = ctypes.c_size_t()
    rc = lib().ta_split_workspace_bytes(B, Hq, Sq, D, num_splits, ctypes.byref(n))
    if rc != TA_OK:
        raise TileAttnError(rc, ta_status_string(rc))
    return n.value


def ta_split_heuristic(B: int, Hq: int, Hkv: int, Sq: int, Sk: int, D: int, causal: bool) -> int:
    n = ctypes.c_int()
    rc = lib().ta_split_heuristic(B, Hq, Hkv, Sq, Sk, D, int(bool(causal)), ctypes.byref(n))
    if rc != TA_OK:
        raise TileAttnError(rc, ta_status_string(rc))
    return n.value


def attn_fwd_split_raw(Q, K, V, O, o_bf16, LSE, B, Hq, Hkv, Sq, Sk, D, causal, scale,
                       num_splits, workspace, workspace_bytes, stream) -> int:
    """attn_fwd_split with integer pointers; returns the status code."""
    return lib().attn_fwd_split(Q, K, V, O, int(bool(o_bf16)), LSE, B, Hq, Hkv, Sq, Sk, D,
                                int(causal), float(scale), int(num_splits), workspace,
                                int(workspace_bytes), stream)


def attn_fwd_split_noalloc_raw(Q, K, V, O, o_bf16, LSE, B, Hq, Hkv, Sq, Sk, D, causal, scale,
                               num_splits, stream) -> int:
    """attn_fwd_split_noalloc with integer pointers; returns the status code."""
    return lib().attn_fwd_split_noalloc(Q, K, V, O, int(bool(o_bf16)), LSE, B, Hq, Hkv, Sq, Sk, D,
                                        int(causal), float(scale), int(num_splits), stream)


def attn_fwd_raw(Q, K, V, O, LSE, B, Hq, Hkv, Sq, Sk, D, causal, scale, stream) -> int:
    """The C call with integer pointers; returns the status code."""
    return lib().attn_fwd(Q, K, V, O, LSE, B, Hq, Hkv, Sq, Sk, D, int(causal), float(scale), stream)


def attn_fwd_bf16out_raw(Q, K, V, O, LSE, B, Hq, Hkv, Sq, Sk, D, causal, scale, stream) -> int:
    """attn_fwd_bf16out with integer pointers; returns the status code."""
    return lib().attn_fwd_bf16out(Q, K, V, O, LSE, B, Hq, Hkv, Sq, Sk, D, int(causal),
                                  float(scale), stream)


def _one_device(*tensors):
    """A context that makes the tensors' device current for the launch (the
    library launches on the current device); raises if they are spread over
    several devices."""
    import torch

    dev = tensors[0].device
    for t in tensors[1:]:
        if t is not None and t.device != dev:
            raise TypeError(f"all tensors must be on one device ({dev} and {t.device} given)")
    return torch.cuda.device(dev)


def _attn(q, k, v, causal, scale, out, lse, stream, o_dtype, raw):
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
        out = torch.empty((B, Hq, Sq, D), dtype=o_dtype, device=q.device)
    if lse is None:
        lse = torch.empty((B, Hq, Sq), dtype=torch.float32, device=q.device)
    for name, t, shape, dt in (("out", out, (B, Hq, Sq, D), o_dtype),
                               ("lse", lse, (B, Hq, Sq), torch.float32)):
        if t.dtype != dt or tuple(t.shape) != shape or not t.is_contiguous():
            raise TypeError(f"{name} must be a contiguous {dt} tensor of shape {shape}")
    if stream is None:
        stream = torch.cuda.current_stream(q.device)
    with _one_device(q, k, v, out, lse):
        rc = raw(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), lse.data_ptr(),
                 B, Hq, Hkv, Sq, Sk, D, causal, scale, stream.cuda_stream)
    if rc != TA_OK:
        raise TileAttnError(rc, ta_status_string(rc))
    return out, lse


def attn_fwd(q, k, v, causal: bool = False, scale: float | None = None, out=None, lse=None,
             stream=None):
    """O, LSE = attention forward of bf16 BHSD tensors q [B,Hq,Sq,D] and
    k, v [B,Hkv,Sk,D] on the GPU.  Returns fp32 O [B,Hq,Sq,D] and
    LSE [B,Hq,Sq].  ``scale`` defaults to 1/sqrt(D).  The launch is
    asynchronous on ``stream`` (default: torch's current stream)."""
    import torch

    return _attn(q, k, v, causal, scale, out, lse, stream, torch.float32, attn_fwd_raw)


def attn_fwd_bf16out(q, k, v, causal: bool = False, scale: float | None = None, out=None,
                     lse=None, stream=None):
    """As attn_fwd, with O returned in bfloat16 (the fp32 result rounded to
    nearest even by the kernel)."""
    import torch

    return _attn(q, k, v, causal, scale, out, lse, stream, torch.bfloat16, attn_fwd_bf16out_raw)


def attn_fwd_split(q, k, v, causal: bool = False, scale: float | None = None,
                   num_splits: int | None = None, out=None, lse=None, workspace=None,
                   out_dtype=None, stream=None):
    """attn_fwd with the key range split over ``num_splits`` workgroups per
    query tile (default: ta_split_heuristic) and the partial results merged
    by a second kernel.  ``workspace`` is a uint8 GPU tensor of at least
    ta_split_workspace_bytes(...) bytes (allocated here if None); it must
    stay alive until the launch has finished on ``stream``.  ``out_dtype``
    is torch.float32 (default) or torch.bfloat16."""
    import torch

    o_dtype = torch.float32 if out_dtype is None else out_dtype
    if o_dtype not in (torch.float32, torch.bfloat16):
        raise TypeError("out_dtype must be torch.float32 or torch.bfloat16")
    B, Hq, Sq, D = q.shape
    Hkv, Sk = k.shape[1], k.shape[2]
    if num_splits is None:
        num_splits = ta_split_heuristic(B, Hq, Hkv, Sq, Sk, D, causal)
    need = ta_split_workspace_bytes(B, Hq, Sq, D, num_splits)
    if stream is None:
        stream = torch.cuda.current_stream(q.device)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=q.device)
        # freed when this call returns: keep the allocator from handing the
        # block to other work before the launch on ``stream`` has finished
        workspace.record_stream(stream)
    if (workspace.dtype != torch.uint8 or workspace.device != q.device
            or not workspace.is_contiguous()):
        raise TypeError("workspace must be a contiguous uint8 tensor on q's device")
    ws_ptr, ws_bytes = workspace.data_ptr(), workspace.numel()

    def raw(Q, K, V, O, LSE, B, Hq, Hkv, Sq, Sk, D, causal, scale, stream):
        return attn_fwd_split_raw(Q, K, V, O, o_dtype == torch.bfloat16, LSE, B, Hq, Hkv, Sq, Sk,
                                  D, causal, scale, num_splits, ws_ptr, ws_bytes, stream)

    return _attn(q, k, v, causal, scale, out, lse, stream, o_dtype, raw)


def attn_fwd_split_noalloc(q, k, v, causal: bool = False, scale: float | None = None,
                           num_splits: int | None = None, out=None, lse=None, out_dtype=None,
                           stream=None):
    """attn_fwd_split with the partial results in the library's static
    per-GPU scratch instead of a workspace (the C call allocates nothing;
    pass ``out`` and ``lse`` to allocate nothing here either).  Calls that
    overlap on one GPU race on that scratch."""
    import torch

    o_dtype = torch.float32 if out_dtype is None else out_dtype
    if o_dtype not in (torch.float32, torch.bfloat16):
        raise TypeError("out_dtype must be torch.float32 or torch.bfloat16")
    if num_splits is None:
        B, Hq, Sq, D = q.shape
        num_splits = ta_split_heuristic(B, Hq, k.shape[1], Sq, k.shape[2], D, causal)

    def raw(Q, K, V, O, LSE, B, Hq, Hkv, Sq, Sk, D, causal, scale, stream):
        return attn_fwd_split_noalloc_raw(Q, K, V, O, o_dtype == torch.bfloat16, LSE, B, Hq, Hkv,
                                          Sq, Sk, D, causal, scale, num_splits, stream)

    return _attn(q, k, v, causal, scale, out, lse, stream, o_dtype, raw)


def mla_workspace_bytes(B: int, H: int, num_splits: int) -> int:
    n = ctypes.c_size_t()
    rc = lib().mla_workspace_bytes(B, H, num_splits, ctypes.byref(n))
    if rc != TA_OK:
        raise TileAttnError(rc, ta_status_string(rc))
    return n.value


def mla_split_heuristic(B: int, H: int, Hkv: int, Skv: int) -> int:
    n = ctypes.c_int()
    rc = lib().mla_split_heuristic(B, H, Hkv, Skv, ctypes.byref(n))
    if rc != TA_OK:
        raise TileAttnError(rc, ta_status_string(rc))
    return n.value


def mla_decode_raw(Q, Q_pe, KV, K_pe, O, LSE, B, H, Hkv, Skv, Dl, Dr, scale, num_splits,
                   workspace, workspace_bytes, stream) -> int:
    """mla_decode with integer pointers; returns the status code."""
    return lib().mla_decode(Q, Q_pe, KV, K_pe, O, LSE, B, H, Hkv, Skv, Dl, Dr, float(scale),
                            int(num_splits), workspace, int(workspace_bytes), stream)


def mla_decode(q, q_pe, kv, k_pe, scale: float | None = None, num_splits: int | None = None,
               out=None, lse=None, workspace=None, stream=None):
    """O [B,H,Dl] fp32, LSE [B,H] fp32 = one MLA decode step of bf16 GPU
    tensors q [B,H,Dl], q_pe [B,H,Dr], kv [B,Skv,Hkv,Dl], k_pe [B,Skv,Hkv,Dr].
    ``scale`` defaults to 1/sqrt(Dl + Dr); ``num_splits`` to
    mla_split_heuristic.  ``workspace`` (uint8 GPU tensor) is allocated here
    if needed and not given; it must stay alive until the launch has
    finished on ``stream``."""
    import torch

    for name, t, nd in (("q", q, 3), ("q_pe", q_pe, 3), ("kv", kv, 4), ("k_pe", k_pe, 4)):
        if t.dtype != torch.bfloat16 or not t.is_cuda or t.dim() != nd or not t.is_contiguous():
            raise TypeError(f"{name} must be a contiguous {nd}-D bfloat16 GPU tensor")
    B, H, Dl = q.shape
    Dr = q_pe.shape[2]
    Skv, Hkv = kv.shape[1], kv.shape[2]
    if (tuple(q_pe.shape[:2]) != (B, H) or tuple(kv.shape) != (B, Skv, Hkv, Dl)
            or tuple(k_pe.shape) != (B, Skv, Hkv, Dr)):
        raise TileAttnError(2, f"inconsistent shapes q{tuple(q.shape)} q_pe{tuple(q_pe.shape)} "
                               f"kv{tuple(kv.shape)} k_pe{tuple(k_pe.shape)}")
    if scale is None:
        scale = 1.0 / math.sqrt(Dl + Dr)
    if num_splits is None:
        num_splits = mla_split_heuristic(B, H, Hkv, Skv)
    if out is None:
        out = torch.empty((B, H, Dl), dtype=torch.float32, device=q.device)
    if lse is None:
        lse = torch.empty((B, H), dtype=torch.float32, device=q.device)
    for name, t, shape in (("out", out, (B, H, Dl)), ("lse", lse, (B, H))):
        if t.dtype != torch.float32 or tuple(t.shape) != shape or not t.is_contiguous():
            raise TypeError(f"{name} must be a contiguous float32 tensor of shape {shape}")
    need = mla_workspace_bytes(B, H, num_splits)
    if stream is None:
        stream = torch.cuda.current_stream(q.device)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=q.device)
        workspace.record_stream(stream)   # as in attn_fwd_split
    if workspace.dtype != torch.uint8 or not workspace.is_cuda or not workspace.is_contiguous():
        raise TypeError("workspace must be a contiguous uint8 GPU tensor")
    with _one_device(q, q_pe, kv, k_pe, out, lse, workspace):
        rc = mla_decode_raw(q.data_ptr(), q_pe.data_ptr(), kv.data_ptr(), k_pe.data_ptr(),
                            out.data_ptr(), lse.data_ptr(), B, H, Hkv, Skv, Dl, Dr, scale,
                            num_splits, workspace.data_ptr(), workspace.numel(),
                            stream.cuda_stream)
    if rc != TA_OK:
        raise TileAttnError(rc, ta_status_string(rc))
    return out, lse


def gemm_bf16_raw(A, B, C, c_bf16, M, N, K, stream) -> int:
    """gemm_bf16 with integer pointers; returns the status code."""
    return lib().gemm_bf16(A, B, C, int(bool(c_bf16)), M, N, K, stream)


def gemm_bf16(a, b, out=None, out_dtype=None, stream=None):
    """C = A B for contiguous bfloat16 GPU matrices a [M, K], b [K, N]; C is
    float32 (default) or bfloat16 (``out_dtype=torch.bfloat16``)."""
    import torch

    for name, t in (("a", a), ("b", b)):
        if t.dtype != torch.bfloat16 or not t.is_cuda or t.dim() != 2 or not t.is_contiguous():
            raise TypeError(f"{name} must be a contiguous 2-D bfloat16 GPU tensor")
    M, K = a.shape
    K2, N = b.shape
    if K2 != K:
        raise TileAttnError(2, f"inconsistent shapes a{tuple(a.shape)} b{tuple(b.shape)}")
    dt = torch.float32 if out_dtype is None else out_dtype
    if dt not in (torch.float32, torch.bfloat16):
        raise TypeError("out_dtype must be torch.float32 or torch.bfloat16")
    if out is None:
        out = torch.empty((M, N), dtype=dt, device=a.device)
    if out.dtype != dt or tuple(out.shape) != (M, N) or not out.is_contiguous():
        raise TypeError(f"out must be a contiguous {dt} tensor of shape {(M, N)}")
    if stream is None:
        stream = torch.cuda.current_stream(a.device)
    with _one_device(a, b, out):
        rc = gemm_bf16_raw(a.data_ptr(), b.data_ptr(), out.data_ptr(), dt == torch.bfloat16, M, N,
                           K, stream.cuda_stream)
    if rc != TA_OK:
        raise TileAttnError(rc, ta_status_string(rc))
    return out


def gemv_split_workspace_bytes(N: int, num_splits: int) -> int:
    n = ctypes.c_size_t()
    rc = lib().gemv_split_workspace_bytes(N, num_splits, ctypes.byref(n))
    if rc != TA_OK:
        raise TileAttnError(rc, ta_status_string(rc))
    return n.value


def gemv_split_heuristic(N: int, K: int) -> int:
    n = ctypes.c_int()
    rc = lib().gemv_split_heuristic(N, K, ctypes.byref(n))
    if rc != TA_OK:
        raise TileAttnError(rc, ta_status_string(rc))
    return n.value


def gemv_bf16_split_raw(A, B, C, c_bf16, N, K, num_splits, workspace, workspace_bytes,
                        stream) -> int:
    """gemv_bf16_split with integer pointers; returns the status code."""
    return lib().gemv_bf16_split(A, B, C, int(bool(c_bf16)), N, K, int(num_splits), workspace,
                                 int(workspace_bytes), stream)


def gemv_bf16_split(a, b, num_splits: int | None = None, out=None, out_dtype=None,
                    workspace=None, stream=None):
    """C [1, N] = a [1, K] b [K, N] for contiguous bfloat16 GPU tensors, with
    K split into ``num_splits`` ranges (default gemv_split_heuristic); C is
    float32 (default) or bfloat16.  ``workspace`` (uint8 GPU tensor) is
    allocated here if needed and not given; it must stay alive until the
    launch has finished on ``stream``."""
    import torch

    for name, t in (("a", a), ("b", b)):
        if t.dtype != torch.bfloat16 or not t.is_cuda or t.dim() != 2 or not t.is_contiguous():
            raise TypeError(f"{name} must be a contiguous 2-D bfloat16 GPU tensor")
    M, K = a.shape
    K2, N = b.shape
    if M != 1 or K2 != K:
        raise TileAttnError(2, f"inconsistent shapes a{tuple(a.shape)} b{tuple(b.shape)}")
    dt = torch.float32 if out_dtype is None else out_dtype
    if dt not in (torch.float32, torch.bfloat16):
        raise TypeError("out_dtype must be torch.float32 or torch.bfloat16")
    if num_splits is None:
        num_splits = gemv_split_heuristic(N, K)
    if out is None:
        out = torch.empty((1, N), dtype=dt, device=a.device)
    if out.dtype != dt or tuple(out.shape) != (1, N) or not out.is_contiguous():
        raise TypeError(f"out must be a contiguous {dt} tensor of shape {(1, N)}")
    need = gemv_split_workspace_bytes(N, num_splits)
    if stream is None:
        stream = torch.cuda.current_stream(a.device)
    if workspace is None:
        workspace = torch.empty(max(need, 16), dtype=torch.uint8, device=a.device)
        workspace.record_stream(stream)   # as in attn_fwd_split
    if workspace.dtype != torch.uint8 or not workspace.is_cuda or not workspace.is_contiguous():
        raise TypeError("workspace must be a contiguous uint8 GPU tensor")
    with _one_device(a, b, out, workspace):
        rc = gemv_bf16_split_raw(a.data_ptr(), b.data_ptr(), out.data_ptr(), dt == torch.bfloat16,
                                 N, K, num_splits, workspace.data_ptr(), workspace.numel(),
                                 stream.cuda_stream)
    if rc != TA_OK:
        raise TileAttnError(rc, ta_status_string(rc))
    return out


# ---------------------------------------------------------------------------
# Mamba-2 SSD chunk functions (include/tileattn.h documents them in full).
# Tensors: x [B, L, H, P] bf16; Bm, Cm [B, L, G, N] bf16; dt [B, L, H],
# A [H], D [H] fp32; cb [B, nc, G, Q, Q], states [B, nc, H, P, N] fp32.

SSD_CHUNK = 256


def _ssd_check(name, t, dtype, shape):
    import torch

    if t.dtype != dtype or not t.is_cuda or tuple(t.shape) != tuple(shape) or not t.is_contiguous():
        raise TypeError(f"{name} must be a contiguous {dtype} GPU tensor of shape {tuple(shape)}")


def _ssd_dims(x, Bm):
    Bsz, L, H, P = x.shape
    G, N = Bm.shape[2], Bm.shape[3]
    return Bsz, L, H, G, P, N, -(-L // SSD_CHUNK)


def _ssd_raise(rc):
    if rc != TA_OK:
        raise TileAttnError(rc, ta_status_string(rc))


def ssd_chunk_state(x, Bm, dt, A, out=None, stream=None):
    """states [B, nc, H, P, N] fp32 of each chunk started from zero."""
    import torch

    Bsz, L, H, G, P, N, nc = _ssd_dims(x, Bm)
    _ssd_check("x", x, torch.bfloat16, (Bsz, L, H, P))
    _ssd_check("Bm", Bm, torch.bfloat16, (Bsz, L, G, N))
    _ssd_check("dt", dt, torch.float32, (Bsz, L, H))
    _ssd_check("A", A, torch.float32, (H,))
    if out is None:
        out = torch.empty((Bsz, nc, H, P, N), dtype=torch.float32, device=x.device)
    _ssd_check("out", out, torch.float32, (Bsz, nc, H, P, N))
    stream = stream or torch.cuda.current_stream(x.device)
    with _one_device(x, Bm, dt, A, out):
        _ssd_raise(lib().ssd_chunk_state(x.data_ptr(), Bm.data_ptr(), dt.data_ptr(), A.data_ptr(),
                                         out.data_ptr(), Bsz, L, H, G, P, N, SSD_CHUNK,
                                         stream.cuda_stream))
    return out


def ssd_state_passing(states, dt, A, prev=None, final=None, stream=None):
    """(prev_states [B, nc, H, P, N], final_states [B, H, P, N]): the state
    each chunk enters with, and the state after the last chunk."""
    import torch

    Bsz, nc, H, P, N = states.shape
    L = dt.shape[1]
    _ssd_check("states", states, torch.float32, (Bsz, nc, H, P, N))
    _ssd_check("dt", dt, torch.float32, (Bsz, L, H))
    _ssd_check("A", A, torch.float32, (H,))
    if -(-L // SSD_CHUNK) != nc:
        raise TileAttnError(2, "states and dt disagree on the number of chunks")
    if prev is None:
        prev = torch.empty_like(states)
    if final is None:
        final = torch.empty((Bsz, H, P, N), dtype=torch.float32, device=states.device)
    _ssd_check("prev", prev, torch.float32, (Bsz, nc, H, P, N))
    _ssd_check("final", final, torch.float32, (Bsz, H, P, N))
    stream = stream or torch.cuda.current_stream(states.device)
    with _one_device(states, dt, A, prev, final):
        _ssd_raise(lib().ssd_state_passing(states.data_ptr(), dt.data_ptr(), A.data_ptr(),
                                           prev.data_ptr(), final.data_ptr(), Bsz, L, H, P, N,
                                           SSD_CHUNK, stream.cuda_stream))
    return prev, final


def ssd_bmm_chunk(Cm, Bm, out=None, stream=None):
    """cb [B, nc, G, Q, Q] fp32: cb[l][s] = Cm_l . Bm_s inside each chunk."""
    import torch

    Bsz, L, G, N = Cm.shape
    nc = -(-L // SSD_CHUNK)
    _ssd_check("Cm", Cm, torch.bfloat16, (Bsz, L, G, N))
    _ssd_check("Bm", Bm, torch.bfloat16, (Bsz, L, G, N))
    if out is None:
        out = torch.empty((Bsz, nc, G, SSD_CHUNK, SSD_CHUNK), dtype=torch.float32, device=Cm.device)
    _ssd_check("out", out, torch.float32, (Bsz, nc, G, SSD_CHUNK, SSD_CHUNK))
    stream = stream or torch.cuda.current_stream(Cm.device)
    with _one_device(Cm, Bm, out):
        _ssd_raise(lib().ssd_bmm_chunk(Cm.data_ptr(), Bm.data_ptr(), out.data_ptr(), Bsz, L, G, N,
                                       SSD_CHUNK, stream.cuda_stream))
    return out


def ssd_chunk_scan(x, Cm, cb, dt, A, prev_states, D=None, out=None, stream=None):
    """y [B, L, H, P] fp32 of the chunk-scan function."""
    import torch

    Bsz, L, H, G, P, N, nc = _ssd_dims(x, Cm)
    _ssd_check("x", x, torch.bfloat16, (Bsz, L, H, P))
    _ssd_check("Cm", Cm, torch.bfloat16, (Bsz, L, G, N))
    _ssd_check("cb", cb, torch.float32, (Bsz, nc, G, SSD_CHUNK, SSD_CHUNK))
    _ssd_check("dt", dt, torch.float32, (Bsz, L, H))
    _ssd_check("A", A, torch.float32, (H,))
    _ssd_check("prev_states", prev_states, torch.float32, (Bsz, nc, H, P, N))
    if D is not None:
        _ssd_check("D", D, torch.float32, (H,))
    if out is None:
        out = torch.empty((Bsz, L, H, P), dtype=torch.float32, device=x.device)
    _ssd_check("out", out, torch.float32, (Bsz, L, H, P))
    stream = stream or torch.cuda.current_stream(x.device)
    with _one_device(x, Cm, cb, dt, A, prev_states, D, out):
        _ssd_raise(lib().ssd_chunk_scan(x.data_ptr(), Cm.data_ptr(), cb.data_ptr(), dt.data_ptr(),
                                        A.data_ptr(), prev_states.data_ptr(),
                                        D.data_ptr() if D is not None else None, out.data_ptr(),
                                        Bsz, L, H, G, P, N, SSD_CHUNK, stream.cuda_stream))
    return out


def ssd_forward(x, dt, A, Bm, Cm, D=None, stream=None):
    """The four SSD functions chained on the GPU: (y [B, L, H, P], final
    states [B, H, P, N])."""
    states = ssd_chunk_state(x, Bm, dt, A, stream=stream)
    prev, final = ssd_state_passing(states, dt, A, stream=stream)
    cb = ssd_bmm_chunk(Cm, Bm, stream=stream)
    return ssd_chunk_scan(x, Cm, cb, dt, A, prev, D, stream=stream), final
