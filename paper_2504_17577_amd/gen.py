"""Seeded synthetic inputs for attention forward: the one module that both the
HIP path (through the tests and the bench) and the CPU oracle consume.

It holds none of attention's arithmetic: it draws i.i.d. normal samples,
rounds them to bfloat16 and applies the input recipe of each workload.  Every
tensor is returned as raw bfloat16 bit patterns (``numpy.uint16``) in the
contiguous BHSD layout ``[batch, heads, seq, head_dim]``.

Random numbers come from numpy's counter-based Philox-4x32-10 generator
(Salmon et al., SC'11).  Each tensor has its own substream, keyed by
``(seed, workload id, tensor id)``, so any tensor can be regenerated alone and
two tensors never share draws.
"""
from __future__ import annotations

import dataclasses
import hashlib
import math

import numpy as np

TENSOR_Q, TENSOR_K, TENSOR_V = 0, 1, 2


@dataclasses.dataclass(frozen=True)
class Workload:
    """One attention-forward problem: shapes, masking and input recipe."""

    name: str
    wid: int          # substream id of the workload
    B: int
    Hq: int
    Hkv: int
    Sq: int
    Sk: int
    D: int
    causal: bool
    peaky_every: int = 0      # 0: no peaky rows; else scale key rows j % peaky_every == 0
    peaky_factor: float = 1.0  # ... by this power of two

    @property
    def scale(self) -> float:
        """Softmax scale 1/sqrt(D), rounded to the fp32 value both sides use."""
        return float(np.float32(1.0 / math.sqrt(self.D)))

    def pairs(self) -> int:
        """Number of visible (query, key) pairs in one head."""
        if not self.causal:
            return self.Sq * self.Sk
        off = self.Sk - self.Sq
        return sum(min(self.Sk, i + 1 + off) for i in range(self.Sq))

    def flops(self) -> int:
        """Matmul flops of the forward pass over visible pairs only: QK^T and
        PV each cost 2*D flops per visible pair."""
        return 4 * self.D * self.B * self.Hq * self.pairs()

    def bytes(self, o_bytes: int = 4) -> int:
        """Algorithmic HBM bytes: bf16 Q, K, V read once, O (``o_bytes`` per
        element: 4 for fp32, 2 for bf16) and fp32 LSE written once."""
        q = self.B * self.Hq * self.Sq * self.D
        kv = self.B * self.Hkv * self.Sk * self.D
        return 2 * (q + 2 * kv) + o_bytes * q + 4 * self.B * self.Hq * self.Sq

    def describe(self) -> str:
        s = (f"B={self.B} Hq={self.Hq} Hkv={self.Hkv} Sq={self.Sq} Sk={self.Sk} "
             f"D={self.D} {'causal' if self.causal else 'non-causal'}")
        if self.peaky_every:
            s += f", key rows j%{self.peaky_every}==0 x{self.peaky_factor:g}"
        return s


# Workloads: a tiny correctness case, a causal D=64 case, the dense D=128
# throughput case, a long causal case with peaky keys, a grouped-query causal
# case, the paper's five FlashAttention benchmark shapes, and two shapes with
# fewer queries than keys.  All draw Q/K/V
# i.i.d. N(0,1) in bf16 with scale 1/sqrt(D).
WORKLOADS = {
    w.name: w
    for w in (
        Workload("tiny_d64_s128", 0, 1, 2, 2, 128, 128, 64, False),
        Workload("causal_d64_s1k", 1, 4, 16, 16, 1024, 1024, 64, True),
        Workload("dense_d128_s2k", 2, 8, 32, 32, 2048, 2048, 128, False),
        Workload("causal_peaky_d128_s8k", 3, 1, 32, 32, 8192, 8192, 128, True,
                 peaky_every=64, peaky_factor=8.0),
        Workload("gqa4_causal_d128_s4k", 4, 2, 32, 8, 4096, 4096, 128, True),
        # the paper's FlashAttention benchmark shapes (table "FlashAttention
        # shapes in our benchmark"): batch 1, 32 heads, head dim 128
        Workload("paper_fa0_s512_causal", 10, 1, 32, 32, 512, 512, 128, True),
        Workload("paper_fa1_s512", 11, 1, 32, 32, 512, 512, 128, False),
        Workload("paper_fa2_s1k_causal", 12, 1, 32, 32, 1024, 1024, 128, True),
        Workload("paper_fa3_s1k", 13, 1, 32, 32, 1024, 1024, 128, False),
        Workload("paper_fa4_s4k_causal", 14, 1, 32, 32, 4096, 4096, 128, True),
        # query and key lengths that differ: a 1k-query chunk of a causal
        # prefill against an 8k-key cache (bottom-right alignment, GQA 4), and
        # 512 queries attending to 4k keys without a mask
        Workload("chunk_causal_d128_q1k_k8k", 20, 1, 32, 8, 1024, 8192, 128, True),
        Workload("cross_d128_q512_k4k", 21, 4, 16, 16, 512, 4096, 128, False),
    )
}


def bf16_from_f32(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 with round-to-nearest-even and return
    the bit patterns.  Inputs here are finite, so no NaN special case."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def f32_from_bf16(u: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bit patterns to float32 (exact)."""
    return (np.asarray(u, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _stream(seed: int, wid: int, tensor: int) -> np.random.Generator:
    key = np.array([seed & 0xFFFFFFFFFFFFFFFF, (wid << 8) | tensor], dtype=np.uint64)
    return np.random.Generator(np.random.Philox(key=key))


def normal_bf16(shape, seed: int, wid: int, tensor: int) -> np.ndarray:
    """i.i.d. N(0,1) samples of the given shape, as bfloat16 bits."""
    g = _stream(seed, wid, tensor)
    x = g.standard_normal(size=int(np.prod(shape)), dtype=np.float32)
    return bf16_from_f32(x).reshape(shape)


def scale_rows_bf16(u: np.ndarray, every: int, factor: float) -> np.ndarray:
    """Multiply rows j % every == 0 (axis -2) by ``factor``.  For a power of
    two this is exact in bfloat16 for the normal samples drawn here."""
    out = u.copy()
    rows = f32_from_bf16(out[..., ::every, :]) * np.float32(factor)
    out[..., ::every, :] = bf16_from_f32(rows)
    return out


def make_inputs(w: Workload, seed: int = 0):
    """(q, k, v) bfloat16 bit arrays for workload ``w``."""
    q = normal_bf16((w.B, w.Hq, w.Sq, w.D), seed, w.wid, TENSOR_Q)
    k = normal_bf16((w.B, w.Hkv, w.Sk, w.D), seed, w.wid, TENSOR_K)
    v = normal_bf16((w.B, w.Hkv, w.Sk, w.D), seed, w.wid, TENSOR_V)
    if w.peaky_every:
        k = scale_rows_bf16(k, w.peaky_every, w.peaky_factor)
    return q, k, v


def random_problem(B, Hq, Hkv, Sq, Sk, D, seed: int, wid: int = 100, std: float = 1.0):
    """(q, k, v) bfloat16 bits for an ad-hoc shape (tests' edge cases)."""
    def one(shape, t):
        g = _stream(seed, wid, t)
        x = g.standard_normal(size=int(np.prod(shape)), dtype=np.float32) * np.float32(std)
        return bf16_from_f32(x).reshape(shape)
    return (one((B, Hq, Sq, D), TENSOR_Q), one((B, Hkv, Sk, D), TENSOR_K),
            one((B, Hkv, Sk, D), TENSOR_V))


def digest(u: np.ndarray) -> str:
    """Short BLAKE2b digest of an array's bytes (records which inputs ran)."""
    return hashlib.blake2b(np.ascontiguousarray(u).view(np.uint8), digest_size=8).hexdigest()


# ---------------------------------------------------------------------------
# Multi-head latent attention (MLA) decode inputs.  One new query token per
# batch element attends to a cache of Skv positions.  Layouts follow the
# paper's MLA listing (appendix "Implementation of FlashMLA with TileLang"):
#   q     [B, H, Dl]         latent part of the query
#   q_pe  [B, H, Dr]         rotary part of the query
#   kv    [B, Skv, Hkv, Dl]  latent cache, used both as key and as value
#   k_pe  [B, Skv, Hkv, Dr]  rotary part of the key
# The paper gives no sizes; the workloads use DeepSeek-V3's published MLA
# dimensions (128 query heads, one latent head of 512, rotary part 64).

TENSOR_QPE, TENSOR_KPE = 3, 4


@dataclasses.dataclass(frozen=True)
class MlaWorkload:
    """One MLA decode problem: shapes and input recipe (i.i.d. N(0,1))."""

    name: str
    wid: int
    B: int
    H: int
    Hkv: int
    Skv: int
    Dl: int = 512
    Dr: int = 64

    @property
    def scale(self) -> float:
        """Softmax scale 1/sqrt(Dl + Dr) (scores then have unit variance),
        rounded to the fp32 value both sides use."""
        return float(np.float32(1.0 / math.sqrt(self.Dl + self.Dr)))

    def flops(self) -> int:
        """Matmul flops: scores over Dl + Dr, then P V over Dl, per (head, key)."""
        return 2 * self.B * self.H * self.Skv * (self.Dl + self.Dr + self.Dl)

    def bytes(self) -> int:
        """Algorithmic HBM bytes: bf16 cache (kv, k_pe) and queries read once,
        fp32 O and LSE written once."""
        cache = self.B * self.Skv * self.Hkv * (self.Dl + self.Dr) * 2
        q = self.B * self.H * (self.Dl + self.Dr) * 2
        return cache + q + self.B * self.H * (self.Dl + 1) * 4

    def describe(self) -> str:
        return (f"B={self.B} H={self.H} Hkv={self.Hkv} Skv={self.Skv} Dl={self.Dl} "
                f"Dr={self.Dr} decode")


MLA_WORKLOADS = {
    w.name: w
    for w in (
        MlaWorkload("mla_tiny_s200", 30, 2, 128, 1, 200),
        MlaWorkload("mla_b64_s8k", 31, 64, 128, 1, 8192),
        MlaWorkload("mla_b128_s4k", 32, 128, 128, 1, 4096),
        MlaWorkload("mla_gqa2_b8_s2k", 33, 8, 64, 2, 2048),
    )
}


def make_mla_inputs(w: MlaWorkload, seed: int = 0):
    """(q, q_pe, kv, k_pe) bfloat16 bit arrays for MLA workload ``w``."""
    q = normal_bf16((w.B, w.H, w.Dl), seed, w.wid, TENSOR_Q)
    q_pe = normal_bf16((w.B, w.H, w.Dr), seed, w.wid, TENSOR_QPE)
    kv = normal_bf16((w.B, w.Skv, w.Hkv, w.Dl), seed, w.wid, TENSOR_K)
    k_pe = normal_bf16((w.B, w.Skv, w.Hkv, w.Dr), seed, w.wid, TENSOR_KPE)
    return q, q_pe, kv, k_pe


def random_mla_problem(B, H, Hkv, Skv, seed: int, Dl: int = 512, Dr: int = 64, wid: int = 101):
    """(q, q_pe, kv, k_pe) bfloat16 bits for an ad-hoc MLA shape."""
    return make_mla_inputs(MlaWorkload("adhoc", wid, B, H, Hkv, Skv, Dl, Dr), seed)


# ---------------------------------------------------------------------------
# Matrix multiplication C = A B (the paper's Matmul listing: A [M, K] and
# B [K, N] row-major, tiles of C accumulated over K).  The shapes are the
# paper's M0-M7 (appendix table "Matrix shapes in our benchmark"); A and B
# i.i.d. N(0,1) in bf16.

@dataclasses.dataclass(frozen=True)
class GemmWorkload:
    name: str
    wid: int
    M: int
    N: int
    K: int

    def flops(self) -> int:
        return 2 * self.M * self.N * self.K

    def bytes(self, c_bytes: int = 2) -> int:
        """A and B read once (bf16), C written once."""
        return 2 * (self.M * self.K + self.K * self.N) + c_bytes * self.M * self.N

    def describe(self) -> str:
        return f"M={self.M} N={self.N} K={self.K}"


GEMM_WORKLOADS = {
    w.name: w
    for w in (
        GemmWorkload("gemm_tiny", 40, 256, 384, 192),
        GemmWorkload("gemm_m0", 41, 4096, 1024, 8192),
        GemmWorkload("gemm_m1", 42, 4096, 8192, 8192),
        GemmWorkload("gemm_m2", 43, 4096, 28672, 8192),
        GemmWorkload("gemm_m3", 44, 4096, 8192, 28672),
        GemmWorkload("gemm_m4", 45, 8192, 1024, 8192),
        GemmWorkload("gemm_m5", 46, 8192, 8192, 8192),
        GemmWorkload("gemm_m6", 47, 8192, 28672, 8192),
        GemmWorkload("gemm_m7", 48, 8192, 8192, 28672),
        # M = 1: the paper's matrix-vector shapes V0-V7 (same table)
        GemmWorkload("gemv_tiny", 60, 1, 320, 200),
        GemmWorkload("gemv_v0", 61, 1, 16384, 16384),
        GemmWorkload("gemv_v1", 62, 1, 43008, 14336),
        GemmWorkload("gemv_v2", 63, 1, 14336, 14336),
        GemmWorkload("gemv_v3", 64, 1, 57344, 14336),
        GemmWorkload("gemv_v4", 65, 1, 14336, 57344),
        GemmWorkload("gemv_v5", 66, 1, 9216, 9216),
        GemmWorkload("gemv_v6", 67, 1, 36864, 9216),
        GemmWorkload("gemv_v7", 68, 1, 9216, 36864),
    )
}

TENSOR_A, TENSOR_B = 5, 6


def make_gemm_inputs(w: GemmWorkload, seed: int = 0):
    """(a [M, K], b [K, N]) bfloat16 bit arrays for GEMM workload ``w``.
    For M = 1 (up to 8.2e8 elements of B) B is drawn block-wise by the
    thread pool of ``normal_bf16_blocks``."""
    a = normal_bf16((w.M, w.K), seed, w.wid, TENSOR_A)
    if w.M == 1:
        return a, normal_bf16_blocks((w.K, w.N), seed, w.wid, TENSOR_B)
    return a, normal_bf16((w.K, w.N), seed, w.wid, TENSOR_B)


def random_gemm_problem(M: int, N: int, K: int, seed: int, wid: int = 102):
    return make_gemm_inputs(GemmWorkload("adhoc", wid, M, N, K), seed)


# ---------------------------------------------------------------------------
# Mamba-2 state-space duality (SSD) chunk kernels, the paper's linear-attention
# workload ("chunk-scan and chunk-state functions from Mamba-2"; appendix
# table "Linear Attention shapes in our benchmark": batch, 64 heads, sequence
# length, head dim 64, state dim 128).  Layouts are Mamba-2's:
#   x      [B, L, H, P]  bf16     per-head input
#   Bm, Cm [B, L, G, N]  bf16     input / output projections, head h uses group h // (H/G)
#   dt     [B, L, H]     fp32     step sizes (> 0)
#   A      [H]           fp32     decay rates (< 0)
#   D      [H]           fp32     skip weights
# Recipe: x, Bm, Cm i.i.d. N(0,1); dt = exp(U(ln 1e-3, ln 1e-1)) and
# A = -exp(U(ln 1, ln 16)), the ranges Mamba-2 initialises them in;
# D ~ U(0.5, 1.5).  x, Bm and Cm are drawn in blocks of 2^23 elements, one
# jumped substream per block, by a thread pool (the largest x is 2^31
# elements).  The chunk-scan function also takes the per-chunk matrix
# cb [B, nc, G, Q, Q] and the entering states [B, nc, H, P, N] (fp32); for
# tests of that function alone they are drawn here too: cb ~ N(0, N) (the
# spread of a dot product of two N-vectors of unit normals), states ~ N(0, 1).

TENSOR_X, TENSOR_BM, TENSOR_CM, TENSOR_DT, TENSOR_A, TENSOR_D = 10, 11, 12, 13, 14, 15
TENSOR_CB, TENSOR_STATES = 16, 17


@dataclasses.dataclass(frozen=True)
class SsdWorkload:
    """One SSD chunk-kernel problem: shapes and input recipe."""

    name: str
    wid: int
    B: int
    L: int
    H: int
    G: int = 1
    P: int = 64
    N: int = 128
    Q: int = 256      # chunk size (Mamba-2's default)

    @property
    def nc(self) -> int:
        return -(-self.L // self.Q)

    def flops_state(self) -> int:
        """Matmul flops of the chunk-state function: 2 P N per position and head."""
        return 2 * self.B * self.H * self.L * self.P * self.N

    def flops_scan(self) -> int:
        """Matmul flops of the chunk-scan function per position and head: the
        entering-state term (2 N P) and the causal within-chunk term
        (2 P per visible earlier position of the chunk)."""
        pairs = 0
        for c in range(self.nc):
            n = min(self.Q, self.L - c * self.Q)
            pairs += n * (n + 1) // 2
        return self.B * self.H * (2 * self.L * self.N * self.P + 2 * pairs * self.P)

    def bytes_state(self) -> int:
        """Algorithmic HBM bytes of chunk-state: x, Bm, dt read once, fp32 states written."""
        return (2 * self.B * self.L * (self.H * self.P + self.G * self.N) + 4 * self.B * self.L * self.H
                + 4 * self.B * self.nc * self.H * self.P * self.N)

    def bytes_scan(self) -> int:
        """Algorithmic HBM bytes of chunk-scan: x, Cm, cb (lower triangle is all
        that is needed, counted whole), dt, entering states read once; fp32 out written."""
        return (2 * self.B * self.L * (self.H * self.P + self.G * self.N)
                + 4 * self.B * self.nc * self.G * self.Q * self.Q + 4 * self.B * self.L * self.H
                + 4 * self.B * self.nc * self.H * self.P * self.N + 4 * self.B * self.L * self.H * self.P)

    def describe(self) -> str:
        return (f"B={self.B} L={self.L} H={self.H} G={self.G} P={self.P} N={self.N} "
                f"chunk={self.Q}")


SSD_WORKLOADS = {
    w.name: w
    for w in (
        SsdWorkload("ssd_tiny_s300", 50, 2, 300, 4, 2),
        SsdWorkload("ssd_b1_s1k", 51, 1, 1024, 64),
        SsdWorkload("ssd_b1_s2k", 52, 1, 2048, 64),
        SsdWorkload("ssd_b1_s8k", 53, 1, 8192, 64),
        SsdWorkload("ssd_b64_s1k", 54, 64, 1024, 64),
        SsdWorkload("ssd_b64_s2k", 55, 64, 2048, 64),
        SsdWorkload("ssd_b64_s8k", 56, 64, 8192, 64),
    )
}


BLOCK = 1 << 23   # elements per independently drawn block of a large tensor


def normal_bf16_blocks(shape, seed: int, wid: int, tensor: int, threads: int = 16) -> np.ndarray:
    """i.i.d. N(0,1) samples as bfloat16 bits, drawn in blocks of BLOCK
    elements: block i comes from the tensor's Philox substream jumped i times
    (2^128 draws apart), so the result does not depend on ``threads``, and
    the blocks are drawn by a thread pool (numpy releases the GIL while it
    fills them)."""
    from concurrent.futures import ThreadPoolExecutor

    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.uint16)
    key = np.array([seed & 0xFFFFFFFFFFFFFFFF, (wid << 8) | tensor], dtype=np.uint64)

    def fill(i):
        g = np.random.Generator(np.random.Philox(key=key).jumped(i))
        m = min(BLOCK, n - i * BLOCK)
        out[i * BLOCK:i * BLOCK + m] = bf16_from_f32(g.standard_normal(size=m, dtype=np.float32))

    with ThreadPoolExecutor(max(1, threads)) as ex:
        list(ex.map(fill, range(-(-n // BLOCK))))
    return out.reshape(shape)


def _uniform_f32(shape, lo, hi, seed, wid, tensor):
    g = _stream(seed, wid, tensor)
    return g.uniform(lo, hi, size=int(np.prod(shape))).astype(np.float32).reshape(shape)


def make_ssd_inputs(w: SsdWorkload, seed: int = 0):
    """dict of x, Bm, Cm (bfloat16 bits), dt, A, D (float32) for workload ``w``."""
    ln = math.log
    return {
        "x": normal_bf16_blocks((w.B, w.L, w.H, w.P), seed, w.wid, TENSOR_X),
        "Bm": normal_bf16_blocks((w.B, w.L, w.G, w.N), seed, w.wid, TENSOR_BM),
        "Cm": normal_bf16_blocks((w.B, w.L, w.G, w.N), seed, w.wid, TENSOR_CM),
        "dt": np.exp(_uniform_f32((w.B, w.L, w.H), ln(1e-3), ln(1e-1), seed, w.wid, TENSOR_DT)),
        "A": -np.exp(_uniform_f32((w.H,), ln(1.0), ln(16.0), seed, w.wid, TENSOR_A)),
        "D": _uniform_f32((w.H,), 0.5, 1.5, seed, w.wid, TENSOR_D),
    }


def make_ssd_scan_extras(w: SsdWorkload, seed: int = 0):
    """(cb [B,nc,G,Q,Q], states [B,nc,H,P,N]) float32 draws for testing the
    chunk-scan function on its own."""
    g = _stream(seed, w.wid, TENSOR_CB)
    cb = g.standard_normal(size=w.B * w.nc * w.G * w.Q * w.Q, dtype=np.float32)
    cb = (cb * np.float32(math.sqrt(w.N))).reshape(w.B, w.nc, w.G, w.Q, w.Q)
    g = _stream(seed, w.wid, TENSOR_STATES)
    st = g.standard_normal(size=w.B * w.nc * w.H * w.P * w.N, dtype=np.float32)
    return cb, st.reshape(w.B, w.nc, w.H, w.P, w.N)


def random_ssd_problem(B, L, H, G, seed: int, P: int = 64, N: int = 128, Q: int = 256,
                       wid: int = 103):
    """(workload, inputs) for an ad-hoc SSD shape (tests' edge cases)."""
    w = SsdWorkload("adhoc", wid, B, L, H, G, P, N, Q)
    return w, make_ssd_inputs(w, seed)
