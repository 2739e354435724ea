"""Host-side checks of libtileattn that need no GPU: the library loads and
exports every function include/tileattn.h declares, argument validation
returns the documented status before any HIP call, and the key-tile schedule
agrees with a brute-force count of visible and masked (query, key) pairs."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2504_17577_amd import tileattn as ta

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_functions():
    text = open(os.path.join(ROOT, "include", "tileattn.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^[A-Za-z_][\w \*]*?\b(\w+)\s*\(", text, flags=re.M)))


def test_exports_every_declared_symbol():
    names = declared_functions()
    assert {"attn_fwd", "ta_schedule", "ta_tile_shape", "ta_status_string", "ta_version"} <= set(names)
    lib = ctypes.CDLL(ta.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), f"{n} declared in include/tileattn.h but not exported"


def test_version_and_strings():
    assert ta.ta_version() >= 400
    for s in range(10):
        assert ta.ta_status_string(s)
    assert ta.ta_status_string(99) == "unknown status"
    assert ta.ta_tile_shape(64) == ta.ta_tile_shape(128)
    with pytest.raises(ta.TileAttnError):
        ta.ta_tile_shape(96)


# Fake, 16-byte aligned, non-overlapping addresses: every call below must
# fail validation, so nothing is ever dereferenced or launched.  A wrong
# expectation in this table would launch a kernel on these addresses, so the
# fake-pointer tests run only where no GPU is present (no /dev/kfd).
no_gpu = pytest.mark.skipif(os.path.exists("/dev/kfd"),
                            reason="fake-pointer validation cases run only without a GPU")
Q, K, V, O, L = 0x10000000, 0x20000000, 0x30000000, 0x40000000, 0x50000000
OK = dict(Q=Q, K=K, V=V, O=O, LSE=L, B=1, Hq=2, Hkv=2, Sq=128, Sk=128, D=64, causal=0,
          scale=0.125, stream=None)

BAD = [
    (dict(Q=0), 1), (dict(K=0), 1), (dict(V=0), 1), (dict(O=0), 1), (dict(LSE=0), 1),
    (dict(B=0), 2), (dict(Hq=0), 2), (dict(Hkv=0), 2), (dict(Sq=0), 2), (dict(Sk=-1), 2),
    (dict(Hq=6, Hkv=4), 2), (dict(causal=1, Sq=129, Sk=128), 2),
    (dict(Sq=1 << 25, D=128), 2),
    (dict(D=96), 3), (dict(D=256), 3), (dict(D=0), 2),
    (dict(Q=Q + 8), 4), (dict(V=V + 2), 4), (dict(O=O + 4), 4), (dict(LSE=L + 4), 4),
    (dict(scale=float("nan")), 5), (dict(scale=float("inf")), 5), (dict(scale=-0.5), 5),
    (dict(O=Q + 16), 6), (dict(LSE=K + 64), 6), (dict(LSE=O + 1024), 6), (dict(O=V - 1024), 6),
]


@no_gpu
@pytest.mark.parametrize("change,status", BAD, ids=[str(c) for c, _ in BAD])
def test_validation_before_any_hip_call(change, status):
    a = dict(OK, **change)
    rc = ta.attn_fwd_raw(a["Q"], a["K"], a["V"], a["O"], a["LSE"], a["B"], a["Hq"], a["Hkv"],
                         a["Sq"], a["Sk"], a["D"], a["causal"], a["scale"], a["stream"])
    assert rc == status, f"{change}: got {ta.STATUS.get(rc, rc)}, want {ta.STATUS[status]}"


def brute_schedule(Sq, Sk, causal, qt, BM, BN):
    """(tiles with a visible key, first tile with a masked pair) by enumeration."""
    q = np.arange(qt * BM, min(qt * BM + BM, Sq))[:, None]
    n_tiles = -(-Sk // BN)
    key = np.arange(n_tiles * BN)[None, :]
    visible = np.broadcast_to((key < Sk) & ((key <= q + (Sk - Sq)) if causal else True),
                              (len(q), n_tiles * BN))
    vis_tile = visible.reshape(len(q), n_tiles, BN).any(axis=(0, 2))
    mask_tile = (~visible).reshape(len(q), n_tiles, BN).any(axis=(0, 2))
    return vis_tile, mask_tile, int(visible.sum())


@pytest.mark.parametrize("D", [64, 128])
def test_schedule_matches_brute_force(D):
    BM, BN = ta.ta_tile_shape(D)
    rng = np.random.default_rng(0)
    shapes = [(1, 1), (37, 37), (128, 128), (129, 200), (1000, 1000), (64, 1000), (200, 129)]
    shapes += [tuple(sorted(rng.integers(1, 700, size=2))) for _ in range(12)]
    for Sq, Sk in shapes:
        for causal in (False, True):
            if causal and Sq > Sk:
                with pytest.raises(ta.TileAttnError):
                    ta.ta_schedule(Sq, Sk, D, causal, 0)
                continue
            total = 0
            for qt in range(-(-Sq // BM)):
                n, fm = ta.ta_schedule(Sq, Sk, D, causal, qt)
                vis, needs_mask, pairs = brute_schedule(Sq, Sk, causal, qt, BM, BN)
                last_vis = int(np.nonzero(vis)[0].max())
                assert n == last_vis + 1, (Sq, Sk, causal, qt, n)
                assert not needs_mask[:fm].any(), f"unmasked tile with masked pairs {Sq, Sk, qt}"
                assert fm == n or needs_mask[fm], f"first_masked not tight {Sq, Sk, qt}"
                total += pairs
            want = sum(min(Sk, i + 1 + Sk - Sq) for i in range(Sq)) if causal else Sq * Sk
            assert total == want
    with pytest.raises(ta.TileAttnError):
        ta.ta_schedule(100, 100, D, False, 1)   # only one query tile


# attn_fwd_split: the same argument errors, plus the split count and the
# workspace.  Sk=128 is two key tiles, so two splits really split and the
# workspace is checked; a fake workspace far from every other buffer.
WS = 0x60000000
WS_OK = dict(OK, splits=2, ws=WS, ws_bytes=1 << 24, o_bf16=0)
BAD_SPLIT = [(c, st) for c, st in BAD] + [
    (dict(splits=0), 2), (dict(splits=129), 2), (dict(splits=-1), 2),
    (dict(ws=0), 8), (dict(ws_bytes=2 * 2 * 128 * 65 * 4 - 1), 8),
    (dict(ws=WS + 8), 4), (dict(ws=Q - 4096), 6), (dict(ws=O + 4096), 6),
    (dict(ws=L - 16), 6), (dict(o_bf16=1, O=L - 2 * 128 * 64 * 2 + 16), 6),
]


@no_gpu
@pytest.mark.parametrize("change,status", BAD_SPLIT, ids=[str(c) for c, _ in BAD_SPLIT])
def test_split_validation_before_any_hip_call(change, status):
    a = dict(WS_OK, **change)
    rc = ta.attn_fwd_split_raw(a["Q"], a["K"], a["V"], a["O"], a["o_bf16"], a["LSE"], a["B"],
                               a["Hq"], a["Hkv"], a["Sq"], a["Sk"], a["D"], a["causal"],
                               a["scale"], a["splits"], a["ws"], a["ws_bytes"], a["stream"])
    assert rc == status, f"{change}: got {ta.STATUS.get(rc, rc)}, want {ta.STATUS[status]}"


BAD_NOALLOC = [(c, st) for c, st in BAD] + [
    (dict(splits=0), 2), (dict(splits=129), 2), (dict(splits=-1), 2),
    # partial results beyond the static scratch: 2 splits of 32 heads x 4096
    # rows x 129 floats = 135 MB
    (dict(Hq=32, Hkv=32, Sq=4096, Sk=4096, D=128), 9),
]


@no_gpu
@pytest.mark.parametrize("change,status", BAD_NOALLOC, ids=[str(c) for c, _ in BAD_NOALLOC])
def test_split_noalloc_validation_before_any_hip_call(change, status):
    a = dict(WS_OK, **change)
    rc = ta.attn_fwd_split_noalloc_raw(a["Q"], a["K"], a["V"], a["O"], a["o_bf16"], a["LSE"],
                                       a["B"], a["Hq"], a["Hkv"], a["Sq"], a["Sk"], a["D"],
                                       a["causal"], a["scale"], a["splits"], a["stream"])
    assert rc == status, f"{change}: got {ta.STATUS.get(rc, rc)}, want {ta.STATUS[status]}"


@no_gpu
def test_bf16out_validation_before_any_hip_call():
    for change, status in BAD:
        a = dict(OK, **change)
        rc = ta.attn_fwd_bf16out_raw(a["Q"], a["K"], a["V"], a["O"], a["LSE"], a["B"], a["Hq"],
                                     a["Hkv"], a["Sq"], a["Sk"], a["D"], a["causal"], a["scale"],
                                     a["stream"])
        assert rc == status, f"{change}: got {ta.STATUS.get(rc, rc)}"


def test_split_workspace_bytes():
    for B, Hq, Sq, D, n in [(1, 2, 128, 64, 2), (3, 5, 77, 128, 7), (1, 32, 1024, 128, 128)]:
        assert ta.ta_split_workspace_bytes(B, Hq, Sq, D, n) == n * B * Hq * Sq * (D + 1) * 4
    assert ta.ta_split_workspace_bytes(2, 2, 100, 64, 1) == 0
    for bad in [(0, 1, 1, 64, 2), (1, 1, 1, 64, 0), (1, 1, 1, 64, 129)]:
        with pytest.raises(ta.TileAttnError):
            ta.ta_split_workspace_bytes(*bad)
    with pytest.raises(ta.TileAttnError):
        ta.ta_split_workspace_bytes(1, 1, 1, 96, 2)


@pytest.mark.parametrize("shape", [
    (1, 32, 32, 512, 512, 128, True), (1, 32, 32, 512, 512, 128, False),
    (1, 32, 32, 1024, 1024, 128, True), (1, 32, 32, 4096, 4096, 128, True),
    (1, 32, 8, 1024, 8192, 128, True), (4, 16, 16, 512, 4096, 128, False),
    (8, 32, 32, 2048, 2048, 128, False), (1, 2, 2, 128, 128, 64, False),
    (1, 1, 1, 1, 100000, 64, False), (1, 1, 1, 1, 1, 128, True),
    (2, 8, 8, 128, 16384, 128, False),
])
def test_split_heuristic_properties(shape):
    B, Hq, Hkv, Sq, Sk, D, causal = shape
    BM, BN = ta.ta_tile_shape(D)
    wg = B * Hq * -(-Sq // BM)
    n_kv = -(-Sk // BN)
    n = ta.ta_split_heuristic(*shape)
    assert 1 <= n <= 128
    if wg >= 512:
        assert n == 1
    elif n > 1:
        assert n <= n_kv // 32                    # at least 32 key tiles per split
        assert (n - 1) * wg < 512                 # no more splits than the target needs
    if n == 1 and wg < 512:
        assert n_kv // 32 <= 1                    # only when the keys are too short to split


# mla_decode: argument errors before any HIP call (fake pointers)
MQ, MQP, MKV, MKP, MO, ML, MWS = (0x10000000, 0x18000000, 0x20000000, 0x30000000, 0x40000000,
                                  0x50000000, 0x60000000)
MLA_OK = dict(Q=MQ, Qpe=MQP, KV=MKV, Kpe=MKP, O=MO, LSE=ML, B=2, H=128, Hkv=1, Skv=256, Dl=512,
              Dr=64, scale=0.04, splits=2, ws=MWS, ws_bytes=1 << 24, stream=None)
BAD_MLA = [
    (dict(Q=0), 1), (dict(Qpe=0), 1), (dict(KV=0), 1), (dict(Kpe=0), 1), (dict(O=0), 1),
    (dict(LSE=0), 1),
    (dict(B=0), 2), (dict(H=0), 2), (dict(Hkv=0), 2), (dict(Skv=0), 2), (dict(H=128, Hkv=3), 2),
    (dict(splits=0), 2), (dict(splits=129), 2),
    (dict(Dl=256), 3), (dict(Dr=32), 3),
    (dict(Q=MQ + 8), 4), (dict(KV=MKV + 2), 4), (dict(O=MO + 4), 4), (dict(ws=MWS + 8), 4),
    (dict(scale=float("nan")), 5), (dict(scale=-1.0), 5),
    (dict(O=MKV + 64), 6), (dict(LSE=MQ + 16), 6), (dict(LSE=MO + 1024), 6),
    (dict(ws=MKP - 64), 6), (dict(ws=ML - 16), 6),
    (dict(ws=0), 8), (dict(ws_bytes=2 * 2 * 128 * 513 * 4 - 1), 8),
]


@no_gpu
@pytest.mark.parametrize("change,status", BAD_MLA, ids=[str(c) for c, _ in BAD_MLA])
def test_mla_validation_before_any_hip_call(change, status):
    a = dict(MLA_OK, **change)
    rc = ta.mla_decode_raw(a["Q"], a["Qpe"], a["KV"], a["Kpe"], a["O"], a["LSE"], a["B"], a["H"],
                           a["Hkv"], a["Skv"], a["Dl"], a["Dr"], a["scale"], a["splits"], a["ws"],
                           a["ws_bytes"], a["stream"])
    assert rc == status, f"{change}: got {ta.STATUS.get(rc, rc)}, want {ta.STATUS[status]}"


def test_mla_workspace_and_heuristic():
    assert ta.mla_workspace_bytes(64, 128, 4) == 4 * 64 * 128 * 513 * 4
    assert ta.mla_workspace_bytes(64, 128, 1) == 0
    with pytest.raises(ta.TileAttnError):
        ta.mla_workspace_bytes(0, 128, 2)
    for B, H, Hkv, Skv in [(64, 128, 1, 8192), (128, 128, 1, 4096), (1, 128, 1, 64),
                           (2, 128, 1, 200), (8, 64, 2, 2048), (512, 128, 1, 4096)]:
        n = ta.mla_split_heuristic(B, H, Hkv, Skv)
        wg = B * Hkv * -(-(H // Hkv) // 128)   # 128 query heads per workgroup
        tiles = -(-Skv // 32)
        assert 1 <= n <= 128
        if wg >= 256:
            assert n == 1
        elif n > 1:
            assert n <= tiles // 8 and (n - 1) * wg < 256
        else:
            assert tiles // 8 <= 1


# gemm_bf16: argument errors before any HIP call (fake pointers)
GA, GB, GC = 0x10000000, 0x30000000, 0x50000000
GEMM_OK = dict(A=GA, B=GB, C=GC, c_bf16=0, M=256, N=256, K=128, stream=None)
BAD_GEMM = [
    (dict(A=0), 1), (dict(B=0), 1), (dict(C=0), 1),
    (dict(M=0), 2), (dict(N=-1), 2), (dict(K=0), 2),
    (dict(M=200), 3), (dict(N=100), 3), (dict(K=96), 3),
    (dict(A=GA + 8), 4), (dict(C=GC + 4), 4),
    (dict(C=GA + 1024), 6), (dict(C=GB - 4096), 6), (dict(c_bf16=1, C=GB - 256 * 256 * 2 + 16), 6),
    # M = 1 (matrix-vector): N % 64 and K % 8; other M still need M % 128
    (dict(M=1, N=96), 3), (dict(M=1, K=12), 3), (dict(M=2), 3), (dict(M=1, C=GC + 4), 4),
    (dict(M=1, C=GA + 128), 6),
    # the tiled kernel's 32-bit offsets: K * N * 2 < 2^31
    (dict(N=65536, K=16384), 2),
]


@no_gpu
@pytest.mark.parametrize("change,status", BAD_GEMM, ids=[str(c) for c, _ in BAD_GEMM])
def test_gemm_validation_before_any_hip_call(change, status):
    a = dict(GEMM_OK, **change)
    rc = ta.gemm_bf16_raw(a["A"], a["B"], a["C"], a["c_bf16"], a["M"], a["N"], a["K"], a["stream"])
    assert rc == status, f"{change}: got {ta.STATUS.get(rc, rc)}, want {ta.STATUS[status]}"


# gemv_bf16_split: argument errors before any HIP call (fake pointers)
GW = 0x60000000
GEMV_OK = dict(A=GA, B=GB, C=GC, c_bf16=0, N=256, K=128, splits=2, ws=GW, ws_bytes=1 << 20,
               stream=None)
BAD_GEMV = [
    (dict(A=0), 1), (dict(B=0), 1), (dict(C=0), 1),
    (dict(N=0), 2), (dict(K=-8), 2), (dict(splits=0), 2), (dict(splits=65), 2),
    (dict(N=96), 3), (dict(K=12), 3),
    (dict(A=GA + 8), 4), (dict(B=GB + 2), 4), (dict(C=GC + 4), 4), (dict(ws=GW + 8), 4),
    (dict(C=GA + 128), 6), (dict(C=GB + 1024), 6), (dict(c_bf16=1, C=GB + 128 * 256 * 2 - 16), 6),
    (dict(ws=GA + 16), 6), (dict(ws=GB - 1024), 6), (dict(ws=GC - 2 * 256 * 4 + 16), 6),
    (dict(ws=0), 8), (dict(ws_bytes=2 * 256 * 4 - 1), 8),
]


@no_gpu
@pytest.mark.parametrize("change,status", BAD_GEMV, ids=[str(c) for c, _ in BAD_GEMV])
def test_gemv_split_validation_before_any_hip_call(change, status):
    a = dict(GEMV_OK, **change)
    rc = ta.gemv_bf16_split_raw(a["A"], a["B"], a["C"], a["c_bf16"], a["N"], a["K"], a["splits"],
                                a["ws"], a["ws_bytes"], a["stream"])
    assert rc == status, f"{change}: got {ta.STATUS.get(rc, rc)}, want {ta.STATUS[status]}"


def test_gemv_split_workspace_and_heuristic():
    assert ta.gemv_split_workspace_bytes(9216, 7) == 7 * 9216 * 4
    assert ta.gemv_split_workspace_bytes(9216, 1) == 0
    for bad in [(0, 2), (64, 0), (64, 65)]:
        with pytest.raises(ta.TileAttnError):
            ta.gemv_split_workspace_bytes(*bad)
    # the paper's V0-V7 (N, K): few 256-column strips split K, many do not
    # (workgroups = 256-column strips x splits: 256, 504, 504, 224, 504, 252, 432, 252)
    expect = {(16384, 16384): 4, (43008, 14336): 3, (14336, 14336): 9, (57344, 14336): 1,
              (14336, 57344): 9, (9216, 9216): 7, (36864, 9216): 3, (9216, 36864): 7}
    for (N, K), n in expect.items():
        assert ta.gemv_split_heuristic(N, K) == n, (N, K)

    def fill(w):   # share of the last round of 256 CU slots the workgroups fill
        return w / (256 * -(-w // 256))

    for N, K in [(64, 8), (64, 1 << 20), (320, 4096), (320, 1 << 20), (1024, 2048),
                 (65536, 1024), (6400, 8192), (36864, 1 << 20), (256, 1 << 16)]:
        n = ta.gemv_split_heuristic(N, K)
        strips = N // 256 if N % 256 == 0 else -(-N // 64)
        assert 1 <= n <= 64, (N, K, n)
        if n > 1:
            assert n * strips <= 512 and K // n >= 1024, (N, K, n)
        # brute force: no allowed count fills the last round better
        for m in range(2, 65):
            if m * strips <= 512 and K // m >= 1024 and m != n:
                assert fill(m * strips) <= fill(n * strips) + 1e-12 or (
                    n == 1 and N % 256 == 0 and strips < 144), (N, K, n, m)


# SSD chunk functions: argument errors before any HIP call (fake pointers).
# Shapes: B=1, L=300, H=4, G=2 -> x 153600 B, Bm/Cm 153600 B, dt 4800 B,
# cb 2 chunks x 2 groups x 256 KiB, states 2 x 4 x 32 KiB.
SX, SB, SC, SDT, SA, SD = 0x10000000, 0x11000000, 0x12000000, 0x13000000, 0x14000000, 0x15000000
SCB, SST, SOUT = 0x20000000, 0x30000000, 0x40000000
SSD_OK = dict(x=SX, Bm=SB, Cm=SC, cb=SCB, dt=SDT, A=SA, prev=SST, D=SD, out=SOUT, B=1, L=300,
              H=4, G=2, P=64, N=128, Q=256)
BAD_SSD = [
    (dict(x=0), 1), (dict(Cm=0), 1), (dict(cb=0), 1), (dict(dt=0), 1), (dict(A=0), 1),
    (dict(prev=0), 1), (dict(out=0), 1),
    (dict(B=0), 2), (dict(L=0), 2), (dict(H=0), 2), (dict(G=0), 2), (dict(H=6, G=4), 2),
    (dict(P=128), 3), (dict(N=64), 3), (dict(Q=128), 3),
    (dict(x=SX + 8), 4), (dict(cb=SCB + 4), 4), (dict(out=SOUT + 8), 4), (dict(dt=SDT + 2), 4),
    (dict(out=SX + 1024), 6), (dict(out=SCB - 4096), 6), (dict(out=SST + 16), 6),
    (dict(out=SD - 16), 6),
]


@no_gpu
@pytest.mark.parametrize("change,status", BAD_SSD, ids=[str(c) for c, _ in BAD_SSD])
def test_ssd_scan_validation_before_any_hip_call(change, status):
    a = dict(SSD_OK, **change)
    rc = ta.lib().ssd_chunk_scan(a["x"], a["Cm"], a["cb"], a["dt"], a["A"], a["prev"], a["D"],
                                 a["out"], a["B"], a["L"], a["H"], a["G"], a["P"], a["N"],
                                 a["Q"], None)
    assert rc == status, f"{change}: got {ta.STATUS.get(rc, rc)}, want {ta.STATUS[status]}"


BAD_SSD_STATE = [
    (dict(x=0), 1), (dict(Bm=0), 1), (dict(out=0), 1), (dict(L=-5), 2), (dict(H=3, G=2), 2),
    (dict(N=256), 3), (dict(Bm=SB + 2), 4), (dict(out=SB + 4096), 6), (dict(out=SDT), 6),
]


@no_gpu
@pytest.mark.parametrize("change,status", BAD_SSD_STATE, ids=[str(c) for c, _ in BAD_SSD_STATE])
def test_ssd_state_validation_before_any_hip_call(change, status):
    a = dict(SSD_OK, **change)
    rc = ta.lib().ssd_chunk_state(a["x"], a["Bm"], a["dt"], a["A"], a["out"], a["B"], a["L"],
                                  a["H"], a["G"], a["P"], a["N"], a["Q"], None)
    assert rc == status, f"{change}: got {ta.STATUS.get(rc, rc)}, want {ta.STATUS[status]}"


@no_gpu
def test_ssd_bmm_and_passing_validation_before_any_hip_call():
    L = ta.lib()
    assert L.ssd_bmm_chunk(SC, SB, 0, 1, 300, 2, 128, 256, None) == 1
    assert L.ssd_bmm_chunk(SC, SB, SCB, 1, 300, 2, 128, 128, None) == 3
    assert L.ssd_bmm_chunk(SC, SB, SC + 64, 1, 300, 2, 128, 256, None) == 6
    assert L.ssd_bmm_chunk(SC + 4, SB, SCB, 1, 300, 2, 128, 256, None) == 4
    assert L.ssd_state_passing(SST, SDT, SA, 0, None, 1, 300, 4, 64, 128, 256, None) == 1
    assert L.ssd_state_passing(SST, SDT, SA, SOUT, None, 1, 300, 4, 32, 128, 256, None) == 3
    assert L.ssd_state_passing(SST, SDT, SA, SST + 1024, None, 1, 300, 4, 64, 128, 256, None) == 6
    assert L.ssd_state_passing(SST, SDT, SA, SOUT, SOUT + 64, 1, 300, 4, 64, 128, 256, None) == 6
