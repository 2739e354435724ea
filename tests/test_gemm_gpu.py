"""GPU parity of gemm_bf16 (C = A B, bf16 inputs, fp32 accumulation) through
the C ABI against the float64 oracle.  Tolerance per element, from the
arithmetic: every bf16 x bf16 product is exact in fp32 and the K-sum is
accumulated in fp32, so |C - C_ref| <= 1e-5 * sum_k |a_ik||b_kj| (a random
rounding walk over K/16 accumulation steps stays two orders of magnitude
below this; a dropped or doubled 16-product step does not); bf16 output adds
its rounding, 2^-8 |C_ref|."""
import numpy as np
import pytest

import oracle
from paper_2504_17577_amd import gen

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

REL_ABS = 1e-5


@pytest.fixture(scope="module")
def ta():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2504_17577_amd import tileattn
    tileattn.lib()
    return tileattn


def dev(x):
    return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).cuda()


def check(tag, c, a, b, rows=None, bf16=False):
    ref = oracle.gemm(a, b, rows=rows)
    scale = oracle.gemm_abs(a, b, rows=rows)
    got = c.float().cpu().numpy() if rows is None else c.float()[torch.tensor(rows)].cpu().numpy()
    tol = REL_ABS * scale + (2.0 ** -8 * np.abs(ref) if bf16 else 0.0)
    err = np.abs(got - ref)
    assert np.isfinite(got).all(), f"{tag}: non-finite output"
    worst = float((err / tol).max())
    print(f"{tag}: max|dC|={err.max():.3e}, worst err/tol={worst:.3f}", flush=True)
    assert worst <= 1.0, tag


# at most 256 tiles of 128 x 128 (all but the last): the four-stage ring,
# with K steps 1, 3 (= stages in flight), 5 and 16; the last one has more
# tiles, but too few of 256 x 256: double-buffered 128 x 128 tiles
SHAPES = [(128, 128, 64), (256, 256, 64), (256, 384, 192), (512, 768, 320), (384, 128, 1024),
          (2304, 2304, 128)]


@pytest.mark.parametrize("shape", SHAPES, ids=[str(s) for s in SHAPES])
def test_gemm_full_compare(ta, shape):
    M, N, K = shape
    print(f"gemm {shape}", flush=True)
    a, b = gen.random_gemm_problem(M, N, K, seed=M + N + K)
    c = torch.full((M, N), float("nan"), device="cuda")
    ta.gemm_bf16(dev(a), dev(b), out=c)
    torch.cuda.synchronize()
    check(f"gemm {shape}", c, a, b)


@pytest.mark.parametrize("name", ["gemm_m0", "gemm_m4", "gemm_m5", "gemm_m3", "gemm_m1",
                                  "gemm_m2", "gemm_m6", "gemm_m7"])
def test_gemm_workload_sampled(ta, name):
    """The paper's shapes at full size (all three tile configurations):
    sampled rows against the oracle, every element finite."""
    w = gen.GEMM_WORKLOADS[name]
    print(f"gemm workload {name} {w.describe()}", flush=True)
    a, b = gen.make_gemm_inputs(w, seed=0)
    c = torch.full((w.M, w.N), float("nan"), device="cuda")
    ta.gemm_bf16(dev(a), dev(b), out=c)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(c).all())
    rng = np.random.default_rng(1)
    rows = sorted({0, 1, 31, 32, 127, 128, 255, 256, w.M - 1} |
                  {int(x) for x in rng.integers(0, w.M, size=24)})
    check(f"gemm {name}", c, a, b, rows=rows)


def test_gemm_bf16_out_is_rounded_fp32_and_deterministic(ta):
    a, b = gen.random_gemm_problem(512, 512, 256, seed=9)
    da, db = dev(a), dev(b)
    c32 = ta.gemm_bf16(da, db)
    c32b = ta.gemm_bf16(da, db)
    c16 = ta.gemm_bf16(da, db, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert torch.equal(c32.view(torch.int32), c32b.view(torch.int32))
    assert torch.equal(c16.view(torch.int16), c32.to(torch.bfloat16).view(torch.int16))
    check("gemm bf16 out", c16, a, b, bf16=True)


def test_gemm_rejects_bad_shapes(ta):
    a, b = gen.random_gemm_problem(128, 128, 96, seed=1)
    with pytest.raises(ta.TileAttnError) as e:
        ta.gemm_bf16(dev(a), dev(b))
    assert e.value.status == 3


# M = 1: the matrix-vector kernel (the paper's V0-V7 shapes)
GEMV_SHAPES = [(64, 8), (320, 200), (1024, 4096), (4096, 1000), (192, 16392), (2048, 3080),
               (36864, 72), (36864, 1048)]


@pytest.mark.parametrize("shape", GEMV_SHAPES, ids=[str(s) for s in GEMV_SHAPES])
def test_gemv_full_compare(ta, shape):
    """N % 64 == 0, K % 8 == 0: strips of 64 columns (and of 256 from
    N = 36864 on), row ranges split unevenly over the 16 waves when K / 8 is
    not a multiple of 16, waves with no rows, and every mix of the two-group
    step, the one-group step and the tail"""
    N, K = shape
    print(f"gemv N={N} K={K}", flush=True)
    a, b = gen.random_gemm_problem(1, N, K, seed=N + K)
    c = torch.full((1, N), float("nan"), device="cuda")
    ta.gemm_bf16(dev(a), dev(b), out=c)
    torch.cuda.synchronize()
    check(f"gemv {shape}", c, a, b)


@pytest.mark.parametrize("name", ["gemv_v5", "gemv_v7", "gemv_v0", "gemv_v6", "gemv_v1",
                                  "gemv_v4", "gemv_v2", "gemv_v3"])
def test_gemv_workload_sampled(ta, name):
    """The paper's matrix-vector shapes at full size: every output finite,
    sampled columns (first and last of strips, random ones) against the
    oracle on the same columns of B."""
    w = gen.GEMM_WORKLOADS[name]
    print(f"gemv workload {name} {w.describe()}", flush=True)
    a, b = gen.make_gemm_inputs(w, seed=0)
    c = torch.full((1, w.N), float("nan"), device="cuda")
    ta.gemm_bf16(dev(a), dev(b), out=c)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(c).all())
    rng = np.random.default_rng(2)
    cols = sorted({0, 1, 63, 64, 127, w.N - 64, w.N - 1} | {int(x) for x in rng.integers(0, w.N, size=40)})
    bs = np.ascontiguousarray(b[:, cols])
    ref, scale = oracle.gemm(a, bs)[0], oracle.gemm_abs(a, bs)[0]
    got = c[0, torch.tensor(cols)].cpu().numpy()
    worst = float((np.abs(got - ref) / (REL_ABS * scale)).max())
    print(f"{name}: worst err/tol={worst:.3f}", flush=True)
    assert worst <= 1.0


def test_gemv_bf16_out_and_deterministic(ta):
    a, b = gen.random_gemm_problem(1, 2048, 3000, seed=11)
    da, db = dev(a), dev(b)
    c32 = ta.gemm_bf16(da, db)
    c32b = ta.gemm_bf16(da, db)
    c16 = ta.gemm_bf16(da, db, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert torch.equal(c32.view(torch.int32), c32b.view(torch.int32))
    assert torch.equal(c16.view(torch.int16), c32.to(torch.bfloat16).view(torch.int16))
    check("gemv bf16 out", c16, a, b, bf16=True)


# gemv_bf16_split: K split over workgroups, fp32 partial sums merged in order.
# (N, K, splits): 256-column strips (N % 256 == 0) and 64-column ones, ranges
# of uneven length, splits with fewer row groups than waves, more splits than
# row groups (empty ranges), and the largest split count
GEMV_SPLIT_SHAPES = [(256, 1024, 4), (320, 200, 3), (1024, 4096, 7), (64, 8, 5), (9216, 2056, 7),
                     (2048, 3080, 64), (4096, 1000, 2), (36864, 1048, 3)]


@pytest.mark.parametrize("shape", GEMV_SPLIT_SHAPES, ids=[str(s) for s in GEMV_SPLIT_SHAPES])
def test_gemv_split_full_compare(ta, shape):
    N, K, S = shape
    print(f"gemv split N={N} K={K} splits={S}", flush=True)
    a, b = gen.random_gemm_problem(1, N, K, seed=N + K + S)
    c = torch.full((1, N), float("nan"), device="cuda")
    # every workspace byte 0xFF (a NaN): a partial sum left unwritten shows
    ws = torch.full((ta.gemv_split_workspace_bytes(N, S),), 255, dtype=torch.uint8, device="cuda")
    ta.gemv_bf16_split(dev(a), dev(b), num_splits=S, out=c, workspace=ws)
    torch.cuda.synchronize()
    check(f"gemv split {shape}", c, a, b)


@pytest.mark.parametrize("name", ["gemv_v7", "gemv_v5", "gemv_v0", "gemv_v6", "gemv_v1", "gemv_v2",
                                  "gemv_v4"])
def test_gemv_split_workload_sampled(ta, name):
    """The matrix-vector shapes the split count heuristic splits, at full
    size: every output finite, sampled columns against the oracle."""
    w = gen.GEMM_WORKLOADS[name]
    S = ta.gemv_split_heuristic(w.N, w.K)
    print(f"gemv split workload {name} {w.describe()} splits={S}", flush=True)
    assert S > 1
    a, b = gen.make_gemm_inputs(w, seed=0)
    c = torch.full((1, w.N), float("nan"), device="cuda")
    ta.gemv_bf16_split(dev(a), dev(b), num_splits=S, out=c)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(c).all())
    rng = np.random.default_rng(3)
    cols = sorted({0, 1, 255, 256, w.N - 256, w.N - 1} | {int(x) for x in rng.integers(0, w.N, size=40)})
    bs = np.ascontiguousarray(b[:, cols])
    ref, scale = oracle.gemm(a, bs)[0], oracle.gemm_abs(a, bs)[0]
    got = c[0, torch.tensor(cols)].cpu().numpy()
    worst = float((np.abs(got - ref) / (REL_ABS * scale)).max())
    print(f"{name} split: worst err/tol={worst:.3f}", flush=True)
    assert worst <= 1.0


def test_gemv_split_bf16_out_and_deterministic(ta):
    """bf16 C is the fp32 result rounded once; repeated calls agree bit for
    bit; one split is gemm_bf16's matrix-vector product, bit for bit."""
    a, b = gen.random_gemm_problem(1, 2048, 6000, seed=12)
    da, db = dev(a), dev(b)
    c32 = ta.gemv_bf16_split(da, db, num_splits=5)
    c32b = ta.gemv_bf16_split(da, db, num_splits=5)
    c16 = ta.gemv_bf16_split(da, db, num_splits=5, out_dtype=torch.bfloat16)
    c1 = ta.gemv_bf16_split(da, db, num_splits=1)
    ref1 = ta.gemm_bf16(da, db)
    torch.cuda.synchronize()
    assert torch.equal(c32.view(torch.int32), c32b.view(torch.int32))
    assert torch.equal(c16.view(torch.int16), c32.to(torch.bfloat16).view(torch.int16))
    assert torch.equal(c1.view(torch.int32), ref1.view(torch.int32))
    check("gemv split fp32", c32, a, b)
    check("gemv split bf16 out", c16, a, b, bf16=True)
