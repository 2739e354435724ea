"""GPU parity of the SSD chunk functions (ssd_chunk_state, ssd_state_passing,
ssd_bmm_chunk, ssd_chunk_scan) through the C ABI against the float64 oracle
(oracle/ssd.py), on the same seeded inputs.

Tolerances, from the arithmetic of the kernels:
  * chunk state / chunk scan: each product has one operand rounded to bf16
    (the weighted x, the weighted cb entry, the entering state), a relative
    error of at most 2^-8 per term; the decays come from an fp32 prefix sum
    and exp2 (relative error ~1e-4 on the terms that matter) and the sums are
    fp32.  So |out - ref| <= 2^-7 * (the same sums over |terms|), which the
    oracle computes (``chunk_state_abs`` / ``chunk_scan_abs``).  A single
    round-to-nearest-even has a relative error of root mean square ~1.5e-3
    (uniform over half an ulp); a sum of several rounded terms averages it
    down, and the decay often leaves one or two terms dominant, so the root
    mean square of err / |terms| over all outputs must stay below 2^-9
    (1.95e-3); a wrong decay index or a lost dt shifts it by far more.
  * chunk matrix: exact bf16 products, fp32 sums of 128 terms:
    1e-5 * sum_n |Cm_l[n]| |Bm_s[n]|.
  * state passing: fp32 multiply-adds over the chunks, 1e-5 of the same
    recurrence over |states|.
  * the four chained: each stage's bound carried through, 2^-6 of the chained
    |terms| sums.
"""
import numpy as np
import pytest

import oracle.ssd as ossd
from paper_2504_17577_amd import gen

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

Q = 256
BOUND = 2.0 ** -7
RMS = 2.0 ** -9


@pytest.fixture(scope="module")
def ta():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2504_17577_amd import tileattn
    tileattn.lib()
    return tileattn


def dev_bf16(x):
    return torch.from_numpy(np.ascontiguousarray(x).view(np.int16)).view(torch.bfloat16).cuda()


def dev_f32(x):
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).cuda()


def check(tag, got, ref, scale, bound=BOUND, rms=RMS):
    got = np.asarray(got, dtype=np.float64)
    assert np.isfinite(got).all(), f"{tag}: non-finite output"
    r = np.abs(got - ref) / np.maximum(scale, 1e-30)
    worst, mean_sq = float(r.max()), float(np.sqrt(np.mean(r ** 2)))
    print(f"{tag}: max|d|={np.abs(got - ref).max():.3e} worst err/scale={worst:.3e} "
          f"rms={mean_sq:.3e}", flush=True)
    assert worst <= bound, f"{tag}: worst err/scale {worst} > {bound}"
    if rms is not None:
        assert mean_sq <= rms, f"{tag}: rms err/scale {mean_sq} > {rms}"


SHAPES = [  # (B, L, H, G)
    (2, 300, 4, 2),      # ragged last chunk, two groups
    (1, 1, 2, 1),        # a single position
    (1, 37, 2, 2),       # one short chunk, one head per group
    (1, 512, 4, 1),      # exact multiple of the chunk
    (2, 1000, 8, 2),     # four chunks, ragged
]


def problem(shape, seed):
    B, L, H, G = shape
    w, inp = gen.random_ssd_problem(B, L, H, G, seed=seed)
    return w, inp


@pytest.mark.parametrize("shape", SHAPES, ids=[str(s) for s in SHAPES])
def test_chunk_state(ta, shape):
    print(f"ssd_chunk_state {shape}", flush=True)
    w, inp = problem(shape, seed=sum(shape))
    out = torch.full((w.B, w.nc, w.H, w.P, w.N), float("nan"), device="cuda")
    ta.ssd_chunk_state(dev_bf16(inp["x"]), dev_bf16(inp["Bm"]), dev_f32(inp["dt"]),
                       dev_f32(inp["A"]), out=out)
    torch.cuda.synchronize()
    ref = ossd.chunk_state(inp["x"], inp["Bm"], inp["dt"], inp["A"], Q)
    scale = ossd.chunk_state_abs(inp["x"], inp["Bm"], inp["dt"], inp["A"], Q)
    check(f"chunk_state {shape}", out.cpu().numpy(), ref, scale)


@pytest.mark.parametrize("shape", SHAPES, ids=[str(s) for s in SHAPES])
def test_chunk_scan(ta, shape):
    print(f"ssd_chunk_scan {shape}", flush=True)
    w, inp = problem(shape, seed=7 + sum(shape))
    cb, prev = gen.make_ssd_scan_extras(w, seed=3)
    out = torch.full((w.B, w.L, w.H, w.P), float("nan"), device="cuda")
    ta.ssd_chunk_scan(dev_bf16(inp["x"]), dev_bf16(inp["Cm"]), dev_f32(cb), dev_f32(inp["dt"]),
                      dev_f32(inp["A"]), dev_f32(prev), dev_f32(inp["D"]), out=out)
    torch.cuda.synchronize()
    args = (inp["x"], inp["Cm"], cb, inp["dt"], inp["A"], prev, inp["D"], Q)
    check(f"chunk_scan {shape}", out.cpu().numpy(), ossd.chunk_scan(*args), ossd.chunk_scan_abs(*args))


def test_chunk_scan_without_skip_term(ta):
    w, inp = problem((1, 300, 2, 1), seed=21)
    cb, prev = gen.make_ssd_scan_extras(w, seed=4)
    y = ta.ssd_chunk_scan(dev_bf16(inp["x"]), dev_bf16(inp["Cm"]), dev_f32(cb), dev_f32(inp["dt"]),
                          dev_f32(inp["A"]), dev_f32(prev), None)
    torch.cuda.synchronize()
    zero = np.zeros_like(inp["D"])
    args = (inp["x"], inp["Cm"], cb, inp["dt"], inp["A"], prev, zero, Q)
    check("chunk_scan D=None", y.cpu().numpy(), ossd.chunk_scan(*args), ossd.chunk_scan_abs(*args))


@pytest.mark.parametrize("shape", SHAPES, ids=[str(s) for s in SHAPES])
def test_bmm_chunk(ta, shape):
    print(f"ssd_bmm_chunk {shape}", flush=True)
    w, inp = problem(shape, seed=11 + sum(shape))
    out = torch.full((w.B, w.nc, w.G, Q, Q), float("nan"), device="cuda")
    ta.ssd_bmm_chunk(dev_bf16(inp["Cm"]), dev_bf16(inp["Bm"]), out=out)
    torch.cuda.synchronize()
    ref = ossd.bmm_chunk(inp["Cm"], inp["Bm"], Q)
    ab = lambda u: np.ascontiguousarray(u) & np.uint16(0x7FFF)
    scale = ossd.bmm_chunk(ab(inp["Cm"]), ab(inp["Bm"]), Q)
    got = out.cpu().numpy()
    # rows and columns of padded positions (past L) are written as exact zeros
    pos = np.arange(w.nc * Q).reshape(w.nc, Q) >= w.L
    pad = pos[None, :, None, :, None] | pos[None, :, None, None, :]
    pad = np.broadcast_to(pad, got.shape)
    assert (got[pad] == 0).all(), "padded rows/columns of cb must be zero"
    check(f"bmm_chunk {shape}", got, ref, np.maximum(scale, 1e-30), bound=1e-5, rms=None)


@pytest.mark.parametrize("shape", SHAPES, ids=[str(s) for s in SHAPES])
def test_state_passing(ta, shape):
    print(f"ssd_state_passing {shape}", flush=True)
    w, inp = problem(shape, seed=13 + sum(shape))
    _, states = gen.make_ssd_scan_extras(w, seed=5)
    prev, final = ta.ssd_state_passing(dev_f32(states), dev_f32(inp["dt"]), dev_f32(inp["A"]))
    torch.cuda.synchronize()
    rp, rf = ossd.state_passing(states, inp["dt"], inp["A"], Q)
    sp, sf = ossd.state_passing(np.abs(states), inp["dt"], inp["A"], Q)
    check(f"state_passing prev {shape}", prev.cpu().numpy(), rp, np.maximum(sp, 1e-30), bound=1e-5,
          rms=None)
    check(f"state_passing final {shape}", final.cpu().numpy(), rf, sf, bound=1e-5, rms=None)


def chained_scale(inp):
    """The chained sums with every term replaced by its magnitude."""
    ab = lambda u: np.ascontiguousarray(u) & np.uint16(0x7FFF)
    s_abs = ossd.chunk_state_abs(inp["x"], inp["Bm"], inp["dt"], inp["A"], Q)
    p_abs, _ = ossd.state_passing(s_abs, inp["dt"], inp["A"], Q)
    cb_abs = ossd.bmm_chunk(ab(inp["Cm"]), ab(inp["Bm"]), Q)
    return ossd.chunk_scan_abs(inp["x"], inp["Cm"], cb_abs, inp["dt"], inp["A"], p_abs, inp["D"], Q)


@pytest.mark.parametrize("shape", [(2, 300, 4, 2), (2, 1000, 8, 2), (1, 2048, 4, 1)],
                         ids=["s300", "s1000", "s2048"])
def test_chained_forward_matches_oracle(ta, shape):
    """The four kernels chained on the GPU reproduce the oracle's chained
    result (pinned to the step-by-step recurrence)."""
    print(f"ssd chained {shape}", flush=True)
    w, inp = problem(shape, seed=17 + sum(shape))
    y, final = ta.ssd_forward(dev_bf16(inp["x"]), dev_f32(inp["dt"]), dev_f32(inp["A"]),
                              dev_bf16(inp["Bm"]), dev_bf16(inp["Cm"]), dev_f32(inp["D"]))
    torch.cuda.synchronize()
    ry, rf = ossd.ssd_forward(inp["x"], inp["dt"], inp["A"], inp["Bm"], inp["Cm"], inp["D"], Q)
    check(f"chained y {shape}", y.cpu().numpy(), ry, chained_scale(inp), bound=2.0 ** -6,
          rms=2.0 ** -8)


def test_workload_b1_s8k_sampled(ta):
    """The paper's longest single-sequence shape (B=1, L=8192, 64 heads):
    chunk state and chunk scan on every chunk and head, checked on a sample of
    heads against the oracle run on those heads alone."""
    w = gen.SSD_WORKLOADS["ssd_b1_s8k"]
    print(f"ssd {w.name}", flush=True)
    inp = gen.make_ssd_inputs(w, seed=0)
    cb, prev = gen.make_ssd_scan_extras(w, seed=0)
    dx, dB, dC = dev_bf16(inp["x"]), dev_bf16(inp["Bm"]), dev_bf16(inp["Cm"])
    ddt, dA, dD = dev_f32(inp["dt"]), dev_f32(inp["A"]), dev_f32(inp["D"])
    st = ta.ssd_chunk_state(dx, dB, ddt, dA)
    y = ta.ssd_chunk_scan(dx, dC, dev_f32(cb), ddt, dA, dev_f32(prev), dD)
    torch.cuda.synchronize()
    heads = [0, 17, 63]
    sub = dict(x=inp["x"][:, :, heads], Bm=inp["Bm"], Cm=inp["Cm"], dt=inp["dt"][:, :, heads],
               A=inp["A"][heads], D=inp["D"][heads])
    ref_s = ossd.chunk_state(sub["x"], sub["Bm"], sub["dt"], sub["A"], Q)
    sc_s = ossd.chunk_state_abs(sub["x"], sub["Bm"], sub["dt"], sub["A"], Q)
    check("b1_s8k chunk_state", st[:, :, heads].cpu().numpy(), ref_s, sc_s)
    args = (sub["x"], sub["Cm"], cb, sub["dt"], sub["A"], prev[:, :, heads], sub["D"], Q)
    check("b1_s8k chunk_scan", y[:, :, heads].cpu().numpy(), ossd.chunk_scan(*args),
          ossd.chunk_scan_abs(*args))


def test_chunk_state_two_heads_per_workgroup(ta):
    """Grids of at least 1024 two-head workgroups run two heads of a group
    per workgroup: both heads of several pairs, both groups, a ragged last
    chunk, against the oracle on those heads alone."""
    shape = (2, 4000, 64, 2)
    print(f"ssd_chunk_state {shape} (two heads per workgroup)", flush=True)
    w, inp = problem(shape, seed=21)
    out = torch.full((w.B, w.nc, w.H, w.P, w.N), float("nan"), device="cuda")
    ta.ssd_chunk_state(dev_bf16(inp["x"]), dev_bf16(inp["Bm"]), dev_f32(inp["dt"]),
                       dev_f32(inp["A"]), out=out)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(out).all())
    heads = [0, 1, 30, 31, 32, 33, 62, 63]
    groups = [h // (w.H // w.G) for h in heads]
    sub_x, sub_dt, sub_A = inp["x"][:, :, heads], inp["dt"][:, :, heads], inp["A"][heads]
    for i, (h, g) in enumerate(zip(heads, groups)):
        bm = inp["Bm"][:, :, [g]]
        ref = ossd.chunk_state(sub_x[:, :, [i]], bm, sub_dt[:, :, [i]], sub_A[[i]], Q)
        scale = ossd.chunk_state_abs(sub_x[:, :, [i]], bm, sub_dt[:, :, [i]], sub_A[[i]], Q)
        check(f"chunk_state {shape} head {h}", out[:, :, [h]].cpu().numpy(), ref, scale)


def test_repeatable_and_stream(ta):
    """Two runs are bitwise identical; a non-default stream gives the same."""
    w, inp = problem((1, 600, 4, 2), seed=31)
    cb, prev = gen.make_ssd_scan_extras(w, seed=6)
    a = [dev_bf16(inp["x"]), dev_bf16(inp["Cm"]), dev_f32(cb), dev_f32(inp["dt"]),
         dev_f32(inp["A"]), dev_f32(prev), dev_f32(inp["D"])]
    y1 = ta.ssd_chunk_scan(*a)
    y2 = ta.ssd_chunk_scan(*a)
    s = torch.cuda.Stream()
    torch.cuda.synchronize()
    with torch.cuda.stream(s):
        y3 = ta.ssd_chunk_scan(*a, stream=s)
    s.synchronize()
    assert torch.equal(y1, y2) and torch.equal(y1, y3)
