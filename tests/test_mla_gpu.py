"""GPU parity of mla_decode (one multi-head latent attention decode step)
through the C ABI against the fp64 MLA oracle, at the attention tolerance:
max |O - O_ref| <= 2e-2 and max |LSE - LSE_ref| <= 1e-3.  Outputs are
pre-filled with NaN so that an unwritten element fails."""
import numpy as np
import pytest

import oracle
from paper_2504_17577_amd import gen

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

O_TOL, LSE_TOL = 2e-2, 1e-3


@pytest.fixture(scope="module")
def ta():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2504_17577_amd import tileattn
    tileattn.lib()
    return tileattn


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()


def run(ta, q, q_pe, kv, k_pe, scale, splits):
    B, H, Dl = q.shape
    o = torch.full((B, H, Dl), float("nan"), dtype=torch.float32, device="cuda")
    lse = torch.full((B, H), float("nan"), dtype=torch.float32, device="cuda")
    t = [dev(x) for x in (q, q_pe, kv, k_pe)]
    ta.mla_decode(*t, scale=scale, num_splits=splits, out=o, lse=lse)
    torch.cuda.synchronize()
    return o, lse


def check(tag, o, lse, ro, rl):
    o, lse = o.cpu().numpy(), lse.cpu().numpy()
    assert np.isfinite(o).all() and np.isfinite(lse).all(), f"{tag}: unwritten or non-finite"
    eo, el = float(np.abs(o - ro).max()), float(np.abs(lse - rl).max())
    print(f"{tag}: max|dO|={eo:.3e} max|dLSE|={el:.3e}", flush=True)
    assert eo <= O_TOL and el <= LSE_TOL, tag


@pytest.mark.parametrize("splits", [1, 3, None])
def test_mla_tiny_full_compare(ta, splits):
    w = gen.MLA_WORKLOADS["mla_tiny_s200"]
    q, q_pe, kv, k_pe = gen.make_mla_inputs(w, seed=0)
    o, lse = run(ta, q, q_pe, kv, k_pe, w.scale, splits)
    ro, rl = oracle.mla_decode(q, q_pe, kv, k_pe, w.scale)
    check(f"mla_tiny_s200 splits={splits}", o, lse, ro, rl)


EDGE = [
    # (B, H, Hkv, Skv, splits)
    (1, 128, 1, 1, 1), (2, 128, 1, 31, 1), (1, 128, 1, 32, 1), (1, 128, 1, 33, 2),
    (3, 16, 1, 65, 1),       # 16 heads: one wave's worth, the other seven waves are padding
    (2, 100, 1, 300, 4),     # 100 heads: one head block, a wave partly and one wholly padding
    (2, 64, 2, 257, 3),      # two latent heads of 32 query heads each
    (1, 128, 1, 1000, 128),  # more splits than tiles
    (1, 256, 1, 96, 2),      # 256 heads: two head blocks
]


@pytest.mark.parametrize("shape", EDGE, ids=[str(s) for s in EDGE])
def test_mla_edge_shapes(ta, shape):
    B, H, Hkv, Skv, splits = shape
    print(f"mla edge {shape}", flush=True)
    q, q_pe, kv, k_pe = gen.random_mla_problem(B, H, Hkv, Skv, seed=7)
    scale = 576 ** -0.5
    o, lse = run(ta, q, q_pe, kv, k_pe, scale, splits)
    ro, rl = oracle.mla_decode(q, q_pe, kv, k_pe, scale)
    check(f"mla edge {shape}", o, lse, ro, rl)


@pytest.mark.parametrize("name", ["mla_b64_s8k", "mla_b128_s4k", "mla_gqa2_b8_s2k"])
def test_mla_workload_sampled(ta, name):
    """Full-size workload with the heuristic split count (the bench's launch
    configuration): sampled heads against the oracle, and every O row inside
    the hull of its latent cache rows (weights sum to 1 within 2^-8)."""
    w = gen.MLA_WORKLOADS[name]
    q, q_pe, kv, k_pe = gen.make_mla_inputs(w, seed=0)
    n = ta.mla_split_heuristic(w.B, w.H, w.Hkv, w.Skv)
    print(f"mla workload {name}: {n} splits", flush=True)
    o, lse = run(ta, q, q_pe, kv, k_pe, w.scale, n)
    assert bool(torch.isfinite(o).all()) and bool(torch.isfinite(lse).all())
    g = w.H // w.Hkv
    kvf = torch.from_numpy(gen.f32_from_bf16(kv)).cuda()          # [B,Skv,Hkv,Dl]
    vmin = kvf.amin(dim=1).repeat_interleave(g, 1)                # [B,H,Dl]
    vmax = kvf.amax(dim=1).repeat_interleave(g, 1)
    margin = 2.0 ** -7 * torch.maximum(vmin.abs(), vmax.abs())
    over = torch.maximum(o - (vmax + margin), (vmin - margin) - o).amax().item()
    assert over <= 0, f"{name}: O outside the widened hull by {over:.3g}"
    rng = np.random.default_rng(2)
    rows = sorted({(int(rng.integers(w.B)), int(rng.integers(w.H))) for _ in range(160)}
                  | {(0, 0), (w.B - 1, w.H - 1)})
    ro, rl = oracle.mla_rows(q, q_pe, kv, k_pe, w.scale, rows)
    idx = tuple(torch.tensor(c) for c in zip(*rows))
    eo = float(np.abs(o[idx].cpu().numpy() - ro).max())
    el = float(np.abs(lse[idx].cpu().numpy() - rl).max())
    print(f"  {len(rows)} heads: max|dO|={eo:.3e} max|dLSE|={el:.3e}", flush=True)
    assert eo <= O_TOL and el <= LSE_TOL


def test_mla_cache_beyond_32_bits(ta):
    """A latent cache of more than 2^31 elements (over 4 GiB), so that any
    32-bit element or byte offset into it would wrap: heads of the batch
    elements on either side of the 2^30- and 2^31-element boundaries, and of
    the last one, against the oracle (each batch element is its own B = 1
    problem there)."""
    B, H, Skv = 132, 128, 32768
    assert B * Skv * 512 > 2 ** 31
    q, q_pe = (gen.normal_bf16_blocks(s, seed=0, wid=111, tensor=t)
               for t, s in ((0, (B, H, 512)), (1, (B, H, 64))))
    kv = gen.normal_bf16_blocks((B, Skv, 1, 512), seed=0, wid=111, tensor=2)
    k_pe = gen.normal_bf16_blocks((B, Skv, 1, 64), seed=0, wid=111, tensor=3)
    scale = 576 ** -0.5
    n = ta.mla_split_heuristic(B, H, 1, Skv)
    print(f"mla cache beyond 32 bits: B={B} H={H} Skv={Skv}, {n} splits", flush=True)
    o, lse = run(ta, q, q_pe, kv, k_pe, scale, n)
    # batch element b starts at element b * Skv * 512 = b * 2^24
    for b in (0, 63, 64, 127, 128, B - 1):
        heads = [0, 1, 31, 32, 63, 64, 100, 127]
        ro, rl = oracle.mla_rows(q[b:b + 1], q_pe[b:b + 1], kv[b:b + 1], k_pe[b:b + 1], scale,
                                 [(0, h) for h in heads])
        eo = float(np.abs(o[b, heads].cpu().numpy() - ro).max())
        el = float(np.abs(lse[b, heads].cpu().numpy() - rl).max())
        print(f"  batch {b}: max|dO|={eo:.3e} max|dLSE|={el:.3e}", flush=True)
        assert eo <= O_TOL and el <= LSE_TOL, b


def test_mla_single_position(ta):
    """One cache position: O is that latent row.  The weight is exp2 of the
    fp32 residual of (score * c) - round(score * c), so it and the row sum are
    1 within a few ulp: O matches to 2^-20 relative."""
    q, q_pe, kv, k_pe = gen.random_mla_problem(2, 128, 1, 1, seed=8)
    o, lse = run(ta, q, q_pe, kv, k_pe, 576 ** -0.5, 1)
    want = np.broadcast_to(gen.f32_from_bf16(kv)[:, 0, 0, None, :], o.shape)
    err = np.abs(o.cpu().numpy() - want)
    assert (err <= 2.0 ** -20 * np.abs(want)).all(), "one position: O must be that latent row"
    _, rl = oracle.mla_decode(q, q_pe, kv, k_pe, 576 ** -0.5)
    assert float(np.abs(lse.cpu().numpy() - rl).max()) <= 1e-5


def test_mla_rotary_inert_without_q_pe_and_deterministic(ta):
    q, q_pe, kv, k_pe = gen.random_mla_problem(2, 128, 1, 500, seed=9)
    zero = np.zeros_like(q_pe)
    other = gen.random_mla_problem(2, 128, 1, 500, seed=10)[3]
    o1, l1 = run(ta, q, zero, kv, k_pe, 0.05, 3)
    o2, l2 = run(ta, q, zero, kv, other, 0.05, 3)
    o3, l3 = run(ta, q, zero, kv, k_pe, 0.05, 3)
    assert torch.equal(o1, o2) and torch.equal(l1, l2), "k_pe must not matter when q_pe = 0"
    assert torch.equal(o1, o3) and torch.equal(l1, l3), "two runs must agree bitwise"


def test_mla_rejects_bad_arguments(ta):
    q, q_pe, kv, k_pe = [dev(x) for x in gen.random_mla_problem(1, 128, 1, 64, seed=1)]
    with pytest.raises(ta.TileAttnError) as e:
        ta.mla_decode(q, q_pe, kv, k_pe, num_splits=2,
                      workspace=torch.empty(16, dtype=torch.uint8, device="cuda"))
    assert e.value.status == 8
    with pytest.raises(TypeError):
        ta.mla_decode(q.float(), q_pe, kv, k_pe)
    q2, qp2, kv2, kp2 = [dev(x) for x in gen.random_mla_problem(1, 4, 1, 64, seed=1, Dl=64, Dr=32)]
    with pytest.raises(ta.TileAttnError) as e:
        ta.mla_decode(q2, qp2, kv2, kp2)
    assert e.value.status == 3
