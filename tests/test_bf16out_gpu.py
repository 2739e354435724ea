"""GPU checks of attn_fwd_bf16out through the C ABI: its O is the fp32 O of
attn_fwd rounded to nearest even, bit for bit, with the same LSE; against the
fp64 oracle it stays within the stated tolerance (max |O - O_ref| <= 2e-2,
max |LSE - LSE_ref| <= 1e-3); and the aliasing check uses the bf16 size of O."""
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


CASES = [
    # (name, B, Hq, Hkv, Sq, Sk, D, causal)
    ("tiny_d64_s128",) + (1, 2, 2, 128, 128, 64, False),
    ("ragged_gqa_causal", 1, 8, 2, 200, 300, 128, True),
    ("ragged_d64", 2, 6, 3, 65, 63, 64, False),
    ("dense_d128_s2k",) + (8, 32, 32, 2048, 2048, 128, False),
    ("chunk_causal_d128_q1k_k8k",) + (1, 32, 8, 1024, 8192, 128, True),
    ("persistent_ragged_gqa_causal", 4, 20, 5, 1000, 1037, 64, True),
    ("persistent_gqa_causal_d128", 5, 24, 3, 777, 900, 128, True),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_bf16out_is_rounded_fp32(ta, case):
    name, B, Hq, Hkv, Sq, Sk, D, causal = case
    if name in gen.WORKLOADS:
        w = gen.WORKLOADS[name]
        q, k, v = gen.make_inputs(w, seed=0)
    else:
        q, k, v = gen.random_problem(B, Hq, Hkv, Sq, Sk, D, seed=5)
    print(f"bf16out {name}: B={B} Hq={Hq} Hkv={Hkv} Sq={Sq} Sk={Sk} D={D} causal={causal}",
          flush=True)
    scale = 1.0 / np.sqrt(D)
    dq, dk, dv = dev(q), dev(k), dev(v)
    o32 = torch.full((B, Hq, Sq, D), float("nan"), dtype=torch.float32, device="cuda")
    l32 = torch.full((B, Hq, Sq), float("nan"), dtype=torch.float32, device="cuda")
    o16 = torch.full((B, Hq, Sq, D), float("nan"), dtype=torch.bfloat16, device="cuda")
    l16 = torch.full((B, Hq, Sq), float("nan"), dtype=torch.float32, device="cuda")
    ta.attn_fwd(dq, dk, dv, causal=causal, scale=scale, out=o32, lse=l32)
    ta.attn_fwd_bf16out(dq, dk, dv, causal=causal, scale=scale, out=o16, lse=l16)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(o16.float()).all())
    assert torch.equal(o16.view(torch.int16), o32.to(torch.bfloat16).view(torch.int16)), name
    assert torch.equal(l16.view(torch.int32), l32.view(torch.int32)), name


def test_bf16out_against_oracle(ta):
    w = gen.WORKLOADS["causal_d64_s1k"]
    q, k, v = gen.make_inputs(w, seed=0)
    o, lse = ta.attn_fwd_bf16out(dev(q), dev(k), dev(v), causal=w.causal, scale=w.scale)
    torch.cuda.synchronize()
    ro, rl = oracle.attn_fwd(q, k, v, w.causal, w.scale)
    eo = float(np.abs(o.float().cpu().numpy() - ro).max())
    el = float(np.abs(lse.cpu().numpy() - rl).max())
    print(f"bf16out causal_d64_s1k: max|dO|={eo:.3e} max|dLSE|={el:.3e}", flush=True)
    assert eo <= O_TOL and el <= LSE_TOL


def test_bf16out_lse_right_after_o(ta):
    """O (bf16) and LSE carved back to back from one allocation: no false
    aliasing report, and LSE is not overwritten by O stores."""
    B, Hq, Hkv, Sq, Sk, D = 1, 4, 4, 96, 160, 128
    q, k, v = gen.random_problem(B, Hq, Hkv, Sq, Sk, D, seed=9)
    n_o = B * Hq * Sq * D            # bf16 elements = 2 * n_o bytes
    n_l = B * Hq * Sq
    buf = torch.full((n_o // 2 + n_l,), float("nan"), dtype=torch.float32, device="cuda")
    o = buf[: n_o // 2].view(torch.bfloat16).view(B, Hq, Sq, D)
    lse = buf[n_o // 2:].view(B, Hq, Sq)
    ta.attn_fwd_bf16out(dev(q), dev(k), dev(v), causal=True, scale=D ** -0.5, out=o, lse=lse)
    torch.cuda.synchronize()
    ro, rl = oracle.attn_fwd(q, k, v, True, D ** -0.5)
    assert float(np.abs(o.float().cpu().numpy() - ro).max()) <= O_TOL
    assert float(np.abs(lse.cpu().numpy() - rl).max()) <= LSE_TOL
