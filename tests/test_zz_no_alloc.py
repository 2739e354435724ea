"""attn_fwd_split_noalloc (partial results in the library's static per-GPU
scratch) against attn_fwd_split (partial results in a caller workspace),
through the C ABI: the two run the same kernels, so their outputs must agree
bit for bit; both are also held to the attention target's tolerances against
the fp64 oracle.  Two calls in a row, the second smaller (the scratch keeps
the first call's contents, which must not leak into the second)."""
import ctypes

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


def both(ta, shape, causal, splits, o_bf16, seed):
    B, Hq, Hkv, Sq, Sk, D = shape
    q, k, v = gen.random_problem(B, Hq, Hkv, Sq, Sk, D, seed=seed)
    scale = 1.0 / np.sqrt(D)
    dq, dk, dv = dev(q), dev(k), dev(v)
    odt = torch.bfloat16 if o_bf16 else torch.float32
    outs = []
    stream = torch.cuda.current_stream()
    n = ta.ta_split_workspace_bytes(B, Hq, Sq, D, splits)
    ws = torch.empty(max(n, 16), dtype=torch.uint8, device="cuda")
    for noalloc in (False, True):
        o = torch.full((B, Hq, Sq, D), float("nan"), dtype=odt, device="cuda")
        lse = torch.full((B, Hq, Sq), float("nan"), dtype=torch.float32, device="cuda")
        if noalloc:
            rc = ta.attn_fwd_split_noalloc_raw(dq.data_ptr(), dk.data_ptr(), dv.data_ptr(),
                                               o.data_ptr(), o_bf16, lse.data_ptr(), B, Hq, Hkv,
                                               Sq, Sk, D, causal, scale, splits, stream.cuda_stream)
        else:
            rc = ta.attn_fwd_split_raw(dq.data_ptr(), dk.data_ptr(), dv.data_ptr(), o.data_ptr(),
                                       o_bf16, lse.data_ptr(), B, Hq, Hkv, Sq, Sk, D, causal, scale,
                                       splits, ws.data_ptr(), ws.numel(), stream.cuda_stream)
        assert rc == 0, ta.STATUS.get(rc, rc)
        torch.cuda.synchronize()
        outs.append((o.float().cpu().numpy(), lse.cpu().numpy()))
    (o_ws, l_ws), (o_st, l_st) = outs
    assert np.isfinite(o_st).all() and np.isfinite(l_st).all()
    assert np.array_equal(o_st, o_ws) and np.array_equal(l_st, l_ws), "noalloc differs from split"
    ro, rl = oracle.attn_fwd(q, k, v, causal, scale)
    eo, el = float(np.abs(o_st - ro).max()), float(np.abs(l_st - rl).max())
    print(f"noalloc {shape} causal={causal} splits={splits} bf16={o_bf16}: "
          f"max|dO|={eo:.3e} max|dLSE|={el:.3e}", flush=True)
    assert eo <= O_TOL and el <= LSE_TOL


def test_noalloc_matches_split_two_calls(ta):
    # first call: 33.8 MB of partial results (4 splits of 32 heads x 512
    # rows x 129 floats); second call smaller, over the stale contents
    both(ta, (1, 32, 8, 512, 4096, 128), True, 4, 0, seed=1)
    both(ta, (2, 4, 2, 200, 1000, 64), False, 3, 1, seed=2)


def test_noalloc_one_split_and_too_large(ta):
    both(ta, (1, 2, 2, 128, 300, 64), True, 1, 0, seed=3)
    B, Hq, Sq, D = 1, 32, 4096, 128
    q = torch.zeros((B, Hq, Sq, D), dtype=torch.bfloat16, device="cuda")
    o = torch.zeros((B, Hq, Sq, D), dtype=torch.float32, device="cuda")
    lse = torch.zeros((B, Hq, Sq), dtype=torch.float32, device="cuda")
    rc = ta.attn_fwd_split_noalloc_raw(q.data_ptr(), q.data_ptr(), q.data_ptr(), o.data_ptr(), 0,
                                       lse.data_ptr(), B, Hq, Hq, Sq, Sq, D, 0, 0.1, 2,
                                       torch.cuda.current_stream().cuda_stream)
    assert ta.STATUS[rc] == "TA_ERR_SCRATCH"
