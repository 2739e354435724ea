"""Pins for the MLA decode oracle (``oracle.mla_decode`` / ``oracle.mla_rows``),
which reduces MLA to the attention oracle (key = [kv | k_pe], value = kv, one
query row per head).  Each ``pin_*`` checks it against something other than
that reduction:

  * a direct float64 numpy evaluation of the MLA formula, written per head
    with the latent and rotary dot products kept separate (brute force on
    small shapes, one and two latent heads);
  * closed forms: a single cache position (O = kv[0], LSE = its score), zero
    scale (O = mean of the latent rows, LSE = ln Skv);
  * invariants: permuting cache positions (kv and k_pe together) changes
    nothing; with q_pe = 0 the result does not depend on k_pe; query heads
    of one latent head are unaffected by the other latent head's cache;
  * the selected-rows entry equals the full one.
"""
from __future__ import annotations

import numpy as np

import oracle
from paper_2504_17577_amd import gen


def _f64(bits):
    return gen.f32_from_bf16(bits).astype(np.float64)


def _direct(q, q_pe, kv, k_pe, scale):
    """The MLA formula in float64, head by head."""
    B, H, Dl = q.shape
    Skv, Hkv = kv.shape[1], kv.shape[2]
    g = H // Hkv
    qf, qp, kvf, kp = _f64(q), _f64(q_pe), _f64(kv), _f64(k_pe)
    o = np.empty((B, H, Dl))
    lse = np.empty((B, H))
    for b in range(B):
        for h in range(H):
            hk = h // g
            s = scale * (kvf[b, :, hk, :] @ qf[b, h] + kp[b, :, hk, :] @ qp[b, h])
            m = s.max()
            e = np.exp(s - m)
            o[b, h] = (e @ kvf[b, :, hk, :]) / e.sum()
            lse[b, h] = m + np.log(e.sum())
    return o, lse


def _close(a, b, tol, what):
    err = float(np.max(np.abs(np.asarray(a) - np.asarray(b))))
    assert err <= tol, f"{what}: max abs diff {err:.3e} > {tol:.1e}"


SHAPES = [  # (B, H, Hkv, Skv, Dl, Dr)
    (2, 4, 1, 7, 16, 8), (1, 6, 2, 33, 16, 8), (2, 8, 1, 1, 32, 16), (1, 4, 2, 65, 512, 64),
]


def pin_direct_formula(lib):
    for i, (B, H, Hkv, Skv, Dl, Dr) in enumerate(SHAPES):
        q, q_pe, kv, k_pe = gen.random_mla_problem(B, H, Hkv, Skv, seed=40 + i, Dl=Dl, Dr=Dr)
        scale = 1.0 / np.sqrt(Dl + Dr)
        o, lse = oracle.mla_decode(q, q_pe, kv, k_pe, scale, lib=lib)
        ro, rl = _direct(q, q_pe, kv, k_pe, scale)
        _close(o, ro, 1e-12, f"O vs direct formula {SHAPES[i]}")
        _close(lse, rl, 1e-12, f"LSE vs direct formula {SHAPES[i]}")


def pin_single_position(lib):
    q, q_pe, kv, k_pe = gen.random_mla_problem(2, 4, 2, 1, seed=50, Dl=32, Dr=16)
    o, lse = oracle.mla_decode(q, q_pe, kv, k_pe, 0.3, lib=lib)
    for b in range(2):
        for h in range(4):
            hk = h // 2
            assert np.array_equal(o[b, h], _f64(kv[b, 0, hk])), "O must equal kv[0]"
            s = 0.3 * (float(np.dot(_f64(q[b, h]), _f64(kv[b, 0, hk])))
                       + float(np.dot(_f64(q_pe[b, h]), _f64(k_pe[b, 0, hk]))))
            _close(lse[b, h], s, 1e-12 * max(1.0, abs(s)), "LSE of one position")


def pin_zero_scale(lib):
    q, q_pe, kv, k_pe = gen.random_mla_problem(1, 4, 1, 37, seed=51, Dl=32, Dr=16)
    o, lse = oracle.mla_decode(q, q_pe, kv, k_pe, 0.0, lib=lib)
    _close(o, np.broadcast_to(_f64(kv)[0, :, 0, :].mean(axis=0), o.shape), 1e-12, "mean of kv")
    _close(lse, np.full(lse.shape, np.log(37.0)), 1e-12, "ln Skv")


def pin_position_permutation(lib):
    q, q_pe, kv, k_pe = gen.random_mla_problem(2, 4, 1, 50, seed=52, Dl=32, Dr=16)
    perm = np.random.default_rng(0).permutation(50)
    o1, l1 = oracle.mla_decode(q, q_pe, kv, k_pe, 0.2, lib=lib)
    o2, l2 = oracle.mla_decode(q, q_pe, kv[:, perm], k_pe[:, perm], 0.2, lib=lib)
    _close(o1, o2, 1e-12, "permuted O")
    _close(l1, l2, 1e-12, "permuted LSE")


def pin_rotary_part_inert_without_q_pe(lib):
    q, q_pe, kv, k_pe = gen.random_mla_problem(1, 4, 1, 40, seed=53, Dl=32, Dr=16)
    zero = np.zeros_like(q_pe)
    other = gen.random_mla_problem(1, 4, 1, 40, seed=54, Dl=32, Dr=16)[3]
    o1, l1 = oracle.mla_decode(q, zero, kv, k_pe, 0.25, lib=lib)
    o2, l2 = oracle.mla_decode(q, zero, kv, other, 0.25, lib=lib)
    assert np.array_equal(o1, o2) and np.array_equal(l1, l2), "k_pe must not matter when q_pe = 0"
    o3, _ = oracle.mla_decode(q, q_pe, kv, k_pe, 0.25, lib=lib)
    assert not np.allclose(o1, o3), "q_pe must matter otherwise"


def pin_latent_head_map(lib):
    q, q_pe, kv, k_pe = gen.random_mla_problem(1, 6, 2, 30, seed=55, Dl=32, Dr=16)
    kv2, kp2 = kv.copy(), k_pe.copy()
    kv2[:, :, 1], kp2[:, :, 1] = kv[:, ::-1, 0], k_pe[:, ::-1, 0]   # change latent head 1 only
    o1, _ = oracle.mla_decode(q, q_pe, kv, k_pe, 0.2, lib=lib)
    o2, _ = oracle.mla_decode(q, q_pe, kv2, kp2, 0.2, lib=lib)
    assert np.array_equal(o1[:, :3], o2[:, :3]), "heads 0..2 read latent head 0"
    assert not np.allclose(o1[:, 3:], o2[:, 3:]), "heads 3..5 read latent head 1"


def pin_rows_entry(lib):
    q, q_pe, kv, k_pe = gen.random_mla_problem(2, 8, 2, 45, seed=56, Dl=32, Dr=16)
    o, lse = oracle.mla_decode(q, q_pe, kv, k_pe, 0.2, lib=lib)
    rows = [(1, 7), (0, 0), (1, 2), (0, 5)]
    ro, rl = oracle.mla_rows(q, q_pe, kv, k_pe, 0.2, rows, lib=lib)
    for n, (b, h) in enumerate(rows):
        assert np.array_equal(ro[n], o[b, h]) and rl[n] == lse[b, h], "rows entry"


PINS = {name[4:]: fn for name, fn in sorted(globals().items()) if name.startswith("pin_")}
