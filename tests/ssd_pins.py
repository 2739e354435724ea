"""Pins of the SSD chunk oracle (oracle/ssd.py) against formulations that share
none of its code: the state-space recurrence stepped one position at a time,
the materialised quadratic ("attention") form of the same model, the no-decay
special case as causal linear attention built from running sums, and closed
forms of single steps.  Each ``pin_*`` takes the oracle module (so the
mutation test can hand in a broken copy) and raises AssertionError on a
mismatch.

The model (Mamba-2, "Transformers are SSMs", Section 3): for each batch
element and head h (group g = h // (H/G)),
    h_t = exp(dt_t A_h) h_{t-1} + dt_t x_t Bm_t^T   (P x N),   h_{-1} = 0
    y_t = h_t Cm_t + D_h x_t
"""
from __future__ import annotations

import math

import numpy as np

from paper_2504_17577_amd import gen

REL = 1e-10


def widen(bits):
    return gen.f32_from_bf16(bits).astype(np.float64)


def recurrence(inp):
    """The SSM stepped one position at a time: (y [B,L,H,P], final h [B,H,P,N])."""
    X, Bw, Cw = widen(inp["x"]), widen(inp["Bm"]), widen(inp["Cm"])
    dt, A, D = (np.asarray(inp[k], dtype=np.float64) for k in ("dt", "A", "D"))
    Bsz, L, H, P = X.shape
    G, N = Bw.shape[2], Bw.shape[3]
    y = np.zeros((Bsz, L, H, P))
    hs = np.zeros((Bsz, H, P, N))
    for t in range(L):
        for h in range(H):
            g = h // (H // G)
            decay = np.exp(dt[:, t, h] * A[h])                              # [B]
            hs[:, h] = decay[:, None, None] * hs[:, h] + \
                dt[:, t, h][:, None, None] * X[:, t, h, :, None] * Bw[:, t, g, None, :]
            y[:, t, h] = np.einsum("bpn,bn->bp", hs[:, h], Cw[:, t, g]) + D[h] * X[:, t, h]
    return y, hs


def quadratic_form(inp):
    """y = (Lmask o (Cm Bm^T)) (dt x) + D x with Lmask[t, s] = prod_{s<r<=t}
    exp(dt_r A) for s <= t: the whole sequence as one masked matrix."""
    X, Bw, Cw = widen(inp["x"]), widen(inp["Bm"]), widen(inp["Cm"])
    dt, A, D = (np.asarray(inp[k], dtype=np.float64) for k in ("dt", "A", "D"))
    Bsz, L, H, P = X.shape
    G = Bw.shape[2]
    y = np.zeros((Bsz, L, H, P))
    for b in range(Bsz):
        for h in range(H):
            g = h // (H // G)
            e = np.exp(dt[b, :, h] * A[h])                                 # per-step decay
            Lm = np.zeros((L, L))
            for t in range(L):
                prod = 1.0
                for s in range(t, -1, -1):
                    Lm[t, s] = prod
                    prod *= e[s]
            M = Lm * (Cw[b, :, g] @ Bw[b, :, g].T)
            y[b, :, h] = M @ (dt[b, :, h, None] * X[b, :, h]) + D[h] * X[b, :, h]
    return y


def _scale(ref):
    return max(1.0, float(np.abs(ref).max()))


def _check(tag, got, ref, rel=REL):
    err = float(np.abs(np.asarray(got) - np.asarray(ref)).max())
    tol = rel * _scale(ref)
    assert err <= tol, f"{tag}: max err {err:.3e} > {tol:.3e}"
    return err


def pin_recurrence(ssd, B=2, L=300, H=4, G=2, Q=64, seed=1):
    """steps 1-4 chained == the recurrence (ragged last chunk when Q does not divide L)"""
    _, inp = gen.random_ssd_problem(B, L, H, G, seed=seed, P=8, N=16, Q=Q)
    y, final = ssd.ssd_forward(inp["x"], inp["dt"], inp["A"], inp["Bm"], inp["Cm"], inp["D"], Q)
    yr, hr = recurrence(inp)
    _check(f"y vs recurrence (Q={Q})", y, yr)
    _check(f"final state vs recurrence (Q={Q})", final, hr)


def pin_quadratic(ssd, L=70, Q=32, seed=2):
    """steps 1-4 chained == the materialised quadratic form"""
    _, inp = gen.random_ssd_problem(1, L, 2, 1, seed=seed, P=4, N=8, Q=Q)
    y, _ = ssd.ssd_forward(inp["x"], inp["dt"], inp["A"], inp["Bm"], inp["Cm"], inp["D"], Q)
    _check("y vs quadratic form", y, quadratic_form(inp))


def pin_chunk_state_from_zero(ssd, seed=3):
    """step 1 alone: S_c is the state the recurrence reaches over chunk c's
    positions when it starts from zero"""
    Q, L = 16, 40
    _, inp = gen.random_ssd_problem(2, L, 2, 1, seed=seed, P=4, N=8, Q=Q)
    S = ssd.chunk_state(inp["x"], inp["Bm"], inp["dt"], inp["A"], Q)
    for c in range(-(-L // Q)):
        lo, hi = c * Q, min(L, c * Q + Q)
        part = {k: (v[:, lo:hi] if k in ("x", "Bm", "Cm", "dt") else v) for k, v in inp.items()}
        _, h = recurrence(part)
        _check(f"chunk {c} state", S[:, c], h)


def pin_no_decay_linear_attention(ssd, seed=4):
    """A = 0: no decay, so y_t = sum_{s<=t} (Cm_t . Bm_s) dt_s x_s + D x_t,
    causal linear attention, built here from a running sum of outer products"""
    Q, L = 16, 50
    _, inp = gen.random_ssd_problem(1, L, 2, 2, seed=seed, P=4, N=8, Q=Q)
    inp["A"] = np.zeros_like(inp["A"])
    y, _ = ssd.ssd_forward(inp["x"], inp["dt"], inp["A"], inp["Bm"], inp["Cm"], inp["D"], Q)
    X, Bw, Cw = widen(inp["x"]), widen(inp["Bm"]), widen(inp["Cm"])
    dt, D = inp["dt"].astype(np.float64), inp["D"].astype(np.float64)
    kv = np.cumsum(dt[0, :, :, None, None] * X[0, :, :, :, None] * Bw[0, :, :, None, :], axis=0)
    ref = np.einsum("thpn,thn->thp", kv, Cw[0]) + D[None, :, None] * X[0]
    _check("no-decay linear attention", y[0], ref)


def pin_bmm_brute_force(ssd, seed=5):
    """step 3: every entry as a math.fsum dot product"""
    Q, L = 8, 19
    _, inp = gen.random_ssd_problem(1, L, 2, 2, seed=seed, P=4, N=8, Q=Q)
    cb = ssd.bmm_chunk(inp["Cm"], inp["Bm"], Q)
    Cw, Bw = widen(inp["Cm"]), widen(inp["Bm"])
    for c in range(cb.shape[1]):
        for g in range(2):
            for l in range(Q):
                for s in range(Q):
                    t, u = c * Q + l, c * Q + s
                    ref = 0.0 if t >= L or u >= L else \
                        math.fsum(Cw[0, t, g, n] * Bw[0, u, g, n] for n in range(8))
                    assert abs(cb[0, c, g, l, s] - ref) <= 1e-12 * max(1.0, abs(ref)), (c, g, l, s)


def pin_scan_entering_state_only(ssd, seed=6):
    """step 4 with cb = 0 and D = 0 leaves the entering state decayed by the
    running product of per-step decays (a product here, a sum of logs in the
    oracle): y_l = (prod_{r<=l} exp(dt_r A)) H Cm_l"""
    Q, L = 16, 40
    w, inp = gen.random_ssd_problem(1, L, 2, 1, seed=seed, P=4, N=8, Q=Q)
    nc = w.nc
    rng = np.random.default_rng(seed)
    Hin = rng.standard_normal((1, nc, 2, 4, 8))
    cb = np.zeros((1, nc, 1, Q, Q))
    y = ssd.chunk_scan(inp["x"], inp["Cm"], cb, inp["dt"], inp["A"], Hin, np.zeros(2), Q)
    Cw = widen(inp["Cm"])
    dt, A = inp["dt"].astype(np.float64), inp["A"].astype(np.float64)
    for c in range(nc):
        for h in range(2):
            prod = 1.0
            for l in range(Q):
                t = c * Q + l
                if t >= L:
                    break
                prod *= math.exp(dt[0, t, h] * A[h])
                ref = prod * (Hin[0, c, h] @ Cw[0, t, 0])
                assert np.abs(y[0, t, h] - ref).max() <= 1e-12 * max(1.0, np.abs(ref).max()), (c, h, l)


def pin_scan_linear_in_inputs(ssd, seed=7):
    """step 4 is linear in (cb, entering states, D) jointly with x fixed:
    scan(cb1 + cb2, H1 + H2, D1 + D2) = scan(cb1, H1, D1) + scan(cb2, H2, D2)"""
    Q, L = 16, 36
    w, inp = gen.random_ssd_problem(1, L, 2, 1, seed=seed, P=4, N=8, Q=Q)
    rng = np.random.default_rng(seed)
    nc = w.nc
    cb1, cb2 = rng.standard_normal((2, 1, nc, 1, Q, Q))
    H1, H2 = rng.standard_normal((2, 1, nc, 2, 4, 8))
    D1, D2 = rng.standard_normal((2, 2))
    f = lambda cb, Hs, D: ssd.chunk_scan(inp["x"], inp["Cm"], cb, inp["dt"], inp["A"], Hs, D, Q)
    _check("scan linearity", f(cb1 + cb2, H1 + H2, D1 + D2), f(cb1, H1, D1) + f(cb2, H2, D2))


def pin_chunk_size_invariance(ssd, seed=8):
    """the chained result does not depend on the chunk size (Q = 1 is the
    recurrence itself, Q >= L the quadratic form)"""
    _, inp = gen.random_ssd_problem(1, 45, 2, 1, seed=seed, P=4, N=8, Q=8)
    ys = [ssd.ssd_forward(inp["x"], inp["dt"], inp["A"], inp["Bm"], inp["Cm"], inp["D"], Q)[0]
          for Q in (1, 7, 16, 64)]
    for y in ys[1:]:
        _check("chunk-size invariance", y, ys[0])


def _flip_signs(rng, bits):
    """bf16 bit array with the sign of a random half of its entries flipped"""
    m = rng.random(bits.shape) < 0.5
    return np.where(m, bits ^ np.uint16(0x8000), bits).astype(np.uint16)


def _nonneg_bits(bits):
    return (np.ascontiguousarray(bits) & np.uint16(0x7FFF)).astype(np.uint16)


def pin_scan_abs_scale(ssd, seed=9):
    """chunk_scan_abs, the scale every chunk-scan tolerance is stated against,
    is the chunk scan with every term replaced by its magnitude.  Three facts
    fix it without restating it: (1) on non-negative x, Cm, cb, entering
    states and D every term already is its magnitude, so it equals the chunk
    scan itself (the decays exp(a) are positive for any sign of A, so a
    flipped A is caught here); (2) it bounds |chunk scan| element by element
    (triangle inequality); (3) it is unchanged when the sign of any input
    entry flips (a dropped magnitude on any operand is caught here)."""
    Q, L = 16, 40
    w, inp = gen.random_ssd_problem(1, L, 4, 2, seed=seed, P=4, N=8, Q=Q)
    rng = np.random.default_rng(seed)
    nc = w.nc
    x, Cm = inp["x"], inp["Cm"]
    cb = rng.standard_normal((1, nc, 2, Q, Q))
    Hs = rng.standard_normal((1, nc, 4, 4, 8))
    D = rng.standard_normal(4)
    dt, A = inp["dt"], inp["A"]
    assert (np.asarray(A) < 0).all(), "the pin needs decaying heads"
    # (1) non-negative operands
    xp, Cp = _nonneg_bits(x), _nonneg_bits(Cm)
    _check("scan_abs == scan on non-negative operands",
           ssd.chunk_scan_abs(xp, Cp, np.abs(cb), dt, A, np.abs(Hs), np.abs(D), Q),
           ssd.chunk_scan(xp, Cp, np.abs(cb), dt, A, np.abs(Hs), np.abs(D), Q))
    # (2) triangle inequality on signed operands
    y = ssd.chunk_scan(x, Cm, cb, dt, A, Hs, D, Q)
    ya = ssd.chunk_scan_abs(x, Cm, cb, dt, A, Hs, D, Q)
    slack = 1e-12 * max(1.0, float(np.abs(ya).max()))
    assert (np.abs(y) <= ya + slack).all(), "|chunk_scan| exceeds chunk_scan_abs"
    # (3) sign flips of every operand leave it unchanged
    flip = lambda a: np.where(rng.random(np.shape(a)) < 0.5, -a, a)
    yf = ssd.chunk_scan_abs(_flip_signs(rng, x), _flip_signs(rng, Cm), flip(cb), dt, A,
                            flip(Hs), flip(D), Q)
    _check("scan_abs under sign flips", yf, ya)


def pin_state_abs_scale(ssd, seed=10):
    """chunk_state_abs, the scale of the chunk-state tolerances: equal to the
    chunk state on non-negative x and Bm, at least |chunk state| on signed
    ones, and unchanged by sign flips of x and Bm entries"""
    Q, L = 16, 40
    _, inp = gen.random_ssd_problem(2, L, 4, 2, seed=seed, P=4, N=8, Q=Q)
    rng = np.random.default_rng(seed)
    x, Bm, dt, A = inp["x"], inp["Bm"], inp["dt"], inp["A"]
    xp, Bp = _nonneg_bits(x), _nonneg_bits(Bm)
    _check("state_abs == state on non-negative operands",
           ssd.chunk_state_abs(xp, Bp, dt, A, Q), ssd.chunk_state(xp, Bp, dt, A, Q))
    s = ssd.chunk_state(x, Bm, dt, A, Q)
    sa = ssd.chunk_state_abs(x, Bm, dt, A, Q)
    slack = 1e-12 * max(1.0, float(np.abs(sa).max()))
    assert (np.abs(s) <= sa + slack).all(), "|chunk_state| exceeds chunk_state_abs"
    _check("state_abs under sign flips",
           ssd.chunk_state_abs(_flip_signs(rng, x), _flip_signs(rng, Bm), dt, A, Q), sa)


ALL_PINS = [pin_recurrence, pin_quadratic, pin_chunk_state_from_zero,
            pin_no_decay_linear_attention, pin_bmm_brute_force, pin_scan_entering_state_only,
            pin_scan_linear_in_inputs, pin_chunk_size_invariance,
            pin_scan_abs_scale, pin_state_abs_scale]
