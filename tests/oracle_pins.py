"""Pins for the fp64 attention oracle: checks against what the mathematics and
libraries other than the oracle fix, never against the oracle's own formula.

Each ``pin_*`` takes a loaded oracle library handle and raises AssertionError
when the oracle behind it is wrong.  ``tests/test_oracle_pins.py`` runs them
on the real oracle; ``tests/test_oracle_mutants.py`` plants plausible
mistakes in the oracle's C source and checks that some pin catches each one.

What pins what:
  * torch's CPU flash-attention kernel in float64 (an independent library
    implementation of softmax(scale*QK^T)V that also returns the natural-log
    LSE) on non-causal, square-causal and grouped-query problems;
  * closed forms: constant V, zero scale (uniform weights), causal row 0,
    a single key, two keys (numpy.logaddexp), the hand-worked cases in
    tests/golden/closed_forms.txt;
  * invariants: key/value permutation, grouped-query == repeated heads,
    causal == non-causal over the visible prefix (bottom-right alignment),
    shifting every key by u shifts LSE by scale*q.u and leaves O alone,
    numerical stability at huge scores;
  * one-hot V: O rows are the attention probabilities, which are >= 0, sum
    to one, vanish on masked keys and equal exp(s_ij - LSE_i) with s from a
    numpy matmul.
"""
from __future__ import annotations

import math
import os

import numpy as np
import torch

import oracle
from paper_2504_17577_amd import gen

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _f64(bits):
    return gen.f32_from_bf16(bits).astype(np.float64)


def _bits(x):
    b = gen.bf16_from_f32(np.asarray(x, dtype=np.float32))
    assert np.array_equal(_f64(b), np.asarray(x, dtype=np.float64)), "value not exact in bf16"
    return b


def _close(a, b, tol, what):
    err = float(np.max(np.abs(np.asarray(a) - np.asarray(b)))) if np.size(a) else 0.0
    assert err <= tol and np.all(np.isfinite(a)), f"{what}: max err {err:.3g} > {tol:.3g}"


def _torch_ref(q, k, v, causal, scale):
    """torch CPU flash attention in float64: (O, LSE)."""
    g = q.shape[1] // k.shape[1]
    tq = torch.from_numpy(_f64(q))
    tk = torch.from_numpy(_f64(k)).repeat_interleave(g, 1)
    tv = torch.from_numpy(_f64(v)).repeat_interleave(g, 1)
    o, lse = torch.ops.aten._scaled_dot_product_flash_attention_for_cpu(
        tq, tk, tv, 0.0, bool(causal), scale=float(scale))[:2]
    return o.numpy(), lse.numpy()


def pin_torch_noncausal(lib):
    for (B, Hq, Hkv, Sq, Sk, D), seed in (((2, 2, 2, 19, 23, 64), 1), ((1, 4, 4, 33, 9, 128), 2),
                                          ((1, 2, 2, 5, 64, 16), 3)):
        q, k, v = gen.random_problem(B, Hq, Hkv, Sq, Sk, D, seed=seed)
        scale = 1.0 / math.sqrt(D)
        o, lse = oracle.attn_fwd(q, k, v, False, scale, lib=lib)
        ro, rl = _torch_ref(q, k, v, False, scale)
        _close(o, ro, 1e-12, "O vs torch")
        _close(lse, rl, 1e-12, "LSE vs torch")


def pin_torch_causal_square(lib):
    # torch aligns its causal mask top-left; for Sq == Sk that is the same mask
    for (B, Hq, Hkv, S, D), seed in (((2, 2, 2, 31, 64), 4), ((1, 3, 3, 17, 32), 5)):
        q, k, v = gen.random_problem(B, Hq, Hkv, S, S, D, seed=seed)
        o, lse = oracle.attn_fwd(q, k, v, True, 0.3, lib=lib)
        ro, rl = _torch_ref(q, k, v, True, 0.3)
        _close(o, ro, 1e-12, "causal O vs torch")
        _close(lse, rl, 1e-12, "causal LSE vs torch")


def pin_torch_gqa(lib):
    q, k, v = gen.random_problem(1, 8, 2, 13, 21, 64, seed=6)
    o, lse = oracle.attn_fwd(q, k, v, False, 0.125, lib=lib)
    ro, rl = _torch_ref(q, k, v, False, 0.125)
    _close(o, ro, 1e-12, "GQA O vs torch")
    _close(lse, rl, 1e-12, "GQA LSE vs torch")
    q, k, v = gen.random_problem(2, 6, 3, 11, 11, 16, seed=7)
    o, lse = oracle.attn_fwd(q, k, v, True, 0.25, lib=lib)
    ro, rl = _torch_ref(q, k, v, True, 0.25)
    _close(o, ro, 1e-12, "GQA causal O vs torch")
    _close(lse, rl, 1e-12, "GQA causal LSE vs torch")


def pin_constant_v(lib):
    q, k, _ = gen.random_problem(1, 2, 2, 9, 14, 32, seed=8)
    for c in (0.75, -3.5):
        v = _bits(np.full(k.shape, c, dtype=np.float32))
        for causal in (False, True):
            o, _ = oracle.attn_fwd(q, k, v, causal, 0.2, lib=lib)
            _close(o, np.full(o.shape, c), 1e-12 * abs(c), f"constant V={c} causal={causal}")


def pin_zero_scale_uniform(lib):
    # scale 0: every visible key weighs 1/n_i, so LSE_i = ln n_i and O_i is
    # the mean of the visible V rows
    B, H, Sq, Sk, D = 1, 2, 6, 10, 8
    q, k, v = gen.random_problem(B, H, H, Sq, Sk, D, seed=9)
    vf = _f64(v)
    for causal in (False, True):
        o, lse = oracle.attn_fwd(q, k, v, causal, 0.0, lib=lib)
        for i in range(Sq):
            n = min(Sk, i + 1 + Sk - Sq) if causal else Sk
            _close(lse[:, :, i], np.full((B, H), math.log(n)), 1e-12, f"ln n row {i}")
            _close(o[:, :, i, :], vf[:, :, :n, :].mean(axis=2), 1e-12, f"mean V row {i}")


def pin_causal_row0(lib):
    # causal, Sq == Sk: query 0 sees key 0 only, so O = V[0] and LSE = s_00
    q, k, v = gen.random_problem(2, 4, 2, 12, 12, 64, seed=10)
    o, lse = oracle.attn_fwd(q, k, v, True, 0.125, lib=lib)
    qf, kf, vf = _f64(q), _f64(k), _f64(v)
    for h in range(4):
        hk = h // 2
        assert np.array_equal(o[:, h, 0, :], vf[:, hk, 0, :]), "causal row 0 O != V[0]"
        s00 = 0.125 * np.einsum("bd,bd->b", qf[:, h, 0, :], kf[:, hk, 0, :])
        _close(lse[:, h, 0], s00, 1e-12, "causal row 0 LSE")


def pin_single_key(lib):
    q, k, v = gen.random_problem(1, 2, 1, 7, 1, 32, seed=11)
    o, lse = oracle.attn_fwd(q, k, v, False, 0.5, lib=lib)
    qf, kf, vf = _f64(q), _f64(k), _f64(v)
    assert np.array_equal(o, np.broadcast_to(vf[:, :1, :1, :], o.shape)), "single key O != V[0]"
    _close(lse, 0.5 * np.einsum("bhid,bd->bhi", qf, kf[:, 0, 0, :]), 1e-12, "single key LSE")


def pin_two_keys(lib):
    # two keys: weight of key 0 is 1/(1+exp(s1-s0)), LSE = logaddexp(s0, s1)
    q, k, v = gen.random_problem(1, 1, 1, 10, 2, 16, seed=12)
    o, lse = oracle.attn_fwd(q, k, v, False, 0.7, lib=lib)
    qf, kf, vf = _f64(q)[0, 0], _f64(k)[0, 0], _f64(v)[0, 0]
    s = 0.7 * (qf @ kf.T)
    w0 = 1.0 / (1.0 + np.exp(s[:, 1] - s[:, 0]))
    _close(lse[0, 0], np.logaddexp(s[:, 0], s[:, 1]), 1e-12, "two-key LSE")
    _close(o[0, 0], w0[:, None] * vf[0] + (1 - w0)[:, None] * vf[1], 1e-12, "two-key O")


def pin_golden_closed_forms(lib):
    for case in load_golden():
        q = _bits(np.array(case["q"], dtype=np.float32)[None, None])
        k = _bits(np.array(case["k"], dtype=np.float32)[None, None])
        v = _bits(np.array(case["v"], dtype=np.float32)[None, None])
        o, lse = oracle.attn_fwd(q, k, v, case["causal"], case["scale"], lib=lib)
        _close(o[0, 0], np.array(case["o"]), case["tol"], f"golden {case['name']} O")
        _close(lse[0, 0], np.array(case["lse"]), case["tol"], f"golden {case['name']} LSE")


def pin_permutation(lib):
    q, k, v = gen.random_problem(1, 2, 2, 8, 27, 32, seed=13)
    perm = np.random.default_rng(0).permutation(27)
    o1, l1 = oracle.attn_fwd(q, k, v, False, 0.3, lib=lib)
    o2, l2 = oracle.attn_fwd(q, k[:, :, perm], v[:, :, perm], False, 0.3, lib=lib)
    _close(o1, o2, 1e-12, "permuted keys O")
    _close(l1, l2, 1e-12, "permuted keys LSE")


def pin_gqa_equals_repeat(lib):
    q, k, v = gen.random_problem(2, 6, 2, 9, 15, 16, seed=14)
    for causal in (False, True):
        o1, l1 = oracle.attn_fwd(q, k, v, causal, 0.4, lib=lib)
        o2, l2 = oracle.attn_fwd(q, np.repeat(k, 3, axis=1), np.repeat(v, 3, axis=1), causal, 0.4,
                                 lib=lib)
        assert np.array_equal(o1, o2) and np.array_equal(l1, l2), "GQA != repeated K/V heads"


def pin_causal_is_prefix(lib):
    # bottom-right alignment: causal row i equals non-causal attention over
    # keys [0, i + Sk - Sq]
    for Sq, Sk in ((7, 7), (5, 12), (1, 9)):
        q, k, v = gen.random_problem(1, 2, 2, Sq, Sk, 16, seed=15 + Sk)
        o, lse = oracle.attn_fwd(q, k, v, True, 0.35, lib=lib)
        for i in range(Sq):
            n = i + 1 + Sk - Sq
            po, pl = oracle.attn_fwd(q[:, :, i:i + 1], k[:, :, :n], v[:, :, :n], False, 0.35,
                                     lib=lib)
            _close(o[:, :, i], po[:, :, 0], 1e-12, f"causal prefix O Sq={Sq} Sk={Sk} i={i}")
            _close(lse[:, :, i], pl[:, :, 0], 1e-12, f"causal prefix LSE Sq={Sq} Sk={Sk} i={i}")


def pin_key_shift(lib):
    # adding u to every key adds scale*q.u to each score of a row: O stays,
    # LSE moves by that amount.  Small integers keep K + u exact in bf16.
    rng = np.random.default_rng(1)
    qf = rng.integers(-3, 4, size=(1, 2, 6, 8)).astype(np.float32)
    kf = rng.integers(-3, 4, size=(1, 2, 10, 8)).astype(np.float32)
    vf = rng.integers(-4, 5, size=(1, 2, 10, 8)).astype(np.float32)
    u = rng.integers(-2, 3, size=(8,)).astype(np.float32)
    q, k, v, k2 = _bits(qf), _bits(kf), _bits(vf), _bits(kf + u)
    o1, l1 = oracle.attn_fwd(q, k, v, False, 0.25, lib=lib)
    o2, l2 = oracle.attn_fwd(q, k2, v, False, 0.25, lib=lib)
    _close(o1, o2, 1e-12, "key shift O")
    _close(l2 - l1, 0.25 * (qf.astype(np.float64) @ u.astype(np.float64)), 1e-12, "key shift LSE")


def pin_large_scores_stable(lib):
    # scores in the thousands: softmax collapses onto the largest score; a
    # version that skips the max subtraction overflows
    qf = np.zeros((1, 1, 3, 4), dtype=np.float32)
    qf[0, 0, :, 0] = [64.0, -64.0, 32.0]
    kf = np.zeros((1, 1, 5, 4), dtype=np.float32)
    kf[0, 0, :, 0] = [1.0, 2.0, 3.0, 4.0, 8.0]
    vf = np.arange(20, dtype=np.float32).reshape(1, 1, 5, 4)
    o, lse = oracle.attn_fwd(_bits(qf), _bits(kf), _bits(vf), False, 8.0, lib=lib)
    best = [4, 0, 4]
    s_best = [8.0 * 64 * 8, 8.0 * -64 * 1, 8.0 * 32 * 8]
    for i in range(3):
        _close(o[0, 0, i], vf[0, 0, best[i]], 1e-12, f"huge-score row {i} O")
        _close(lse[0, 0, i], s_best[i], 1e-9, f"huge-score row {i} LSE")


def pin_onehot_v_probabilities(lib):
    # V = identity rows (D >= Sk): O row i is the probability row P_i
    for causal, (Sq, Sk) in ((False, (7, 16)), (True, (9, 16)), (True, (16, 16))):
        q, k, _ = gen.random_problem(1, 2, 2, Sq, Sk, 32, seed=30 + Sq)
        eye = np.zeros((1, 2, Sk, 32), dtype=np.float32)
        eye[0, :, np.arange(Sk), np.arange(Sk)] = 1.0
        o, lse = oracle.attn_fwd(q, k, _bits(eye), causal, 0.3, lib=lib)
        s = 0.3 * np.matmul(_f64(q), np.swapaxes(_f64(k), -1, -2))
        for i in range(Sq):
            n = min(Sk, i + 1 + Sk - Sq) if causal else Sk
            p = o[0, :, i, :]
            assert np.all(p >= 0), "negative probability"
            assert np.all(p[:, n:] == 0), f"masked keys carry weight (row {i})"
            _close(p.sum(axis=1), np.ones(2), 1e-12, f"row {i} sums to one")
            _close(p[:, :n], np.exp(s[0, :, i, :n] - lse[0, :, i, None]), 1e-12,
                   f"row {i} P = exp(s - LSE)")


def pin_rows_entry(lib):
    q, k, v = gen.random_problem(2, 4, 2, 21, 30, 32, seed=16)
    o, lse = oracle.attn_fwd(q, k, v, True, 0.2, lib=lib)
    rows = [(1, 3, 20), (0, 0, 0), (1, 1, 7), (0, 2, 13)]
    ro, rl = oracle.attn_rows(q, k, v, True, 0.2, rows, lib=lib)
    for r, (b, h, i) in enumerate(rows):
        assert np.array_equal(ro[r], o[b, h, i]) and rl[r] == lse[b, h, i], "rows entry differs"


def pin_thread_count_invariant(lib):
    q, k, v = gen.random_problem(1, 3, 3, 25, 25, 16, seed=17)
    a = oracle.attn_fwd(q, k, v, True, 0.3, nthreads=1, lib=lib)
    b = oracle.attn_fwd(q, k, v, True, 0.3, nthreads=7, lib=lib)
    assert all(np.array_equal(x, y) for x, y in zip(a, b)), "result depends on thread count"


def load_golden():
    """Hand-worked closed-form cases from tests/golden/closed_forms.txt.

    Each block is ``key: value`` lines; q/k/v/o are row lists separated by
    ``;``, scalars are Python expressions over ``math`` (e.g. ``math.log(4)``).
    """
    path = os.path.join(GOLDEN, "closed_forms.txt")
    cases, cur = [], {}
    env = {"math": math, "__builtins__": {}}

    def rows(text):
        return [[float(eval(x, env)) for x in r.split(",")] for r in text.split(";")]

    with open(path) as f:
        for raw in f:
            if not raw.strip():          # a blank line ends a case
                if cur:
                    cases.append(cur)
                    cur = {}
                continue
            line = raw.split("#", 1)[0].strip()
            if not line:                 # comment line
                continue
            key, val = (t.strip() for t in line.split(":", 1))
            if key in ("q", "k", "v", "o"):
                cur[key] = rows(val)
            elif key == "lse":
                cur[key] = [float(eval(x, env)) for x in val.split(",")]
            elif key == "causal":
                cur[key] = val == "true"
            elif key == "name":
                cur[key] = val
            else:
                cur[key] = float(eval(val, env))
    if cur:
        cases.append(cur)
    return cases


PINS = {name[4:]: fn for name, fn in sorted(globals().items()) if name.startswith("pin_")}
