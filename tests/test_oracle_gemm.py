"""Pins of the GEMM oracle (oracle.gemm, float64 numpy matmul of the widened
bf16 inputs): exact integer products, an independent math.fsum evaluation,
the transpose identity, the rows entry, and the |A||B| scale."""
import math

import numpy as np

import oracle
from paper_2504_17577_amd import gen


def _bits(x):
    return gen.bf16_from_f32(np.asarray(x, dtype=np.float32))


def test_integer_inputs_exact():
    """Small integers are exact in bf16; their products and sums are exact
    in float64, so C must equal the int64 matrix product exactly."""
    rng = np.random.default_rng(0)
    ai = rng.integers(-8, 9, size=(37, 53))
    bi = rng.integers(-8, 9, size=(53, 29))
    c = oracle.gemm(_bits(ai), _bits(bi))
    assert np.array_equal(c, (ai @ bi).astype(np.float64))


def test_against_fsum():
    a, b = gen.random_gemm_problem(9, 7, 300, seed=3)
    c = oracle.gemm(a, b)
    A, B = gen.f32_from_bf16(a).astype(float), gen.f32_from_bf16(b).astype(float)
    for i in range(9):
        for j in range(7):
            ref = math.fsum(A[i, k] * B[k, j] for k in range(300))
            assert abs(c[i, j] - ref) <= 1e-12 * math.fsum(abs(A[i, k] * B[k, j]) for k in range(300))


def test_transpose_identity_and_rows():
    a, b = gen.random_gemm_problem(31, 17, 64, seed=4)
    c = oracle.gemm(a, b)
    ct = oracle.gemm(np.ascontiguousarray(b.T), np.ascontiguousarray(a.T))
    assert np.allclose(c.T, ct, rtol=0, atol=1e-12 * np.abs(c).max())
    rows = [30, 0, 7]
    assert np.array_equal(oracle.gemm(a, b, rows=rows), c[rows])


def test_abs_scale_bounds_result():
    a, b = gen.random_gemm_problem(12, 10, 100, seed=5)
    assert (np.abs(oracle.gemm(a, b)) <= oracle.gemm_abs(a, b) + 1e-12).all()
    ones = _bits(np.ones((3, 4)))
    assert np.array_equal(oracle.gemm_abs(ones, _bits(-np.ones((4, 2)))), np.full((3, 2), 4.0))


def test_matrix_vector_is_dot_products():
    """M = 1 (the paper's V0-V7 shapes): each output is one dot product,
    evaluated here with math.fsum, and the column-sliced call the GPU tests
    use gives the same values as the full one."""
    a, b = gen.random_gemm_problem(1, 24, 520, seed=6)
    c = oracle.gemm(a, b)
    A, B = gen.f32_from_bf16(a).astype(float), gen.f32_from_bf16(b).astype(float)
    assert c.shape == (1, 24)
    for j in range(24):
        ref = math.fsum(A[0, k] * B[k, j] for k in range(520))
        assert abs(c[0, j] - ref) <= 1e-12 * math.fsum(abs(A[0, k] * B[k, j]) for k in range(520))
    cols = [23, 0, 5]
    assert np.array_equal(oracle.gemm(a, np.ascontiguousarray(b[:, cols]))[0], c[0, cols])
