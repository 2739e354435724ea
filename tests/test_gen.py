"""Seeded input generator: determinism, distribution, bf16 rounding and the
peaky-key recipe."""
import numpy as np

from paper_2504_17577_amd import gen


def test_same_seed_same_bytes_and_streams_differ():
    a = gen.normal_bf16((3, 5, 7), seed=0, wid=1, tensor=gen.TENSOR_Q)
    b = gen.normal_bf16((3, 5, 7), seed=0, wid=1, tensor=gen.TENSOR_Q)
    c = gen.normal_bf16((3, 5, 7), seed=0, wid=1, tensor=gen.TENSOR_K)
    d = gen.normal_bf16((3, 5, 7), seed=1, wid=1, tensor=gen.TENSOR_Q)
    e = gen.normal_bf16((3, 5, 7), seed=0, wid=2, tensor=gen.TENSOR_Q)
    assert a.dtype == np.uint16 and np.array_equal(a, b)
    assert not np.array_equal(a, c) and not np.array_equal(a, d) and not np.array_equal(a, e)


def test_moments():
    x = gen.f32_from_bf16(gen.normal_bf16((1 << 20,), seed=3, wid=0, tensor=0)).astype(np.float64)
    n = x.size
    assert abs(x.mean()) < 5 / np.sqrt(n)
    assert abs(x.var() - 1.0) < 5 * np.sqrt(2.0 / n)


def test_bf16_round_to_nearest_even():
    cases = {
        0x3F808000: 0x3F80,  # exactly halfway, even below -> stays
        0x3F818000: 0x3F82,  # exactly halfway, odd below -> rounds up to even
        0x3F808001: 0x3F81,  # just above halfway -> up
        0x3F807FFF: 0x3F80,  # just below halfway -> down
        0xBF818000: 0xBF82,  # negative, halfway to even
        0x7F7FFFFF: 0x7F80,  # largest float rounds to +inf in bf16
        0x00000000: 0x0000,
    }
    src = np.array(list(cases), dtype=np.uint32).view(np.float32)
    assert gen.bf16_from_f32(src).tolist() == list(cases.values())
    u = np.array([0x3F80, 0xC040, 0x0001], dtype=np.uint16)
    assert gen.f32_from_bf16(u).tolist() == [1.0, -3.0, np.float32(2.0 ** -133)]


def test_peaky_rows_exactly_x8():
    w = gen.Workload("t", 9, 1, 2, 2, 130, 130, 16, True, peaky_every=64, peaky_factor=8.0)
    q, k, v = gen.make_inputs(w, seed=5)
    plain = gen.normal_bf16(k.shape, 5, 9, gen.TENSOR_K)
    rows = np.arange(130) % 64 == 0
    kf, pf = gen.f32_from_bf16(k), gen.f32_from_bf16(plain)
    assert np.array_equal(kf[:, :, rows], pf[:, :, rows] * 8)
    assert np.array_equal(k[:, :, ~rows], plain[:, :, ~rows])
    assert np.array_equal(q, gen.normal_bf16(q.shape, 5, 9, gen.TENSOR_Q))


def test_workload_counts():
    W = gen.WORKLOADS
    assert W["dense_d128_s2k"].flops() == 4 * 128 * 8 * 32 * 2048 * 2048
    assert W["causal_d64_s1k"].pairs() == 1024 * 1025 // 2
    assert W["gqa4_causal_d128_s4k"].flops() == 274945015808
    assert W["dense_d128_s2k"].bytes() == 673185792
    # bottom-right causal pair count when Sk > Sq
    w = gen.Workload("t", 0, 1, 1, 1, 3, 5, 8, True)
    assert w.pairs() == 3 + 4 + 5
    assert gen.WORKLOADS["tiny_d64_s128"].scale == 0.125
