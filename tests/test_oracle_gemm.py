"""Pins of the oracle's integer MMA and dequantized linear layer (Section 4.4:
per-group integer MMA with a power-of-two per subgroup; Appendix C: per-group
16-bit scales on both operands) against numpy matmuls (library routines) of
independently decoded operands, special cases and closed-form ranges."""
import numpy as np
import pytest

import oracle
import workloads as W


def _rand_act(seed, M, K, gs, flags_max=4):
    g = np.random.Generator(np.random.PCG64(seed))
    c = g.integers(-7, 8, size=(M, K)).astype(np.int8)
    flags = g.integers(0, flags_max + 1, size=(M, K // gs)).astype(np.uint8)
    scales = np.abs(g.normal(0, 0.01, size=(M, K // 64))).astype(np.float16).view(np.uint16)
    return oracle.ActQuant(None, c, flags, scales, np.zeros((M, K // 64), np.int8), gs)


def _rand_w(seed, N, K):
    g = np.random.Generator(np.random.PCG64(seed))
    wq = g.integers(-7, 8, size=(N, K)).astype(np.int8)
    sw = np.abs(g.normal(0, 0.002, size=(N, K // 64))).astype(np.float16).view(np.uint16)
    return wq, sw


def test_flag_zero_reduces_to_integer_matmul():
    a = _rand_act(1, 9, 128, 16, flags_max=0)
    wq, _ = _rand_w(2, 11, 128)
    ref = a.c.astype(np.int64) @ wq.astype(np.int64).T
    np.testing.assert_array_equal(oracle.gemm_i32(a, wq), ref)


@pytest.mark.parametrize("gs", [8, 16, 32, 64])
def test_integer_accumulator_matches_decoded_matmul(gs):
    a = _rand_act(3 + gs, 13, 192, gs)
    wq, _ = _rand_w(4, 17, 192)
    f = np.repeat(a.flags.astype(np.int64), gs, axis=1)
    d = a.c.astype(np.int64) * (2 ** f)
    np.testing.assert_array_equal(oracle.gemm_i32(a, wq), d @ wq.astype(np.int64).T)


def test_per_subgroup_shift_form_equals_decoded_form():
    """Section 4.4's form sum_sub 2^FLAG * (sum c*w) equals the decoded form."""
    a = _rand_act(5, 6, 128, 16)
    wq, _ = _rand_w(6, 7, 128)
    c = a.c.astype(np.int64).reshape(6, -1, 16)
    w = wq.astype(np.int64).reshape(7, -1, 16)
    part = np.einsum("msk,nsk->mns", c, w)          # per-subgroup integer MMA
    shifted = (part * (2 ** a.flags.astype(np.int64))[:, None, :]).sum(axis=2)
    np.testing.assert_array_equal(oracle.gemm_i32(a, wq), shifted)


def test_integer_range_bound():
    g = np.random.Generator(np.random.PCG64(7))
    K = 12288
    c = np.full((1, K), 7, np.int8)
    flags = np.full((1, K // 16), 4, np.uint8)
    a = oracle.ActQuant(None, c, flags, np.zeros((1, K // 64), np.uint16), None, 16)
    wq = np.full((1, K), 7, np.int8)
    I = oracle.gemm_i32(a, wq)
    assert I[0, 0] == 112 * 7 * K < 2 ** 24
    # one 64-group: |P| <= 112 * 7 * 64 = 50176 < 2^24
    assert 112 * 7 * 64 == 50176
    del g


@pytest.mark.parametrize("epilogue", [0, 1])
def test_linear_matches_dequantized_matmul(epilogue):
    a = _rand_act(8, 10, 256, 16)
    wq, sw = _rand_w(9, 12, 256)
    bias = W.to_bf16_bits(np.linspace(-0.1, 0.1, 12))
    y, S = oracle.linear_f64(a, wq, sw, bias, epilogue=epilogue)
    sa = np.repeat(a.scales.view(np.float16).astype(np.float64), 64, axis=1)
    swf = np.repeat(sw.view(np.float16).astype(np.float64), 64, axis=1)
    f = np.repeat(a.flags.astype(np.int64), 16, axis=1)
    xt = sa * (a.c.astype(np.float64) * 2.0 ** f)
    wt = swf * wq.astype(np.float64)
    ref = xt @ wt.T + W.bf16_bits_to_f32(bias).astype(np.float64)[None, :]
    if epilogue == 1:
        import torch
        ref = torch.nn.functional.gelu(torch.tensor(ref), approximate="tanh").numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-12)
    assert np.all(S >= np.abs(ref if epilogue == 0 else y * 0) - 1e-12)


def test_no_bias_and_sampled_outputs():
    a = _rand_act(10, 20, 128, 32)
    wq, sw = _rand_w(11, 24, 128)
    y, S = oracle.linear_f64(a, wq, sw, None)
    rows = np.array([0, 5, 19, 7])
    cols = np.array([3, 0, 23, 7])
    ys, Ss = oracle.linear_f64_sampled(a, wq, sw, None, rows, cols)
    np.testing.assert_array_equal(ys, y[rows, cols])
    np.testing.assert_array_equal(Ss, S[rows, cols])


def test_end_to_end_on_workload_rows():
    """Quantized layer output approximates the full-precision product."""
    x = W.make_x(1, 0, rows=32)
    w = W.make_w(1, 0, rows=64)
    a = oracle.quantize_act(x, 16)
    wq, sw = oracle.quantize_weight(w)
    y, _ = oracle.linear_f64(a, wq, sw, None)
    ref = W.bf16_bits_to_f32(x).astype(np.float64) @ W.bf16_bits_to_f32(w).astype(np.float64).T
    rel = np.linalg.norm(y - ref) / np.linalg.norm(ref)
    assert rel < 0.25
