"""Pins of the oracle's fused output quantization: the layer's bf16 output
run through the next layer's activation quantizer (Eq. 1, Eq. 2 and the
right shift of Section 3, applied on the fly to the producing layer's result,
Appendix C).

The exact case builds activations and weights whose group scales are powers
of two (every group holds an element of magnitude 127 * 2^e, resp. 7 * 2^f),
so that Stage 1 and the weight quantizer return the integers themselves and
the layer output is 2^(e_m + f_n) times an integer matmul computed here with
numpy; its bf16 rounding is then exact arithmetic plus one rounding, done
here on numpy's float32 bit patterns."""
import numpy as np
import pytest
import torch

import oracle
import workloads as W


def _exact_case(seed, M, N, K, gs):
    c = W.make_exact_case(seed, M, N, K)
    assert np.array_equal(W.bf16_bits_to_f32(c.bias).astype(np.float64), c.bias_val)
    return c.A, c.Wi, c.e, c.f, c.x, c.w, c.bias, c.bias_val


@pytest.mark.parametrize("gs,out_gs", [(16, 16), (8, 32), (64, 8)])
def test_exact_power_of_two_case(gs, out_gs):
    M, N, K = 12, 192, 256
    A, Wi, e, f, x, w, bias, bias_val = _exact_case(100 + gs, M, N, K, gs)
    a = oracle.quantize_act(x, gs)
    wq, sw = oracle.quantize_weight(w)
    # Stage 1 and the weight quantizer return the integers and the powers of two
    np.testing.assert_array_equal(a.q8.astype(np.int64), A)
    np.testing.assert_array_equal(wq.astype(np.int64), Wi)
    np.testing.assert_array_equal(a.scales.view(np.float16).astype(np.float64),
                                  np.repeat(np.ldexp(1.0, e)[:, None], K // 64, axis=1))
    np.testing.assert_array_equal(sw.view(np.float16).astype(np.float64),
                                  np.repeat(np.ldexp(1.0, f)[:, None], K // 64, axis=1))
    # the decoded activations from the codes, independently of the oracle's GEMM
    fl = np.repeat(a.flags.astype(np.int64), gs, axis=1)
    d = a.c.astype(np.int64) << fl
    I = d @ Wi.T
    y = np.ldexp(I.astype(np.float64), e[:, None] + f[None, :]) + bias_val[None, :]
    # every value is an integer times a power of two below 2^24 of it: exact in fp32
    assert np.array_equal(y.astype(np.float32).astype(np.float64), y)
    expect = oracle.quantize_act(W.to_bf16_bits(y), out_gs)
    got = oracle.linear_quantize(a, wq, sw, bias, 0, out_gs)
    np.testing.assert_array_equal(got.c, expect.c)
    np.testing.assert_array_equal(got.flags, expect.flags)
    np.testing.assert_array_equal(got.scales, expect.scales)
    np.testing.assert_array_equal(got.q8, expect.q8)


def test_gelu_case_quantizes_the_rounded_activation():
    M, N, K = 6, 128, 192
    _, _, e, f, x, w, bias, _ = _exact_case(7, M, N, K, 16)
    a = oracle.quantize_act(x, 16)
    wq, sw = oracle.quantize_weight(w)
    y, _ = oracle.linear_f64(a, wq, sw, bias, epilogue=0)
    g = torch.nn.functional.gelu(torch.tensor(y, dtype=torch.float64), approximate="tanh").numpy()
    bits = np.vectorize(oracle.f64_to_bf16_rne, otypes=[np.uint16])(g)
    expect = oracle.quantize_act(bits, 32)
    got = oracle.linear_quantize(a, wq, sw, bias, 1, 32)
    np.testing.assert_array_equal(got.c, expect.c)
    np.testing.assert_array_equal(got.flags, expect.flags)
    np.testing.assert_array_equal(got.scales, expect.scales)


def test_round_bf16_array():
    g = np.random.Generator(np.random.PCG64(11))
    # values exact in float32: the float32 -> bf16 bit rounding of numpy patterns
    v32 = (g.standard_normal(20000) * np.exp(g.uniform(-40, 40, 20000))).astype(np.float32)
    np.testing.assert_array_equal(oracle.round_bf16(v32.astype(np.float64)), W.to_bf16_bits(v32))
    # arbitrary doubles: the scalar rounding, elementwise; ties and signed zeros
    v = g.standard_normal(2000) * np.exp(g.uniform(-20, 20, 2000))
    v = np.concatenate([v, [0.0, -0.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -(1.0 + 2.0 ** -8)]])
    ref = np.array([oracle.f64_to_bf16_rne(t) for t in v], np.uint16)
    np.testing.assert_array_equal(oracle.round_bf16(v), ref)
    assert list(oracle.round_bf16(np.array([1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8]))) == [0x3F80, 0x3F82]
