"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Bit-exact: activation codes / flags / scales / zeros, unpacked weight codes and
weight scales, the integer accumulator.  Within tolerance (tests/helpers.py):
the bf16 output of the linear layer.  Inputs come from workloads.py (the
seeded recipes of each layer, truncated to oracle-friendly row counts that
still span several tiles and a ragged tail) plus edge cases.
"""
import numpy as np
import pytest

import oracle
import workloads as W
from helpers import (bf16_bits_to_f64, bf16_ulp_distance, to_dev_bf16, to_host_u16,
                     y_tolerance)

pytestmark = pytest.mark.gpu

LAYERS = [(c, i) for c in (1, 2, 3, 5) for i in range(len(W.CONFIGS[c].layers))] + [(4, 0)]


def _q():
    import paper_2509_26436_amd as q
    return q


def _act_parity(xb, gs, ldx_pad=0, with_zeros=True):
    import torch
    q = _q()
    M, K = xb.shape
    if ldx_pad:
        full = np.zeros((M, K + ldx_pad), np.uint16)
        full[:, :K] = xb
        xd = to_dev_bf16(full)[:, :K]
    else:
        xd = to_dev_bf16(xb)
    got = q.quantize_act(xd, lzs_group=gs, with_zeros=with_zeros)
    torch.cuda.synchronize()
    ref = oracle.quantize_act(xb, lzs_group=gs)
    np.testing.assert_array_equal(got.codes.cpu().numpy(), ref.codes)
    np.testing.assert_array_equal(got.flags.cpu().numpy(), ref.abi_flags)
    np.testing.assert_array_equal(to_host_u16(got.scales), ref.abi_scales)
    if with_zeros:
        np.testing.assert_array_equal(got.zeros.cpu().numpy(), ref.abi_zeros)
    return got, ref


@pytest.mark.parametrize("cfg,layer", LAYERS)
@pytest.mark.parametrize("gs", [8, 16, 32, 64])
def test_quantize_bit_exact_workloads(cfg, layer, gs):
    rows = 200 if cfg != 5 else 130          # several waves and a ragged tail
    xb = W.make_x(cfg, layer, rows=rows)
    _act_parity(xb, gs)


@pytest.mark.parametrize("M,K", [(1, 64), (1, 128), (3, 192), (7, 1152), (33, 64)])
def test_quantize_small_and_ragged(M, K):
    xb = W.make_random_x(1000 + M * K, M, K, "t3", 0.1)
    for gs in (8, 16, 32, 64):
        _act_parity(xb, gs)


def test_quantize_strided_rows():
    xb = W.make_random_x(77, 45, 576, "laplace", 0.3)
    _act_parity(xb, 16, ldx_pad=64)
    _act_parity(xb, 8, ldx_pad=8)


def test_quantize_edge_values():
    x = np.zeros((6, 256))
    x[1] = 1e-9                                   # fp16 scale underflows to 0
    x[2, :64] = 1e-5                              # subnormal fp16 scale
    x[2, 64:] = np.linspace(-1e-4, 1e-4, 192)
    x[3] = np.linspace(-8e6, 8e6, 256)            # near the top of the fp16 scale range
    x[4, ::2] = 3.0                               # exact ties after scaling
    x[4, 1::2] = -2.5
    x[5] = np.ldexp(1.0, np.arange(256) % 40 - 20)
    xb = W.to_bf16_bits(x)
    xb[0, :8] = 0x8000                            # negative zeros
    for gs in (8, 16, 32, 64):
        _act_parity(xb, gs)


def test_quantize_all_bf16_magnitudes_as_group_max():
    """Every finite positive bf16 value is the maximum of one group (so alpha/127
    and 1/s are exercised over the whole input range, fp16 saturation included);
    the rest of the group holds v * k/64 for k = 1..63."""
    mags = np.arange(0x0001, 0x7F80, dtype=np.uint32).astype(np.uint16)
    v = W.bf16_bits_to_f32(mags).astype(np.float64)
    frac = np.arange(64) / 64.0
    frac[0] = 1.0
    with np.errstate(over="ignore"):
        x = v[:, None] * frac[None, :]
    xb = W.to_bf16_bits(x)
    xb[:, 1::3] |= 0x8000
    for gs in (16, 64):
        _act_parity(xb, gs)


def test_quantize_empty():
    import torch
    q = _q()
    xd = torch.empty((0, 128), dtype=torch.bfloat16, device="cuda")
    out = q.quantize_act(xd, 16)
    assert out.codes.shape == (2, 0, 32)


@pytest.mark.parametrize("cfg,layer", LAYERS)
def test_pack_weight_bit_exact(cfg, layer):
    import torch
    q = _q()
    L = W.CONFIGS[cfg].layers[layer]
    n_rows = min(L.N, 200)
    wb = W.make_w(cfg, layer, rows=n_rows)
    pw = q.pack_weight(to_dev_bf16(wb))
    wq = q.unpack_weight(pw)
    torch.cuda.synchronize()
    wq_ref, sw_ref = oracle.quantize_weight(wb)
    np.testing.assert_array_equal(wq.cpu().numpy(), wq_ref)
    np.testing.assert_array_equal(to_host_u16(pw.scales), sw_ref)


def test_pack_weight_edges():
    import torch
    q = _q()
    w = np.zeros((70, 128))
    w[1] = 1e-9
    w[2] = np.linspace(-3, 3, 128)
    w[3, :64] = 0.5                                   # exact ties: 0.5/(0.5/7) = 7
    w[4] = np.ldexp(1.0, np.arange(128) % 30 - 15)
    w[5:] = np.random.Generator(np.random.PCG64(3)).normal(0, 0.02, (65, 128))
    wb = W.to_bf16_bits(w)
    pw = q.pack_weight(to_dev_bf16(wb))
    wq = q.unpack_weight(pw)
    torch.cuda.synchronize()
    wq_ref, sw_ref = oracle.quantize_weight(wb)
    np.testing.assert_array_equal(wq.cpu().numpy(), wq_ref)
    np.testing.assert_array_equal(to_host_u16(pw.scales), sw_ref)


def _gemm_case(xb, wb, gs):
    import torch
    q = _q()
    a_ref = oracle.quantize_act(xb, lzs_group=gs)
    wq_ref, sw_ref = oracle.quantize_weight(wb)
    # the GPU consumes the oracle's packed codes (no oracle input from the GPU path)
    M, K = xb.shape
    qa = q.QuantizedAct(
        codes=torch.from_numpy(a_ref.codes).cuda(),
        flags=torch.from_numpy(a_ref.abi_flags).cuda(),
        scales=torch.from_numpy(a_ref.abi_scales.view(np.int16)).cuda(),
        zeros=None, M=M, K=K, lzs_group=gs)
    pw = q.pack_weight(to_dev_bf16(wb))
    return qa, pw, a_ref, wq_ref, sw_ref


@pytest.mark.parametrize("gs", [8, 16, 32, 64])
@pytest.mark.parametrize("M,N,K", [(200, 136, 192), (130, 320, 2880 // 5), (1, 64, 64),
                                   (129, 129, 128), (256, 384, 1152)])
def test_gemm_i32_bit_exact(M, N, K, gs):
    import torch
    q = _q()
    xb = W.make_random_x(M * 7 + N, M, K, "t3", 0.05)
    wb = W.to_bf16_bits(np.random.Generator(np.random.PCG64(N + K)).normal(0, 0.02, (N, K)))
    qa, pw, a_ref, wq_ref, _ = _gemm_case(xb, wb, gs)
    acc = q.w4a4_gemm_i32(qa, pw)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(acc.cpu().numpy(), oracle.gemm_i32(a_ref, wq_ref))


def _linear_check(qa, pw, a_ref, wq_ref, sw_ref, bias_b, epi, ldy_pad=0):
    import torch
    q = _q()
    M, N, K = qa.M, pw.N, qa.K
    if ldy_pad:
        ybuf = torch.full((M, N + ldy_pad), 7.0, dtype=torch.bfloat16, device="cuda")
        y = q.w4a4_linear(qa, pw, None if bias_b is None else to_dev_bf16(bias_b), epi,
                          out=ybuf[:, :N])
    else:
        y = q.w4a4_linear(qa, pw, None if bias_b is None else to_dev_bf16(bias_b), epi)
    torch.cuda.synchronize()
    if ldy_pad:
        assert torch.all(ybuf[:, N:] == 7.0)
    y_bits = to_host_u16(y.contiguous())
    y64, S = oracle.linear_f64(a_ref, wq_ref, sw_ref, bias_b, epilogue=epi)
    tol = y_tolerance(y64, S, K, gelu=(epi == 1))
    err = np.abs(bf16_bits_to_f64(y_bits) - y64)
    bad = err > tol
    assert not bad.any(), (f"{bad.sum()} outputs out of tolerance; worst excess "
                           f"{(err - tol).max():.3e}")
    ulp = bf16_ulp_distance(y_bits, oracle.to_bf16_bits(y64))
    assert np.mean(ulp <= 1) > 0.99
    return y


@pytest.mark.parametrize("cfg,layer", [(1, 0), (2, 0), (2, 3), (3, 1), (4, 0), (5, 0), (5, 2)])
def test_linear_workload_layers(cfg, layer):
    L = W.CONFIGS[cfg].layers[layer]
    M = 160
    N = min(L.N, 448)
    K = L.K
    xb = W.make_x(cfg, layer, rows=M)
    wb = W.make_w(cfg, layer, rows=N)
    bias = W.make_bias(cfg, layer, cols=N)
    qa, pw, a_ref, wq_ref, sw_ref = _gemm_case(xb, wb, 16)
    _linear_check(qa, pw, a_ref, wq_ref, sw_ref, bias, L.epilogue)


@pytest.mark.parametrize("gs", [8, 32, 64])
def test_linear_group_sizes(gs):
    xb = W.make_x(3, 0, rows=96)
    wb = W.make_w(3, 0, rows=200)
    bias = W.make_bias(3, 0, cols=200)
    qa, pw, a_ref, wq_ref, sw_ref = _gemm_case(xb, wb, gs)
    _linear_check(qa, pw, a_ref, wq_ref, sw_ref, bias, 0)


def test_linear_no_bias_gelu_and_strided_output():
    xb = W.make_x(1, 0, rows=70)
    wb = W.make_w(1, 0, rows=130)
    qa, pw, a_ref, wq_ref, sw_ref = _gemm_case(xb, wb, 16)
    _linear_check(qa, pw, a_ref, wq_ref, sw_ref, None, 0)
    _linear_check(qa, pw, a_ref, wq_ref, sw_ref, None, 1)
    bias = W.make_bias(1, 0, cols=130)
    _linear_check(qa, pw, a_ref, wq_ref, sw_ref, bias, 1, ldy_pad=6)


def test_quantize_then_linear_end_to_end():
    """The GPU's own quantizer output feeds the GPU GEMM (the product path)."""
    import torch
    q = _q()
    xb = W.make_x(2, 2, rows=256)
    wb = W.make_w(2, 2, rows=320)
    bias = W.make_bias(2, 2, cols=320)
    qa = q.quantize_act(to_dev_bf16(xb), 16)
    pw = q.pack_weight(to_dev_bf16(wb))
    y = q.w4a4_linear(qa, pw, to_dev_bf16(bias))
    torch.cuda.synchronize()
    a_ref = oracle.quantize_act(xb, 16)
    wq_ref, sw_ref = oracle.quantize_weight(wb)
    y64, S = oracle.linear_f64(a_ref, wq_ref, sw_ref, bias)
    err = np.abs(bf16_bits_to_f64(to_host_u16(y)) - y64)
    assert np.all(err <= y_tolerance(y64, S, xb.shape[1]))
