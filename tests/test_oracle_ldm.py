"""Pins of the oracle's LDM setting (the experimental-details appendix:
per-channel weight quantization, static per-tensor activation quantization,
4-bit compression on the fly; reading R8): a search over all levels, special
cases that reduce to the per-group functions (themselves pinned elsewhere),
round-trip bounds, and the layer against a float64 numpy matmul of the
dequantized operands."""
import numpy as np
import pytest

import oracle
import workloads as W


def _f32(bits):
    return W.bf16_bits_to_f32(bits)


def _nearest_even(p, lo, hi):
    """The nearest integer level in [lo, hi] to each float64 in p, ties to even."""
    levels = np.arange(lo, hi + 1, dtype=np.float64)
    dist = np.abs(p.reshape(-1)[:, None] - levels[None, :])
    best = dist.min(axis=1)
    out = []
    for i in range(dist.shape[0]):
        c = levels[dist[i] == best[i]]
        if c.size > 1:
            c = c[c % 2 == 0]
        out.append(c[0])
    return np.array(out).reshape(p.shape)


@pytest.mark.parametrize("gs", [8, 16, 64])
def test_static_codes_by_search_and_clipping(gs):
    xb = W.make_random_x(31 + gs, 6, 128, "t3", 0.05)
    x = _f32(xb).astype(np.float64)
    s = np.float32(np.abs(x).max() / 127.0 * 0.5)       # a calibrated range half the data's
    a = oracle.quantize_act_static(xb, float(s), gs)
    r = np.float32(1.0) / s
    p = (_f32(xb) * r).astype(np.float32).astype(np.float64)
    np.testing.assert_array_equal(a.q8.astype(np.float64), _nearest_even(p, -127, 127))
    # values inside the range round-trip within half a step; outside, they saturate
    inside = np.abs(x) <= 127 * float(s)
    assert inside.mean() > 0.9 and (~inside).any()
    err = np.abs(x - float(s) * a.q8)
    assert np.all(err[inside] <= 0.5 * float(s) * (1 + 2.0 ** -20))
    assert np.all(np.abs(a.q8[~inside]) == 127)
    # Stage 2 is the subgroup LZS of the Stage-1 codes
    for m in range(2):
        for j in range(128 // gs):
            f, c = oracle.lzs_subgroup(a.q8[m, j * gs:(j + 1) * gs])
            assert f == a.flags[m, j]
            np.testing.assert_array_equal(c, a.c[m, j * gs:(j + 1) * gs])


def test_static_with_the_groups_own_scale_is_the_dynamic_quantizer():
    """A row that is one 64-group, quantized with its own fp16 group scale as
    the static scale, gives the dynamic quantizer's codes and flags."""
    xb = W.make_random_x(41, 10, 64, "laplace", 0.1)
    dyn = oracle.quantize_act(xb, 16)
    for m in range(xb.shape[0]):
        s = float(dyn.scales[m:m + 1].view(np.float16)[0, 0])
        st = oracle.quantize_act_static(xb[m:m + 1], s, 16)
        np.testing.assert_array_equal(st.q8[0], dyn.q8[m])
        np.testing.assert_array_equal(st.c[0], dyn.c[m])
        np.testing.assert_array_equal(st.flags[0], dyn.flags[m])


def test_per_channel_weights():
    w = W.make_w(1, 0, rows=24)[:, :256].copy()
    wq, sw = oracle.quantize_weight_per_channel(w)
    beta = np.abs(_f32(w)).max(axis=1)
    ref = (beta / np.float32(7.0)).astype(np.float32).astype(np.float16).view(np.uint16)
    np.testing.assert_array_equal(sw, ref)
    s = sw.view(np.float16).astype(np.float32)
    r = np.float32(1.0) / s
    p = (_f32(w) * r[:, None]).astype(np.float32).astype(np.float64)
    np.testing.assert_array_equal(wq.astype(np.float64), _nearest_even(p, -7, 7))
    # the row maximum maps to +-7; K = 64 reduces to the per-group quantizer
    idx = np.abs(_f32(w)).argmax(axis=1)
    assert np.all(np.abs(wq[np.arange(24), idx]) == 7)
    wq64, sw64 = oracle.quantize_weight_per_channel(w[:, :64].copy())
    wqg, swg = oracle.quantize_weight(w[:, :64].copy())
    np.testing.assert_array_equal(wq64, wqg)
    np.testing.assert_array_equal(sw64, swg[:, 0])


@pytest.mark.parametrize("epilogue", [0, 1])
def test_static_linear_against_dequantized_matmul(epilogue):
    xb = W.make_random_x(51, 9, 192, "laplace", 0.1)
    s = 0.0031
    a = oracle.quantize_act_static(xb, s, 16)
    wb = W.make_w(1, 0, rows=13)[:, :192].copy()
    wq, sw = oracle.quantize_weight_per_channel(wb)
    bias = W.to_bf16_bits(np.linspace(-0.2, 0.2, 13))
    y, S = oracle.linear_static_f64(a, s, wq, sw, bias, epilogue)
    d = a.c.astype(np.float64) * 2.0 ** np.repeat(a.flags.astype(np.int64), 16, axis=1)
    ref = (float(np.float32(s)) * d) @ (sw.view(np.float16).astype(np.float64)[:, None] * wq).T
    ref = ref + W.bf16_bits_to_f32(bias).astype(np.float64)[None, :]
    if epilogue == 1:
        import torch
        ref = torch.nn.functional.gelu(torch.tensor(ref), approximate="tanh").numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-15)
    assert np.all(S > 0)


def test_static_linear_equals_per_group_linear_with_equal_scales():
    """With every group scale equal (the static s on the activation side, the
    channel scale repeated on the weight side) the per-group layer and the
    LDM-setting layer agree (two separate code paths of the oracle)."""
    xb = W.make_random_x(61, 7, 256, "t3", 0.05)
    s16 = np.array([0.004], np.float16)
    s = float(s16[0])
    a = oracle.quantize_act_static(xb, s, 32)
    wb = W.make_w(3, 0, rows=11)[:, :256].copy()
    wq, sw = oracle.quantize_weight_per_channel(wb)
    y_st, _ = oracle.linear_static_f64(a, s, wq, sw, None, 0)
    a_pg = oracle.ActQuant(a.q8, a.c, a.flags, np.full((7, 4), s16.view(np.uint16)[0], np.uint16),
                           np.zeros((7, 4), np.int8), 32)
    sw_pg = np.repeat(sw[:, None], 4, axis=1)
    y_pg, _ = oracle.linear_f64(a_pg, wq, sw_pg, None, 0)
    np.testing.assert_allclose(y_st, y_pg, rtol=1e-14, atol=0)
