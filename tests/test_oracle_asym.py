"""Pins of the oracle's asymmetric mode (Eq. 1's zero point, repaired so the
255 signed levels cover each group's range including 0; reading R9): scale
and zero point through numpy's conversions, codes by search over all levels,
the half-step round trip, the fixed points of the mapping (0 -> z, the range
ends -> +-127), the one-signed-group special case, the weight group sums
against numpy, and the layer against a float64 matmul of the dequantized
operands s (d - z)."""
import numpy as np
import pytest

import oracle
import workloads as W


def _f32(bits):
    return W.bf16_bits_to_f32(bits)


def _ref_scale_zero(xg):
    lo = np.float32(min(float(xg.min()), 0.0))
    hi = np.float32(max(float(xg.max()), 0.0))
    span = np.float32(hi - lo)
    with np.errstate(over="ignore"):
        s16 = np.array([span / np.float32(254.0)], np.float32).astype(np.float16)
    bits = int(s16.view(np.uint16)[0])
    if bits == 0x7C00:
        bits = 0x7BFF
    s = np.float32(np.array([bits], np.uint16).view(np.float16)[0])
    r = np.float32(0.0) if s == 0 else np.float32(1.0) / s
    z = -127 - int(np.rint(np.float32(lo * r)))
    return bits, s, r, int(np.clip(z, -127, 127))


@pytest.mark.parametrize("kind,gs", [("laplace", 16), ("t3", 8), ("normal", 64)])
def test_scale_zero_and_codes_by_search(kind, gs):
    xb = W.make_random_x(71 + gs, 8, 128, kind, 0.1)
    a = oracle.quantize_act_asym(xb, gs)
    x = _f32(xb)
    levels = np.arange(-254, 255, dtype=np.float64)
    for m in range(x.shape[0]):
        for g in range(2):
            xg = x[m, 64 * g:64 * g + 64]
            bits, s, r, z = _ref_scale_zero(xg)
            assert int(a.scales[m, g]) == bits
            assert int(a.zeros[m, g]) == z
            p = (xg * r).astype(np.float32).astype(np.float64)
            dist = np.abs(p[:, None] - levels[None, :])
            best = dist.min(axis=1)
            q_ref = []
            for i in range(64):
                c = levels[dist[i] == best[i]]
                if c.size > 1:
                    c = c[c % 2 == 0]
                q_ref.append(np.clip(c[0] + z, -127, 127))
            np.testing.assert_array_equal(a.q8[m, 64 * g:64 * g + 64], np.array(q_ref, np.int8))


def test_round_trip_and_fixed_points():
    xb = W.make_random_x(81, 16, 256, "laplace", 0.2)
    a = oracle.quantize_act_asym(xb, 16)
    x = _f32(xb).astype(np.float64)
    s = np.repeat(a.scales.view(np.float16).astype(np.float64), 64, axis=1)
    z = np.repeat(a.zeros.astype(np.float64), 64, axis=1)
    q = a.q8.astype(np.float64)
    # half a step (plus the rounding of r), wherever the code did not clip
    inside = np.abs(q) < 127
    assert np.all(np.abs(x - s * (q - z))[inside] <= s[inside] * (0.5 + 2.0 ** -20 * 256))
    # the group minimum maps to -127; 0 would map to z exactly
    xg = x.reshape(16, 4, 64)
    qg = q.reshape(16, 4, 64)
    idx = xg.argmin(axis=2)
    assert np.all(np.take_along_axis(qg, idx[..., None], axis=2) == -127)
    zero_bits = np.zeros((1, 64), np.uint16)
    zero_bits[0, 5] = W.to_bf16_bits(np.array([0.3]))[0]
    zero_bits[0, 9] = W.to_bf16_bits(np.array([-0.7]))[0]
    az = oracle.quantize_act_asym(zero_bits, 64)
    assert int(az.q8[0, 0]) == int(az.zeros[0, 0])


def test_one_signed_group_has_zero_point_minus_127():
    """A group with no negative value (post-ReLU-like): lo = 0, z = -127,
    q = rne(x / s) - 127, s = fp16(max / 254)."""
    x = np.abs(W.bf16_bits_to_f32(W.make_random_x(91, 3, 64, "laplace", 0.1)))
    xb = W.to_bf16_bits(x)
    a = oracle.quantize_act_asym(xb, 16)
    assert np.all(a.zeros == -127)
    s = a.scales.view(np.float16).astype(np.float32)
    ref_s = (x.max(axis=1) / np.float32(254.0)).astype(np.float16).astype(np.float32)
    np.testing.assert_array_equal(s[:, 0], ref_s)
    r = (np.float32(1.0) / s).astype(np.float32)
    qref = np.clip(np.rint((x * r).astype(np.float32)) - 127, -127, 127)
    np.testing.assert_array_equal(a.q8, qref.astype(np.int8))


def test_weight_group_sums():
    wq = np.random.Generator(np.random.PCG64(5)).integers(-7, 8, (9, 192)).astype(np.int8)
    np.testing.assert_array_equal(oracle.weight_group_sums(wq),
                                  wq.astype(np.int64).reshape(9, 3, 64).sum(axis=2))


@pytest.mark.parametrize("epilogue", [0, 1])
def test_asym_linear_against_dequantized_matmul(epilogue):
    xb = W.make_random_x(101, 10, 192, "t3", 0.05)
    a = oracle.quantize_act_asym(xb, 16)
    wb = W.make_w(1, 0, rows=12)[:, :192].copy()
    wq, sw = oracle.quantize_weight(wb)
    bias = W.to_bf16_bits(np.linspace(-0.1, 0.1, 12))
    y, S = oracle.linear_asym_f64(a, wq, sw, bias, epilogue)
    d = a.c.astype(np.float64) * 2.0 ** np.repeat(a.flags.astype(np.int64), 16, axis=1)
    sa = np.repeat(a.scales.view(np.float16).astype(np.float64), 64, axis=1)
    z = np.repeat(a.zeros.astype(np.float64), 64, axis=1)
    swf = np.repeat(sw.view(np.float16).astype(np.float64), 64, axis=1)
    ref = (sa * (d - z)) @ (swf * wq).T + W.bf16_bits_to_f32(bias).astype(np.float64)[None, :]
    if epilogue == 1:
        import torch
        ref = torch.nn.functional.gelu(torch.tensor(ref), approximate="tanh").numpy()
    np.testing.assert_allclose(y, ref, rtol=1e-12, atol=1e-14)
    assert np.all(S > 0)


def test_zero_points_of_zero_reduce_to_the_symmetric_layer():
    """With every zero point 0 the asymmetric layer is the per-group layer
    (two separate code paths of the oracle)."""
    xb = W.make_random_x(111, 6, 128, "laplace", 0.1)
    a = oracle.quantize_act(xb, 16)
    wb = W.make_w(1, 0, rows=7)[:, :128].copy()
    wq, sw = oracle.quantize_weight(wb)
    y0, _ = oracle.linear_f64(a, wq, sw, None)
    a.zeros = np.zeros_like(a.scales, dtype=np.int8)
    y1, _ = oracle.linear_asym_f64(a, wq, sw, None)
    np.testing.assert_allclose(y1, y0, rtol=1e-14, atol=0)
