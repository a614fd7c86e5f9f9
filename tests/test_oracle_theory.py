"""Statistical pin of the oracle against the error-bound theorem (Section 4.1)
and its derivation (Appendix A), per element (G_s = 1, the derivation's own
setting) and per subgroup (G_s = 16, where the subgroup maximum sets FLAG)."""
import numpy as np
import pytest

import oracle
import workloads as W


def _f16_val(bits):
    return np.asarray(bits, np.uint16).view(np.float16).astype(np.float64)


@pytest.mark.parametrize("cfg,layer", [(1, 0), (2, 0), (3, 0), (3, 3), (5, 0)])
def test_theorem_on_workload_distributions(cfg, layer):
    x = W.make_x(cfg, layer, rows=64)
    xf = W.bf16_bits_to_f32(x).astype(np.float64)
    a = oracle.quantize_act(x, lzs_group=1)
    s8 = np.repeat(_f16_val(a.scales), 64, axis=1)
    nz = s8 > 0
    q = np.abs(a.q8.astype(np.int64))
    d = np.abs(a.decoded().astype(np.int64))
    # Appendix A: per-magnitude truncation error <= 2^(H-3) - 1 (in 8-bit steps)
    H = np.vectorize(lambda m: int(m).bit_length())(q)
    bound = np.where(H >= 4, 2 ** np.maximum(H - 3, 0) - 1, 0)
    assert np.all(q - d <= bound)
    # expected LZS error is at most s8 * sum_k P_k (2^(k-3) - 1) (empirical P_k)
    Pk = np.array([np.mean(H[nz] == k) for k in range(8)])
    e_lzs = np.mean((q - d)[nz])
    assert e_lzs <= sum(Pk[k] * (2 ** (k - 3) - 1) for k in range(4, 8)) + 1e-12
    # worst-case reduction: E_LZS <= 15 P(|J| >= 8)
    p8 = np.mean(q[nz] >= 8)
    assert e_lzs <= 15 * p8 + 1e-12
    # theorem: if P(|J| >= 8) < 1/2, the total error stays below s4/2 = 8 s8
    err = np.abs(xf - s8 * np.sign(a.q8) * d)[nz] / s8[nz]
    if p8 < 0.5:
        assert err.mean() < 8.0


def test_lzs_beats_naive_int4_on_small_values():
    """The random-value study (Section 4.3): on data concentrated near zero
    with a few large values, QuaRTZ keeps the low bits that a direct 4-bit
    min-max quantizer rounds away."""
    g = np.random.Generator(np.random.PCG64(5))
    x = g.laplace(0, 0.05, size=(256, 256))
    x[:, ::97] *= 40
    xb = W.to_bf16_bits(x)
    xf = W.bf16_bits_to_f32(xb).astype(np.float64)
    a = oracle.quantize_act(xb, lzs_group=16)
    s8 = np.repeat(_f16_val(a.scales), 64, axis=1)
    quartz = s8 * a.decoded()
    # naive symmetric INT4 per 64-group: s4 = max|x| / 7
    amax = np.abs(xf).reshape(256, -1, 64).max(axis=2)
    s4 = np.repeat(amax / 7.0, 64, axis=1)
    naive = s4 * np.clip(np.rint(xf / s4), -7, 7)
    small = np.abs(xf) < np.repeat(amax, 64, axis=1) / 16
    assert np.mean(np.abs(xf - quartz)[small]) < np.mean(np.abs(xf - naive)[small])
    assert np.mean(np.abs(xf - quartz)) < np.mean(np.abs(xf - naive))
