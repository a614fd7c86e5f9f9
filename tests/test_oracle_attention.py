"""Pins of the oracle's LZS attention (reading R11 of the attention setting of
the hardware appendix, Table 8): softmax(Q K^T / sqrt(d)) V per head with the
activation quantizer (Eq. 1, Eq. 2) on Q and K along d, on V^T along the
keys and on the binary32 softmax output per query row.

  * the binary32-input quantizer equals the (pinned) bf16 one on values a
    bf16 holds exactly;
  * the softmax against scipy's, and its invariants;
  * scores, the PV product and the whole head against a numpy composition
    that dequantizes the codes itself (c * 2^FLAG * s) and multiplies in
    float64;
  * closed forms: equal scores give every probability the code 127 -> 112 of
    its own group scale, and a dominant key passes 112/127 of its value row.
"""
import numpy as np
import pytest

import oracle
import workloads as W


def dequant(a: oracle.ActQuant) -> np.ndarray:
    """x~ = s * c * 2^FLAG, written out with numpy from the raw fields."""
    M, K = a.c.shape
    f = np.repeat(a.flags.astype(np.int64), a.lzs_group, axis=1)
    s = np.repeat((a.scales.astype(np.uint16)).view(np.float16).astype(np.float64), 64, axis=1)
    return a.c.astype(np.float64) * (2.0 ** f) * s


def rand_bf16(seed, shape, scale=1.0):
    return W.to_bf16_bits(np.random.Generator(np.random.PCG64(seed)).normal(0, scale, shape))


@pytest.mark.parametrize("gs", [8, 16, 32, 64])
def test_f32_quantizer_equals_bf16_quantizer_on_bf16_values(gs):
    xb = rand_bf16(1 + gs, (37, 256), 0.3)
    xb[3, :64] = 0                       # a zero group
    xb[5, 64:128] = W.to_bf16_bits(np.full(64, 1e-7))    # subnormal fp16 scale
    x32 = (xb.astype(np.uint32) << 16).view(np.float32)
    a = oracle.quantize_act(xb, gs)
    b = oracle.quantize_f32(x32, gs)
    np.testing.assert_array_equal(a.c, b.c)
    np.testing.assert_array_equal(a.flags, b.flags)
    np.testing.assert_array_equal(a.scales, b.scales)


def test_softmax_against_scipy_and_invariants():
    from scipy.special import softmax
    rng = np.random.Generator(np.random.PCG64(7))
    S = rng.normal(0, 3, (19, 300))
    P = oracle.softmax_rows(S)
    ref = softmax(S, axis=1).astype(np.float32)
    np.testing.assert_allclose(P, ref, rtol=2 ** -23, atol=0)
    np.testing.assert_allclose(P.astype(np.float64).sum(1), 1.0, atol=1e-6)
    np.testing.assert_array_equal(oracle.softmax_rows(S + 5.0), P)           # shift invariance
    perm = rng.permutation(300)
    np.testing.assert_array_equal(oracle.softmax_rows(S[:, perm]), P[:, perm])


@pytest.mark.parametrize("gs", [8, 16, 32])
def test_scores_and_pv_against_numpy(gs):
    L, d = 96, 128
    qa = oracle.quantize_act(rand_bf16(10, (L, d)), gs)
    ka = oracle.quantize_act(rand_bf16(11, (L + 32, d)), gs)
    S, _ = oracle.attn_scores_f64(qa, ka, 1.0 / np.sqrt(d))
    np.testing.assert_allclose(S, dequant(qa) @ dequant(ka).T / np.sqrt(d), rtol=1e-12, atol=1e-12)
    P = oracle.softmax_rows(S)
    pa = oracle.quantize_f32(P, gs)
    vta = oracle.quantize_act(rand_bf16(12, (d, L + 32)), gs)
    O, _ = oracle.attn_pv_f64(pa, vta)
    np.testing.assert_allclose(O, dequant(pa) @ dequant(vta).T, rtol=1e-12, atol=1e-15)
    rows = np.array([0, 5, L - 1]); cols = np.array([1, 2, d - 1])
    Os, _ = oracle.attn_pv_f64(pa, vta, rows, cols)
    np.testing.assert_allclose(Os, O[rows, cols], rtol=1e-14)


def test_head_against_numpy_composition():
    from scipy.special import softmax
    L, d, gs = 128, 128, 16
    qb, kb, vb = rand_bf16(20, (L, d)), rand_bf16(21, (L, d)), rand_bf16(22, (L, d))
    O, parts = oracle.lzs_attention_f64(qb, kb, vb, gs)
    q = dequant(oracle.quantize_act(qb, gs))
    k = dequant(oracle.quantize_act(kb, gs))
    vt = dequant(oracle.quantize_act(np.ascontiguousarray(vb.T), gs))
    P = softmax(q @ k.T / np.sqrt(d), axis=1).astype(np.float32)
    np.testing.assert_allclose(parts["P"], P, rtol=2 ** -22, atol=0)
    pq = dequant(oracle.quantize_f32(parts["P"], gs))
    np.testing.assert_allclose(O, pq @ vt.T, rtol=1e-12, atol=1e-15)


def test_equal_scores_closed_form():
    """Q = 0: every score is 0 and every probability 1/L; each 64-key group
    of a row holds 64 equal values, so q = 127 for all of them, FLAG = 4 and
    d = 127 >> 4 << 4 = 112: O[i][c] = 112 s16 sum_j V~[j][c] with s16 =
    fp16(fp32(1/L) / 127)."""
    L, d, gs = 256, 128, 16
    qb = np.zeros((L, d), np.uint16)
    kb, vb = rand_bf16(30, (L, d)), rand_bf16(31, (L, d))
    O, parts = oracle.lzs_attention_f64(qb, kb, vb, gs)
    assert (parts["p"].c == 7).all() and (parts["p"].flags == 4).all()
    s16 = float(np.float32(1.0 / L) / np.float32(127.0))
    s16 = float(np.float16(s16))
    assert (parts["p"].scales.view(np.float16).astype(np.float64) == s16).all()
    vt = dequant(parts["vt"])
    np.testing.assert_allclose(O, np.broadcast_to(112 * s16 * vt.sum(1), (L, d)), rtol=1e-12)


def test_dominant_key_passes_its_value_row():
    """One key's score exceeds the others by about 30 (after quantization of
    the keys), so its probability rounds to 1 in binary32: its code is
    127 -> 112 at the group scale fp16(1/127), the others' codes are 0, and
    O[i] = 112 fp16(1/127) V~[j]."""
    L, d, gs = 128, 128, 16
    rng = np.random.Generator(np.random.PCG64(40))
    qb = W.to_bf16_bits(np.tile(rng.normal(0, 1, d), (L, 1)))
    k = rng.normal(0, 0.01, (L, d))
    k[17] = 40.0 * np.sqrt(d) * W.bf16_bits_to_f32(qb[0]) / np.sum(W.bf16_bits_to_f32(qb[0]) ** 2)
    kb = W.to_bf16_bits(k)
    vb = rand_bf16(41, (L, d))
    O, parts = oracle.lzs_attention_f64(qb, kb, vb, gs)
    assert (parts["P"][:, 17].astype(np.float64) > 1 - 1e-12).all()
    c = parts["p"].c
    assert (c[:, 17] == 7).all() and (np.delete(c, 17, axis=1) == 0).all()
    s = float(np.float16(np.float32(parts["P"][0, 17]) / np.float32(127.0)))
    vt = dequant(parts["vt"])
    np.testing.assert_allclose(O, np.broadcast_to(112 * s * vt[:, 17], (L, d)), rtol=1e-12)
