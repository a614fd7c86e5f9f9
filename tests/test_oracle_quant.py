"""Pins of the oracle's activation quantizer (Eq. 1 + Eq. 2 + right shift) and
weight quantizer (Appendix C, round-to-nearest int4) against a hand-worked
fixture, brute-force searches, numpy's fp16 conversion, round-trip bounds and
metamorphic relations."""
import os

import numpy as np
import pytest

import oracle
import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _bf16(a):
    return W.to_bf16_bits(np.asarray(a, np.float64))


def _f32(bits):
    return W.bf16_bits_to_f32(bits)


def _f16_val(bits):
    return np.asarray(bits, np.uint16).view(np.float16).astype(np.float32)


def test_worked_group_fixture():
    x = np.zeros(64)
    expect_c = np.zeros(64, np.int8)
    expect_q = np.zeros(64, np.int32)
    flags = None
    scale_bits = None
    with open(os.path.join(GOLDEN, "worked_group.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            parts = line.split()
            if parts[0] == "flags":
                flags = [int(v) for v in parts[1:]]
            elif parts[0] == "c":
                expect_c[int(parts[1])] = int(parts[2])
            elif parts[0] == "scale_bits":
                scale_bits = int(parts[1])
            else:
                k = int(parts[0])
                x[k] = float(parts[1])
                expect_q[k] = int(parts[2])
    a = oracle.quantize_act(_bf16(x[None, :]), lzs_group=16)
    assert int(a.scales[0, 0]) == scale_bits
    np.testing.assert_array_equal(a.q8[0].astype(np.int32), expect_q)
    assert list(a.flags[0]) == flags
    np.testing.assert_array_equal(a.c[0], expect_c)
    assert a.zeros[0, 0] == 0


def _x_sample(seed, M=48, K=256, kind="laplace", scale=0.1):
    return W.make_random_x(seed, M, K, kind, scale)


@pytest.mark.parametrize("lzs_group", [1, 8, 16, 32, 64])
def test_stage1_scale_and_codes_by_search(lzs_group):
    """Scale: fp16(max|x| / 127) via numpy's conversion; codes: the nearest
    level to fp32(x * (1/s)) found by searching all 255 levels (ties to even)."""
    xb = _x_sample(21 + lzs_group, M=12, K=128, kind="t3", scale=0.05)
    a = oracle.quantize_act(xb, lzs_group=lzs_group)
    x = _f32(xb)
    levels = np.arange(-127, 128, dtype=np.float64)
    for m in range(x.shape[0]):
        for g in range(x.shape[1] // 64):
            xg = x[m, 64 * g:64 * g + 64]
            alpha = np.float32(np.abs(xg).max())
            with np.errstate(over="ignore"):
                s16 = np.array([alpha / np.float32(127.0)], np.float32).astype(np.float16)
            bits = int(s16.view(np.uint16)[0])
            if bits == 0x7C00:
                bits = 0x7BFF
            assert int(a.scales[m, g]) == bits
            s = np.float32(s16[0])
            r = np.float32(0.0) if s == 0 else np.float32(1.0) / s
            p = (xg * r).astype(np.float32).astype(np.float64)
            dist = np.abs(p[:, None] - levels[None, :])
            best = dist.min(axis=1)
            q_ref = []
            for i in range(64):
                cands = levels[dist[i] == best[i]]
                if cands.size > 1:                  # a tie: take the even level
                    cands = cands[cands % 2 == 0]
                q_ref.append(cands[0])
            q_ref = np.array(q_ref)
            np.testing.assert_array_equal(a.q8[m, 64 * g:64 * g + 64], q_ref.astype(np.int8))


def test_half_step_round_trip_and_group_max():
    """|x - s q| <= s/2 (midtread quantizer, Appendix A) up to the fp32
    rounding of x * (1/s) (relative 2^-23 of |x/s| <= 127); the group maximum
    maps to +-127 when the fp16 scale is normal."""
    xb = _x_sample(31, M=64, K=512, kind="laplace", scale=0.2)
    a = oracle.quantize_act(xb, lzs_group=16)
    x = _f32(xb).astype(np.float64)
    s = np.repeat(_f16_val(a.scales).astype(np.float64), 64, axis=1)
    err = np.abs(x - s * a.q8)
    assert np.all(err <= s * (0.5 + 127 * 2.0 ** -22))
    normal = _f16_val(a.scales) >= 2.0 ** -14
    xg = x.reshape(x.shape[0], -1, 64)
    qg = a.q8.reshape(a.q8.shape[0], -1, 64)
    idx = np.abs(xg).argmax(axis=2)
    qmax = np.take_along_axis(qg, idx[..., None], axis=2)[..., 0]
    assert np.all(np.abs(qmax[normal]) == 127)
    # hence some subgroup of every non-zero group has FLAG 4
    fg = a.flags.reshape(a.flags.shape[0], -1, 4)
    assert np.all(fg.max(axis=2)[normal] == 4)


def test_combined_bound_and_lossless_invariant():
    xb = _x_sample(41, M=64, K=512, kind="t3", scale=0.05)
    for gs in (8, 16, 32, 64):
        a = oracle.quantize_act(xb, lzs_group=gs)
        x = _f32(xb).astype(np.float64)
        s = np.repeat(_f16_val(a.scales).astype(np.float64), 64, axis=1)
        f = np.repeat(a.flags.astype(np.int64), gs, axis=1)
        d = a.decoded()
        # |x - s d| <= s/2 + s (2^FLAG - 1)   (triangle inequality, Appendix A)
        assert np.all(np.abs(x - s * d) <= s * (0.5 + 127 * 2.0 ** -22) + s * ((1 << f) - 1))
        # an element is kept exactly iff its magnitude is a multiple of 2^FLAG
        q = a.q8.astype(np.int64)
        np.testing.assert_array_equal(d == q, (np.abs(q) % (1 << f)) == 0)
        # a subgroup whose magnitudes all fit 3 bits has FLAG 0 and is lossless
        qs = np.abs(q).reshape(q.shape[0], -1, gs).max(axis=2)
        np.testing.assert_array_equal(a.flags == 0, qs <= 7)
        assert np.all(np.abs(a.c) <= 7)


def test_sign_symmetry():
    xb = _x_sample(51, M=32, K=256)
    a = oracle.quantize_act(xb, lzs_group=16)
    b = oracle.quantize_act(xb ^ np.uint16(0x8000), lzs_group=16)
    np.testing.assert_array_equal(b.c, -a.c)
    np.testing.assert_array_equal(b.q8, -a.q8)
    np.testing.assert_array_equal(b.flags, a.flags)
    np.testing.assert_array_equal(b.scales, a.scales)


def test_power_of_two_scaling_is_equivariant():
    xb = _x_sample(61, M=32, K=256, scale=0.5)
    a = oracle.quantize_act(xb, lzs_group=16)
    for k in (-3, -1, 1, 4):
        xk = W.to_bf16_bits(_f32(xb).astype(np.float64) * 2.0 ** k)
        b = oracle.quantize_act(xk, lzs_group=16)
        ok = (_f16_val(a.scales) >= 2.0 ** -14) & (_f16_val(b.scales) >= 2.0 ** -14)
        assert ok.all()
        np.testing.assert_array_equal(b.c, a.c)
        np.testing.assert_array_equal(b.flags, a.flags)
        np.testing.assert_array_equal(_f16_val(b.scales), _f16_val(a.scales) * np.float32(2.0 ** k))


def test_permutations():
    xb = _x_sample(71, M=8, K=128)
    a = oracle.quantize_act(xb, lzs_group=16)
    g = np.random.Generator(np.random.PCG64(72))
    # permuting elements inside one subgroup permutes its codes
    perm = g.permutation(16)
    xp = xb.copy()
    xp[:, 16:32] = xb[:, 16:32][:, perm]
    b = oracle.quantize_act(xp, lzs_group=16)
    np.testing.assert_array_equal(b.c[:, 16:32], a.c[:, 16:32][:, perm])
    np.testing.assert_array_equal(b.flags, a.flags)
    # permuting whole subgroups inside a group permutes the flags
    xs = xb.copy()
    xs[:, 0:16], xs[:, 48:64] = xb[:, 48:64], xb[:, 0:16]
    c = oracle.quantize_act(xs, lzs_group=16)
    assert list(c.flags[0, :4]) == [a.flags[0, 3], a.flags[0, 1], a.flags[0, 2], a.flags[0, 0]]


def test_zero_groups_and_tiny_scales():
    x = np.zeros((3, 128))
    x[1, 64:] = 1e-9          # fp16(alpha/127) underflows to 0
    x[2, :64] = 1e-5          # subnormal fp16 scale (1e-5 / 127 ~ 7.9e-8)
    a = oracle.quantize_act(_bf16(x), lzs_group=16)
    assert np.all(a.scales[0] == 0) and np.all(a.c[0] == 0) and np.all(a.flags[0] == 0)
    assert a.scales[1, 1] == 0 and np.all(a.c[1] == 0)
    assert 0 < a.scales[2, 0] < 0x0400


def test_full_group_lzs_degenerates_to_top_three_bits():
    xb = _x_sample(81, M=16, K=256)
    a = oracle.quantize_act(xb, lzs_group=64)
    assert np.all(a.flags == 4)
    q = a.q8.astype(np.int32)
    np.testing.assert_array_equal(a.decoded(), np.sign(q) * (np.abs(q) & 0x70))


def test_pack_unpack_layout():
    g = np.random.Generator(np.random.PCG64(91))
    c = g.integers(-7, 8, size=(5, 64)).astype(np.int8)
    codes = oracle.pack_codes(c)
    assert codes.shape == (1, 5, 32)
    np.testing.assert_array_equal(oracle.unpack_codes(codes, 5, 64), c)
    c2 = g.integers(-7, 8, size=(3, 192)).astype(np.int8)
    np.testing.assert_array_equal(oracle.unpack_codes(oracle.pack_codes(c2), 3, 192), c2)
    # element 8j+i -> nibble (i/2) + 4(i%2) of little-endian word j; sign-magnitude
    c1 = np.zeros((2, 128), np.int8)
    c1[1, 64 + 1] = -3     # row 1, group 1, odd element 1 -> nibble 4 (byte 2): 0xB
    c1[1, 64 + 6] = 5      # even element 6 -> nibble 3 (byte 1, high nibble): 0x5
    c1[0, 8 + 2] = 7       # row 0, group 0, word 1, element 2 -> nibble 1 of word 1
    out = oracle.pack_codes(c1)
    # K-group-major: (group 1, row 1) is the fourth 32-byte block
    assert list(out[1, 1, :4]) == [0x00, 0x50, 0x0B, 0x00]
    assert list(out[0, 0, 4:8]) == [0x70, 0x00, 0x00, 0x00]
    assert out.sum() == 0x50 + 0x0B + 0x70


def test_weight_quantizer():
    w = W.make_w(1, 0, rows=40)
    wq, sw = oracle.quantize_weight(w)
    wf = _f32(w).astype(np.float64)
    s = np.repeat(_f16_val(sw).astype(np.float64), 64, axis=1)
    assert np.all(np.abs(wq) <= 7)
    assert np.all(np.abs(wf - s * wq) <= s * (0.5 + 7 * 2.0 ** -22))
    # the group maximum maps to +-7
    wg = wf.reshape(40, -1, 64)
    qg = wq.reshape(40, -1, 64)
    idx = np.abs(wg).argmax(axis=2)
    assert np.all(np.abs(np.take_along_axis(qg, idx[..., None], axis=2)) == 7)
    # scale = fp16(max|w| / 7) through numpy's conversion
    beta = np.abs(W.bf16_bits_to_f32(w)).reshape(40, -1, 64).max(axis=2)
    ref = (beta / np.float32(7.0)).astype(np.float32).astype(np.float16).view(np.uint16)
    np.testing.assert_array_equal(sw, ref)
    # sign symmetry
    wq2, sw2 = oracle.quantize_weight(w ^ np.uint16(0x8000))
    np.testing.assert_array_equal(wq2, -wq)
    np.testing.assert_array_equal(sw2, sw)


def test_memory_ratio_fixture():
    vals = {}
    with open(os.path.join(GOLDEN, "memory_ratio.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            k, v = line.split()
            vals[k] = float(v)
    ratio = 16.0 / (vals["value_bits"] + vals["scale_bits"] / vals["group"])
    assert round(ratio, 1) == vals["printed_ratio"]
    # the oracle's storage: K/2 code bytes + K/64 fp16 scales per weight row
    K = 1152
    w = W.make_w(1, 0, rows=2)
    wq, sw = oracle.quantize_weight(w)
    stored_bits = (K // 2 + 2 * sw.shape[1]) * 8
    assert round(16 * K / stored_bits, 1) == vals["printed_ratio"]
