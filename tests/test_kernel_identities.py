"""Exhaustive checks of the arithmetic identities the HIP quantizer relies on
to skip work while staying bit-exact with the definition of Eq. 1 (symmetric
reading): s = fp16_rne(fp32(alpha / 127)), r = fp32(1 / s),
q = min(rne(fp32(|x| * r)), 127).

Both identities are checked over every finite positive bf16 group maximum
alpha (the whole input domain of the scale).  The GPU side of the same facts
(including the hardware reciprocal plus one Newton step equalling 1/s) is
exercised bit-exactly against the oracle by the GPU parity test that makes
every bf16 magnitude a group maximum.
"""
import numpy as np


def _all_alpha():
    bits = np.arange(1, 0x7F80, dtype=np.uint32) << 16
    return bits.view(np.float32)


def test_scale_by_reciprocal_constant_equals_division():
    a = _all_alpha()
    with np.errstate(over="ignore"):
        by_div = (a / np.float32(127)).astype(np.float16).view(np.uint16)
        by_mul = (a * np.float32(1.0 / 127.0)).astype(np.float16).view(np.uint16)
    np.testing.assert_array_equal(by_div, by_mul)


def test_code_never_exceeds_127_for_normal_unsaturated_scales():
    a = _all_alpha()
    with np.errstate(over="ignore"):
        s16 = np.minimum((a / np.float32(127)).astype(np.float16).view(np.uint16), 0x7BFF)
    s = s16.view(np.float16).astype(np.float32)
    normal = (s16 >= 0x0400) & (s16 < 0x7BFF)
    r = (np.float32(1) / s[normal]).astype(np.float32)
    q = np.rint((a[normal] * r).astype(np.float32))
    assert normal.sum() == 30 * 128          # 30 binades of bf16 alpha
    assert q.max() == 127.0
    # and the clamp does bind for some subnormal scales, so it cannot be dropped there
    sub = (s16 > 0) & (s16 < 0x0400)
    r_sub = (np.float32(1) / s[sub]).astype(np.float32)
    assert np.rint((a[sub] * r_sub).astype(np.float32)).max() > 127.0
