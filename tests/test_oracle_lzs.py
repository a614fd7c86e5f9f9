"""Pins of the oracle's Stage 2 (leading-zero suppression, Eq. 2 and the right
shift of Section 3) by brute force over every int8 input and by the closed-form
bounds that Appendix A prints."""
import os

import numpy as np

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _appendix_a():
    bounds, keys = {}, {}
    with open(os.path.join(GOLDEN, "appendix_a_bounds.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            a, b = line.split()
            if a.isdigit():
                bounds[int(a)] = int(b)
            else:
                keys[a] = float(b)
    return bounds, keys


def _single(q):
    f, c = oracle.lzs_subgroup(np.array([q], np.int8))
    return f, int(c[0])


def test_all_int8_values_single_element_subgroups():
    """G_s = 1: each value's own bit length sets its shift (Appendix A setup)."""
    bounds, keys = _appendix_a()
    lossless = 0
    max_err = {}
    total = 0
    for q in range(-127, 128):
        f, c = _single(q)
        m = abs(q)
        h = m.bit_length()
        d = c * (1 << f)
        err = abs(q - d)
        # the sign is kept and the magnitude is truncated toward zero
        assert (c == 0) or (np.sign(c) == np.sign(q))
        assert abs(d) <= m < abs(d) + (1 << f)
        assert err <= bounds[h]
        max_err[h] = max(max_err.get(h, 0), err)
        if q >= 0:
            total += err
        lossless += (err == 0)
    # Appendix A: for H >= 4 the bound 2^(H-3) - 1 is attained (e.g. m = 2^H - 1)
    for h in range(4, 8):
        assert max_err[h] == bounds[h] == 2 ** (h - 3) - 1
        f, c = _single(2 ** h - 1)
        assert (2 ** h - 1) - c * (1 << f) == bounds[h]
    for h in range(0, 4):
        assert max_err.get(h, 0) == 0
    assert max(bounds.values()) == keys["worst_case"]
    # values with a sign and at most three significant magnitude bits are lossless
    assert lossless == 47
    assert total == 620


def test_lossless_iff_at_most_three_significant_bits():
    for q in range(-127, 128):
        m = abs(q)
        sig = 0 if m == 0 else m.bit_length() - (len(bin(m)) - len(bin(m).rstrip("0")))
        f, c = _single(q)
        assert (c * (1 << f) == q) == (sig <= 3)


def test_minus_128_saturates_to_flag_four():
    f, c = _single(-128)
    assert f == 4 and c == -7


def test_truncation_toward_zero_not_arithmetic_shift():
    # q = -5 in a subgroup with FLAG 1 (another member has bit length 4)
    f, c = oracle.lzs_subgroup(np.array([-5, 9], np.int8))
    assert f == 1
    assert list(c) == [-2, 4]          # -5 -> -(5 >> 1) = -2, decoded -4 (not -6)


def test_subgroup_flag_brute_force_and_or_equals_max():
    g = np.random.Generator(np.random.PCG64(11))
    for n in (2, 8, 16, 32, 64):
        for _ in range(300):
            scale = int(g.integers(0, 8))
            q = g.integers(-(2 ** scale) + 1, 2 ** scale, size=n).clip(-127, 127).astype(np.int8)
            f, c = oracle.lzs_subgroup(q)
            mags = np.abs(q.astype(np.int32))
            # smallest shift that brings every magnitude under 8
            f_ref = min(s for s in range(8) if (mags >> s).max() <= 7)
            assert f == f_ref
            # OR aggregation and max aggregation give the same bit length
            assert int(mags.max()).bit_length() == int(np.bitwise_or.reduce(mags)).bit_length()
            np.testing.assert_array_equal(np.abs(c.astype(np.int32)), mags >> f)
            np.testing.assert_array_equal(np.sign(c) * (c != 0), np.sign(q) * (c != 0))


def test_expected_error_formula_matches_brute_force():
    """Appendix A: E[E_LZS] = s8 * sum_{k=4..7} P_k (2^(k-3) - 1) is the mean of
    the per-magnitude bound; for magnitudes at the top of each bit length the
    bound is the exact error, so the mean error equals the formula there."""
    bounds, keys = _appendix_a()
    mags = [2 ** h - 1 for h in range(4, 8)]
    P = {h: 0.25 for h in range(4, 8)}
    errs = []
    for m in mags:
        f, c = _single(m)
        errs.append(m - c * (1 << f))
    assert np.mean(errs) == sum(P[k] * (2 ** (k - 3) - 1) for k in range(4, 8))
    # worst case reduction: 15 * P(|J| >= 8) < 7.5  <=>  P(|J| >= 8) < 1/2
    assert keys["worst_case"] * keys["prob_threshold"] == keys["threshold_s8"]
    assert keys["threshold_s8"] == (keys["s4_over_s8"] - 1) / 2
