"""Pins of the oracle's scalar building blocks against library routines and
closed forms (none of them re-types the oracle's own code).

- fp16 encode/decode against numpy's IEEE binary16 conversion (Appendix C:
  16-bit scales), with overflow saturating to 65504.
- round-half-to-even against numpy.rint (tie rule of the rounding in Eq. 1).
- clz against Python's int.bit_length (Eq. 2's clz on a 32-bit word).
- the FLAG table of Eq. 2 from a hand-worked fixture.
- GELU-tanh against torch's implementation in float64.
"""
import math
import os

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def _np_f16_sat(v: np.float32) -> int:
    with np.errstate(over="ignore"):
        h = np.array([v], np.float32).astype(np.float16)
    bits = int(h.view(np.uint16)[0])
    if (bits & 0x7FFF) == 0x7C00:          # overflow -> saturate
        bits = (bits & 0x8000) | 0x7BFF
    return bits


def test_f16_encode_matches_numpy_random():
    g = _rng(1)
    e = g.uniform(-30, 17, size=4000)
    v = (np.sign(g.uniform(-1, 1, size=e.size)) * np.exp2(e)).astype(np.float32)
    for x in v:
        assert oracle.f32_to_f16_rne_sat(float(x)) == _np_f16_sat(x), float(x)


def test_f16_encode_ties_and_edges():
    vals = []
    for e in range(-24, 16):
        base = 2.0 ** e
        for frac in (0.0, 2.0 ** -11, 3 * 2.0 ** -11, 5 * 2.0 ** -11, 2.0 ** -12, 1 - 2.0 ** -12,
                     0.5 + 2.0 ** -11):
            vals.append(base * (1 + frac))
    vals += [65504.0, 65519.0, 65519.99, 65520.0, 65536.0, 1e6, 3e38,
             2.0 ** -25, 3 * 2.0 ** -26, 2.0 ** -26, 2.0 ** -14 * (1 - 2.0 ** -11)]
    for x in vals:
        for s in (1.0, -1.0):
            f = np.float32(s * x)
            assert oracle.f32_to_f16_rne_sat(float(f)) == _np_f16_sat(f), float(f)


def test_f16_decode_all_finite_patterns():
    bits = np.arange(0, 1 << 16, dtype=np.uint32).astype(np.uint16)
    ref = bits.view(np.float16).astype(np.float32)
    finite = np.isfinite(ref)
    got = np.array([oracle.f16_to_f32(int(b)) for b in bits[finite][::7]], np.float32)
    np.testing.assert_array_equal(got, ref[finite][::7])


def test_bf16_decode():
    g = _rng(2)
    bits = g.integers(0, 1 << 16, size=2000).astype(np.uint16)
    ref = (bits.astype(np.uint32) << 16).view(np.float32)
    for b, r in zip(bits, ref):
        if np.isfinite(r):
            assert oracle.bf16_to_f32(int(b)) == r


def test_rne_matches_rint():
    g = _rng(3)
    v = np.concatenate([g.uniform(-300, 300, 3000),
                        np.arange(-260, 261) + 0.5,
                        np.arange(-260, 261).astype(np.float64),
                        np.arange(-10, 11) + 0.4999999,
                        np.arange(-10, 11) + 0.5000001])
    for x in v:
        assert oracle.rne(float(x)) == float(np.rint(x)), x


def test_clz_matches_bitlength():
    g = _rng(4)
    vals = [0, 1, 2, 3, 0x7FFFFFFF, 0x80000000, 0xFFFFFFFF] + list(g.integers(0, 1 << 32, 500))
    vals += [1 << b for b in range(32)]
    for v in vals:
        assert oracle.clz32(int(v)) == 32 - int(v).bit_length()


def _load_flag_table():
    rows = []
    with open(os.path.join(GOLDEN, "eq2_flag_table.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            lo, hi, clz, flag = map(int, line.split())
            rows.append((lo, hi, clz, flag))
    return rows


def test_eq2_flag_table_golden():
    rows = _load_flag_table()
    covered = set()
    for lo, hi, clz, flag in rows:
        for m in range(lo, hi + 1):
            assert oracle.clz32(m) == clz
            assert oracle.lzs_flag(m) == flag
            covered.add(m)
    assert covered == set(range(128))


def test_flag_is_smallest_shift_that_fits_three_bits():
    # Brute-force characterization: FLAG is the least f >= 0 with m >> f <= 7,
    # i.e. "preserve the bottom 3 bits when mag < 8" (Section 3).
    for m in range(128):
        f = min(f for f in range(8) if (m >> f) <= 7)
        assert oracle.lzs_flag(m) == f
        assert f <= 4


def test_gelu_tanh_matches_torch():
    torch = pytest.importorskip("torch")
    xs = np.linspace(-8, 8, 401)
    ref = torch.nn.functional.gelu(torch.tensor(xs, dtype=torch.float64), approximate="tanh").numpy()
    got = np.array([oracle.gelu_tanh(float(x)) for x in xs])
    np.testing.assert_allclose(got, ref, rtol=1e-14, atol=1e-15)
    # odd-part identity of GELU: gelu(x) - gelu(-x) = x
    for x in (0.3, 1.7, 4.2):
        assert math.isclose(oracle.gelu_tanh(x) - oracle.gelu_tanh(-x), x, rel_tol=1e-14)


def test_bf16_rounding_of_double():
    g = _rng(5)
    v = g.standard_normal(3000) * np.exp2(g.uniform(-20, 20, 3000))
    for x in v:
        m, e = math.frexp(float(x))                 # x = m * 2^e, |m| in [0.5, 1)
        ref = np.float64(np.rint(m * 256.0)) * 2.0 ** (e - 8)   # 8 significant bits
        ref_bits = int((np.array([ref], np.float32).view(np.uint32)[0]) >> 16)
        assert oracle.f64_to_bf16_rne(float(x)) == ref_bits
