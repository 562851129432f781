"""Pins of the group-wise 4-bit KV-cache quantizer oracle (Section 4.2, Eq. 1-3).

Each pin is a fact other than the oracle's own formula: values on an exact
grid whose codes are known in advance, the end points of the range, the
Eq. 3 error bound, the uniform-noise energy behind Eq. 17, invariances under
exact shifts and power-of-two scaling, independence of the groups, and the
correctly rounded quotient against exact rational arithmetic.
"""

from fractions import Fraction

import numpy as np
import pytest

from oracle.kv import kv_quant_ref, kv_dequant_ref, pack_u4, unpack_u4
from test_oracle_quant import _round_to_f32, _rne_int


def _f16(a):
    return np.asarray(a, dtype=np.float16)


@pytest.mark.parametrize("group", [16, 128])
def test_exact_grid_gives_known_codes(group):
    # x = m0 + k * 2^e with k covering 0..15: s = 2^e exactly, codes = k and
    # the reconstruction is exact.  Catches 16 levels instead of 15, a missing
    # or mis-signed offset, and a swapped nibble order.
    rng = np.random.default_rng(group)
    T = 6
    k = np.stack([np.resize(rng.permutation(16), group) for _ in range(T * 2)])
    k = k.reshape(T, 2 * group)
    e = rng.integers(-6, 4, size=(T, 2))
    m0 = rng.integers(-40, 40, size=(T, 2)).astype(np.float64) / 4
    x = m0.repeat(group, 1) + k * np.exp2(e).repeat(group, 1)
    x16 = _f16(x)
    assert np.array_equal(x16.astype(np.float64), x)          # the grid is exact in fp16
    codes, s, m = kv_quant_ref(x16, group)
    assert np.array_equal(unpack_u4(codes), k)
    assert np.array_equal(s, np.exp2(e).astype(np.float32))
    assert np.array_equal(m, m0.astype(np.float32))
    assert np.array_equal(kv_dequant_ref(codes, s, m, group), x16)


def test_range_end_points():
    rng = np.random.default_rng(1)
    x = _f16(rng.standard_normal((9, 512)) * rng.uniform(0.01, 300, (9, 1)))
    codes, s, m = kv_quant_ref(x, 128)
    c = unpack_u4(codes).reshape(9, 4, 128)
    g = x.astype(np.float32).reshape(9, 4, 128)
    assert np.all(s > 0)
    assert np.all(c[np.arange(9)[:, None], np.arange(4)[None], g.argmin(2)] == 0)
    assert np.all(c[np.arange(9)[:, None], np.arange(4)[None], g.argmax(2)] == 15)
    assert c.min() >= 0 and c.max() <= 15


def test_error_bound_eq3():
    # |x - xhat| <= s/2 plus the fp32 roundings of x - m, d / s, code * s and
    # the sum, plus the final fp16 rounding.
    rng = np.random.default_rng(2)
    x = rng.standard_normal((64, 1024))
    x[:, 7] *= 500.0                                     # a massive channel
    x16 = _f16(x)
    codes, s, m = kv_quant_ref(x16, 128)
    xhat = kv_dequant_ref(codes, s, m, 128).astype(np.float64)
    xv = x16.astype(np.float64)
    S = np.repeat(s.astype(np.float64), 128, axis=1)
    Mn = np.repeat(m.astype(np.float64), 128, axis=1)
    u = 2.0 ** -24
    bound = S * (0.5 + 4 * u * 16) + 4 * u * (np.abs(Mn) + 15 * S) + 2.0 ** -11 * np.abs(xhat) + 2.0 ** -25
    assert np.all(np.abs(xv - xhat) <= bound)
    # and the step really is the range over 15 intervals
    g = xv.reshape(64, 8, 128)
    np.testing.assert_allclose(s, (g.max(2) - g.min(2)) / 15, rtol=2 ** -22)


def test_uniform_noise_energy():
    # With a step small against the spread, the rounding error is close to
    # uniform on [-s/2, s/2]: mean squared error s^2 / 12 (the model of Eq. 17).
    rng = np.random.default_rng(3)
    x = _f16(rng.uniform(-1, 1, (256, 1024)))
    codes, s, m = kv_quant_ref(x, 128)
    # fp32 reconstruction, so that the fp16 output rounding does not add noise
    q = unpack_u4(codes).reshape(256, 8, 128).astype(np.float64)
    xhat = q * s[..., None].astype(np.float64) + m[..., None].astype(np.float64)
    err = (x.astype(np.float64).reshape(256, 8, 128) - xhat) ** 2
    ratio = err.mean() / np.mean(s.astype(np.float64) ** 2 / 12)
    assert abs(ratio - 1) < 0.05


def test_shift_and_scale_invariance():
    rng = np.random.default_rng(4)
    x = rng.integers(-500, 500, size=(5, 256)).astype(np.float64)
    c0, s0, m0 = kv_quant_ref(_f16(x), 128)
    # an exact shift moves the minimum and keeps the codes and the step
    c1, s1, m1 = kv_quant_ref(_f16(x + 1024), 128)
    assert np.array_equal(c0, c1) and np.array_equal(s0, s1) and np.array_equal(m1, m0 + 1024)
    # power-of-two scaling scales the step and the minimum
    for e in (-8, 3):
        c2, s2, m2 = kv_quant_ref(_f16(x * 2.0 ** e), 128)
        assert np.array_equal(c0, c2)
        assert np.array_equal(s2, s0 * np.float32(2.0 ** e)) and np.array_equal(m2, m0 * np.float32(2.0 ** e))


def test_constant_groups():
    x = np.zeros((3, 256), np.float16)
    x[1, :128] = 3.5
    x[1, 128:] = -70000 / 2
    x[2] = np.float16(6e-8)                               # fp16 subnormal
    codes, s, m = kv_quant_ref(x, 128)
    assert np.all(s == 0) and np.all(codes == 0)
    assert np.array_equal(kv_dequant_ref(codes, s, m, 128), x)


def test_groups_are_independent():
    rng = np.random.default_rng(5)
    x = _f16(rng.standard_normal((4, 512)))
    c0, s0, m0 = kv_quant_ref(x, 128)
    y = x.copy()
    y[2, 300] = np.float16(50.0)                          # group 2 of token 2
    c1, s1, m1 = kv_quant_ref(y, 128)
    changed = np.argwhere(s0 != s1)
    assert changed.tolist() == [[2, 2]]
    u0, u1 = unpack_u4(c0), unpack_u4(c1)
    diff = np.argwhere(u0 != u1)
    assert np.all(diff[:, 0] == 2) and np.all((diff[:, 1] >= 256) & (diff[:, 1] < 384))


def test_quotient_matches_exact_rational():
    rng = np.random.default_rng(6)
    x = _f16(rng.standard_normal((12, 64)) * rng.uniform(1e-3, 1e3, (12, 1)) + rng.normal(0, 5, (12, 1)))
    codes, s, m = kv_quant_ref(x, 32)
    got = unpack_u4(codes)
    for t in range(12):
        for g in range(2):
            vals = [Fraction(float(v)) for v in x[t, 32 * g: 32 * (g + 1)].astype(np.float32)]
            lo = min(vals)
            sc = _round_to_f32(Fraction(_round_to_f32(max(vals) - lo)) / 15)
            assert s[t, g] == sc and m[t, g] == float(lo)
            for j, v in enumerate(vals):
                d = _round_to_f32(v - lo) if v != lo else 0.0
                q = _round_to_f32(Fraction(d) / Fraction(sc)) if d else 0.0
                assert got[t, 32 * g + j] == min(15, max(0, _rne_int(Fraction(q))))


def test_pack_unpack_all_bytes():
    b = np.arange(256, dtype=np.uint8).reshape(1, 256)
    c = unpack_u4(b)
    assert c.min() == 0 and c.max() == 15
    assert np.array_equal(pack_u4(c), b)
    assert np.array_equal(c[0, :4], [0, 0, 1, 0])        # byte 1: low nibble (even element) = 1
    with pytest.raises(ValueError):
        pack_u4(np.array([[16, 0]]))


def test_bad_group():
    with pytest.raises(ValueError):
        kv_quant_ref(np.zeros((2, 200), np.float16), 128)


def test_reconstruction_rounds_twice():
    # xhat = fl16(fl32(fl32(code * s) + m)).  With s = 1 + 2^-23, code 15 and
    # m = 196569 * 2^-24: fl32(15 s) = 15 + 2^-19, the fp32 sum is exactly the
    # fp16 tie 15 + 3 * 2^-8, which rounds to the even 15 + 2^-6.  One rounding
    # of the exact 15 s + m (a fused multiply-add) gives 15 + 12287 * 2^-20 and
    # then 15 + 2^-7.
    s = np.array([[np.float32(1 + 2.0 ** -23)]], dtype=np.float32)
    m = np.array([[np.float32(196569 * 2.0 ** -24)]], dtype=np.float32)
    codes = pack_u4(np.full((1, 16), 15))
    xhat = kv_dequant_ref(codes, s, m, 16)
    assert np.all(xhat == np.float16(15 + 2.0 ** -6))
