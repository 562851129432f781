"""Pins for the oracle's quantizer, packing and weight preparation.

The quantizer is checked against exact rational arithmetic (fractions), the
closed forms the paper's equations imply (Eq. 2-3 error bound, one-hot rows,
scale invariance) and the statistical laws it states (Eq. 17 uniform-noise
energy, Eq. 22 step ratio between 4 and 8 bits).
"""

from fractions import Fraction

import numpy as np
import pytest

from oracle.hadamard import rotate_rows, hadamard
from oracle.quant import (quantize_rows, pack_int4, unpack_int4, qmax_for_bits,
                          rotate_quant_ref, prepare_weights_ref, dequant_rows)


def _round_to_f32(fr):
    """Correctly rounded (nearest-even) fp32 value of a Fraction (normal range)."""
    if fr == 0:
        return 0.0
    sign = -1 if fr < 0 else 1
    a = abs(fr)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    # a in [2^e, 2^(e+1)); fp32 has 24 significant bits.
    ulp = Fraction(2) ** (e - 23)
    q, r = divmod(a, ulp)
    if r * 2 > ulp or (r * 2 == ulp and q % 2 == 1):
        q += 1
    return sign * float(q * ulp)


def _rne_int(fr):
    """Round a Fraction to the nearest integer, ties to even."""
    fl = fr.numerator // fr.denominator
    rem = fr - fl
    if rem > Fraction(1, 2) or (rem == Fraction(1, 2) and fl % 2 == 1):
        fl += 1
    return fl


def _brute_force_quantize(row, bits):
    """Exact-rational quantizer of one fp32 row: s = fl32(a/qmax), t = fl32(y/s)."""
    qmax = qmax_for_bits(bits)
    a = max(abs(Fraction(float(v))) for v in row)
    if a == 0:
        return [0] * len(row), 0.0
    s = _round_to_f32(a / qmax)
    codes = []
    for v in row:
        t = _round_to_f32(Fraction(float(v)) / Fraction(s))
        c = _rne_int(Fraction(t))
        codes.append(max(-(1 << (bits - 1)), min((1 << (bits - 1)) - 1, c)))
    return codes, s


@pytest.mark.parametrize("bits", [4, 8])
def test_quantizer_matches_exact_rational(bits):
    rng = np.random.default_rng(bits)
    y = (rng.standard_normal((6, 64)) * rng.uniform(0.01, 100, (6, 1))).astype(np.float32)
    y[2, 7] = -y[2].max() * 3   # negative absmax
    codes, scales = quantize_rows(y, bits)
    for m in range(y.shape[0]):
        bc, bs = _brute_force_quantize(y[m], bits)
        assert float(scales[m]) == bs
        assert codes[m].tolist() == bc


def test_rne_tie_cases():
    # Round-half-to-even on exact ties (Eq. 2 rounding; ties pinned to even).
    y = np.array([[7.0, 0.5, 1.5, 2.5, -0.5, -1.5, -2.5, 3.5]], dtype=np.float32)
    codes, s = quantize_rows(y, 4)          # absmax 7 -> s = 1 exactly
    assert float(s[0]) == 1.0
    assert codes[0].tolist() == [7, 0, 2, 2, 0, -2, -2, 4]


@pytest.mark.parametrize("bits", [4, 8])
def test_code_range_and_absmax_hits_qmax(bits):
    rng = np.random.default_rng(100 + bits)
    y = (rng.standard_t(3, size=(64, 512)) * 10).astype(np.float32)
    codes, scales = quantize_rows(y, bits)
    qmax = qmax_for_bits(bits)
    assert np.abs(codes.astype(np.int64)).max() <= qmax
    assert np.all(np.abs(codes.astype(np.int64)).max(axis=1) == qmax)
    assert codes.min() >= -qmax      # the clamp never binds at -2^(b-1)


@pytest.mark.parametrize("bits", [4, 8])
def test_dequant_error_bound(bits):
    # Eq. 3: |e| = |y - Q_b(y)| <= s/2, up to the fp32 rounding of the quotient
    # (relative 2^-24 of |t| <= qmax, well inside 2^-20 * s).
    rng = np.random.default_rng(200 + bits)
    y = (rng.standard_normal((32, 1024)) * rng.uniform(1e-3, 1e3, (32, 1))).astype(np.float32)
    codes, scales = quantize_rows(y, bits)
    err = np.abs(y.astype(np.float64) - dequant_rows(codes, scales))
    bound = scales.astype(np.float64)[:, None] * (0.5 + 2.0 ** -20)
    assert np.all(err <= bound)


@pytest.mark.parametrize("bits", [4, 8])
def test_one_hot_gives_all_qmax(bits):
    # Closed form: a one-hot token rotates to a row of +-1, so s = 1/qmax
    # (rounded) and every code is +-qmax with the sign of the Hadamard row.
    h = 256
    x = np.zeros((2, h), dtype=np.float16)
    x[0, 3] = 1
    x[1, 200] = -2
    codes, scales = rotate_quant_ref(x, h, bits)
    c = unpack_int4(codes) if bits == 4 else codes
    H = hadamard(h)
    qmax = qmax_for_bits(bits)
    assert np.array_equal(c[0].astype(np.int64), qmax * H[3])
    assert np.array_equal(c[1].astype(np.int64), -qmax * H[200])
    assert float(scales[0]) == float(np.float32(1) / np.float32(qmax))
    assert float(scales[1]) == float(np.float32(2) / np.float32(qmax))


def test_zero_row():
    x = np.zeros((3, 256), dtype=np.float16)
    x[1, 5] = 0.25
    for bits in (4, 8):
        codes, scales = rotate_quant_ref(x, 256, bits)
        assert scales[0] == 0 and scales[2] == 0 and scales[1] > 0
        c = unpack_int4(codes) if bits == 4 else codes
        assert np.all(c[0] == 0) and np.all(c[2] == 0)


@pytest.mark.parametrize("bits", [4, 8])
def test_power_of_two_scale_invariance(bits):
    rng = np.random.default_rng(7)
    x = rng.standard_normal((8, 512)).astype(np.float16)
    c0, s0 = rotate_quant_ref(x, 512, bits)
    for e in (-3, 2, 5):
        c1, s1 = rotate_quant_ref((x.astype(np.float32) * 2.0 ** e).astype(np.float16), 512, bits)
        assert np.array_equal(c0, c1)
        assert np.array_equal(s1, (s0 * np.float32(2.0 ** e)).astype(np.float32))


@pytest.mark.parametrize("h", [256, 1024, 4096])
def test_unnormalised_equals_orthonormal_codes_for_h_power_of_4(h):
    # For h = 4^j the orthonormal R = B / sqrt(h) is B times a power of two,
    # so quantizing x B or x B / sqrt(h) gives the same codes.
    rng = np.random.default_rng(h)
    x = (rng.standard_normal((4, h)) * 3).astype(np.float16)
    y = rotate_rows(x, h)
    yn = (y / np.float32(np.sqrt(h))).astype(np.float32)
    for bits in (4, 8):
        assert np.array_equal(quantize_rows(y, bits)[0], quantize_rows(yn, bits)[0])


def test_pack_unpack_all_bytes():
    b = np.arange(256, dtype=np.uint8)[None, :]
    codes = unpack_int4(b)
    assert codes.shape == (1, 512)
    lo, hi = codes[0, 0::2], codes[0, 1::2]
    for v in range(256):
        l, u = v & 0xF, v >> 4
        assert lo[v] == (l - 16 if l >= 8 else l)
        assert hi[v] == (u - 16 if u >= 8 else u)
    assert np.array_equal(pack_int4(codes), b)


def test_pack_layout_low_nibble_even_k():
    c = np.array([[1, -1, -8, 7]], dtype=np.int8)
    assert pack_int4(c).tolist() == [[0xF1, 0x78]]
    with pytest.raises(ValueError):
        pack_int4(np.array([[8, 0]]))


def test_step_ratio_eq22():
    # Eq. 22: going from 4 to 8 bits shrinks the step by qmax4/qmax8 = 7/127 and
    # the error variance by about its square.
    rng = np.random.default_rng(22)
    x = rng.standard_normal((256, 1024)).astype(np.float16)
    y = rotate_rows(x, 1024)
    mse = {}
    for bits in (4, 8):
        c, s = quantize_rows(y, bits)
        mse[bits] = np.mean((y - dequant_rows(c, s)) ** 2)
        if bits == 8:
            s8 = s
        else:
            s4 = s
    np.testing.assert_allclose(s8 / s4, 7 / 127, rtol=1e-6)
    assert 0.8 < (mse[8] / mse[4]) / (7 / 127) ** 2 < 1.25


def test_uniform_noise_energy_eq17():
    # Eq. 17 (uniform noise model): E||eps||^2 = d s^2 / 12 at 8 bits, where
    # the grid is fine relative to the data.
    rng = np.random.default_rng(17)
    x = rng.standard_normal((128, 2048)).astype(np.float16)
    y = rotate_rows(x, 2048)
    c, s = quantize_rows(y, 8)
    err2 = ((y - dequant_rows(c, s)) ** 2).sum(axis=1)
    ratio = err2 / (2048 * s.astype(np.float64) ** 2 / 12)
    assert 0.9 < ratio.mean() < 1.1


def test_prepare_weights_matches_definition():
    rng = np.random.default_rng(3)
    w = (rng.standard_normal((16, 512)) * 0.02).astype(np.float32)
    wp, ws = prepare_weights_ref(w, 512)
    z = rotate_rows(w, 512)
    for n in range(16):
        codes, s = _brute_force_quantize(z[n], 4)
        assert unpack_int4(wp[n:n + 1])[0].tolist() == codes
        assert float(ws[n]) == float(np.float32(np.float32(s) / np.float32(512)))


@pytest.mark.parametrize("bits", [4, 8])
def test_near_tie_quotients_match_exact_rational(bits):
    # Values whose quotient y/s lies within a few fp32 ulps of a half-integer:
    # here fl32(y/s) and cheaper stand-ins (y * fl32(1/s), fma variants) round
    # to different codes, so only the correctly rounded quotient passes.
    rng = np.random.default_rng(300 + bits)
    qmax = qmax_for_bits(bits)
    rows = []
    for _ in range(24):
        a = np.float32(rng.uniform(0.5, 4.0))
        s = np.float32(a / np.float32(qmax))
        vals = [a]
        for k in range(-qmax, qmax):
            centre = np.float32((k + 0.5) * float(s))
            for d in (-2, -1, 0, 1, 2):
                v = centre
                step = np.float32(np.inf) if d > 0 else np.float32(-np.inf)
                for _ in range(abs(d)):
                    v = np.nextafter(v, step)
                if abs(v) <= a:
                    vals.append(v)
        rows.append(vals)
    width = max(len(r) for r in rows)
    y = np.zeros((len(rows), width), dtype=np.float32)
    for i, r in enumerate(rows):
        y[i, :len(r)] = r
    codes, scales = quantize_rows(y, bits)
    for m in range(y.shape[0]):
        bc, bs = _brute_force_quantize(y[m], bits)
        assert float(scales[m]) == bs
        assert codes[m].tolist() == bc


# --------------------------------------------------------------------------
# the weight byte order of the W4A8 GEMM (a storage order: same codes)
# --------------------------------------------------------------------------
def test_a8order_worked_examples():
    from oracle import pack_int4_a8order, unpack_int4_a8order
    # k = 0..7 -> byte j = k_j | k_{j+4} << 4, worked by hand.
    assert pack_int4_a8order(np.arange(8)[None, :]).tolist() == [[0x40, 0x51, 0x62, 0x73]]
    # Negative codes are 4-bit two's complement: -8 -> 8, -1 -> 15, -2 -> 14.
    c = np.array([[-8, -1, 7, -2, 1, -8, 0, 3]])
    assert pack_int4_a8order(c).tolist() == [[0x18, 0x8F, 0x07, 0x3E]]
    assert unpack_int4_a8order(np.array([[0x18, 0x8F, 0x07, 0x3E]], np.uint8)).tolist() == c.tolist()


def test_a8order_round_trip_and_gemm_invariance():
    from oracle import pack_int4_a8order, unpack_int4_a8order
    rng = np.random.default_rng(41)
    w = rng.integers(-8, 8, size=(6, 256))
    p = pack_int4_a8order(w)
    assert p.shape == (6, 128) and p.dtype == np.uint8
    assert np.array_equal(unpack_int4_a8order(p), w)
    # Relative to the canonical packing, only the nibbles inside each 4-byte
    # group move: the multiset of nibbles per group is unchanged.
    canon = pack_int4(w)
    for g in range(0, 128, 4):
        a = sorted([b & 15 for b in canon[0, g:g + 4]] + [b >> 4 for b in canon[0, g:g + 4]])
        b = sorted([x & 15 for x in p[0, g:g + 4]] + [x >> 4 for x in p[0, g:g + 4]])
        assert a == b
    # A dot product read through either order is the same integer.
    a8 = rng.integers(-128, 128, size=256)
    assert int(np.dot(a8, unpack_int4_a8order(p)[2].astype(np.int64))) == \
        sum(int(a8[k]) * int(w[2, k]) for k in range(256))
