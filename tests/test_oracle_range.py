"""Pins for the range-based (zero-point) quantizer oracle, Eq. 1-3.

Each check is fixed by the definition or by arithmetic, not by retyping the
oracle: exact integer grids the quantizer must reproduce, the error bound of
Eq. 3, zero as an exact level, degenerate rows, and brute-force integer dot
products for the zero-point GEMM.
"""

import numpy as np
import pytest

import workloads
from oracle import (quantize_rows_range, rotate_quant_range_ref, dequant_rows_range,
                    weight_sums_ref, zero_point_acc_ref, qlinear_range_ref, qlinear_acc_ref,
                    unpack_int4, rotate_rows)


def _q(codes, bits):
    """Unsigned levels q from the stored codes c = q - 2^(b-1)."""
    return np.asarray(codes, np.int64) + (1 << (bits - 1))


def test_worked_example():
    # Row (1, -2, 0.5, 3) at 4 bits: range 5 over 15 steps, s = 1/3; the
    # zero point is -(-2) / s = 6; levels 1*3+6 = 9, 0, round(1.5)+6 = 8
    # (half to even), 9+6 = 15.
    codes, s, z = quantize_rows_range(np.array([[1.0, -2.0, 0.5, 3.0]], np.float32), 4)
    assert s[0] == np.float32(5.0) / np.float32(15.0)
    assert z[0] == 6
    assert _q(codes, 4).tolist() == [[9, 0, 8, 15]]


@pytest.mark.parametrize("bits", [4, 8])
def test_exact_integer_grid_is_reproduced(bits):
    # Rows that are exactly s0 * (k - z0) with integer levels k covering 0 and
    # 2^b - 1 and a power-of-two step: the range is exactly s0 (2^b - 1), so
    # the step, the zero point and every level come back exactly.
    rng = np.random.default_rng(3)
    L = (1 << bits) - 1
    for trial in range(50):
        s0 = np.float32(2.0 ** rng.integers(-12, 4))
        z0 = int(rng.integers(1, L))            # zero strictly inside: min < 0 < max
        k = rng.integers(0, L + 1, size=64)
        k[:2] = (0, L)
        k = rng.permutation(k)
        y = (s0 * (k - z0)).astype(np.float32)[None, :]
        codes, s, z = quantize_rows_range(y, bits)
        assert s[0] == s0, trial
        assert z[0] == z0, trial
        assert np.array_equal(_q(codes, bits)[0], k), trial


@pytest.mark.parametrize("bits", [4, 8])
@pytest.mark.parametrize("gen", ["gauss_outliers", "student_t"])
def test_error_bound_and_exact_zero(bits, gen):
    # Eq. 3: |y - Q_b(y)| <= s / 2 for every element (a hair more for the fp32
    # rounding of s and of y / s), including the clamped extremes; values that
    # are exactly 0 reconstruct exactly (zero is a level).
    rng = np.random.default_rng(11 + bits)
    x = getattr(workloads, gen)(rng, 24, 512)
    y = rotate_rows(x, 512)
    y[:, ::37] = 0.0
    codes, s, z = quantize_rows_range(y, bits)
    q = _q(codes, bits)
    assert np.all((q >= 0) & (q <= (1 << bits) - 1))
    assert np.all((z >= 0) & (z <= (1 << bits) - 1))
    rec = dequant_rows_range(codes, s, z, bits)
    err = np.abs(y.astype(np.float64) - rec)
    assert np.all(err <= s[:, None].astype(np.float64) * (0.5 + 2.0 ** -18))
    assert np.all(rec[:, ::37] == 0.0)
    # The row minimum sits on level 0 (RNE is odd, so round(mn/s) + round(-mn/s) = 0).
    amin = np.argmin(y, axis=1)
    assert np.all(q[np.arange(len(q)), amin] == 0)


@pytest.mark.parametrize("bits", [4, 8])
def test_error_energy_matches_uniform_model(bits):
    # Smooth rows: the rounding error is close to uniform on a step, so its
    # mean square is s^2 / 12 (to within sampling noise).
    rng = np.random.default_rng(5)
    y = rng.uniform(-3.0, 5.0, size=(64, 4096)).astype(np.float32)
    codes, s, z = quantize_rows_range(y, bits)
    rec = dequant_rows_range(codes, s, z, bits)
    mse = np.mean((y - rec) ** 2, axis=1)
    ratio = mse / (s.astype(np.float64) ** 2 / 12.0)
    assert np.all(np.abs(ratio - 1.0) < 0.12)


def test_degenerate_rows():
    y = np.zeros((4, 16), np.float32)
    y[1] = 2.5      # positive constant: range [0, 2.5]
    y[2] = -0.75    # negative constant: range [-0.75, 0]
    for bits in (4, 8):
        L = (1 << bits) - 1
        codes, s, z = quantize_rows_range(y, bits)
        q = _q(codes, bits)
        assert s[0] == 0 and z[0] == 0 and np.all(q[0] == 0)
        assert z[1] == 0 and np.all(q[1] == L)
        assert z[2] == L and np.all(q[2] == 0)
        rec = dequant_rows_range(codes, s, z, bits)
        assert np.all(rec[0] == 0)
        assert np.allclose(rec[1], 2.5, rtol=1e-6) and np.allclose(rec[2], -0.75, rtol=1e-6)


def test_weight_sums_brute_force():
    rng = np.random.default_rng(8)
    wp = workloads.random_weight_bytes(rng, 5, 64)
    # Nibbles decoded by hand: low nibble = even k, two's complement.
    expect = []
    for row in wp:
        tot = 0
        for byte in row.tolist():
            for nib in (byte & 0xF, byte >> 4):
                tot += nib - 16 if nib >= 8 else nib
        expect.append(tot)
    assert weight_sums_ref(wp).tolist() == expect


@pytest.mark.parametrize("bits", [4, 8])
def test_zero_point_gemm_brute_force(bits):
    # The corrected accumulator is sum_k (q_k - z) w_k, formed here with
    # Python integers one product at a time from the levels and weights.
    rng = np.random.default_rng(21 + bits)
    M, K, N = 3, 256, 4
    x = workloads.gauss_outliers(rng, M, K)
    codes, s, z = rotate_quant_range_ref(x, 256, bits)
    wp = workloads.random_weight_bytes(rng, N, K)
    c = unpack_int4(codes) if bits == 4 else np.asarray(codes)
    q = _q(c, bits)
    w = unpack_int4(wp)
    got = zero_point_acc_ref(qlinear_acc_ref(codes, bits, wp), z, bits, weight_sums_ref(wp))
    for m in range(M):
        for n in range(N):
            ref = sum((int(q[m, k]) - int(z[m])) * int(w[n, k]) for k in range(K))
            assert got[m, n] == ref


@pytest.mark.parametrize("bits", [4, 8])
def test_range_linear_close_to_fp64(bits):
    # y = s_m w_s[n] acc' in fp64, against the fp32-then-fp16 epilogue: within
    # half an fp16 ulp plus the two fp32 roundings.
    rng = np.random.default_rng(30 + bits)
    M, K, N = 4, 512, 32
    x = workloads.student_t(rng, M, K)
    codes, s, z = rotate_quant_range_ref(x, 512, bits)
    wp = workloads.random_weight_bytes(rng, N, K)
    ws = workloads.random_scales(rng, N)
    y = qlinear_range_ref(codes, s, z, bits, wp, ws).astype(np.float64)
    c = unpack_int4(codes) if bits == 4 else np.asarray(codes)
    q = _q(c, bits)
    w = unpack_int4(wp).astype(np.float64)
    exact = ((q - z[:, None]).astype(np.float64) @ w.T) * s[:, None].astype(np.float64) * \
        ws[None, :].astype(np.float64)
    ulp = np.spacing(np.abs(exact).astype(np.float16)).astype(np.float64)
    assert np.all(np.abs(y - exact) <= 0.5 * ulp + np.abs(exact) * 2.0 ** -22 + 1e-30)
