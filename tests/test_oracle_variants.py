"""Pins of the randomized-sign rotation oracle (CPU).

The randomized rotation y = (x * d) . B_h (QuaRot-style online Hadamard,
Section 4.2; Eq. 4) is checked against facts that do not come from the oracle
itself: the bitmask convention bit by bit, the identity at d = +1, the joint
sign-flip symmetry, exact integer products, Parseval (Eq. 12), the closed form
for a single massive channel, and the cancellation of the signs in the weight
absorption of Eq. 5.
"""

import numpy as np
import pytest

import workloads
from oracle import (signs_from_bits, apply_signs, rotate_quant_signed_ref,
                    prepare_weights_signed_ref, rotate_quant_ref, prepare_weights_ref,
                    rotate_rows, unpack_int4, sylvester)


def _bits_of(d):
    """+-1 vector -> bitmask (independent of signs_from_bits)."""
    K = len(d)
    out = np.zeros((K + 7) // 8, dtype=np.uint8)
    for k in range(K):
        if d[k] < 0:
            out[k // 8] |= np.uint8(1 << (k % 8))
    return out


def test_bitmask_convention_exhaustive_byte():
    for byte in range(256):
        d = signs_from_bits(np.array([byte], dtype=np.uint8), 8)
        for b in range(8):
            assert d[b] == (-1.0 if (byte >> b) & 1 else 1.0)


def test_no_signs_is_the_plain_rotation():
    rng = np.random.default_rng(0)
    x = workloads.gauss_outliers(rng, 5, 512)
    zero = np.zeros(512 // 8, dtype=np.uint8)
    for bits in (4, 8):
        c0, s0 = rotate_quant_ref(x, 512, bits)
        c1, s1 = rotate_quant_signed_ref(x, 512, bits, zero)
        assert np.array_equal(c0, c1) and np.array_equal(s0.view(np.uint32), s1.view(np.uint32))


def test_joint_sign_flip_symmetry():
    # (x * s) * (d * s) = x * d for any +-1 vector s: codes and scales unchanged.
    rng = np.random.default_rng(1)
    K = 1024
    x = workloads.gauss_outliers(rng, 4, K)
    d = np.where(rng.random(K) < 0.5, -1.0, 1.0)
    s = np.where(rng.random(K) < 0.5, -1.0, 1.0)
    xs = np.where(s < 0, -x, x).astype(np.float16)
    for bits in (4, 8):
        c0, s0 = rotate_quant_signed_ref(x, 256, bits, _bits_of(d))
        c1, s1 = rotate_quant_signed_ref(xs, 256, bits, _bits_of(d * s))
        assert np.array_equal(c0, c1) and np.array_equal(s0, s1)


def test_integer_inputs_give_the_exact_signed_product():
    rng = np.random.default_rng(2)
    K = 256
    x = rng.integers(-30, 31, size=(3, K)).astype(np.float16)
    d = np.where(rng.random(K) < 0.5, -1, 1)
    y = rotate_rows(apply_signs(x, _bits_of(d)), K).astype(np.float64)
    exact = (x.astype(np.int64) * d[None, :]) @ sylvester(K)
    assert np.array_equal(y, exact.astype(np.float64))


def test_parseval_with_signs():
    rng = np.random.default_rng(3)
    K = 4096
    x = workloads.gauss_outliers(rng, 3, K)
    bits = workloads.random_sign_bits(rng, K)
    y = rotate_rows(apply_signs(x, bits), K).astype(np.float64)
    xn = np.sum(x.astype(np.float64) ** 2, axis=1)
    yn = np.sum(y ** 2, axis=1)
    assert np.allclose(yn, K * xn, rtol=1e-5)


def test_single_massive_channel_spreads_evenly():
    # x = v e_k: every output of the signed rotation is +-v (closed form), so
    # every code has magnitude qmax whatever the signs.
    rng = np.random.default_rng(4)
    K = 512
    x = np.zeros((2, K), dtype=np.float16)
    x[0, 17] = 300.0
    x[1, 400] = -0.125
    bits = workloads.random_sign_bits(rng, K)
    y = rotate_rows(apply_signs(x, bits), K)
    assert np.all(np.abs(y[0]) == 300.0) and np.all(np.abs(y[1]) == 0.125)
    c, _ = rotate_quant_signed_ref(x, K, 8, bits)
    assert np.all(np.abs(c.astype(np.int64)) == 127)


def test_signs_cancel_in_the_weight_absorption():
    # Eq. 5 with D B on both sides: the dequantized layer approximates X W^T as
    # well as the unsigned one does, and much better than a mismatched D.
    rng = np.random.default_rng(5)
    M, K, N, h = 16, 512, 64, 512
    x = workloads.gauss_outliers(rng, M, K)
    w = workloads.weights(rng, N, K)
    bits = workloads.random_sign_bits(rng, K)
    other = workloads.random_sign_bits(rng, K)
    exact = x.astype(np.float64) @ w.astype(np.float64).T

    def layer(xb, wb):
        c, s = rotate_quant_signed_ref(x, h, 8, xb)
        wp, ws = prepare_weights_signed_ref(w, h, wb)
        acc = unpack_int4(wp).astype(np.float64)
        return (c.astype(np.float64) * s[:, None].astype(np.float64)) @ \
            (acc * ws[:, None].astype(np.float64)).T

    zero = np.zeros_like(bits)
    err = np.linalg.norm(layer(bits, bits) - exact) / np.linalg.norm(exact)
    plain = np.linalg.norm(layer(zero, zero) - exact) / np.linalg.norm(exact)
    bad = np.linalg.norm(layer(bits, other) - exact) / np.linalg.norm(exact)
    # matched signs: the same 4-bit-weight error level as the plain rotation;
    # mismatched signs: no longer an approximation of X W^T at all
    assert err < 1.25 * plain and bad > 0.7, (err, plain, bad)


def test_weight_preparation_without_signs_is_unchanged():
    rng = np.random.default_rng(6)
    w = workloads.weights(rng, 8, 256)
    a = prepare_weights_ref(w, 256)
    b = prepare_weights_signed_ref(w, 256, np.zeros(32, dtype=np.uint8))
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
