"""Pins of the residual-dynamics oracle (Section 3.1 Eq. 8-11, Section 3.2, Eq. 20).

Each test checks the oracle against something other than its own formula:
closed forms, invariances the paper states, the scaling trends of Eq. 19 and
Eq. 22, and brute-force tables.
"""

import numpy as np
import pytest

import workloads
from oracle import hadamard, rotate_rows
from oracle.residual import (DEFAULT_EPS, hist_snr_tokens_ref, inverse_rotate_f64,
                             jump_ratio_tokens_ref, reconstructed_history_ref,
                             residual_dynamics_ref, select_sensitive_layers_ref)
from oracle.quant import quantize_rows


def _f16(a):
    return np.asarray(a, dtype=np.float16)


def test_jump_ratio_closed_forms():
    rng = np.random.default_rng(0)
    x = _f16(rng.standard_normal((5, 256)))
    # dx = c x (exact in fp16 for powers of two): JR = c ||x|| / (||x|| + eps).
    for c in (0.25, 1.0, 8.0):
        dx = _f16(c * x.astype(np.float32))
        nx = np.linalg.norm(x.astype(np.float64), axis=1)
        jr = jump_ratio_tokens_ref(x, dx)
        assert np.allclose(jr, c * nx / (nx + DEFAULT_EPS), rtol=1e-14, atol=0)
    # No update: JR = 0; no history: JR = ||dx|| / eps.
    assert np.all(jump_ratio_tokens_ref(x, np.zeros_like(x)) == 0)
    z = np.zeros((1, 256), np.float16)
    d = _f16(np.full((1, 256), 0.5))
    assert jump_ratio_tokens_ref(z, d, eps=1e-3)[0] == pytest.approx(0.5 * 16 / 1e-3, rel=1e-14)


def test_jump_ratio_rotation_invariant():
    # Eq. 13: the same orthonormal rotation of x and dx leaves JR unchanged.
    rng = np.random.default_rng(1)
    h = 512
    x = rng.standard_normal((4, h))
    dx = 3.0 * rng.standard_normal((4, h))
    R = hadamard(h).astype(np.float64) / np.sqrt(h)
    jr = jump_ratio_tokens_ref(x, dx)
    jr_rot = jump_ratio_tokens_ref(x @ R, dx @ R)
    assert np.allclose(jr, jr_rot, rtol=1e-12, atol=0)


@pytest.mark.parametrize("h", [64, 28 * 8, 4096, 28 * 512])
def test_inverse_rotation_undoes_the_rotation(h):
    # (I (x) H_h) (I (x) H_h) / h = I, with H_h the integer matrix of the path.
    rng = np.random.default_rng(h)
    K = 2 * h if h <= 1024 else h
    v = rng.standard_normal((3, K))
    if h <= 1024:
        H = hadamard(h).astype(np.float64)
        y = (v.reshape(3, K // h, h) @ H).reshape(3, K)
    else:
        y = np.asarray(rotate_rows(v.astype(np.float32), h), np.float64)
        v = v.astype(np.float32).astype(np.float64)
    back = inverse_rotate_f64(y, h)
    tol = 1e-12 if h <= 1024 else 1e-4   # fp32 forward rotation for the large sizes
    assert np.allclose(back, v, rtol=0, atol=tol * np.abs(v).max())


def test_reconstruction_error_is_the_rotated_quantization_error():
    # Eq. 10 and Eq. 16: xhat - x = Q_b(u) - u (up to the fp32 rounding of
    # u = x + dx), and its norm is ||code * s - y|| / sqrt(h) in the rotated
    # space.  Fails if dx is not subtracted or the inverse misses its 1/h.
    rng = np.random.default_rng(2)
    T, h = 6, 1024
    x = _f16(rng.standard_normal((T, h)))
    dx = _f16(4.0 * rng.standard_normal((T, h)))
    xhat = reconstructed_history_ref(x, dx, h, 4)
    u = x.astype(np.float32) + dx.astype(np.float32)
    y = rotate_rows(u, h)
    codes, s = quantize_rows(y, 4)
    err_rot = codes.astype(np.float64) * s.astype(np.float64)[:, None] - y.astype(np.float64)
    lhs = np.sum((xhat - x.astype(np.float64)) ** 2, axis=1)
    rhs = np.sum(err_rot ** 2, axis=1) / h
    assert np.allclose(lhs, rhs, rtol=1e-6)


def test_snr_exact_grid_closed_form():
    # One-hot rows a * e_k with a = qmax * 2^e and no update: the rotated row
    # is +-a everywhere, s = a / qmax is exact and the codes reproduce it, so
    # the error is 0 and SNR = 10 log10(a^2 / eps).
    h = 256
    for bits, qmax in ((4, 7), (8, 127)):
        x = np.zeros((3, h), np.float16)
        x[0, 5] = qmax * 2.0 ** -3
        x[1, 200] = -qmax * 2.0 ** 2
        x[2, 0] = qmax
        snr = hist_snr_tokens_ref(x, np.zeros_like(x), h, bits)
        a2 = np.sum(x.astype(np.float64) ** 2, axis=1)
        assert np.allclose(snr, 10 * np.log10(a2 / DEFAULT_EPS), rtol=1e-12)


def test_snr_bits_trend():
    # Eq. 19 / Eq. 22: the error energy scales with s^2, s ~ 1/qmax, so going
    # from 4 to 8 bits raises the SNR by about 20 log10(127 / 7) = 25.2 dB.
    rng = np.random.default_rng(3)
    x = _f16(rng.standard_normal((8, 1024)))
    dx = _f16(rng.standard_normal((8, 1024)))
    gain = np.mean(hist_snr_tokens_ref(x, dx, 1024, 8) - hist_snr_tokens_ref(x, dx, 1024, 4))
    assert abs(gain - 20 * np.log10(127 / 7)) < 1.5


def test_snr_jump_trend():
    # Eq. 19: once the update dominates the range, the SNR falls by about
    # 20 dB per decade of Jump Ratio.
    rng = np.random.default_rng(4)
    x = rng.standard_normal((8, 1024))
    g = rng.standard_normal((8, 1024))
    snr = {}
    for c in (10.0, 100.0):
        snr[c] = np.mean(hist_snr_tokens_ref(_f16(x), _f16(c * g), 1024, 4))
    assert abs((snr[100.0] - snr[10.0]) + 20.0) < 1.5


def test_layer_means():
    rng = np.random.default_rng(5)
    x = _f16(rng.standard_normal((7, 256)))
    dx = _f16(0.5 * rng.standard_normal((7, 256)))
    jr, snr, jr_l, snr_l = residual_dynamics_ref(x, dx, 256, 4)
    assert jr.shape == snr.shape == (7,)
    assert jr_l == pytest.approx(sum(jr) / 7, rel=1e-14)
    assert snr_l == pytest.approx(sum(snr) / 7, rel=1e-14)


def test_selection_rule_table():
    # Eq. 20, both inequalities strict.
    jr = [0.9, 0.9, 0.2, 0.5, 0.9, 0.5]
    snr = [10.0, 20.0, 10.0, 10.0, 15.0, 14.9]
    sel, bits = select_sensitive_layers_ref(jr, snr, tau_jr=0.5, tau_snr=15.0)
    assert sel == [0]
    sel, bits = select_sensitive_layers_ref(jr, snr, tau_jr=0.4, tau_snr=15.0)
    assert sel == [0, 3, 5]
    assert bits == [8, 4, 4, 8, 4, 8]
    assert select_sensitive_layers_ref([], [], 0.0, 0.0) == ([], [])
    with pytest.raises(ValueError):
        select_sensitive_layers_ref([1.0], [], 0.0, 0.0)


def test_three_phase_stream_selects_phase_boundaries():
    # On a synthetic residual stream with the three-phase pattern of Section 2
    # (large updates while massive activations emerge in the first layers and
    # are redistributed in the last one, small ones in between), the rule
    # marks the early layers and the last layer.
    L, T, d = 12, 8, 256
    stream = workloads.residual_stream(np.random.default_rng(6), L, T, d)
    jr_l, snr_l = [], []
    for x, dx in stream:
        _, _, j, s = residual_dynamics_ref(x, dx, d, 4)
        jr_l.append(j)
        snr_l.append(s)
    sel, _ = select_sensitive_layers_ref(jr_l, snr_l, tau_jr=0.5, tau_snr=float(np.median(snr_l)))
    assert sel == [0, 1, 2, L - 1]
