"""Residual-dynamics calibration metrics and the sensitive-layer rule (oracle; test infrastructure).

What the paper fixes:
* Eq. 6: x^(l+1) = x^(l) + dx^(l); x^(l) is the historical residual state of a
  token entering layer l, dx^(l) the update the layer adds.
* Eq. 8-9: Jump Ratio JR_{l,t} = ||dx_t||_2 / (||x_t||_2 + eps) per token, and
  the layer value JR_l is its mean over the T tokens.
* Eq. 10: the history reconstructed from the quantized updated state is
  xhat_t = Q_b(x_t + dx_t) - dx_t.
* Eq. 11: SNR_hist,l = mean over t of 10 log10(||x_t||^2 / (||xhat_t - x_t||^2 + eps)).
* Eq. 20: S = {l : JR_l > tau_JR and SNR_hist,l < tau_SNR}.
* Section 3.2 (Eq. 14-16): quantization happens in the rotated space and its
  result is mapped back by the inverse rotation.

Readings taken where the paper is silent:
* Q_b is the quantizer the path deploys: u = fl32(x + dx) is rotated by B_h in
  the pinned fp32 order, quantized per token with the symmetric quantizer
  (s = fl32(absmax / qmax), round half to even), dequantized as code * s and
  rotated back by the inverse of the unnormalized B_h, which is B_h / h.  Every
  step after the codes is fp64.
* The historical state in Eq. 10 is the full-precision x^(l) of the
  calibration run: each layer's sensitivity is measured on its own, not through
  the recursion of Eq. 7.
* b = 4 (the precision the rule guards) and eps = 1e-8 unless given.  The paper
  gives no values for eps, tau_JR or tau_SNR; they are inputs here.
* Norms, logarithms and means are fp64.
"""

import numpy as np

from .hadamard import paley28, rotate_rows, split_had_size
from .quant import quantize_rows

__all__ = ["jump_ratio_tokens_ref", "inverse_rotate_f64", "reconstructed_history_ref",
           "hist_snr_tokens_ref", "residual_dynamics_ref", "select_sensitive_layers_ref"]

DEFAULT_EPS = 1e-8


def jump_ratio_tokens_ref(x, dx, eps=DEFAULT_EPS):
    """Eq. 8: ||dx_t|| / (||x_t|| + eps) for every token row, fp64 [T]."""
    x = np.asarray(x, dtype=np.float64)
    dx = np.asarray(dx, dtype=np.float64)
    return np.linalg.norm(dx, axis=1) / (np.linalg.norm(x, axis=1) + eps)


def inverse_rotate_f64(y, had_size):
    """Rows of y (fp64 [T, K]) times (I (x) H_h)^-1 = (I (x) H_h) / h, in fp64."""
    y = np.asarray(y, dtype=np.float64)
    T, K = y.shape
    f, p = split_had_size(had_size)
    h = f * p
    # H_h = H_f (x) H_p with the H_f index slow: H_p by its Sylvester recursion
    # on the fast index, then H_28 (symmetric) on the slow one.
    v = y.reshape(T, K // h, f, p).copy()
    half = 1
    while half < p:
        v = v.reshape(T, K // h, f, p // (2 * half), 2, half)
        a, c = v[..., 0, :].copy(), v[..., 1, :].copy()
        v[..., 0, :], v[..., 1, :] = a + c, a - c
        half *= 2
    v = v.reshape(T, K // h, f, p)
    if f == 28:
        v = np.einsum("ab,tkbp->tkap", paley28().astype(np.float64), v)
    return (v / h).reshape(T, K)


def reconstructed_history_ref(x, dx, had_size, bits=4):
    """Eq. 10: xhat = Q_b(x + dx) - dx in the original space (fp64 [T, K])."""
    x16 = np.asarray(x, dtype=np.float16)
    dx16 = np.asarray(dx, dtype=np.float16)
    u = x16.astype(np.float32) + dx16.astype(np.float32)           # fl32(x + dx)
    y = rotate_rows(u, had_size)                                   # pinned fp32 rotation
    codes, s = quantize_rows(y, bits)
    yq = codes.astype(np.float64) * s.astype(np.float64)[:, None]  # Q_b in the rotated space
    return inverse_rotate_f64(yq, had_size) - dx16.astype(np.float64)


def hist_snr_tokens_ref(x, dx, had_size, bits=4, eps=DEFAULT_EPS):
    """Eq. 11 per token: 10 log10(||x_t||^2 / (||xhat_t - x_t||^2 + eps)), fp64 [T]."""
    x64 = np.asarray(x, dtype=np.float16).astype(np.float64)
    xhat = reconstructed_history_ref(x, dx, had_size, bits)
    num = np.sum(x64 * x64, axis=1)
    err = xhat - x64
    den = np.sum(err * err, axis=1) + eps
    with np.errstate(divide="ignore"):       # a zero history has SNR -inf
        return 10.0 * np.log10(num / den)


def residual_dynamics_ref(x, dx, had_size, bits=4, eps=DEFAULT_EPS):
    """Per-token JR and SNR_hist (dB) and their layer means (Eq. 8-11).

    x, dx: float16 [T, K], one layer's residual states and updates.
    Returns (jr_tokens, snr_tokens, jr_layer, snr_layer), fp64.
    """
    jr = jump_ratio_tokens_ref(np.asarray(x, np.float16), np.asarray(dx, np.float16), eps)
    snr = hist_snr_tokens_ref(x, dx, had_size, bits, eps)
    return jr, snr, float(np.mean(jr)), float(np.mean(snr))


def select_sensitive_layers_ref(jr_layers, snr_layers, tau_jr, tau_snr):
    """Eq. 20: the (0-indexed) layers with JR_l > tau_JR and SNR_hist,l < tau_SNR,
    and the activation bits of every layer (8 for those, 4 otherwise)."""
    jr = [float(v) for v in jr_layers]
    snr = [float(v) for v in snr_layers]
    if len(jr) != len(snr):
        raise ValueError("one JR and one SNR value per layer")
    sel = [l for l in range(len(jr)) if jr[l] > tau_jr and snr[l] < tau_snr]
    return sel, [8 if l in sel else 4 for l in range(len(jr))]
