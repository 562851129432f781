"""Range-based (asymmetric) activation quantizer with a zero point (oracle; test
infrastructure).

What the paper fixes:
* Eq. 1: the step of a b-bit uniform quantizer is the token's range over
  2^b - 1, s = (max(x) - min(x)) / (2^b - 1).
* Eq. 2: values are divided by the step and rounded element-wise; Eq. 3: the
  error is x - Q_b(x).
* Algorithm 1 (calibration step) lists zero points among the quantizer
  parameters; Eq. 4-5: quantization happens on the rotated activations.

Readings taken where the paper is silent:
* Eq. 2 has no zero point, yet a range step spans 2^b - 1 intervals from the
  minimum, not from zero.  The integer zero point of the asymmetric
  quantizers in the PTQ baselines is used: the range is taken over the row
  and 0 (mn = min(min y, 0), mx = max(max y, 0)), so that zero is a level and
  the zero point lies in [0, 2^b - 1]:
      s = fl32(fl32(mx - mn) / (2^b - 1))            (Eq. 1, one IEEE division)
      z = clamp(RNE(fl32(-mn / s)), 0, 2^b - 1)
      q = clamp(RNE(fl32(y / s)) + z, 0, 2^b - 1)     (Eq. 2, half to even)
      Q_b(y) = s * (q - z)
* A row with mx = mn = 0 (all zero) gets s = 0, z = 0, q = 0.
* Storage: the stored code is c = q - 2^(b-1), in [-2^(b-1), 2^(b-1) - 1], so
  the codes pack exactly like the symmetric path's (two's complement nibbles
  at 4 bits, int8 at 8 bits) and feed the same signed integer GEMM.
* GEMM with a zero point: sum_k (q_k - z) w_k = acc + (2^(b-1) - z) wsum,
  with acc = sum_k c_k w_k (the path's exact integer accumulator) and
  wsum[n] = sum_k w[n, k] over the weight codes.  The corrected sum is an
  exact integer; the epilogue is the symmetric path's,
  y = fl16(fl32(fl32(fl32(acc') * s_m) * w_s[n])).
"""

import numpy as np

from .hadamard import rotate_rows
from .quant import pack_int4, unpack_int4
from .gemm import qlinear_acc_ref, epilogue_ref

__all__ = ["range_levels", "quantize_rows_range", "rotate_quant_range_ref",
           "dequant_rows_range", "weight_sums_ref", "zero_point_acc_ref",
           "qlinear_range_ref"]


def range_levels(bits):
    """2^b - 1, the number of steps between the lowest and highest level."""
    if bits not in (4, 8):
        raise ValueError(f"bits must be 4 or 8, got {bits}")
    return (1 << bits) - 1


def quantize_rows_range(y, bits):
    """Per-row range quantization of fp32 rows.

    Returns (codes int8 [M, K] holding q - 2^(b-1), scales float32 [M],
    zeros int32 [M]).
    """
    y = np.asarray(y, dtype=np.float32)
    L = range_levels(bits)
    half = 1 << (bits - 1)
    M = y.shape[0]
    if y.shape[1]:
        mx = np.maximum(y.max(axis=1), np.float32(0))
        mn = np.minimum(y.min(axis=1), np.float32(0))
    else:
        mx = np.zeros(M, np.float32)
        mn = np.zeros(M, np.float32)
    width = (mx - mn).astype(np.float32)                    # fl32(mx - mn)
    scales = (width / np.float32(L)).astype(np.float32)      # Eq. 1
    zeros = np.zeros(M, dtype=np.int32)
    q = np.zeros(y.shape, dtype=np.int64)
    nz = scales != 0
    if np.any(nz):
        zq = (-mn[nz] / scales[nz]).astype(np.float32)       # fl32(-mn / s)
        zeros[nz] = np.clip(np.rint(zq), 0, L).astype(np.int32)
        t = (y[nz] / scales[nz, None]).astype(np.float32)    # fl32(y / s)
        q[nz] = np.clip(np.rint(t).astype(np.int64) + zeros[nz, None], 0, L)
    codes = (q - half).astype(np.int8)
    return codes, scales, zeros


def rotate_quant_range_ref(x, had_size, bits):
    """Online rotation + per-token range quantization (Eq. 4, Eq. 1-2).

    x: float16 [M, K].  Returns (codes, scales, zeros): codes uint8 [M, K/2]
    (A4, packed) or int8 [M, K] (A8); scales float32 [M]; zeros int32 [M].
    """
    y = rotate_rows(x, had_size)
    codes, scales, zeros = quantize_rows_range(y, bits)
    if bits == 4:
        return pack_int4(codes), scales, zeros
    return codes, scales, zeros


def dequant_rows_range(codes, scales, zeros, bits):
    """Q_b(y) = s * (q - z) per row in float64, from stored codes c = q - 2^(b-1)."""
    q = np.asarray(codes, dtype=np.int64) + (1 << (bits - 1))
    return (q - np.asarray(zeros, np.int64)[:, None]).astype(np.float64) * \
        np.asarray(scales, np.float64)[:, None]


def weight_sums_ref(w_packed):
    """wsum[n] = sum_k w[n, k] over the 4-bit weight codes (int64 [N])."""
    return unpack_int4(w_packed).astype(np.int64).sum(axis=1)


def zero_point_acc_ref(acc, zeros, bits, w_sums):
    """acc'[m, n] = acc[m, n] + (2^(b-1) - z[m]) * wsum[n], exact (int64)."""
    off = (1 << (bits - 1)) - np.asarray(zeros, dtype=np.int64)
    return np.asarray(acc, dtype=np.int64) + off[:, None] * np.asarray(w_sums, np.int64)[None, :]


def qlinear_range_ref(a_codes, a_scales, a_zeros, bits, w_packed, w_scales):
    """Quantized linear on range-quantized activations: exact integer GEMM,
    zero-point correction, then the pinned epilogue (fp16 [M, N])."""
    acc = qlinear_acc_ref(a_codes, bits, w_packed)
    acc = zero_point_acc_ref(acc, a_zeros, bits, weight_sums_ref(w_packed))
    return epilogue_ref(acc, a_scales, w_scales)
