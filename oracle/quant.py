"""Symmetric quantizer, nibble packing and weight preparation (oracle; test infrastructure).

What the paper fixes:
* Eq. 2: Q_b(x) = s * round(x / s), element-wise rounding; Eq. 3: e = x - Q_b(x).
* Section 4.2: weights are quantized per output channel and activations per
  token, both symmetric; weights use round-to-nearest (RTN).
* Algorithm 1 steps 1-2: weights at 4 bits, activations at 4 or 8 bits.

Readings taken where the paper is silent or at odds with itself:
* Eq. 1 gives a range step (max - min) / (2^b - 1), but Section 4.2 says the
  quantizers are symmetric and Eq. 2 has no zero point.  The symmetric step is
  used: s = fl32(absmax / qmax) with qmax = 2^(b-1) - 1 (7 or 127), one IEEE
  fp32 division; no clipping ratio.
* A row whose absmax is 0 gets s = 0 and all codes 0.
* The quotient is the correctly rounded fp32 t = fl32(y / s); the code is
  round-half-to-even of t, clamped to [-2^(b-1), 2^(b-1) - 1].  (With
  s = absmax / qmax the clamp never binds; it is kept as the definition.)
* A4 packing: byte j of a row holds code[2j] in its low nibble and code[2j+1]
  in its high nibble, both as 4-bit two's complement.  A8 codes are int8.
* Weights are rotated by the same B_h (Eq. 5), quantized with the 4-bit
  symmetric quantizer per output row, and the stored per-channel scale is
  fl32(s_w / h), which folds in the 1/h of the unnormalised rotation.
"""

import numpy as np

from .hadamard import rotate_rows, split_had_size

__all__ = ["qmax_for_bits", "quantize_rows", "pack_int4", "unpack_int4",
           "pack_int4_a8order", "unpack_int4_a8order",
           "rotate_quant_ref", "prepare_weights_ref", "dequant_rows"]


def qmax_for_bits(bits):
    if bits not in (4, 8):
        raise ValueError(f"bits must be 4 or 8, got {bits}")
    return (1 << (bits - 1)) - 1


def quantize_rows(y, bits):
    """Per-row symmetric quantization of fp32 rows.

    Returns (codes int8 [M, K], scales float32 [M]).
    """
    y = np.asarray(y, dtype=np.float32)
    qmax = qmax_for_bits(bits)
    lo, hi = -(1 << (bits - 1)), (1 << (bits - 1)) - 1
    absmax = np.max(np.abs(y), axis=1) if y.shape[1] else np.zeros(y.shape[0], np.float32)
    scales = (absmax / np.float32(qmax)).astype(np.float32)       # IEEE fp32 divide
    codes = np.zeros(y.shape, dtype=np.int8)
    nz = scales != 0
    if np.any(nz):
        t = (y[nz] / scales[nz, None]).astype(np.float32)           # fl32(y / s)
        r = np.rint(t)                                              # half to even
        codes[nz] = np.clip(r, lo, hi).astype(np.int8)
    return codes, scales


def pack_int4(codes):
    """[M, K] int codes in [-8, 7] -> uint8 [M, K/2]; low nibble = even k."""
    c = np.asarray(codes).astype(np.int64)
    if c.shape[-1] % 2:
        raise ValueError("K must be even to pack int4")
    if c.size and (c.min() < -8 or c.max() > 7):
        raise ValueError("int4 codes must lie in [-8, 7]")
    lo = c[..., 0::2] & 0xF
    hi = c[..., 1::2] & 0xF
    return (lo | (hi << 4)).astype(np.uint8)


def unpack_int4(packed):
    """uint8 [..., K/2] -> int8 [..., K]: nibbles as 4-bit two's complement."""
    p = np.asarray(packed, dtype=np.uint8)
    nib = np.arange(16)
    value = np.where(nib >= 8, nib - 16, nib).astype(np.int8)    # nibble -> -8..7
    out = np.empty(p.shape[:-1] + (2 * p.shape[-1],), dtype=np.int8)
    out[..., 0::2] = value[p & 0xF]
    out[..., 1::2] = value[p >> 4]
    return out


def pack_int4_a8order(codes):
    """Weight codes [N, K] in [-8, 7] (K % 8 == 0) -> uint8 [N, K/2] in the
    order the W4A8 GEMM takes: in each group of eight k (4 bytes), byte j
    holds k = 8g + j in its low nibble and k = 8g + j + 4 in its high one.
    A storage order only; the GEMM's result does not depend on it."""
    c = np.asarray(codes).astype(np.int64)
    if c.shape[-1] % 8:
        raise ValueError("K must be a multiple of 8")
    if c.size and (c.min() < -8 or c.max() > 7):
        raise ValueError("int4 codes must lie in [-8, 7]")
    g = c.reshape(c.shape[:-1] + (c.shape[-1] // 8, 8)) & 0xF
    out = g[..., 0:4] | (g[..., 4:8] << 4)
    return out.reshape(c.shape[:-1] + (c.shape[-1] // 2,)).astype(np.uint8)


def unpack_int4_a8order(packed):
    """Inverse of pack_int4_a8order: uint8 [N, K/2] -> int8 [N, K]."""
    p = np.asarray(packed, dtype=np.uint8).astype(np.int64)
    g = p.reshape(p.shape[:-1] + (p.shape[-1] // 4, 4))
    lo = g & 0xF
    hi = (g >> 4) & 0xF
    both = np.concatenate([lo, hi], axis=-1)
    both = np.where(both >= 8, both - 16, both)
    return both.reshape(p.shape[:-1] + (2 * p.shape[-1],)).astype(np.int8)


def rotate_quant_ref(x, had_size, bits):
    """Online rotation + per-token quantization of activations (Eq. 4, Eq. 2).

    x: float16 [M, K].  Returns (codes, scales): codes are uint8 [M, K/2]
    (A4, packed) or int8 [M, K] (A8); scales float32 [M].
    """
    y = rotate_rows(x, had_size)
    codes, scales = quantize_rows(y, bits)
    if bits == 4:
        return pack_int4(codes), scales
    return codes, scales


def prepare_weights_ref(w, had_size):
    """Offline weight preparation (Eq. 5 absorption, per-channel symmetric RTN, 4 bits).

    w: float32 [N, K].  Returns (w_packed uint8 [N, K/2], w_scales float32 [N])
    with w_scales = fl32(fl32(absmax(W_n B) / 7) / h).
    """
    f, p = split_had_size(had_size)
    h = f * p
    z = rotate_rows(np.asarray(w, dtype=np.float32), h)
    codes, s_w = quantize_rows(z, 4)
    w_scales = (s_w / np.float32(h)).astype(np.float32)
    return pack_int4(codes), w_scales


def dequant_rows(codes, scales):
    """Q_b(y) = code * s per row, in float64 (for error checks, Eq. 2-3)."""
    return np.asarray(codes, dtype=np.float64) * np.asarray(scales, np.float64)[:, None]
