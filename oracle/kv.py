"""Group-wise 4-bit KV-cache quantizer (oracle; test infrastructure).

What the paper fixes:
* Section 4.2: the KV cache is quantized group-wise to 4 bits with a group
  size of 128.
* Algorithm 1 (precision step): the KV cache stays at 4 bits on every layer,
  whatever activation bits the policy gives the layer.
* Eq. 1: the step of a b-bit uniform quantizer is the range of the values
  divided by 2^b - 1; Eq. 2: values are divided by the step and rounded.

Readings taken where the paper is silent:
* Symmetric or asymmetric is not stated for the KV cache.  Eq. 1's range step
  spans 2^b - 1 = 15 intervals from the minimum to the maximum, so the 16
  levels are placed from the group minimum: m = min(x), s = fl32(fl32(max(x) - m) / 15),
  code = clamp(RNE(fl32(fl32(x - m) / s)), 0, 15), i.e. Eq. 2's rounding applied
  to the offset from the minimum (the zero point is the fp32 minimum).
* A group is `group` consecutive elements of one token's K (or V) vector; with
  head_dim 128 a group of 128 is one head of one token.
* A constant group (max = min) gets s = 0 and codes 0, and reconstructs exactly.
* Reconstruction: xhat = fl16(fl32(fl32(code * s) + m)), two fp32 roundings.
* Packing: byte j of a token row holds code[2j] in its low nibble and
  code[2j+1] in its high nibble, as unsigned nibbles.  s and m are fp32, one
  pair per group, in group order.
* No rotation inside the codec: the rotation the PTQ baselines apply to K and
  V happens upstream of the cache.
"""

import numpy as np

__all__ = ["kv_quant_ref", "kv_dequant_ref", "pack_u4", "unpack_u4", "KV_LEVELS"]

KV_LEVELS = 15        # 2^4 - 1 intervals (Eq. 1 at b = 4)


def pack_u4(codes):
    """[T, D] codes in [0, 15] -> uint8 [T, D/2]; low nibble = even element."""
    c = np.asarray(codes).astype(np.int64)
    if c.shape[-1] % 2:
        raise ValueError("row length must be even")
    if np.any((c < 0) | (c > 15)):
        raise ValueError("codes must lie in [0, 15]")
    return (c[..., 0::2] | (c[..., 1::2] << 4)).astype(np.uint8)


def unpack_u4(packed):
    """uint8 [T, D/2] -> int64 [T, D] codes in [0, 15]."""
    p = np.asarray(packed, dtype=np.uint8).astype(np.int64)
    out = np.empty(p.shape[:-1] + (2 * p.shape[-1],), dtype=np.int64)
    out[..., 0::2] = p & 0xF
    out[..., 1::2] = p >> 4
    return out


def _groups(x, group):
    T, D = x.shape
    if group <= 0 or D % group:
        raise ValueError("the row length must be a multiple of the group size")
    return x.reshape(T, D // group, group)


def kv_quant_ref(kv, group=128):
    """fp16 [T, D] -> (codes uint8 [T, D/2], scales fp32 [T, D/group], mins fp32 [T, D/group])."""
    x = _groups(np.asarray(kv, dtype=np.float16).astype(np.float32), group)
    T, G, _ = x.shape
    m = x.min(axis=2)                                        # exact (fp16 values)
    r = (x.max(axis=2) - m).astype(np.float32)              # fl32(max - min)
    s = (r / np.float32(KV_LEVELS)).astype(np.float32)     # Eq. 1, one IEEE division
    codes = np.zeros(x.shape, dtype=np.int64)
    nz = s != 0
    if np.any(nz):
        d = (x[nz] - m[nz][:, None]).astype(np.float32)     # fl32(x - m)
        t = (d / s[nz][:, None]).astype(np.float32)         # fl32(d / s)
        codes[nz] = np.clip(np.rint(t), 0, KV_LEVELS).astype(np.int64)   # Eq. 2, half to even
    return pack_u4(codes.reshape(T, G * group)), s, m


def kv_dequant_ref(codes, scales, mins, group=128):
    """Reconstruct fp16 [T, D] from the packed codes and per-group (s, m)."""
    c = unpack_u4(codes)
    T, D = c.shape
    q = _groups(c.astype(np.float32), group)
    s = np.asarray(scales, dtype=np.float32).reshape(T, D // group, 1)
    m = np.asarray(mins, dtype=np.float32).reshape(T, D // group, 1)
    t = (q * s).astype(np.float32)                          # fl32(code * s)
    t = (t + m).astype(np.float32)                          # fl32(. + m)
    return t.astype(np.float16).reshape(T, D)
