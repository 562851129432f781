"""Variants of the rotated quantizer (oracle; test infrastructure).

Randomized-sign rotation.  Section 4.2 uses a QuaRot-style online Hadamard
rotation.  QuaRot's rotation is a randomized Hadamard transform: a fixed
diagonal of random +-1 signs applied before the Hadamard matrix, R = D H (up
to normalisation), which keeps R orthogonal and spreads a massive channel
over every output (Section 2, Eq. 4).  Reading taken here:

* y = (x * d) . B_h with d_k in {+1, -1}; the signs are an input (drawn once,
  seeded, by the caller), stored as a bitmask: bit (k & 7) of byte k >> 3 set
  means d_k = -1.  Negation is exact in fp16 and fp32, so x * d is formed
  first and the rotation then follows the pinned order of the hadamard module.
* Weight absorption (Eq. 5) applies the same signs to the weight rows:
  (x D B)(W D B)^T = h x D D W^T = h x W^T, because D D = I and B B^T = h I.
"""

import numpy as np

from .quant import rotate_quant_ref, prepare_weights_ref

__all__ = ["signs_from_bits", "apply_signs", "rotate_quant_signed_ref",
           "prepare_weights_signed_ref"]


def signs_from_bits(sign_bits, K):
    """Bitmask uint8 [ceil(K/8)] -> float64 [K] of +1 / -1 (bit set = -1)."""
    b = np.asarray(sign_bits, dtype=np.uint8)
    if b.size * 8 < K:
        raise ValueError("sign bitmask shorter than K bits")
    bits = (b[:, None] >> np.arange(8, dtype=np.uint8)[None, :]) & 1    # [bytes, 8], bit k & 7
    flat = bits.reshape(-1)[:K]
    return np.where(flat == 1, -1.0, 1.0)


def apply_signs(x, sign_bits):
    """x * diag(d) row-wise; exact (a sign flip), dtype preserved."""
    x = np.asarray(x)
    d = signs_from_bits(sign_bits, x.shape[1])
    return np.where(d[None, :] < 0, -x, x).astype(x.dtype)


def rotate_quant_signed_ref(x, had_size, bits, sign_bits):
    """Randomized-sign online rotation + per-token quantization: the codes and
    scales of (x * d) . B_h (Eq. 4, Eq. 2; the rotation of Section 4.2)."""
    return rotate_quant_ref(apply_signs(x, sign_bits), had_size, bits)


def prepare_weights_signed_ref(w, had_size, sign_bits):
    """Weight preparation with the same signs (Eq. 5 absorption of D B)."""
    return prepare_weights_ref(apply_signs(np.asarray(w, dtype=np.float32), sign_bits), had_size)
