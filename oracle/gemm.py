"""Exact integer GEMM and dequant epilogue (oracle; test infrastructure).

What the paper fixes: the linear projection Y = X W^T with X [tokens, in] and
W [out, in] (Section 2, "Low-Bit Quantization of LLMs"), computed on the
rotated operands (Eq. 5), with per-token activation scales and per-output-
channel weight scales (Section 4.2).

Readings:
* The accumulator is the exact integer sum acc[m, n] = sum_k a[m, k] * w[n, k]
  (|acc| <= K * 128 * 8 stays far below 2^31 for every supported K, so a
  32-bit accumulator is exact as well).  It is formed with a float64 library
  matmul on the integer codes: every product and partial sum is an integer
  below 2^53, so the result is exact in any summation order.
* Epilogue order: y = fl16(fl32(fl32(fl32(acc) * a_s[m]) * w_s[n])), every
  conversion and product rounded to nearest-even.
"""

import numpy as np

from .quant import unpack_int4

__all__ = ["qlinear_acc_ref", "qlinear_acc_entries", "epilogue_ref", "qlinear_ref"]


def _as_codes(codes, bits):
    if bits == 4:
        return unpack_int4(codes).astype(np.int64)
    if bits == 8:
        return np.asarray(codes, dtype=np.int8).astype(np.int64)
    raise ValueError(f"bits must be 4 or 8, got {bits}")


def qlinear_acc_ref(a_codes, bits, w_packed, cols=8192):
    """acc[m, n] = sum_k a[m, k] * w[n, k] exactly (int64 [M, N]).

    The weight rows are taken `cols` output channels at a time; every entry is
    one exact float64 dot product whatever the grouping."""
    a = _as_codes(a_codes, bits).astype(np.float64)
    K = a.shape[1]
    if 2 * np.asarray(w_packed).shape[1] != K:
        raise ValueError("K mismatch between activation codes and weights")
    if K * 128 * 8 >= 2 ** 53:
        raise ValueError("K too large for an exact float64 accumulation")
    N = np.asarray(w_packed).shape[0]
    out = np.empty((a.shape[0], N), dtype=np.int64)
    for n0 in range(0, N, cols):
        w = unpack_int4(w_packed[n0:n0 + cols]).astype(np.float64)
        out[:, n0:n0 + cols] = (a @ w.T).astype(np.int64)
    return out


def qlinear_acc_entries(a_codes, bits, w_packed, rows, cols):
    """acc[rows[i], cols[i]] computed one entry at a time (int64 [len(rows)])."""
    a = _as_codes(a_codes, bits)
    w = unpack_int4(w_packed).astype(np.int64)
    rows = np.asarray(rows)
    cols = np.asarray(cols)
    return np.array([int(np.dot(a[m], w[n])) for m, n in zip(rows, cols)],
                    dtype=np.int64)


def epilogue_ref(acc, a_scales, w_scales):
    """fl16(fl32(fl32(fl32(acc) * a_s[m]) * w_s[n])) for an [M, N] accumulator."""
    acc32 = np.asarray(acc, dtype=np.int64).astype(np.float32)
    a_s = np.asarray(a_scales, dtype=np.float32)
    w_s = np.asarray(w_scales, dtype=np.float32)
    t = (acc32 * a_s[:, None]).astype(np.float32)
    t = (t * w_s[None, :]).astype(np.float32)
    return t.astype(np.float16)


def qlinear_ref(a_codes, a_scales, bits, w_packed, w_scales):
    """Full quantized linear: exact integer GEMM then the pinned epilogue."""
    return epilogue_ref(qlinear_acc_ref(a_codes, bits, w_packed), a_scales, w_scales)
