"""Helpers shared by the GPU parity tests (not collected by pytest).

Everything that computes an expected value calls the oracle; this module only
splits work over token rows or output columns (rows and columns of the
quantized linear are independent by definition), draws output-safe weight
scales, and holds the reference encoder of the FP6 block layout, written from
the e2m3 definition.
"""

import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np

from oracle import (rotate_rows, quantize_rows, pack_int4, qlinear_acc_ref, epilogue_ref,
                    unpack_int4)

WORKERS = max(1, min(16, os.cpu_count() or 1))


def sample_rows(M, n, seed):
    """n sorted distinct rows of range(M), always including 0 and M - 1."""
    if M <= n:
        return np.arange(M)
    rows = {0, M - 1}
    rows.update(np.random.default_rng(seed).choice(M, n - 2, replace=False).tolist())
    return np.array(sorted(rows))


def oracle_rotate(x, h):
    """oracle.rotate_rows over row chunks on a thread pool; fp32 [M, K]."""
    M = x.shape[0]
    if M <= 2:
        return rotate_rows(x, h)
    chunks = [c for c in np.array_split(np.arange(M), min(M, 4 * WORKERS)) if c.size]
    with ThreadPoolExecutor(WORKERS) as ex:
        parts = list(ex.map(lambda r: rotate_rows(x[r[0]:r[-1] + 1], h), chunks))
    return np.concatenate(parts)


def oracle_codes(y, bits):
    """Codes and scales of rotated rows y at `bits`, in the library's layout."""
    codes, scales = quantize_rows(y, bits)
    return (pack_int4(codes) if bits == 4 else codes), scales


def oracle_acc(a_codes, bits, w_packed):
    """Exact accumulators [M, N] (int64): the oracle's float64 product."""
    return qlinear_acc_ref(a_codes, bits, w_packed)


def oracle_y(acc, a_scales, w_scales):
    """The pinned epilogue; asserts that every expected output is finite."""
    y = epilogue_ref(acc, a_scales, w_scales)
    assert np.isfinite(y.astype(np.float32)).all(), "expected outputs overflow fp16"
    return y


def safe_w_scales(rng, N, K, a_scales, bits, limit=30000.0):
    """Positive weight scales drawn so that no output can leave fp16 range:
    |acc| <= K * qmax_a * 8, so |y| <= K * qmax_a * 8 * max(a_s) * w_s."""
    qmax = 7 if bits == 4 else 127
    top = float(np.max(a_scales)) if np.size(a_scales) else 1.0
    bound = limit / (K * (qmax + 1) * 8 * max(top, 1e-30))
    return (rng.uniform(0.5, 1.0, N) * bound).astype(np.float32)


def assert_bytes(got, ref, what):
    g = np.ascontiguousarray(got)
    r = np.ascontiguousarray(ref)
    assert g.shape == r.shape, f"{what}: shape {g.shape} vs {r.shape}"
    bad = np.nonzero(g.reshape(g.shape[0], -1).view(np.uint8)
                     != r.reshape(r.shape[0], -1).view(np.uint8))
    assert bad[0].size == 0, f"{what}: {bad[0].size} bytes differ, first in row {bad[0][0]}"


def assert_f16(got, ref, what):
    g, r = got.view(np.uint16), ref.view(np.uint16)
    if np.array_equal(g, r):
        return
    gf, rf = got.astype(np.float64), ref.astype(np.float64)
    rel = np.max(np.abs(gf - rf) / np.maximum(np.abs(rf), 1e-30))
    raise AssertionError(f"{what}: {(g != r).sum()} outputs differ (max rel err {rel:.3g})")


def _e2m3_value(bits6):
    s = -1.0 if bits6 & 0x20 else 1.0
    e, m = (bits6 >> 3) & 3, bits6 & 7
    return s * (m / 8.0 if e == 0 else 2.0 ** (e - 1) * (1.0 + m / 8.0))


def e2m3_table():
    """Encoding of c / 2 for c = -8..7, found by decoding all 64 patterns."""
    table = {}
    for c in range(-8, 8):
        hits = [b for b in range(64) if _e2m3_value(b) == c / 2.0 and not (c == 0 and b & 0x20)]
        assert len(hits) == 1, (c, hits)
        table[c] = hits[0]
    return table


def fp6_layout_ref(packed, K):
    """Reference FP6 block layout of packed 4-bit codes [R, K/2] -> uint8 bytes."""
    codes = unpack_int4(packed).astype(np.int64)             # [R, K], -8..7
    R = codes.shape[0]
    Rp = (R + 31) // 32 * 32
    full = np.zeros((Rp, K), dtype=np.int64)
    full[:R] = codes
    tab = e2m3_table()
    lut = np.array([tab[c] for c in range(-8, 8)], dtype=np.uint64)
    enc = lut[full + 8]                                      # [Rp, K] six-bit fields
    nkb = K // 128
    # k = 128 kb + 64 g + 32 s + j ; lane l = 32 g + r
    e = enc.reshape(Rp // 32, 32, nkb, 2, 2, 32)             # rb, r, kb, g, s, j
    e = e.transpose(0, 2, 4, 3, 1, 5).reshape(Rp // 32, nkb, 2, 64, 32)   # rb, kb, s, l, j
    words = np.zeros(e.shape[:-1] + (3,), dtype=np.uint64)
    for j in range(32):
        pos = 6 * j
        w, off = pos // 64, pos % 64
        words[..., w] |= e[..., j] << np.uint64(off)
        if off > 58:
            words[..., w + 1] |= e[..., j] >> np.uint64(64 - off)
    # plane c of half s holds bytes 8c..8c+7 (word c) of every lane, lane-major
    planes = words.transpose(0, 1, 2, 4, 3).copy()           # rb, kb, s, c, l
    blocks = planes.view(np.uint8).reshape(Rp // 32, nkb, 2 * 3 * 64 * 8)   # rb, kb, 3072
    # blocks are stored k-block major: (kb, rb)
    return blocks.transpose(1, 0, 2).reshape(-1)


def fp6_layout_decode(buf, R, K):
    """Codes int8 [R, K] held by an FP6 block-layout buffer (the inverse of
    fp6_layout_ref); also returns the codes of the padding rows [Rp - R, K]."""
    Rp = (R + 31) // 32 * 32
    nkb = K // 128
    b = np.ascontiguousarray(buf).reshape(nkb, Rp // 32, 2, 3, 64, 8)   # kb, rb, s, c, l, byte
    words = b.transpose(0, 1, 2, 4, 3, 5).copy().view(np.uint64)[..., 0]  # kb, rb, s, l, c
    fields = np.empty(words.shape[:-1] + (32,), dtype=np.uint64)
    for j in range(32):
        pos = 6 * j
        w, off = pos // 64, pos % 64
        v = words[..., w] >> np.uint64(off)
        if off > 58:
            v = v | (words[..., w + 1] << np.uint64(64 - off))
        fields[..., j] = v & np.uint64(0x3F)
    inv = np.full(64, 127, dtype=np.int64)
    for c, bits6 in e2m3_table().items():
        inv[bits6] = c
    codes = inv[fields.astype(np.int64)]                    # kb, rb, s, l, j
    assert (codes != 127).all(), "FP6 field that is no 4-bit code"
    # lane l = 32 g + r, k = 128 kb + 64 g + 32 s + j
    c6 = codes.reshape(nkb, Rp // 32, 2, 2, 32, 32)          # kb, rb, s, g, r, j
    c6 = c6.transpose(1, 4, 0, 3, 2, 5).reshape(Rp, K)       # rb, r, kb, g, s, j
    return c6[:R].astype(np.int8), c6[R:].astype(np.int8)


def oracle_prepare(w, h):
    """oracle.prepare_weights_ref over row chunks on a thread pool."""
    from oracle import prepare_weights_ref
    N = w.shape[0]
    chunks = [c for c in np.array_split(np.arange(N), min(N, 4 * WORKERS)) if c.size]
    with ThreadPoolExecutor(WORKERS) as ex:
        parts = list(ex.map(lambda r: prepare_weights_ref(w[r[0]:r[-1] + 1], h), chunks))
    return np.concatenate([p[0] for p in parts]), np.concatenate([p[1] for p in parts])


def assert_acc(got, ref, what):
    """int32 accumulators against the oracle's, naming where they differ."""
    g = np.asarray(got).astype(np.int64)
    if np.array_equal(g, ref):
        return
    bad = np.nonzero(g != ref)
    rows, cols = bad
    raise AssertionError(
        f"{what}: {rows.size} accumulators differ; rows {np.unique(rows)[:12]} "
        f"({np.unique(rows).size} rows, 256-row tiles {np.unique(rows // 256)[:12]}), "
        f"cols {np.unique(cols)[:12]} ({np.unique(cols).size} cols, 192-col tiles "
        f"{np.unique(cols // 192)[:12]}); got {g[bad][:6]} want {ref[bad][:6]}")


def decode_layout_ref(w_packed):
    """The decode layout written out from its definition: for 16-row block b,
    128-k chunk c, 16-byte piece g of the chunk and row r of the block, the
    piece sits at 16-byte position ((b * (K / 128) + c) * 4 + g) * 16 + r."""
    w = np.ascontiguousarray(w_packed)
    N, half = w.shape
    K = half * 2
    pieces = w.reshape(N // 16, 16, K // 128, 4, 16)        # [b, r, c, g, byte]
    return np.ascontiguousarray(pieces.transpose(0, 2, 3, 1, 4)).reshape(-1)
