"""Hadamard matrices and the block rotation y = x . B_h  (oracle; test infrastructure).

What the paper fixes (Section 2, Eq. 4 and Eq. 5): activations are quantized in
a rotated space X R with R^T R = I, and the rotation is absorbed into the weight
offline.  It names Hadamard rotations (QuaRot-style) as the fixed choice.  It
fixes neither the matrix for non-power-of-two sizes, nor the normalisation, nor
an arithmetic order.  The readings used here:

* H_{2^j}: Sylvester's construction in natural order,
  H_1 = [1], H_{2m} = [[H_m, H_m], [H_m, -H_m]].
* H_28: Paley's second construction with q = 13 (13 = 1 mod 4):
  Q_ij = chi(j - i) (quadratic character mod 13), the symmetric conference
  matrix C = [[0, 1^T], [1, Q]] (14x14), and
  H_28 = C (x) [[1, 1], [1, -1]] + I_14 (x) [[1, -1], [-1, -1]].
* H_{28 * 2^j} = H_28 (x) H_{2^j}: H_28 acts on the slow index a of
  i = a * 2^j + c, H_{2^j} on the fast index c.
* B_h = I_{K/h} (x) H_h, unnormalised (+-1 entries); the 1/h that makes
  (xB)(WB)^T = h X W^T exact is folded into the weight scale (quant module).
* Arithmetic: the input is widened to fp32 (exact), every product x_i * H_id is
  exact (+-x_i), and the sum over i is taken in fp32 in this pinned order:
    - over the fast index c: a pairwise tree in index order (adjacent pairs
      first: P[0::2] + P[1::2], repeated), one fp32 rounding per add;
    - for 28 * 2^j sizes, the 28 partial results over the slow index a are
      then added sequentially, a = 0, 1, ..., 27.
  The tree order is the one a radix-2 fast Walsh-Hadamard transform produces
  when it processes index bit 0 first, then bit 1, and so on.
"""

import functools

import numpy as np

__all__ = ["sylvester", "sylvester_columns", "paley28", "hadamard", "split_had_size",
           "rotate_rows"]


def sylvester(n):
    """Sylvester Hadamard matrix of order n = 2^j, natural order, int64."""
    return _sylvester_i8(int(n)).astype(np.int64)


@functools.lru_cache(maxsize=8)
def _sylvester_i8(n):
    if n < 1 or (n & (n - 1)) != 0:
        raise ValueError(f"Sylvester order must be a power of two, got {n}")
    H = np.ones((1, 1), dtype=np.int8)
    while H.shape[0] < n:
        m = H.shape[0]
        G = np.empty((2 * m, 2 * m), dtype=np.int8)
        G[:m, :m] = H
        G[:m, m:] = H
        G[m:, :m] = H
        G[m:, m:] = -H
        H = G
    H.setflags(write=False)
    return H


def sylvester_columns(n, d0, d1):
    """Columns d0..d1-1 of the natural-order Sylvester matrix of order n, fp32,
    from the closed form H[c, d] = (-1)^popcount(c AND d) (equal to the
    recursive construction; used so large orders never materialise n x n)."""
    c = np.arange(n, dtype=np.uint32)[:, None]
    d = np.arange(d0, d1, dtype=np.uint32)[None, :]
    parity = np.bitwise_count(c & d) & 1
    return (1 - 2 * parity.astype(np.int8)).astype(np.float32)


def _quadratic_character(a, q):
    """chi(a) for prime q: 0 if a = 0 mod q, +1 if a is a nonzero square, else -1."""
    a %= q
    if a == 0:
        return 0
    squares = {(x * x) % q for x in range(1, q)}
    return 1 if a in squares else -1


def paley28():
    """Order-28 Hadamard matrix from Paley's construction II with q = 13, int64."""
    q = 13
    Q = np.array([[_quadratic_character(j - i, q) for j in range(q)]
                  for i in range(q)], dtype=np.int64)
    C = np.zeros((q + 1, q + 1), dtype=np.int64)
    C[0, 1:] = 1
    C[1:, 0] = 1
    C[1:, 1:] = Q
    H2 = np.array([[1, 1], [1, -1]], dtype=np.int64)
    G = np.array([[1, -1], [-1, -1]], dtype=np.int64)
    return np.kron(C, H2) + np.kron(np.eye(q + 1, dtype=np.int64), G)


def split_had_size(h):
    """Return (f, p) with h = f * p, f in {1, 28}, p a power of two; else ValueError."""
    h = int(h)
    if h >= 1 and (h & (h - 1)) == 0:
        return 1, h
    if h >= 28 and h % 28 == 0:
        p = h // 28
        if (p & (p - 1)) == 0:
            return 28, p
    raise ValueError(f"unsupported Hadamard size {h}: need 2^j or 28*2^j")


def hadamard(h):
    """The order-h Hadamard matrix used by the rotation (int64, symmetric)."""
    f, p = split_had_size(h)
    Hp = sylvester(p)
    if f == 1:
        return Hp
    return np.kron(paley28(), Hp)


@functools.lru_cache(maxsize=4)
def _column_chunks(p, chunk_elems=1 << 20):
    cols = max(1, chunk_elems // p)
    out = []
    for d0 in range(0, p, cols):
        d1 = min(p, d0 + cols)
        H = sylvester_columns(p, d0, d1)
        H.setflags(write=False)
        out.append((d0, d1, H))
    return tuple(out) if p * p <= (1 << 26) else None


def _rotate_fast_index(xa, p, chunk_elems=1 << 20, batch_elems=1 << 20):
    """z[r, d] = sum_c xa[r, c] * H_p[c, d] for every row r, pairwise tree over c
    in index order (fp32).  Rows are independent; they are only grouped so
    that one array operation covers several of them."""
    B = xa.shape[0]
    z = np.empty((B, p), dtype=np.float32)
    chunks = _column_chunks(p)
    if chunks is None:   # large orders: regenerate columns instead of caching them
        cols = max(1, chunk_elems // p)
        chunks = ((d0, min(p, d0 + cols), None) for d0 in range(0, p, cols))
    for d0, d1, H in chunks:
        if H is None:
            H = sylvester_columns(p, d0, d1)
        rb = max(1, batch_elems // (p * (d1 - d0)))
        for r0 in range(0, B, rb):
            P = xa[r0:r0 + rb, :, None] * H[None]       # exact: entries are +-1
            while P.shape[1] > 1:                       # adjacent pairs first
                P = P[:, 0::2] + P[:, 1::2]
            z[r0:r0 + rb, d0:d1] = P[:, 0]
    return z


def rotate_rows(x, h):
    """y = x . (I_{K/h} (x) H_h) for every row of x, in fp32 with the pinned order.

    x: [M, K] float16 or float32 (K a multiple of h).  Returns float32 [M, K].
    Every length-h block of every row is rotated on its own; the blocks are
    only stacked so that the same sums run as whole-array operations.
    """
    x = np.asarray(x)
    if x.ndim != 2:
        raise ValueError("x must be 2-D [M, K]")
    M, K = x.shape
    f, p = split_had_size(h)
    if K % h != 0:
        raise ValueError(f"K={K} is not a multiple of the Hadamard size {h}")
    xb = x.astype(np.float32).reshape(M * (K // h), f, p)   # fp16 -> fp32 is exact; i = a*p + c
    z = np.stack([_rotate_fast_index(np.ascontiguousarray(xb[:, a, :]), p) for a in range(f)],
                 axis=1)                                     # [blocks, f, p]
    if f == 1:
        return z.reshape(M, K)
    H28 = paley28().astype(np.float32)
    out = np.empty_like(z)
    for b in range(f):
        acc = H28[0, b] * z[:, 0]
        for a in range(1, f):                                # sequential over a = 0..27
            acc = acc + H28[a, b] * z[:, a]
        out[:, b] = acc
    return out.reshape(M, K)
