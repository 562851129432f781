"""Pins for the oracle's Hadamard matrices and pinned-order rotation.

Each test checks the oracle against something other than itself: a library
routine (scipy's Sylvester matrix), the defining property H H^T = h I, exact
integer arithmetic, an independent butterfly algorithm, Parseval (Eq. 12) and
the pairwise-summation error bound.
"""

import numpy as np
import pytest
import scipy.linalg

import oracle
from oracle.hadamard import (paley28, sylvester, sylvester_columns, hadamard,
                             rotate_rows, split_had_size)

POW2 = [1, 2, 4, 8, 16, 32, 64, 128, 256, 512, 1024, 2048, 4096]


@pytest.mark.parametrize("n", POW2)
def test_sylvester_matches_scipy(n):
    # scipy.linalg.hadamard builds the same natural-order Sylvester matrix.
    assert np.array_equal(sylvester(n), scipy.linalg.hadamard(n).astype(np.int64))


@pytest.mark.parametrize("n", POW2)
def test_closed_form_columns_match_recursion(n):
    # The rotation draws column chunks from (-1)^popcount(c & d); it must be
    # the recursive Sylvester matrix.
    H = sylvester(n)
    assert np.array_equal(sylvester_columns(n, 0, n).astype(np.int64), H)
    if n >= 4:
        assert np.array_equal(sylvester_columns(n, n // 4, n // 2).astype(np.int64),
                              H[:, n // 4:n // 2])


def test_paley28_is_hadamard():
    H = paley28()
    assert H.shape == (28, 28)
    assert set(np.unique(H)) == {-1, 1}
    assert np.array_equal(H @ H.T, 28 * np.eye(28, dtype=np.int64))
    assert np.array_equal(H, H.T)          # Paley II with q = 1 mod 4 is symmetric


def test_paley_quadratic_residues_mod13():
    # The nonzero squares mod 13 are {1, 3, 4, 9, 10, 12}: the first row of the
    # Jacobsthal block Q (row index 1 of C) must be +1 exactly there.
    H = paley28()
    # Recover C[1, 1:] = Q[0, :] from the (row 2, even column) entries of
    # C (x) H2 + I (x) G: for blocks p != q, H[2p, 2q] = C[p, q].
    q_row = np.array([H[2, 2 * (1 + j)] for j in range(1, 13)])
    expect = np.array([1 if j in (1, 3, 4, 9, 10, 12) else -1 for j in range(1, 13)])
    assert np.array_equal(q_row, expect)


def test_paley28_diagonal_blocks_by_hand():
    # The conference matrix C has a zero diagonal, so the 2 x 2 diagonal blocks
    # of C (x) [[1,1],[1,-1]] + I_14 (x) G are G itself, G = [[1,-1],[-1,-1]].
    # Negating G (or dropping it) still gives a symmetric Hadamard matrix, so
    # only this literal pins the sign of the identity term.
    H = paley28()
    G = np.array([[1, -1], [-1, -1]])
    for p in range(14):
        assert np.array_equal(H[2 * p:2 * p + 2, 2 * p:2 * p + 2], G), f"diagonal block {p}"


def test_paley28_rows_written_out():
    # Rows 2 and 3 (block row 1) worked by hand: C[1, :] = [1, chi(0), ...,
    # chi(12)] = [1, 0, 1,-1, 1, 1,-1,-1,-1,-1, 1, 1,-1, 1] (squares mod 13 are
    # 1, 3, 4, 9, 10, 12); block q contributes C[1,q]*[1, 1] and C[1,q]*[1,-1]
    # off the diagonal and G's rows [1,-1], [-1,-1] on it (q = 1).  Row 0 is
    # [1,-1] followed by thirteen [1, 1] blocks.
    def parse(s):
        return np.array([1 if ch == "+" else -1 for ch in s.replace(" ", "")])
    H = paley28()
    assert np.array_equal(H[0], parse("+- ++ ++ ++ ++ ++ ++ ++ ++ ++ ++ ++ ++ ++"))
    assert np.array_equal(H[2], parse("++ +- ++ -- ++ ++ -- -- -- -- ++ ++ -- ++"))
    assert np.array_equal(H[3], parse("+- -- +- -+ +- +- -+ -+ -+ -+ +- +- -+ +-"))


@pytest.mark.parametrize("h", [28, 56, 112, 448, 896, 28 * 128])
def test_kronecker_hadamard_orthogonal(h):
    # fp64 products of +-1 matrices are exact (sums of at most h < 2^53 terms).
    H = hadamard(h).astype(np.float64)
    assert np.array_equal(H @ H.T, h * np.eye(h))


@pytest.mark.parametrize("h", [3, 12, 20, 36, 84, 0, -4, 28 * 3])
def test_split_rejects_unsupported(h):
    with pytest.raises(ValueError):
        split_had_size(h)


def _int_inputs(rng, M, K, lim):
    return rng.integers(-lim, lim + 1, size=(M, K)).astype(np.float32)


@pytest.mark.parametrize("h,K", [(2, 8), (16, 64), (256, 256), (256, 1024),
                                 (4096, 4096), (28, 56), (28 * 16, 28 * 32),
                                 (28 * 64, 28 * 64)])
def test_rotation_exact_on_integers(h, K):
    # Small integers keep every partial sum exact in fp32, so the pinned-order
    # rotation must equal the int64 matrix product with I (x) H exactly.  A
    # dropped term, a wrong sign or a wrong index breaks this.
    rng = np.random.default_rng(h * 7 + K)
    x = _int_inputs(rng, 5, K, 50)
    y = rotate_rows(x, h)
    B = np.kron(np.eye(K // h, dtype=np.int64), hadamard(h))
    expect = (x.astype(np.float64) @ B.astype(np.float64)).astype(np.int64)  # exact
    assert np.array_equal(y.astype(np.int64), expect)
    assert np.array_equal(y, expect.astype(np.float32))


def _fwht_bit0_first(x):
    """Radix-2 in-place Walsh-Hadamard butterflies in fp32, index bit 0 first."""
    y = np.array(x, dtype=np.float32, copy=True)
    n = y.shape[-1]
    half = 1
    while half < n:
        v = y.reshape(y.shape[:-1] + (n // (2 * half), 2, half))
        a = v[..., 0, :].copy()
        b = v[..., 1, :].copy()
        v[..., 0, :] = a + b
        v[..., 1, :] = a - b
        half *= 2
    return y


@pytest.mark.parametrize("h", [2, 8, 64, 256, 1024, 4096])
def test_tree_order_equals_bit0_first_fwht(h):
    # The pinned pairwise-tree order is the order of a radix-2 FWHT that
    # processes bit 0 first; on random fp32 data the two agree bit for bit.
    rng = np.random.default_rng(h)
    x = rng.standard_normal((3, h)).astype(np.float32) * np.float32(3.0)
    y = rotate_rows(x, h)
    assert np.array_equal(y.view(np.uint32) & 0x7FFFFFFF,
                          _fwht_bit0_first(x).view(np.uint32) & 0x7FFFFFFF)
    assert np.array_equal(y, _fwht_bit0_first(x))


def test_tree_order_differs_from_sequential_order():
    # The order matters: a sequential left-to-right sum gives different bits
    # on random data, so the pin above is not vacuous.
    rng = np.random.default_rng(11)
    x = rng.standard_normal((1, 1024)).astype(np.float32)
    H = sylvester(1024).astype(np.float32)
    seq = np.zeros(1024, dtype=np.float32)
    for i in range(1024):
        seq = seq + x[0, i] * H[i]
    assert not np.array_equal(seq, rotate_rows(x, 1024)[0])


@pytest.mark.parametrize("h,K", [(256, 256), (4096, 4096), (28 * 64, 28 * 64),
                                 (256, 1024)])
def test_parseval_and_error_bound(h, K):
    # Eq. 12: an orthogonal rotation preserves the norm; with the unnormalised
    # B_h this reads ||x B||^2 = h ||x||^2 per block.  The fp32 result must sit
    # within the pairwise (and, for the 28-point stage, recursive) summation
    # bound of the exact product: |err| <= gamma_n * sum|x| with
    # n = log2(p) + (f - 1) rounding steps (Higham, Accuracy and Stability of
    # Numerical Algorithms, Sec. 4.2), u = 2^-24.
    rng = np.random.default_rng(K + h)
    x = (rng.standard_t(3, size=(4, K)) * 4).astype(np.float16)
    y = rotate_rows(x, h).astype(np.float64)
    x64 = x.astype(np.float64)
    B = np.kron(np.eye(K // h), hadamard(h).astype(np.float64))
    exact = x64 @ B
    f, p = split_had_size(h)
    n = int(np.log2(p)) + (f - 1)
    u = 2.0 ** -24
    gamma = n * u / (1 - n * u)
    for blk in range(K // h):
        sl = slice(blk * h, (blk + 1) * h)
        bound = gamma * np.abs(x64[:, sl]).sum(axis=1, keepdims=True)
        assert np.all(np.abs(y[:, sl] - exact[:, sl]) <= bound)
        np.testing.assert_allclose((y[:, sl] ** 2).sum(1),
                                   h * (x64[:, sl] ** 2).sum(1), rtol=1e-5)


def test_block_diagonal_locality():
    # B_h = I (x) H_h: input confined to one block stays in that block.
    rng = np.random.default_rng(5)
    x = np.zeros((1, 1024), dtype=np.float32)
    x[0, 512:768] = rng.standard_normal(256)
    y = rotate_rows(x, 256)
    assert np.all(y[0, :512] == 0) and np.all(y[0, 768:] == 0)
    assert np.any(y[0, 512:768] != 0)


def test_one_hot_rows_give_unit_magnitudes():
    # x = e_i gives the i-th row of H: every entry +-1 (closed form).
    for h in (256, 28 * 8):
        for i in (0, 5, h - 1):
            x = np.zeros((1, h), dtype=np.float16)
            x[0, i] = 1
            y = rotate_rows(x, h)
            assert np.array_equal(y[0], hadamard(h)[i].astype(np.float32))


def test_jump_ratio_rotation_invariant():
    # Eq. 12-13: with the orthonormal R = B / sqrt(h), ||xR|| = ||x|| and the
    # per-token Jump Ratio ||dx R|| / (||x R|| + eps) is unchanged.
    rng = np.random.default_rng(9)
    h = 256
    x = rng.standard_normal((6, h)).astype(np.float32)
    dx = (rng.standard_normal((6, h)) * 5).astype(np.float32)
    R = hadamard(h).astype(np.float64) / np.sqrt(h)
    eps = 1e-6
    jr = np.linalg.norm(dx, axis=1) / (np.linalg.norm(x, axis=1) + eps)
    jr_rot = (np.linalg.norm(rotate_rows(dx, h) / np.sqrt(h), axis=1)
              / (np.linalg.norm(rotate_rows(x, h) / np.sqrt(h), axis=1) + eps))
    np.testing.assert_allclose(jr_rot, jr, rtol=1e-5)
    np.testing.assert_allclose(R @ R.T, np.eye(h), atol=1e-12)


@pytest.mark.parametrize("p", [1, 8, 64, 512])
def test_28_stage_is_sequential_over_slow_index(p):
    # Independent route to the pinned 28 * 2^j order: bit-0-first butterflies
    # over the fast index c, then numpy's sequential running sum
    # (np.add.accumulate) over the slow index a = 0..27.
    rng = np.random.default_rng(p + 28)
    h = 28 * p
    x = (rng.standard_normal((2, h)) * 7).astype(np.float32)
    z = _fwht_bit0_first(x.reshape(2, 28, p))                # [m, a, d]
    H28 = paley28().astype(np.float32)
    terms = H28[None, :, :, None] * z[:, :, None, :]          # [m, a, b, d]
    expect = np.add.accumulate(terms, axis=1)[:, -1]          # [m, b, d]
    assert np.array_equal(rotate_rows(x, h), expect.reshape(2, h))
