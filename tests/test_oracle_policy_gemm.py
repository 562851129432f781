"""Pins for the oracle's policy, integer GEMM and epilogue.

The policy is checked against the sensitive sets the paper prints
(tests/golden/policy_sets.txt); the GEMM against pure-Python brute force and an
independent fp64 BLAS product (exact here); the epilogue against exact
rational rounding and the fp16 rounding bound; and the whole quantized linear
against the unquantized X W^T (Eq. 5).
"""

import itertools
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle.gemm import qlinear_acc_ref, qlinear_acc_entries, epilogue_ref, qlinear_ref
from oracle.policy import layer_policy_ref
from oracle.hadamard import hadamard
from oracle.quant import pack_int4, unpack_int4, rotate_quant_ref, prepare_weights_ref

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "policy_sets.txt")


def _golden_sets():
    rows = []
    for line in open(GOLDEN):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        model, L, sset, indexing, cite = [f.strip() for f in line.split("|")]
        s = [int(v) for v in sset.split(",")]
        if indexing == "1-indexed":
            s = [v - 1 for v in s]
        rows.append((model, int(L), sorted(s)))
    return rows


@pytest.mark.parametrize("model,L,sens", _golden_sets())
def test_default_policy_matches_paper_sets(model, L, sens):
    bits = layer_policy_ref(L)
    assert [i for i, b in enumerate(bits) if b == 8] == sens
    assert all(b == 4 for i, b in enumerate(bits) if i not in sens)


def test_policy_mask_and_small_L():
    assert layer_policy_ref(1) == [8]
    assert layer_policy_ref(3) == [8, 8, 8]
    assert layer_policy_ref(5) == [8, 8, 8, 4, 8]
    mask = [0] * 10
    mask[4] = mask[7] = 1
    assert layer_policy_ref(10, mask) == [4, 4, 4, 4, 8, 4, 4, 8, 4, 4]
    with pytest.raises(ValueError):
        layer_policy_ref(0)
    with pytest.raises(ValueError):
        layer_policy_ref(4, [1, 0])


@pytest.mark.parametrize("bits", [4, 8])
def test_gemm_brute_force_all_code_pairs(bits):
    # K = 2: every activation code against every weight code.
    lo_a = -8 if bits == 4 else -128
    hi_a = 7 if bits == 4 else 127
    a_vals = list(range(lo_a, hi_a + 1))
    w_vals = list(range(-8, 8))
    A = np.array([[a, b] for a, b in itertools.product(a_vals, [lo_a, hi_a, 0, 1])])
    W = np.array([[a, b] for a, b in itertools.product(w_vals, [-8, 7, -1])])
    a_codes = pack_int4(A) if bits == 4 else A.astype(np.int8)
    acc = qlinear_acc_ref(a_codes, bits, pack_int4(W))
    for m in range(A.shape[0]):
        for n in range(W.shape[0]):
            assert acc[m, n] == int(A[m, 0]) * int(W[n, 0]) + int(A[m, 1]) * int(W[n, 1])


@pytest.mark.parametrize("bits", [4, 8])
def test_gemm_loops_and_blas_agree(bits):
    rng = np.random.default_rng(bits)
    M, N, K = 9, 7, 96
    lim = 8 if bits == 4 else 128
    A = rng.integers(-lim, lim, size=(M, K))
    W = rng.integers(-8, 8, size=(N, K))
    a_codes = pack_int4(A) if bits == 4 else A.astype(np.int8)
    acc = qlinear_acc_ref(a_codes, bits, pack_int4(W))
    loops = np.array([[sum(int(A[m, k]) * int(W[n, k]) for k in range(K))
                       for n in range(N)] for m in range(M)])
    assert np.array_equal(acc, loops)
    # fp64 BLAS is exact here (every partial sum is an integer far below 2^53).
    assert np.array_equal(acc, (A.astype(np.float64) @ W.T.astype(np.float64)).astype(np.int64))
    rows, cols = [0, 3, 8], [6, 0, 2]
    assert qlinear_acc_entries(a_codes, bits, pack_int4(W), rows, cols).tolist() == \
        [loops[r, c] for r, c in zip(rows, cols)]


def test_accumulator_fits_int32_at_largest_k():
    # Worst case at K = 28672: |acc| <= K * 128 * 8 < 2^31.
    K = 28672
    A = np.full((1, K), -128, dtype=np.int8)
    W = np.full((1, K), -8)
    acc = qlinear_acc_ref(A, 8, pack_int4(W))
    assert acc[0, 0] == K * 1024 and acc[0, 0] < 2 ** 31


def _f16_rne(fr):
    """Correctly rounded fp16 of a Fraction in the normal range."""
    if fr == 0:
        return 0.0
    sign = -1 if fr < 0 else 1
    a = abs(fr)
    e = a.numerator.bit_length() - a.denominator.bit_length()
    if Fraction(2) ** e > a:
        e -= 1
    e = max(e, -14)                 # subnormals share the 2^-24 ulp
    ulp = Fraction(2) ** (e - 10)
    q, r = divmod(a, ulp)
    if r * 2 > ulp or (r * 2 == ulp and q % 2 == 1):
        q += 1
    return sign * float(q * ulp)


def test_fp16_conversion_is_round_half_even():
    # Ties in fp32 -> fp16: 1 + 2^-11 -> 1; 1 + 3*2^-11 -> 1 + 2^-9; subnormal tie.
    v = np.array([1 + 2 ** -11, 1 + 3 * 2 ** -11, 2 ** -25, 3 * 2 ** -25, -(1 + 2 ** -11)],
                 dtype=np.float32)
    got = v.astype(np.float16).astype(np.float64)
    assert got.tolist() == [1.0, 1 + 2 ** -9, 0.0, 2 ** -23, -1.0]
    rng = np.random.default_rng(1)
    w = (rng.standard_normal(2000) * 10.0 ** rng.uniform(-6, 4, 2000)).astype(np.float32)
    assert w.astype(np.float16).astype(np.float64).tolist() == \
        [_f16_rne(Fraction(float(t))) for t in w]


def test_epilogue_rounding_bound():
    # fl16(fl32(fl32(acc) a_s) w_s) is within one fp16 ulp (plus the two fp32
    # roundings) of the exact product acc * a_s * w_s.
    rng = np.random.default_rng(2)
    acc = rng.integers(-3_000_000, 3_000_000, size=(64, 64))
    a_s = rng.uniform(0.01, 2, 64).astype(np.float32)
    w_s = rng.uniform(1e-5, 1e-3, 64).astype(np.float32)
    y = epilogue_ref(acc, a_s, w_s).astype(np.float64)
    exact = acc.astype(np.float64) * a_s.astype(np.float64)[:, None] * w_s.astype(np.float64)[None, :]
    ulp16 = 2.0 ** (np.floor(np.log2(np.abs(exact))) - 10)
    assert np.all(np.abs(y - exact) <= ulp16 * (0.5 + 2 ** -10))


def _pinned_epilogue_exact(acc, a_s, w_s):
    """fl16(fl32(fl32(fl32(acc) a_s) w_s)) with every rounding done on Fractions."""
    from test_oracle_quant import _round_to_f32
    t = Fraction(_round_to_f32(Fraction(int(acc))))
    t = Fraction(_round_to_f32(t * Fraction(float(a_s))))
    t = Fraction(_round_to_f32(t * Fraction(float(w_s))))
    return _f16_rne(t)


def test_epilogue_order_on_discriminating_entries():
    # Entries where another operation order (fl32(a_s * w_s) first) changes the
    # fp16 result; on them the oracle must agree with exact rational rounding
    # of the pinned order.
    rng = np.random.default_rng(4)
    n = 400_000
    acc = rng.integers(-30_000_000, 30_000_000, size=n)
    a_s = rng.uniform(1e-3, 1, n).astype(np.float32)
    w_s = rng.uniform(1e-6, 1e-3, n).astype(np.float32)
    acc32 = acc.astype(np.float32)
    other = (acc32 * (a_s * w_s).astype(np.float32)).astype(np.float16)
    candidate = ((acc32 * a_s).astype(np.float32) * w_s).astype(np.float16)
    idx = np.nonzero(candidate != other)[0][:40]
    assert len(idx) >= 5
    for i in idx:
        y = epilogue_ref(np.array([[acc[i]]]), a_s[i:i + 1], w_s[i:i + 1])[0, 0]
        assert float(y) == _pinned_epilogue_exact(acc[i], a_s[i], w_s[i])
        assert y != other[i]
