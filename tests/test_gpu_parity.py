"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Bar (all bit for bit): activation and weight codes and scales, int32
accumulators, and fp16 outputs (the epilogue order is pinned, so the graded
1-ulp / 1e-3 tolerance is reported but exact equality is required).  Inputs
are seeded; GEMM inputs are seeded random code bytes so that no oracle input
comes from the HIP path.  Full-size shapes are checked on sampled rows the
oracle computes one by one.
"""

import numpy as np
import pytest

import workloads
from oracle import (rotate_quant_ref, prepare_weights_ref, qlinear_acc_ref,
                    epilogue_ref, unpack_int4)
from oracle.gemm import qlinear_acc_entries

torch = pytest.importorskip("torch")
dptq = pytest.importorskip("paper_2606_12487_amd")

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    dptq.lib()
    return torch.device("cuda:0")


def _d(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def _h(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def _sample_rows(M, n, rng):
    if M <= n:
        return np.arange(M)
    rows = set([0, M - 1])
    rows.update(rng.choice(M, n - 2, replace=False).tolist())
    return np.array(sorted(rows))


def _assert_codes(got, ref, what):
    bad = np.nonzero(got != ref)
    assert bad[0].size == 0, f"{what}: {bad[0].size} code bytes differ, first at {bad[0][0]},{bad[1][0]}"


def _assert_f32(got, ref, what):
    assert np.array_equal(got.view(np.uint32), ref.view(np.uint32)), \
        f"{what}: {(got.view(np.uint32) != ref.view(np.uint32)).sum()} scales differ"


def _assert_f16(got, ref, what):
    assert np.isfinite(ref.astype(np.float32)).all(), f"{what}: expected outputs overflow fp16"
    g, r = got.view(np.uint16), ref.view(np.uint16)
    if np.array_equal(g, r):
        return
    gf, rf = got.astype(np.float64), ref.astype(np.float64)
    rel = np.max(np.abs(gf - rf) / np.maximum(np.abs(rf), 1e-30))
    raise AssertionError(f"{what}: {(g != r).sum()} outputs differ (max rel err {rel:.3g})")


# --------------------------------------------------------------------------
# rotate + quantize
# --------------------------------------------------------------------------
ROT_CASES = [
    # (M, K, h)  small, ragged and edge shapes; every row checked
    (1, 8, 8), (3, 16, 1), (5, 64, 2), (7, 256, 256), (37, 1024, 1024),
    (33, 1024, 256), (9, 896, 28 * 32), (4, 224, 28 * 8), (6, 56, 28),
    (3, 112, 28 * 4), (130, 2048, 2048),
    (2, 28672, 28 * 1024), (2, 36864, 4096), (3, 8192, 8192),
    (2, 11008, 256), (16, 256, 256), (2, 28672, 28 * 512),
    (3, 4096, 512), (2, 16384, 16384), (5, 12288, 4096), (4, 4160, 64),
    (3, 4224, 128), (2, 4104, 8), (3, 4120, 8),
    # more than 64 rows so long that one compute unit holds one of them
    # (1024 threads per row in four groups; 7 and 6 segments, so the groups
    # take unequal shares)
    (70, 28672, 28 * 1024), (66, 24576, 8192),
    # more such rows than compute units: each workgroup touches the next row
    # of its XCD into the L2 once its own row is staged
    (300, 28672, 28 * 1024), (257, 24576, 8192),
    # more rows than resident 256-thread workgroups (four per compute unit
    # at this size): the same touch one round of residents ahead
    (1030, 8192, 8192),
    # more than 64 rows of up to 16384 with h = 28 * 2^j or 2^j above 4096
    # (a partial last 4096-element segment, block-diagonal sizes); at
    # h = 16384 the segmented kernel
    (65, 8192, 8192), (100, 14336, 28 * 512), (72, 16384, 16384), (80, 7168, 28 * 256),
    (66, 3584, 28 * 128), (67, 16384, 8192), (129, 12544, 28 * 64),
]


@pytest.mark.parametrize("bits", [4, 8])
@pytest.mark.parametrize("M,K,h", ROT_CASES)
def test_rotate_quant_shapes(dev, M, K, h, bits):
    rng = np.random.default_rng(M * 1000 + K + h)
    x = workloads.gauss_outliers(rng, M, K, n_channels=min(4, K))
    codes, scales = dptq.rotate_quant(_d(x, dev), h, bits)
    c_ref, s_ref = rotate_quant_ref(x, h, bits)
    _assert_f32(_h(scales), s_ref, f"scales M={M} K={K} h={h}")
    _assert_codes(_h(codes), c_ref, f"codes M={M} K={K} h={h}")


def _exact_fwht(x):
    """Walsh-Hadamard transform of integer-valued rows in float64 (every sum is
    an exact integer here, so any order gives the exact x . H)."""
    y = x.astype(np.float64).copy()
    n = y.shape[1]
    half = 1
    while half < n:
        v = y.reshape(y.shape[0], n // (2 * half), 2, half)
        a, b = v[:, :, 0, :].copy(), v[:, :, 1, :].copy()
        v[:, :, 0, :], v[:, :, 1, :] = a + b, a - b
        half *= 2
    return y


@pytest.mark.parametrize("bits", [4, 8])
def test_rotate_quant_largest_hadamard(dev, bits):
    # h = 32768 (the largest supported size) on integer-valued rows: every
    # partial sum is exact in fp32, so the rotation is the exact x . H in any
    # order and the oracle quantizes that exact product.
    from oracle import quantize_rows, pack_int4
    rng = np.random.default_rng(32768 + bits)
    x = rng.integers(-8, 9, size=(3, 32768)).astype(np.float16)
    codes, scales = dptq.rotate_quant(_d(x, dev), 32768, bits)
    y = _exact_fwht(x).astype(np.float32)
    c_ref, s_ref = quantize_rows(y, bits)
    if bits == 4:
        c_ref = pack_int4(c_ref)
    _assert_f32(_h(scales), s_ref, "h=32768 scales")
    _assert_codes(_h(codes), c_ref, "h=32768 codes")


@pytest.mark.parametrize("bits", [4, 8])
def test_rotate_quant_special_rows(dev, bits):
    K, h = 512, 512
    x = np.zeros((8, K), dtype=np.float16)
    x[1, 7] = 1.0                       # one-hot: all codes +-qmax
    x[2, 300] = -3.5
    x[3, :] = 2.0                       # constant row: energy in one output
    x[4, ::2] = 1.0
    x[4, 1::2] = -1.0
    x[5, 0] = 65504.0                   # largest fp16
    x[6, 100] = 6e-8                    # fp16 subnormal
    # row 0 and 7 stay zero: scale 0, codes 0
    codes, scales = dptq.rotate_quant(_d(x, dev), h, bits)
    c_ref, s_ref = rotate_quant_ref(x, h, bits)
    _assert_f32(_h(scales), s_ref, "special scales")
    _assert_codes(_h(codes), c_ref, "special codes")


@pytest.mark.parametrize("bits", [4, 8])
@pytest.mark.parametrize("K,h", [(4096, 4096), (4096, 256), (14336, 28 * 512), (8192, 8192)])
def test_rotate_quant_subnormal_inputs(dev, bits, K, h):
    # Rows of fp16 subnormals and near-subnormal values (exact in fp32): the
    # rotation must not flush them.
    rng = np.random.default_rng(K + h + bits)
    mag = np.exp(rng.uniform(np.log(6e-8), np.log(2e-4), size=(4, K)))
    x = (mag * rng.choice([-1.0, 1.0], size=(4, K))).astype(np.float16)
    x[1] = (rng.integers(-1023, 1024, size=K) * 2.0 ** -24).astype(np.float16)   # all subnormal
    codes, scales = dptq.rotate_quant(_d(x, dev), h, bits)
    c_ref, s_ref = rotate_quant_ref(x, h, bits)
    _assert_f32(_h(scales), s_ref, "subnormal scales")
    _assert_codes(_h(codes), c_ref, "subnormal codes")


@pytest.mark.parametrize("bits", [4, 8])
def test_rotate_quant_exact_ties(dev, bits):
    # With h = 1 the rotation is the identity.  Rows whose absmax is 2*qmax
    # have s = 2 exactly, so odd integers divide to exact halves: ties must go
    # to even (Eq. 2 rounding, pinned half-to-even).
    qmax = 7 if bits == 4 else 127
    K = 256 if bits == 8 else 16
    vals = np.arange(-(2 * qmax - 1), 2 * qmax, 2, dtype=np.float32)
    x = np.zeros((2, K), dtype=np.float16)
    x[0, 0] = 2 * qmax
    x[0, 1:1 + vals.size] = vals[:K - 1]
    x[1, 0] = -2 * qmax
    x[1, 1:1 + vals.size] = -vals[:K - 1]
    codes, scales = dptq.rotate_quant(_d(x, dev), 1, bits)
    c_ref, s_ref = rotate_quant_ref(x, 1, bits)
    assert float(s_ref[0]) == 2.0
    _assert_f32(_h(scales), s_ref, "tie scales")
    _assert_codes(_h(codes), c_ref, "tie codes")


# --------------------------------------------------------------------------
# offline weight preparation (same kernel on fp32 rows)
# --------------------------------------------------------------------------
@pytest.mark.parametrize("N,K,h,nsample", [
    (512, 256, 256, 512), (272, 1024, 1024, 272), (64, 896, 28 * 32, 64),
    (12288, 4096, 4096, 12), (4096, 14336, 28 * 512, 12)])
def test_prepare_weights(dev, N, K, h, nsample):
    rng = np.random.default_rng(N + K)
    w = workloads.weights(rng, N, K)
    wp, ws = dptq.prepare_weights(_d(w, dev), h)
    rows = _sample_rows(N, nsample, rng)
    wp_ref, ws_ref = prepare_weights_ref(w[rows], h)
    _assert_f32(_h(ws)[rows], ws_ref, "w_scales")
    _assert_codes(_h(wp)[rows], wp_ref, "w codes")


def test_prepare_weights_near_ties(dev):
    # fp32 inputs whose quotient lies within a few ulps of a half-integer
    # exercise the correctly rounded division (h = 1: identity rotation).
    rng = np.random.default_rng(77)
    K = 256
    rows = []
    for _ in range(16):
        a = np.float32(rng.uniform(0.5, 4.0))
        s = np.float32(a / np.float32(7))
        vals = [a]
        for k in range(-7, 7):
            c = np.float32((k + 0.5) * float(s))
            for d in range(-4, 5):
                v = c
                for _ in range(abs(d)):
                    v = np.nextafter(v, np.float32(np.inf if d > 0 else -np.inf))
                if abs(v) <= a and len(vals) < K:
                    vals.append(v)
        rows.append(vals + [0.0] * (K - len(vals)))
    w = np.array(rows, dtype=np.float32)
    wp, ws = dptq.prepare_weights(_d(w, dev), 1)
    wp_ref, ws_ref = prepare_weights_ref(w, 1)
    _assert_f32(_h(ws), ws_ref, "near-tie scales")
    _assert_codes(_h(wp), wp_ref, "near-tie codes")


# --------------------------------------------------------------------------
# GEMM: exact accumulators and the epilogue
# --------------------------------------------------------------------------
GEMM_CASES = [
    # (M, K, N, sampled rows or None for all)
    (16, 256, 512, None), (17, 128, 16, None), (300, 1024, 272, None),
    (1, 14336, 4096, None), (4, 14336, 4096, None), (8, 8192, 1024, None),
    (16, 14336, 4096, None), (5, 11008, 64, None), (129, 4096, 528, None),
    (256, 512, 192, None), (511, 640, 400, None),
    (2048, 4096, 12288, 48), (2048, 14336, 4096, 32), (4096, 8192, 1024, 32),
    (2100, 1024, 12304, 48),
    # decode workgroups of two blocks of 16 channels (wide N, M * bits >= 64:
    # both widths at 16 tokens, A8 at 8) and of one block just below that
    (4, 256, 32768, None), (16, 128, 57344, None), (8, 1024, 16384, None), (7, 384, 24576, None),
    (3, 512, 32768, None),
]

# Every kernel must return the same bits; each case runs the automatic
# choice and every kernel whose range covers the shape.
KERNELS = (dptq.GEMM_DECODE, dptq.GEMM_TILE_256X128, dptq.GEMM_TILE_192X256)


def _fits(kernel, M, K, N):
    if kernel == dptq.GEMM_DECODE:
        return M <= 16
    if kernel == dptq.GEMM_TILE_192X256:
        return M >= 256 and N >= 192 and K >= 512
    return True


def _kernels_for(M, K, N):
    return [dptq.GEMM_AUTO] + [k for k in KERNELS if _fits(k, M, K, N)]


def _gemm_inputs(M, K, N, bits, seed):
    rng = np.random.default_rng(seed)
    a = workloads.random_code_bytes(rng, M, K, bits)
    w = workloads.random_weight_bytes(rng, N, K)
    a_s = workloads.random_scales(rng, M, 1e-3, 1.0)
    w_s = workloads.random_scales(rng, N, 1e-6, 1e-3)
    return a, w, a_s, w_s


@pytest.mark.parametrize("bits", [4, 8])
@pytest.mark.parametrize("M,K,N,ns", GEMM_CASES)
def test_gemm_acc_and_output(dev, M, K, N, ns, bits):
    a, w, a_s, w_s = _gemm_inputs(M, K, N, bits, M + K + N + bits)
    ad, wd, asd, wsd = _d(a, dev), _d(w, dev), _d(a_s, dev), _d(w_s, dev)
    rows = np.arange(M) if ns is None else _sample_rows(M, ns, np.random.default_rng(M))
    acc_ref = qlinear_acc_ref(a[rows], bits, w)
    y_ref = epilogue_ref(acc_ref, a_s[rows], w_s)
    for kernel in _kernels_for(M, K, N):
        acc = _h(dptq.qlinear_acc(ad, bits, wd, kernel=kernel))
        y = _h(dptq.qlinear(ad, asd, bits, wd, wsd, kernel=kernel))
        assert np.array_equal(acc[rows].astype(np.int64), acc_ref), \
            f"kernel {kernel}: {(acc[rows] != acc_ref).sum()} accumulators differ"
        _assert_f16(y[rows], y_ref, f"kernel {kernel}: y M={M} K={K} N={N}")


@pytest.mark.parametrize("bits", [4, 8])
@pytest.mark.parametrize("M,N", [(3, 32), (40, 32), (256, 192)])
def test_gemm_extreme_accumulators(dev, bits, M, N):
    # Largest magnitudes at the largest K: all activation codes at their
    # minimum and all weights at -8 give acc = K * 8 * |a_min| per entry.
    K = 65536
    a = (np.full((M, K // 2), 0x88, np.uint8) if bits == 4
         else np.full((M, K), -128, np.int8))
    w = np.full((N, K // 2), 0x88, np.uint8)
    w[1::2] = 0x77                      # +7 rows: negative accumulators
    ref = qlinear_acc_ref(a, bits, w)
    assert int(np.abs(ref).max()) == K * 8 * (8 if bits == 4 else 128)
    for kernel in _kernels_for(M, K, N):
        acc = _h(dptq.qlinear_acc(_d(a, dev), bits, _d(w, dev), kernel=kernel))
        assert np.array_equal(acc.astype(np.int64), ref), f"kernel {kernel}"


def test_gemm_entries_cross_check(dev):
    # One-by-one oracle entries at the full configuration size.
    M, K, N, bits = 2048, 4096, 12288, 4
    a, w, a_s, w_s = _gemm_inputs(M, K, N, bits, 5)
    acc = _h(dptq.qlinear_acc(_d(a, dev), bits, _d(w, dev)))
    rng = np.random.default_rng(6)
    rows = rng.integers(0, M, 200)
    cols = rng.integers(0, N, 200)
    ref = qlinear_acc_entries(a, bits, w, rows, cols)
    assert np.array_equal(acc[rows, cols].astype(np.int64), ref)


# --------------------------------------------------------------------------
# end to end: x -> rotate_quant -> qlinear, against the oracle pipeline
# --------------------------------------------------------------------------
_WEIGHT_CACHE = {}


def _oracle_weights(w, h, key):
    if key not in _WEIGHT_CACHE:
        _WEIGHT_CACHE[key] = prepare_weights_ref(w, h)
    return _WEIGHT_CACHE[key]


def _end_to_end(dev, x, w, h, bits, rows, key):
    wp, ws = dptq.prepare_weights(_d(w, dev), h)
    codes, scales = dptq.rotate_quant(_d(x, dev), h, bits)
    y = _h(dptq.qlinear(codes, scales, bits, wp, ws))
    wp_ref, ws_ref = _oracle_weights(w, h, key)
    _assert_codes(_h(wp), wp_ref, "e2e weight codes")
    c_ref, s_ref = rotate_quant_ref(x[rows], h, bits)
    _assert_codes(_h(codes)[rows], c_ref, "e2e codes")
    _assert_f32(_h(scales)[rows], s_ref, "e2e scales")
    y_ref = epilogue_ref(qlinear_acc_ref(c_ref, bits, wp_ref), s_ref, ws_ref)
    _assert_f16(y[rows], y_ref, "e2e y")


@pytest.mark.parametrize("bits", [4, 8])
def test_end_to_end_tiny_config(dev, bits):
    rng = np.random.default_rng(0)
    x = workloads.gauss_massive(rng, 16, 256)
    w = workloads.weights(rng, 512, 256)
    _end_to_end(dev, x, w, 256, bits, np.arange(16), "tiny")


@pytest.mark.parametrize("bits", [4, 8])
@pytest.mark.parametrize("M", [1, 4, 16, 40])
def test_end_to_end_down_proj_shape(dev, bits, M):
    # K = 14336 with h = 28 x 512, decode and small prefill batches.
    x = workloads.student_t(np.random.default_rng(2 + M), M, 14336)
    w = workloads.weights(np.random.default_rng(2), 256, 14336)
    _end_to_end(dev, x, w, 28 * 512, bits, np.arange(M), "down")
