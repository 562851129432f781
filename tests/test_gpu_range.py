"""GPU parity of the range-based quantizer with an integer zero point (Eq. 1-2)
and its zero-point-corrected linear, through the C ABI.

Bar: codes, scales, zero points, weight sums and fp16 outputs bit for bit
against the oracle on seeded inputs, over every rotation family (register
phases, passes across segments, 28 * 2^j), ragged row counts, rows of zeros
and one-signed rows; the full LLaMA-2-7B QKV shape is checked on sampled
outputs the oracle computes one by one.
"""

import numpy as np
import pytest

import workloads
from paritylib import safe_w_scales
from oracle import (rotate_quant_range_ref, weight_sums_ref, qlinear_range_ref,
                    qlinear_acc_entries, zero_point_acc_ref, epilogue_ref)

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


RQ_CASES = [
    # (M, K, h): tiny h, one register phase, three phases, K not a multiple of
    # 4096, two passes across segments, 28 * 2^j with j = 0, 9, 10, and 43
    # blocks of 256
    (5, 128, 8), (16, 256, 256), (33, 4096, 4096), (9, 6144, 2048), (3, 16384, 16384),
    (7, 896, 28), (4, 14336, 28 * 512), (2, 28672, 28 * 1024), (6, 11008, 256),
    # the longest row (nine segments, the largest staging) and a batch of
    # more rows than compute units
    (2, 36864, 4096), (300, 1024, 1024),
]


def _rows(rng, M, K, h):
    x = workloads.student_t(rng, M, K) if h % 28 == 0 else workloads.gauss_outliers(rng, M, K)
    if M > 2:
        x[1] = 0.0                          # a row of zeros: s = 0, z = 0
        x[2] = np.abs(x[2])                 # one-signed before the rotation
    return x


@pytest.mark.parametrize("bits", [4, 8])
@pytest.mark.parametrize("M,K,h", RQ_CASES)
def test_rotate_quant_range_matches_oracle(dev, M, K, h, bits):
    rng = np.random.default_rng(M * 7 + K + h + bits)
    x = _rows(rng, M, K, h)
    c_ref, s_ref, z_ref = rotate_quant_range_ref(x, h, bits)
    codes, scales, zeros = dptq.rotate_quant_range(_d(x, dev), h, bits)
    assert np.array_equal(_h(scales).view(np.uint32), s_ref.view(np.uint32))
    assert np.array_equal(_h(zeros), z_ref)
    got = _h(codes)
    assert np.array_equal(got, c_ref), f"{(got != c_ref).sum()} code bytes differ"


def test_rotate_quant_range_one_signed_rows(dev):
    # A constant row rotates to (128 c, 0, ..., 0) per block of h = 128: the
    # range is one-sided and the zero point lands on an end level; a row of
    # zeros gets s = 0 and z = 0.
    M, K, h = 4, 256, 128
    x = np.zeros((M, K), np.float16)
    x[0] = 0.5
    x[1] = -0.25
    x[2, ::2] = 1.0
    for bits in (4, 8):
        c_ref, s_ref, z_ref = rotate_quant_range_ref(x, h, bits)
        codes, scales, zeros = dptq.rotate_quant_range(_d(x, dev), h, bits)
        assert np.array_equal(_h(scales).view(np.uint32), s_ref.view(np.uint32))
        assert np.array_equal(_h(zeros), z_ref)
        assert np.array_equal(_h(codes), c_ref)
        assert z_ref[0] == 0 and z_ref[1] == (1 << bits) - 1 and z_ref[3] == 0


@pytest.mark.parametrize("N,K", [(1, 32), (5, 256), (100, 4096), (4096, 14336)])
def test_weight_sums_match_oracle(dev, N, K):
    rng = np.random.default_rng(N + K)
    wp = workloads.random_weight_bytes(rng, N, K)
    got = _h(dptq.weight_sums(_d(wp, dev)))
    assert np.array_equal(got.astype(np.int64), weight_sums_ref(wp))


LINEAR_CASES = [
    # (M, K, N, h): the correction in the epilogue of the decode GEMM (M <= 16,
    # one and two channel blocks per workgroup), of the 256 x 128 tiles
    # (ragged M) and of the 192 x 256 tiles (every output checked), either
    # side of the decode boundary, the tiny workload
    (1, 4096, 512, 4096), (16, 256, 512, 256), (16, 256, 16384, 256), (17, 512, 128, 512),
    (70, 4096, 320, 4096), (300, 1024, 256, 1024), (2048, 512, 12288, 512),
    # 192 x 256 tiles with shifted edge tiles in m and n (every output checked)
    (2100, 256, 12304, 256),
    (5, 14336, 64, 28 * 512),
]


@pytest.mark.parametrize("bits", [4, 8])
@pytest.mark.parametrize("M,K,N,h", LINEAR_CASES)
def test_qlinear_range_matches_oracle(dev, M, K, N, h, bits):
    rng = np.random.default_rng(3 * M + K + N + bits)
    x = _rows(rng, M, K, h)
    w = workloads.weights(rng, N, K)
    wp, ws = dptq.prepare_weights(_d(w, dev), h)
    wp_h, ws_h = _h(wp), _h(ws)
    c_ref, s_ref, z_ref = rotate_quant_range_ref(x, h, bits)
    y_ref = qlinear_range_ref(c_ref, s_ref, z_ref, bits, wp_h, ws_h)
    codes, scales, zeros = dptq.rotate_quant_range(_d(x, dev), h, bits)
    y = dptq.qlinear_range(codes, scales, zeros, bits, wp, ws, dptq.weight_sums(wp))
    got = _h(y)
    assert np.array_equal(got.view(np.uint16), y_ref.view(np.uint16)), \
        f"{(got.view(np.uint16) != y_ref.view(np.uint16)).sum()} outputs differ"


@pytest.mark.parametrize("bits", [4, 8])
def test_qlinear_range_full_shape_sampled(dev, bits):
    # LLaMA-2-7B fused QKV at M = 2048: every code, scale and zero point
    # against the oracle, and 4096 sampled outputs computed one by one.
    M, K, N, h = 2048, 4096, 12288, 4096
    rng = np.random.default_rng(40 + bits)
    x = workloads.gauss_outliers(rng, M, K)
    wp = workloads.random_weight_bytes(rng, N, K)
    c_ref, s_ref, z_ref = rotate_quant_range_ref(x, h, bits)
    # |q - z| < 2^b, twice the symmetric bound on |code|: halve the output limit
    ws = safe_w_scales(rng, N, K, s_ref, bits, limit=15000.0)
    wpd = _d(wp, dev)
    codes, scales, zeros = dptq.rotate_quant_range(_d(x, dev), h, bits)
    assert np.array_equal(_h(codes), c_ref)
    assert np.array_equal(_h(scales).view(np.uint32), s_ref.view(np.uint32))
    assert np.array_equal(_h(zeros), z_ref)
    y = _h(dptq.qlinear_range(codes, scales, zeros, bits, wpd, _d(ws, dev), dptq.weight_sums(wpd)))
    rows = rng.integers(0, M, 4096)
    cols = rng.integers(0, N, 4096)
    acc = qlinear_acc_entries(c_ref, bits, wp, rows, cols)
    sums = weight_sums_ref(wp)
    accz = acc + ((1 << (bits - 1)) - z_ref[rows].astype(np.int64)) * sums[cols]
    want = np.array([epilogue_ref(np.array([[a]]), s_ref[[m]], ws[[n]])[0, 0]
                     for a, m, n in zip(accz, rows, cols)])
    assert np.isfinite(want.astype(np.float32)).all()
    assert np.array_equal(y[rows, cols].view(np.uint16), want.view(np.uint16))
