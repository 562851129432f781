"""GPU parity of the path's variants through the C ABI: the randomized-sign
(QuaRot-style) rotation of Section 4.2, for activations at 4 and 8 bits in
both code layouts and for the weights it is absorbed into (Eq. 5).

Bar: codes, scales and outputs bit for bit against the oracle on seeded
inputs; the signs are seeded random bitmasks drawn by the test.
"""

import numpy as np
import pytest

import workloads
from paritylib import safe_w_scales, oracle_y
from oracle import (rotate_quant_signed_ref, prepare_weights_signed_ref, qlinear_acc_ref,
                    epilogue_ref)

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


SIGNED_CASES = [
    # (M, K, h): every kernel family (register phases h <= 4096 incl. tiny h,
    # 28 * 2^j, power of two above 4096, block-diagonal), ragged rows
    (3, 64, 8), (5, 256, 256), (33, 4096, 4096), (7, 4104, 8), (2, 14336, 28 * 512),
    (3, 896, 28 * 32), (2, 8192, 8192), (70, 1024, 128), (130, 4096, 4096),
]


@pytest.mark.parametrize("bits", [4, 8])
@pytest.mark.parametrize("M,K,h", SIGNED_CASES)
def test_signed_rotate_quant(dev, M, K, h, bits):
    rng = np.random.default_rng(M * 7 + K + h + bits)
    x = workloads.gauss_outliers(rng, M, K, n_channels=min(4, K))
    signs = workloads.random_sign_bits(rng, K)
    codes, scales = dptq.rotate_quant(_d(x, dev), h, bits, signs=_d(signs, dev))
    c_ref, s_ref = rotate_quant_signed_ref(x, h, bits, signs)
    assert np.array_equal(_h(scales).view(np.uint32), s_ref.view(np.uint32))
    got = _h(codes)
    bad = np.nonzero(got != c_ref)
    assert bad[0].size == 0, f"{bad[0].size} code bytes differ, first at {bad[0][0]},{bad[1][0]}"


@pytest.mark.parametrize("M,K,h", [(5, 256, 256), (33, 4096, 4096), (2, 14336, 28 * 512),
                                   (70, 8192, 8192)])
def test_signed_rotate_quant_fp6_layout(dev, M, K, h):
    from paritylib import fp6_layout_ref
    rng = np.random.default_rng(K + h + M)
    x = workloads.gauss_outliers(rng, M, K)
    signs = workloads.random_sign_bits(rng, K)
    out, scales = dptq.rotate_quant_fp6(_d(x, dev), h, signs=_d(signs, dev))
    c_ref, s_ref = rotate_quant_signed_ref(x, h, 4, signs)
    assert np.array_equal(_h(scales).view(np.uint32), s_ref.view(np.uint32))
    assert np.array_equal(_h(out), fp6_layout_ref(c_ref, K))


@pytest.mark.parametrize("N,K,h", [(16, 256, 256), (64, 4096, 4096), (8, 14336, 28 * 512),
                                   (32, 1024, 64)])
def test_signed_weight_preparation(dev, N, K, h):
    rng = np.random.default_rng(N + K + h)
    w = workloads.weights(rng, N, K)
    signs = workloads.random_sign_bits(rng, K)
    wp, ws = dptq.prepare_weights(_d(w, dev), h, signs=_d(signs, dev))
    wp_ref, ws_ref = prepare_weights_signed_ref(w, h, signs)
    assert np.array_equal(_h(wp), wp_ref)
    assert np.array_equal(_h(ws).view(np.uint32), ws_ref.view(np.uint32))


@pytest.mark.parametrize("bits", [4, 8])
def test_signed_layer_end_to_end(dev, bits):
    # The tiny workload with randomized signs on both sides: y bitwise against
    # the oracle, and through the FP6 path at 4 bits as well.
    rng = np.random.default_rng(0)
    M, K, N, h = 16, 256, 512, 256
    x = workloads.gauss_massive(rng, M, K)
    w = workloads.weights(rng, N, K)
    signs = workloads.random_sign_bits(rng, K)
    sd = _d(signs, dev)
    c_ref, s_ref = rotate_quant_signed_ref(x, h, bits, signs)
    wp_ref, ws_ref = prepare_weights_signed_ref(w, h, signs)
    y_ref = epilogue_ref(qlinear_acc_ref(c_ref, bits, wp_ref), s_ref, ws_ref)
    codes, scales = dptq.rotate_quant(_d(x, dev), h, bits, signs=sd)
    wp, ws = dptq.prepare_weights(_d(w, dev), h, signs=sd)
    y = _h(dptq.qlinear(codes, scales, bits, wp, ws))
    assert np.array_equal(y.view(np.uint16), y_ref.view(np.uint16))
    if bits == 4:
        a6, s6 = dptq.rotate_quant_fp6(_d(x, dev), h, signs=sd)
        y6 = _h(dptq.qlinear_fp6(a6, s6, dptq.pack_fp6(wp), ws, M, K, N))
        assert np.array_equal(y6.view(np.uint16), y_ref.view(np.uint16))


FUSED_CASES = [
    # (M, K, N, h, bits): LLaMA decode shapes (7B QKV, 8B down with h = 28 x 512,
    # 7B down with 43 blocks of 256, 70B QKV at h = 8192, 70B down at
    # h = 28 x 1024 with N cut to keep the oracle quick), the tiny workload,
    # odd M (the second row slot idle), a K that is not a multiple of 4096,
    # M = 16 with one row in flight, h = 28 (no butterflies), h = 2^14 (two
    # passes across segments)
    (1, 4096, 12288, 4096, 4), (4, 14336, 4096, 28 * 512, 4), (16, 256, 512, 256, 8),
    (8, 11008, 4096, 256, 4), (8, 8192, 1024, 8192, 8), (3, 512, 32, 512, 4),
    (16, 1024, 16, 1024, 8), (16, 4096, 12288, 4096, 8), (16, 11008, 4096, 256, 4),
    (5, 6144, 256, 2048, 8), (2, 7168, 512, 28 * 256, 8), (1, 28672, 64, 28 * 1024, 4),
    (3, 896, 32, 28, 8), (2, 16384, 64, 16384, 8), (1, 14336, 4096, 28 * 512, 8),
    # one row on both thread groups: segments split by parity (2 and 3 of
    # them), and three rows that do not fit two at a time
    (1, 8192, 256, 8192, 4), (1, 11008, 256, 256, 8), (3, 14336, 128, 28 * 512, 4),
]
# Shapes whose rows do not fit on chip: the two-launch path only.
TWO_LAUNCH_ONLY = [(16, 14336, 4096, 28 * 512, 8), (8, 28672, 256, 28 * 1024, 4),
                   (16, 14336, 512, 28 * 512, 4)]


def _fused_case(dev, M, K, N, h, bits, mode):
    from oracle import rotate_quant_ref
    rng = np.random.default_rng(M * 31 + K + N + bits)
    x = workloads.student_t(rng, M, K) if h % 28 == 0 else workloads.gauss_outliers(rng, M, K)
    wp = workloads.random_weight_bytes(rng, N, K)
    c_ref, s_ref = rotate_quant_ref(x, h, bits)
    ws = safe_w_scales(rng, N, K, s_ref, bits)
    y_ref = oracle_y(qlinear_acc_ref(c_ref, bits, wp), s_ref, ws)
    y, codes, scales = dptq.qlinear_decode_fused(_d(x, dev), h, bits, _d(wp, dev), _d(ws, dev),
                                                 mode=mode)
    assert np.array_equal(_h(scales).view(np.uint32), s_ref.view(np.uint32))
    assert np.array_equal(_h(codes), c_ref)
    got = _h(y)
    assert np.array_equal(got.view(np.uint16), y_ref.view(np.uint16)), \
        f"{(got.view(np.uint16) != y_ref.view(np.uint16)).sum()} outputs differ"


@pytest.mark.parametrize("M,K,N,h,bits", FUSED_CASES)
def test_fused_decode_one_launch_matches_oracle(dev, M, K, N, h, bits):
    _fused_case(dev, M, K, N, h, bits, dptq.DECODE_ONE_LAUNCH)


@pytest.mark.parametrize("M,K,N,h,bits", FUSED_CASES[:4] + TWO_LAUNCH_ONLY)
def test_fused_decode_two_launches_matches_oracle(dev, M, K, N, h, bits):
    _fused_case(dev, M, K, N, h, bits, dptq.DECODE_TWO_LAUNCHES)


@pytest.mark.parametrize("M,K,N,h,bits", [(1, 4096, 4096, 4096, 4), (2, 8192, 512, 8192, 8),
                                          (16, 14336, 512, 28 * 512, 8), (1, 14336, 512, 28 * 512, 4)])
def test_fused_decode_auto_matches_oracle(dev, M, K, N, h, bits):
    _fused_case(dev, M, K, N, h, bits, dptq.DECODE_AUTO)


def test_fused_decode_one_launch_rejects_rows_that_do_not_fit(dev):
    x = torch.zeros((16, 14336), dtype=torch.float16, device=dev)
    wp = torch.zeros((64, 7168), dtype=torch.uint8, device=dev)
    ws = torch.ones((64,), dtype=torch.float32, device=dev)
    with pytest.raises(dptq.DptqError):
        dptq.qlinear_decode_fused(x, 28 * 512, 8, wp, ws, mode=dptq.DECODE_ONE_LAUNCH)


def test_fused_decode_consecutive_calls(dev):
    # Consecutive decode steps with different inputs, M and bits on the same
    # weights are all exact on the one-launch path.
    from oracle import rotate_quant_ref
    K, N, h = 4096, 2048, 4096
    rng = np.random.default_rng(77)
    wp = workloads.random_weight_bytes(rng, N, K)
    # a rotated entry is at most the L1 norm of its row's block (about 3.3e3
    # for these rows), so 2e4 bounds the absmax of all four steps at once
    ws = safe_w_scales(rng, N, K, np.array([20000.0 / 7.0], np.float32), 4)
    wpd, wsd = _d(wp, dev), _d(ws, dev)
    for step, M in enumerate([4, 1, 16, 7]):
        x = workloads.gauss_outliers(rng, M, K)
        bits = 4 if step % 2 == 0 else 8
        y, _, scales = dptq.qlinear_decode_fused(_d(x, dev), h, bits, wpd, wsd,
                                                 mode=dptq.DECODE_ONE_LAUNCH)
        c_ref, s_ref = rotate_quant_ref(x, h, bits)
        y_ref = oracle_y(qlinear_acc_ref(c_ref, bits, wp), s_ref, ws)
        assert np.array_equal(_h(y).view(np.uint16), y_ref.view(np.uint16)), f"step {step}"
        assert np.array_equal(_h(scales).view(np.uint32), s_ref.view(np.uint32))
