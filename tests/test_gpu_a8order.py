"""GPU parity of the W4A8 linear against weights in the 8-bit activation order
(dptq_pack_w4_a8 + dptq_qlinear_a8), through the C ABI.

The order is a storage layout of the same 4-bit weight codes, so the bar is
the canonical path's: the repacked bytes bit for bit against the oracle's
packing of the oracle's codes, and every output of every kernel bit for bit
against the oracle's exact integer GEMM and epilogue (Section 2, Eq. 5,
Section 4.2) on the same seeded inputs.
"""

import numpy as np
import pytest

import workloads
from oracle import (pack_int4_a8order, unpack_int4, qlinear_acc_ref, epilogue_ref,
                    rotate_quant_ref, prepare_weights_ref)

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


def _assert_f16(got, ref, what):
    assert np.isfinite(ref.astype(np.float32)).all(), f"{what}: expected outputs overflow fp16"
    g, r = got.view(np.uint16), ref.view(np.uint16)
    assert np.array_equal(g, r), f"{what}: {(g != r).sum()} outputs differ"


@pytest.mark.parametrize("N,K", [(16, 128), (48, 1024), (272, 4096), (1, 128 * 3)])
def test_pack_matches_oracle(dev, N, K):
    rng = np.random.default_rng(N + K)
    w = workloads.random_weight_bytes(rng, N, K)
    got = _h(dptq.pack_w4_a8(_d(w, dev)))
    ref = pack_int4_a8order(unpack_int4(w))
    assert np.array_equal(got, ref), f"{(got != ref).sum()} bytes differ"


KERNELS = (dptq.GEMM_DECODE, dptq.GEMM_TILE_256X128, dptq.GEMM_TILE_192X256)


def _fits(kernel, M, K, N):
    if kernel == dptq.GEMM_DECODE:
        return M <= 16
    if kernel == dptq.GEMM_TILE_192X256:
        return M >= 256 and N >= 192 and K >= 512
    return True


CASES = [
    # (M, K, N): decode rows (1, ragged, 16), small and ragged tiles, wide
    # tiles with shifted edge tiles, several tiles per compute unit
    (1, 128, 16), (5, 1024, 48), (16, 4096, 272), (17, 256, 32), (130, 1024, 400),
    (256, 512, 192), (300, 640, 208), (511, 1024, 400), (1024, 4096, 2048),
    # decode workgroups of two blocks of 16 channels
    (8, 512, 32768), (12, 256, 16384),
    # 192 x 256 tiles with shifted edge tiles in m and n, several per compute unit
    (2100, 256, 12304),
]


@pytest.mark.parametrize("M,K,N", CASES)
def test_qlinear_a8_every_kernel(dev, M, K, N):
    rng = np.random.default_rng(3 * M + K + N)
    a = workloads.random_code_bytes(rng, M, K, 8)
    w = workloads.random_weight_bytes(rng, N, K)
    a_s = workloads.random_scales(rng, M, 1e-3, 1.0)
    w_s = workloads.random_scales(rng, N, 1e-6, 1e-3)
    y_ref = epilogue_ref(qlinear_acc_ref(a, 8, w), a_s, w_s)
    ad, asd, wsd = _d(a, dev), _d(a_s, dev), _d(w_s, dev)
    w8 = dptq.pack_w4_a8(_d(w, dev))
    for kernel in [dptq.GEMM_AUTO] + [k for k in KERNELS if _fits(k, M, K, N)]:
        y = _h(dptq.qlinear_a8(ad, asd, w8, wsd, kernel=kernel))
        _assert_f16(y, y_ref, f"kernel {kernel} M={M} K={K} N={N}")


def test_qlinear_a8_extreme_accumulators(dev):
    # All activation codes -128 against weights of -8 (and +7 rows) at the
    # largest K: |acc| = K * 8 * 128 = 2^26, on every kernel.
    K, N = 65536, 192
    for M in (3, 256):
        a = np.full((M, K), -128, np.int8)
        w = np.full((N, K // 2), 0x88, np.uint8)
        w[1::2] = 0x77
        a_s = np.full(M, 2.0 ** -20, np.float32)
        w_s = np.full(N, 2.0 ** -10, np.float32)
        y_ref = epilogue_ref(qlinear_acc_ref(a, 8, w), a_s, w_s)
        w8 = dptq.pack_w4_a8(_d(w, dev))
        for kernel in [dptq.GEMM_AUTO] + [k for k in KERNELS if _fits(k, M, K, N)]:
            y = _h(dptq.qlinear_a8(_d(a, dev), _d(a_s, dev), w8, _d(w_s, dev), kernel=kernel))
            _assert_f16(y, y_ref, f"kernel {kernel} M={M}")


def test_qlinear_a8_full_size_sampled(dev):
    # The LLaMA-2-7B fused-QKV layer at M = 2048 (K = 4096, N = 12288) in the
    # launch configuration the benchmark times: x -> rotate_quant (A8) ->
    # qlinear_a8 on the repacked weights, against the oracle pipeline on
    # sampled rows and output channels.
    cfg = workloads.CONFIGS["llama2_7b_qkv"]
    rng = np.random.default_rng(cfg["seed"])
    x = workloads.gauss_outliers(rng, cfg["M"], cfg["K"])
    w = workloads.weights(rng, cfg["N"], cfg["K"])
    wp, ws = dptq.prepare_weights(_d(w, dev), cfg["h"])
    w8 = dptq.pack_w4_a8(wp)
    codes, scales = dptq.rotate_quant(_d(x, dev), cfg["h"], 8)
    y = _h(dptq.qlinear_a8(codes, scales, w8, ws))
    y_canon = _h(dptq.qlinear(codes, scales, 8, wp, ws))
    _assert_f16(y, y_canon, "qlinear_a8 against qlinear at full size")
    srng = np.random.default_rng(13)
    rows = np.unique(np.concatenate([[0, cfg["M"] - 1], srng.choice(cfg["M"], 6, replace=False)]))
    wrows = np.unique(np.concatenate([[0, cfg["N"] - 1], srng.choice(cfg["N"], 6, replace=False)]))
    c_ref, s_ref = rotate_quant_ref(x[rows], cfg["h"], 8)
    wp_ref, ws_ref = prepare_weights_ref(w[wrows], cfg["h"])
    assert np.array_equal(_h(w8)[wrows], pack_int4_a8order(unpack_int4(wp_ref)))
    y_ref = epilogue_ref(qlinear_acc_ref(c_ref, 8, wp_ref), s_ref, ws_ref)
    _assert_f16(y[np.ix_(rows, wrows)], y_ref, "sampled rows against the oracle")
