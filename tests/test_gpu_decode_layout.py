"""GPU parity of the decode weight layout (dptq_prepack_weights with
DPTQ_WEIGHTS_DECODE) and of the decode GEMM that reads it
(dptq_qlinear_decode_native), through the C ABI.

Bar: the layout byte for byte against its definition (written out in numpy);
the int32 accumulators and fp16 outputs bit for bit against the oracle's exact
GEMM and pinned epilogue, at one and two 16-channel blocks per workgroup,
4- and 8-bit activations, M = 1 .. 16.
"""

import numpy as np
import pytest

import workloads
from paritylib import decode_layout_ref, oracle_acc, oracle_y, safe_w_scales, assert_acc

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


@pytest.mark.parametrize("N,K", [(16, 128), (48, 384), (272, 4096), (4096, 14336)])
def test_decode_layout_bytes(dev, N, K):
    rng = np.random.default_rng(N + K)
    w = workloads.random_weight_bytes(rng, N, K)
    got = _h(dptq.prepack_weights(_d(w, dev), dptq.WEIGHTS_DECODE))
    assert np.array_equal(got, decode_layout_ref(w))


CASES = [
    # (M, K, N, bits): the LLaMA-3-8B down decode (K = 14336, N = 4096), LLaMA-2-7B QKV,
    # a 70B-shaped row count at 8 tokens, small and ragged shapes, and the
    # two-block workgroups (M * bits >= 64 with N >= 16384)
    (1, 14336, 4096, 4), (4, 14336, 4096, 8), (16, 14336, 4096, 4), (1, 4096, 12288, 8),
    (8, 8192, 1024, 4), (3, 256, 16, 8), (7, 1152, 208, 4), (16, 128, 48, 8),
    (8, 1024, 16384, 8), (16, 1024, 16384, 4), (12, 2048, 16384, 8),
    # eight chunks in flight per wavefront: exactly 12 chunks per wavefront,
    # 12 or 13 (a ragged split), and the largest M and grid that take it
    (1, 12288, 4096, 4), (3, 12416, 2048, 8), (4, 28672, 4096, 4),
]


@pytest.mark.parametrize("M,K,N,bits", CASES)
def test_decode_native_matches_oracle(dev, M, K, N, bits):
    rng = np.random.default_rng([M, K, N, bits])
    a = workloads.random_code_bytes(rng, M, K, bits)
    w = workloads.random_weight_bytes(rng, N, K)
    a_s = workloads.random_scales(rng, M, 1e-3, 1.0)
    w_s = safe_w_scales(rng, N, K, a_s, bits)
    wd = dptq.prepack_weights(_d(w, dev), dptq.WEIGHTS_DECODE)
    ad = _d(a, dev)
    if bits == 8:
        ad = ad.view(torch.int8)
    acc_ref = oracle_acc(a, bits, w)
    assert_acc(_h(dptq.qlinear_decode_native_acc(ad, bits, wd, N)), acc_ref, f"{M}x{K}x{N} A{bits}")
    y = _h(dptq.qlinear_decode_native(ad, _d(a_s, dev), bits, wd, _d(w_s, dev)))
    y_ref = oracle_y(acc_ref, a_s, w_s)
    assert np.array_equal(y.view(np.uint16), y_ref.view(np.uint16))
    # and the same bits as the canonical-layout decode GEMM
    y0 = _h(dptq.qlinear(ad, _d(a_s, dev), bits, _d(w, dev), _d(w_s, dev), kernel=dptq.GEMM_DECODE))
    assert np.array_equal(y.view(np.uint16), y0.view(np.uint16))


def test_decode_native_rejects_prefill_batches(dev):
    a = torch.zeros((17, 512), dtype=torch.uint8, device=dev)
    wd = torch.zeros((64 * 512,), dtype=torch.uint8, device=dev)
    with pytest.raises(dptq.DptqError):
        dptq.qlinear_decode_native_acc(a, 4, wd, 64)
