"""GPU parity of the residual-dynamics calibration (Eq. 8-11, Eq. 20) through the C ABI.

The per-token Jump Ratio and historical SNR come from fp32 sums on the GPU
and from fp64 in the oracle, so they are compared within tolerances derived
from that arithmetic:

* every squared norm is a sum of non-negative fp32 terms, each thread adding
  at most K / 256 <= 144 of them in sequence before a tree of at most 10
  levels, so its relative error is below (144 + 10) * 2^-24 < 1e-5; the norm
  (square root) halves that and the ratio of two norms adds them:
  JR rtol = 2e-5;
* the error energy is the same kind of sum of (code * s - y)^2 terms, each
  exact up to one fused rounding, so 10 log10 of it moves by at most
  4.35 * 1.2e-5 dB; the oracle's fp64 inverse rotation differs from the
  kernel's rotated-space identity only by the fp32 rounding of the rotation,
  orders of magnitude below the quantization error: SNR atol = 1e-3 dB.

The codes that decide the quantization error are bit-exact (the same kernel
that the rotate + quantize parity tests check), so no tolerance covers a
flipped code.
"""

import numpy as np
import pytest

import workloads
from oracle.residual import residual_dynamics_ref, select_sensitive_layers_ref

torch = pytest.importorskip("torch")
dptq = pytest.importorskip("paper_2606_12487_amd")

pytestmark = pytest.mark.gpu

JR_RTOL = 2e-5
SNR_ATOL = 1e-3


@pytest.fixture(scope="module")
def dev():
    dptq.lib()
    return torch.device("cuda:0")


def _d(a, dev):
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev)


def _h(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def _compare(jr, snr, jr_ref, snr_ref, what):
    jr = jr.astype(np.float64)
    snr = snr.astype(np.float64)
    fin = np.isfinite(jr_ref)
    assert np.array_equal(fin, np.isfinite(jr)), f"{what}: JR finiteness differs"
    np.testing.assert_allclose(jr[fin], jr_ref[fin], rtol=JR_RTOL, atol=0, err_msg=f"{what}: JR")
    fin = np.isfinite(snr_ref)
    assert np.array_equal(fin, np.isfinite(snr)), f"{what}: SNR finiteness differs"
    assert np.array_equal(snr[~fin], snr_ref[~fin]), f"{what}: infinite SNR of the wrong sign"
    np.testing.assert_allclose(snr[fin], snr_ref[fin], rtol=0, atol=SNR_ATOL, err_msg=f"{what}: SNR")


def _stream_layer(T, K, seed):
    """One layer of a seeded residual stream: an early (massive) layer for even
    seeds, a middle (small-update) layer for odd ones."""
    stream = workloads.residual_stream(np.random.default_rng(seed), 5, T, K)
    return stream[1] if seed % 2 == 0 else stream[3]


CASES = [
    # (T, K, h): power-of-two and 28 * 2^j sizes, block-diagonal rotations,
    # ragged token counts, K tails of 8 halfs and the largest sizes.
    (1, 8, 8), (5, 256, 256), (37, 1024, 1024), (9, 896, 28 * 32), (6, 56, 28),
    (3, 4096, 4096), (70, 4096, 4096), (130, 2048, 2048), (2, 11008, 256),
    (4, 4160, 64), (2, 4104, 8), (3, 8192, 8192), (2, 16384, 16384),
    (2, 28672, 28 * 1024), (2, 14336, 28 * 512), (2, 36864, 4096),
]


@pytest.mark.parametrize("bits", [4, 8])
@pytest.mark.parametrize("T,K,h", CASES)
def test_residual_dynamics_matches_oracle(dev, T, K, h, bits):
    x, dx = _stream_layer(T, K, seed=T + K + h)
    jr, snr, means = dptq.residual_dynamics(_d(x, dev), _d(dx, dev), h, bits)
    jr, snr, means = _h(jr), _h(snr), _h(means)
    jr_ref, snr_ref, jr_l, snr_l = residual_dynamics_ref(x, dx, h, bits)
    _compare(jr, snr, jr_ref, snr_ref, f"T={T} K={K} h={h} b={bits}")
    assert means[0] == pytest.approx(jr_l, rel=JR_RTOL)
    assert means[1] == pytest.approx(snr_l, abs=SNR_ATOL)
    # The layer means are the fp64 means of the per-token values handed out.
    assert means[0] == pytest.approx(float(np.mean(jr.astype(np.float64))), rel=1e-12)
    assert means[1] == pytest.approx(float(np.mean(snr.astype(np.float64))), rel=1e-12, abs=1e-12)


@pytest.mark.parametrize("eps", [0.0, 1e-3, 1.0])
def test_residual_dynamics_eps(dev, eps):
    x, dx = _stream_layer(12, 1024, seed=4)
    jr, snr, _ = dptq.residual_dynamics(_d(x, dev), _d(dx, dev), 1024, 4, eps=eps)
    jr_ref, snr_ref, _, _ = residual_dynamics_ref(x, dx, 1024, 4, eps=eps)
    _compare(_h(jr), _h(snr), jr_ref, snr_ref, f"eps={eps}")


@pytest.mark.parametrize("bits", [4, 8])
@pytest.mark.parametrize("K,h", [(4096, 4096), (28 * 512, 28 * 512), (2048, 256)])
def test_residual_dynamics_special_rows(dev, K, h, bits):
    # Zero history and zero update (JR = 0, SNR = -inf), zero history alone
    # (JR = ||dx|| / eps, SNR = -inf), no update, fp16-extreme magnitudes and
    # one-hot rows that land exactly on the quantization grid.
    rng = np.random.default_rng(K + bits)
    T = 8
    x = rng.standard_normal((T, K)).astype(np.float16)
    dx = (0.1 * rng.standard_normal((T, K))).astype(np.float16)
    x[0] = 0
    dx[0] = 0
    x[1] = 0
    dx[2] = 0
    x[3] = np.float16(60000.0) * np.sign(rng.standard_normal(K)).astype(np.float16)
    dx[3] = np.float16(-30000.0)
    x[4] = 0
    x[4, 3] = np.float16(7.0 if bits == 4 else 127.0)
    dx[4] = 0
    x[5] = np.float16(1e-7)                   # subnormal history
    jr, snr, means = dptq.residual_dynamics(_d(x, dev), _d(dx, dev), h, bits)
    jr, snr, means = _h(jr), _h(snr), _h(means)
    jr_ref, snr_ref, _, _ = residual_dynamics_ref(x, dx, h, bits)
    _compare(jr, snr, jr_ref, snr_ref, f"special K={K} h={h} b={bits}")
    assert jr[0] == 0 and snr[0] == -np.inf and snr[1] == -np.inf and jr[2] == 0
    assert means[1] == -np.inf


def test_residual_dynamics_empty_and_no_means(dev):
    x = torch.empty((0, 256), dtype=torch.float16, device=dev)
    jr, snr, _ = dptq.residual_dynamics(x, x, 256, 4)
    assert jr.numel() == 0 and snr.numel() == 0
    # layer_means may be NULL: the per-token values alone.
    xs, dxs = _stream_layer(3, 256, seed=0)
    xd, dxd = _d(xs, dev), _d(dxs, dev)
    jr = torch.empty(3, dtype=torch.float32, device=dev)
    snr = torch.empty(3, dtype=torch.float32, device=dev)
    rc = dptq.lib().dptq_residual_dynamics(xd.data_ptr(), dxd.data_ptr(), 3, 256, 256, 4,
                                           1e-8, jr.data_ptr(), snr.data_ptr(), None, None)
    assert rc == 0
    jr_ref, snr_ref, _, _ = residual_dynamics_ref(xs, dxs, 256, 4)
    _compare(_h(jr), _h(snr), jr_ref, snr_ref, "no means")


@pytest.mark.parametrize("bits", [4, 8])
def test_residual_dynamics_full_size_sampled(dev, bits):
    # A 2048-token calibration batch of a 4096-wide stream (the LLaMA-2-7B
    # hidden size); the oracle recomputes sampled tokens one by one.
    T, K, h = 2048, 4096, 4096
    x, dx = _stream_layer(T, K, seed=bits)
    jr, snr, means = dptq.residual_dynamics(_d(x, dev), _d(dx, dev), h, bits)
    jr, snr, means = _h(jr), _h(snr), _h(means)
    rows = np.sort(np.random.default_rng(9).choice(T, 48, replace=False))
    rows[0] = 0
    jr_ref, snr_ref, _, _ = residual_dynamics_ref(x[rows], dx[rows], h, bits)
    _compare(jr[rows], snr[rows], jr_ref, snr_ref, f"full size b={bits}")
    assert means[0] == pytest.approx(float(np.mean(jr.astype(np.float64))), rel=1e-12)
    assert means[1] == pytest.approx(float(np.mean(snr.astype(np.float64))), rel=1e-12)


def test_calibrated_policy_matches_oracle(dev):
    # The whole calibration: per-layer statistics of a synthetic 12-layer
    # stream on the GPU, then the Eq. 20 rule; the same selection as the
    # oracle's, which marks the phase-boundary layers.
    L, T, d = 12, 64, 1024
    stream = workloads.residual_stream(np.random.default_rng(6), L, T, d)
    jr_g, snr_g, jr_o, snr_o = [], [], [], []
    for x, dx in stream:
        _, _, m = dptq.residual_dynamics(_d(x, dev), _d(dx, dev), d, 4)
        m = _h(m)
        jr_g.append(float(m[0]))
        snr_g.append(float(m[1]))
        _, _, j, s = residual_dynamics_ref(x, dx, d, 4)
        jr_o.append(j)
        snr_o.append(s)
    np.testing.assert_allclose(jr_g, jr_o, rtol=JR_RTOL)
    np.testing.assert_allclose(snr_g, snr_o, atol=SNR_ATOL)
    tau_snr = float(np.median(snr_o))
    sel, bits = select_sensitive_layers_ref(jr_o, snr_o, 0.5, tau_snr)
    assert sel == [0, 1, 2, L - 1]
    assert dptq.select_layers(jr_g, snr_g, 0.5, tau_snr) == bits
