"""GPU parity of the group-wise 4-bit KV-cache codec through the C ABI.

Codes, scales and minima are compared bit for bit with the oracle, and the
reconstruction is compared bit for bit on the oracle's own codes (so that no
oracle input comes from the GPU).  Shapes cover every supported group size,
ragged token counts, the KV rows of LLaMA-3-8B and LLaMA-2-70B (8 KV heads of
128 channels) at prefill lengths, and a large cache fill checked in full.
"""

import numpy as np
import pytest

from oracle.kv import kv_quant_ref, kv_dequant_ref, pack_u4

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


def _eq(got, ref, what):
    g = np.ascontiguousarray(got).view(np.uint8)
    r = np.ascontiguousarray(ref).view(np.uint8)
    assert g.shape == r.shape, what
    bad = int(np.count_nonzero(g != r))
    assert bad == 0, f"{what}: {bad} bytes differ"


def _kv_rows(rng, T, D):
    """K/V-like rows: N(0,1) per channel times a per-channel spread, a few
    outlier channels (keys carry channel outliers) and a per-token offset."""
    x = rng.standard_normal((T, D)).astype(np.float32)
    x *= rng.uniform(0.2, 3.0, D).astype(np.float32)
    x[:, rng.choice(D, max(1, D // 128), replace=False)] *= 20.0
    x += rng.normal(0, 1.0, (T, 1)).astype(np.float32)
    return x.astype(np.float16)


def _check(dev, x, group, what):
    codes, s, m = dptq.kv_quant(_d(x, dev), group)
    c_ref, s_ref, m_ref = kv_quant_ref(x, group)
    _eq(_h(codes), c_ref, what + " codes")
    _eq(_h(s), s_ref, what + " scales")
    _eq(_h(m), m_ref, what + " mins")
    out = dptq.kv_dequant(_d(c_ref, dev), _d(s_ref, dev), _d(m_ref, dev), group)
    _eq(_h(out), kv_dequant_ref(c_ref, s_ref, m_ref, group), what + " reconstruction")


CASES = [
    (1, 128, 128), (7, 1024, 128), (33, 4096, 128), (5, 256, 16), (9, 96, 32),
    (3, 512, 512), (11, 640, 64), (2, 1536, 256), (2048, 1024, 128), (4096, 1024, 128),
    (1000, 128 * 40, 128),
]


@pytest.mark.parametrize("T,D,group", CASES)
def test_kv_codec_matches_oracle(dev, T, D, group):
    x = _kv_rows(np.random.default_rng(T * 7 + D + group), T, D)
    _check(dev, x, group, f"T={T} D={D} g={group}")


def test_kv_codec_random_bit_patterns(dev):
    # Every finite fp16 bit pattern class: subnormals, huge values, mixed
    # exponents inside one group (large quotients and tiny steps).
    rng = np.random.default_rng(1)
    bits = rng.integers(0, 1 << 16, size=(512, 1024), dtype=np.uint16)
    x = bits.view(np.float16).copy()
    x[~np.isfinite(x)] = 0
    _check(dev, x, 128, "random fp16 bits")


def test_kv_codec_special_groups(dev):
    rng = np.random.default_rng(2)
    T, D, g = 8, 512, 128
    x = _kv_rows(rng, T, D)
    x[0] = 0                                              # all-zero row
    x[1, :128] = np.float16(3.5)                          # constant group
    x[2] = np.float16(6e-8)                               # constant subnormal row
    x[3, :64] = np.float16(65504.0)                       # fp16 extremes, range 131008
    x[3, 64:128] = np.float16(-65504.0)
    # exact ties: m + (k + 1/2) s with s = 2^-3; the ends make the range 15 s
    k = rng.integers(0, 15, 128)
    x[4, 128:256] = np.float16(-1.0) + (k + 0.5) * np.float16(0.125)
    x[4, 128] = np.float16(-1.0)
    x[4, 129] = np.float16(-1.0 + 15 * 0.125)
    x[5, 256:384] = np.float16(6e-8) * rng.integers(0, 40, 128)   # subnormal steps
    _check(dev, x, g, "special groups")
    codes, s, m = kv_quant_ref(x, g)
    assert s[0].max() == 0 and s[1, 0] == 0 and s[4, 1] == 0.125


def test_kv_dequant_double_rounding(dev):
    # fl16(fl32(fl32(15 s) + m)) with s = 1 + 2^-23, m = 196569 * 2^-24 is the
    # fp16 tie that rounds to 15 + 2^-6; one fused rounding would give 15 + 2^-7.
    s = np.full((4, 2), np.float32(1 + 2.0 ** -23), np.float32)
    m = np.full((4, 2), np.float32(196569 * 2.0 ** -24), np.float32)
    codes = pack_u4(np.full((4, 32), 15))
    out = _h(dptq.kv_dequant(_d(codes, dev), _d(s, dev), _d(m, dev), 16))
    assert np.all(out == np.float16(15 + 2.0 ** -6))
    _eq(out, kv_dequant_ref(codes, s, m, 16), "double rounding")


def test_kv_append_at_offset(dev):
    # Quantizing new tokens into an existing cache through offset views leaves
    # the earlier rows untouched.
    rng = np.random.default_rng(3)
    T0, T1, D = 100, 37, 1024
    x = _kv_rows(rng, T0 + T1, D)
    codes = torch.zeros((T0 + T1, D // 2), dtype=torch.uint8, device=dev)
    s = torch.zeros((T0 + T1, D // 128), dtype=torch.float32, device=dev)
    m = torch.zeros_like(s)
    xd = _d(x, dev)
    dptq.kv_quant(xd[:T0], 128, codes[:T0], s[:T0], m[:T0])
    dptq.kv_quant(xd[T0:], 128, codes[T0:], s[T0:], m[T0:])
    c_ref, s_ref, m_ref = kv_quant_ref(x, 128)
    _eq(_h(codes), c_ref, "appended codes")
    _eq(_h(s), s_ref, "appended scales")
    _eq(_h(m), m_ref, "appended mins")


def test_kv_codec_empty(dev):
    x = torch.empty((0, 1024), dtype=torch.float16, device=dev)
    codes, s, m = dptq.kv_quant(x, 128)
    assert codes.numel() == 0 and s.numel() == 0
    assert dptq.kv_dequant(codes, s, m, 128).numel() == 0


def test_kv_codec_large_cache_fill(dev):
    # A 32-sequence x 2048-token prefill of one layer's keys for LLaMA-3-8B
    # (8 KV heads x 128), checked in full.
    T, D = 32 * 2048, 1024
    x = _kv_rows(np.random.default_rng(4), T, D)
    _check(dev, x, 128, "large cache fill")
