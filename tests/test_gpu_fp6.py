"""GPU parity of the FP6 operand path: the 4-bit x 4-bit GEMM computed on the
FP6 (e2m3) matrix cores, through the C ABI, against the CPU oracle.

Bar: int32 accumulators and fp16 outputs bit for bit against the oracle's
exact integer GEMM and pinned epilogue (the FP6 path computes the same exact
integer product, so nothing looser applies), and the FP6 block layout byte for
byte against a reference encoder written here from the e2m3 definition (sign,
two exponent bits with bias 1, three mantissa bits; subnormals m / 8).  Inputs
are seeded random code bytes (every nibble value, -8 included) so no oracle
input comes from the HIP path.  Full-size shapes are checked whole against the
int8 path (itself parity-tested against the oracle) and on sampled entries
against the oracle directly.
"""

import numpy as np
import pytest

import workloads
from oracle import (rotate_quant_ref, prepare_weights_ref, qlinear_acc_ref, epilogue_ref,
                    unpack_int4)
from oracle.gemm import qlinear_acc_entries
from paritylib import e2m3_table as _e2m3_table, fp6_layout_ref

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


def test_e2m3_table_closed_form():
    # c / 2 for the 16 codes: the table found by search is the one the layout
    # states (sign bit 5, exponent bits 3-4, mantissa bits 0-2).
    tab = _e2m3_table()
    assert tab[0] == 0 and tab[1] == 0b000100 and tab[7] == 0b010110 and tab[-8] == 0b111000
    for c in range(1, 8):
        assert tab[-c] == tab[c] | 0x20


@pytest.mark.parametrize("R,K", [(1, 128), (31, 256), (32, 128), (33, 640), (70, 384), (5, 4096)])
def test_pack_fp6_layout(dev, R, K):
    rng = np.random.default_rng(R * 7 + K)
    packed = workloads.random_weight_bytes(rng, R, K)
    got = _h(dptq.pack_fp6(_d(packed, dev)))
    ref = fp6_layout_ref(packed, K)
    assert got.shape == ref.shape == (dptq.fp6_bytes(R, K),)
    bad = np.nonzero(got != ref)[0]
    assert bad.size == 0, f"{bad.size} layout bytes differ, first at {bad[0]}"


def _fp6_operands(dev, a_packed, w_packed):
    return dptq.pack_fp6(_d(a_packed, dev)), dptq.pack_fp6(_d(w_packed, dev))


GEMM_CASES = [
    # (M, N, K): single tiles, ragged tiles in m and n, one and many stages,
    # odd stage counts, several tiles per workgroup
    (1, 16, 128), (17, 48, 256), (32, 192, 128), (255, 192, 384), (256, 192, 512),
    (300, 208, 1024), (513, 400, 640), (600, 1008, 2048), (1024, 2304, 1152),
    (257, 16, 4096), (2048, 768, 896),
]


@pytest.mark.parametrize("M,N,K", GEMM_CASES)
def test_fp6_acc_random_codes(dev, M, N, K):
    rng = np.random.default_rng(M * 131 + N * 7 + K)
    a = workloads.random_weight_bytes(rng, M, K)
    w = workloads.random_weight_bytes(rng, N, K)
    a6, w6 = _fp6_operands(dev, a, w)
    acc = _h(dptq.qlinear_fp6_acc(a6, w6, M, K, N))
    ref = qlinear_acc_ref(a, 4, w)
    bad = np.nonzero(acc.astype(np.int64) != ref)
    assert bad[0].size == 0, f"{bad[0].size} accumulators differ, first at {bad[0][0]},{bad[1][0]}"


@pytest.mark.parametrize("M,N,K", GEMM_CASES[:8])
def test_fp6_y_random_codes(dev, M, N, K):
    rng = np.random.default_rng(M * 17 + N + K * 3)
    a = workloads.random_weight_bytes(rng, M, K)
    w = workloads.random_weight_bytes(rng, N, K)
    a_s = workloads.random_scales(rng, M)
    w_s = workloads.random_scales(rng, N)
    a6, w6 = _fp6_operands(dev, a, w)
    y = _h(dptq.qlinear_fp6(a6, _d(a_s, dev), w6, _d(w_s, dev), M, K, N))
    ref = epilogue_ref(qlinear_acc_ref(a, 4, w), a_s, w_s)
    assert np.array_equal(y.view(np.uint16), ref.view(np.uint16)), \
        f"{(y.view(np.uint16) != ref.view(np.uint16)).sum()} outputs differ"


@pytest.mark.parametrize("ca,cw", [(-8, -8), (7, 7), (-8, 7), (7, -8)])
def test_fp6_extreme_accumulators(dev, ca, cw):
    # Every code at an extreme and the largest K: |acc| = 64 K = 2^22 (the
    # largest magnitude the fp32 accumulator must hold exactly), closed form.
    M, N, K = 64, 32, 65536
    nib = lambda c: (c & 15) | ((c & 15) << 4)
    a = np.full((M, K // 2), nib(ca), dtype=np.uint8)
    w = np.full((N, K // 2), nib(cw), dtype=np.uint8)
    a6, w6 = _fp6_operands(dev, a, w)
    acc = _h(dptq.qlinear_fp6_acc(a6, w6, M, K, N))
    assert np.all(acc == ca * cw * K)


def test_fp6_large_k_mixed(dev):
    # A large accumulator followed by small terms: the rows hold +7 codes
    # except a random tail, so exactness needs every low-order bit.
    M, N, K = 96, 64, 65536
    rng = np.random.default_rng(65536)
    ca = np.full((M, K), 7, dtype=np.int64)
    cw = np.full((N, K), 7, dtype=np.int64)
    ca[:, -256:] = rng.integers(-8, 8, size=(M, 256))
    cw[:, -256:] = rng.integers(-8, 8, size=(N, 256))
    from oracle import pack_int4
    a, w = pack_int4(ca), pack_int4(cw)
    a6, w6 = _fp6_operands(dev, a, w)
    acc = _h(dptq.qlinear_fp6_acc(a6, w6, M, K, N))
    assert np.array_equal(acc.astype(np.int64), ca @ cw.T)


def test_fp6_end_to_end_tiny(dev):
    # The tiny workload (M=16, K=256, N=512, h=256) from fp16 activations and
    # fp32 weights: rotate+quantize, pack both operands, FP6 GEMM.
    rng = np.random.default_rng(0)
    M, K, N, h = 16, 256, 512, 256
    x = workloads.gauss_massive(rng, M, K)
    w = workloads.weights(rng, N, K)
    wp_ref, ws_ref = prepare_weights_ref(w, h)
    c_ref, s_ref = rotate_quant_ref(x, h, 4)
    codes, scales = dptq.rotate_quant(_d(x, dev), h, 4)
    wp, ws = dptq.prepare_weights(_d(w, dev), h)
    y = _h(dptq.qlinear_fp6(dptq.pack_fp6(codes), scales, dptq.pack_fp6(wp), ws, M, K, N))
    ref = epilogue_ref(qlinear_acc_ref(c_ref, 4, wp_ref), s_ref, ws_ref)
    assert np.array_equal(y.view(np.uint16), ref.view(np.uint16))


PARTIAL_ROUND_CASES = [
    # (M, N, K): tile counts (256 x 192 tiles) that leave the last round over
    # the compute units partly empty or run below one round: 128, 150 and 176
    # tiles, and one whole round plus 64 or 96 tiles
    (512, 12288, 4096), (1280, 5760, 4096), (2048, 4096, 4096), (2048, 7680, 4096),
    (256, 67584, 4096),
]


@pytest.mark.parametrize("M,N,K", PARTIAL_ROUND_CASES)
def test_fp6_partial_round_matches_oracle(dev, M, N, K):
    from paritylib import assert_acc, oracle_y, safe_w_scales
    rng = np.random.default_rng([M, N, K])
    a = workloads.random_weight_bytes(rng, M, K)
    w = workloads.random_weight_bytes(rng, N, K)
    a_s = workloads.random_scales(rng, M, 1e-3, 1.0)
    w_s = safe_w_scales(rng, N, K, a_s, 4)
    a6, w6 = _fp6_operands(dev, a, w)
    acc_ref = qlinear_acc_ref(a, 4, w)
    assert_acc(_h(dptq.qlinear_fp6_acc(a6, w6, M, K, N)), acc_ref, f"{M}x{N}x{K} acc")
    y = _h(dptq.qlinear_fp6(a6, _d(a_s, dev), w6, _d(w_s, dev), M, K, N))
    y_ref = oracle_y(acc_ref, a_s, w_s)
    bad = np.nonzero(y.view(np.uint16) != y_ref.view(np.uint16))
    assert bad[0].size == 0, f"{bad[0].size} outputs differ, first at {bad[0][0]},{bad[1][0]}"


FULL_SHAPES = [
    # (name, M, K, N): LLaMA-2-7B fused QKV, LLaMA-3-8B down_proj prefill,
    # LLaMA-2-70B qkv and down_proj prefill
    ("llama2_7b_qkv", 2048, 4096, 12288),
    ("llama3_8b_down", 2048, 14336, 4096),
    ("llama2_70b_qkv", 4096, 8192, 10240),
    ("llama2_70b_down", 4096, 28672, 8192),
]


@pytest.mark.parametrize("name,M,K,N", FULL_SHAPES)
def test_fp6_full_size_vs_int8_path_and_oracle(dev, name, M, K, N):
    g = torch.Generator(device=dev)
    g.manual_seed(M + K + N)
    a = torch.randint(0, 256, (M, K // 2), dtype=torch.uint8, device=dev, generator=g)
    w = torch.randint(0, 256, (N, K // 2), dtype=torch.uint8, device=dev, generator=g)
    a_s = torch.rand(M, device=dev, generator=g) * 1e-2 + 1e-3
    w_s = torch.rand(N, device=dev, generator=g) * 1e-3 + 1e-4
    a6, w6 = dptq.pack_fp6(a), dptq.pack_fp6(w)
    y6 = dptq.qlinear_fp6(a6, a_s, w6, w_s, M, K, N)
    y8 = dptq.qlinear(a, a_s, 4, w, w_s)
    acc6 = dptq.qlinear_fp6_acc(a6, w6, M, K, N)
    torch.cuda.synchronize()
    if not torch.equal(y6.view(torch.int16), y8.view(torch.int16)):
        # name the path that disagrees with the oracle on the differing entries
        diff = torch.nonzero(y6.view(torch.int16) != y8.view(torch.int16)).cpu().numpy()
        pick = diff[:: max(1, len(diff) // 16)][:16]
        rows_d, cols_d = pick[:, 0], pick[:, 1]
        ref = qlinear_acc_entries(_h(a), 4, _h(w), rows_d, cols_d)
        y_ref = np.array([epilogue_ref(np.array([[r]]), _h(a_s)[[m]], _h(w_s)[[n]])[0, 0]
                          for r, m, n in zip(ref, rows_d, cols_d)])
        ok6 = np.array_equal(_h(y6)[rows_d, cols_d].view(np.uint16), y_ref.view(np.uint16))
        ok8 = np.array_equal(_h(y8)[rows_d, cols_d].view(np.uint16), y_ref.view(np.uint16))
        raise AssertionError(f"{name}: {len(diff)} outputs differ between the paths "
                             f"(rows {sorted(set(diff[:, 0].tolist()))[:8]}..., "
                             f"cols {sorted(set(diff[:, 1].tolist()))[:8]}...); "
                             f"fp6 matches the oracle there: {ok6}, int8: {ok8}")
    # sampled entries against the oracle, computed one by one
    rng = np.random.default_rng(7)
    rows = np.concatenate([[0, M - 1], rng.integers(0, M, 30)])
    cols = np.concatenate([[0, N - 1], rng.integers(0, N, 30)])
    a_h, w_h = _h(a), _h(w)
    ref = qlinear_acc_entries(a_h, 4, w_h, rows, cols)
    got = _h(acc6)[rows, cols].astype(np.int64)
    assert np.array_equal(got, ref), f"{name}: sampled accumulators differ"
    ys = _h(y6)[rows, cols]
    y_ref = np.array([epilogue_ref(np.array([[r]]), _h(a_s)[[m]], _h(w_s)[[n]])[0, 0]
                      for r, m, n in zip(ref, rows, cols)])
    assert np.array_equal(ys.view(np.uint16), y_ref.view(np.uint16)), f"{name}: sampled y differs"


RQ6_CASES = [
    # (M, K, h): every kernel family (power-of-two register phases, 28 * 2^j,
    # power of two above 4096, block-diagonal), ragged M (padding rows)
    (1, 128, 128), (5, 256, 16), (33, 1024, 1024), (64, 4096, 4096), (70, 4096, 256),
    (3, 14336, 28 * 512), (40, 3584, 28 * 128), (2, 8192, 8192), (31, 11008 - 11008 % 128, 128),
    (130, 4096, 4096),
    # more than 64 rows (28 * 2^j, 2^j above 4096, a partial last 4096-element
    # segment, ragged 32-row blocks)
    (70, 8192, 8192), (100, 14336, 28 * 512), (97, 12544, 28 * 64),
    # rows that leave room for one per compute unit (four thread groups)
    (66, 28672, 28 * 1024), (65, 24576, 8192),
    # more of them than compute units (the next row touched into the L2)
    (260, 28672, 28 * 1024), (1030, 8192, 8192),
]


@pytest.mark.parametrize("M,K,h", RQ6_CASES)
def test_rotate_quant_fp6_matches_oracle_codes(dev, M, K, h):
    from oracle import pack_int4
    rng = np.random.default_rng(M * 10 + K + h)
    x = workloads.gauss_outliers(rng, M, K, n_channels=4)
    out, scales = dptq.rotate_quant_fp6(_d(x, dev), h)
    c_ref, s_ref = rotate_quant_ref(x, h, 4)
    assert np.array_equal(_h(scales).view(np.uint32), s_ref.view(np.uint32))
    ref = fp6_layout_ref(c_ref, K)
    got = _h(out)
    bad = np.nonzero(got != ref)[0]
    assert bad.size == 0, f"{bad.size} FP6 bytes differ, first at {bad[0]}"


def test_rotate_quant_fp6_then_gemm_bench_shape(dev):
    # The LLaMA-2-7B fused QKV layer through the FP6 path end to end equals
    # the int8 path (rotate_quant at 4 bits + qlinear) bit for bit.
    rng = np.random.default_rng(1)
    M, K, N, h = 2048, 4096, 12288, 4096
    x = _d(workloads.gauss_outliers(rng, M, K), dev)
    g = torch.Generator(device=dev)
    g.manual_seed(5)
    w = torch.randint(0, 256, (N, K // 2), dtype=torch.uint8, device=dev, generator=g)
    w_s = torch.rand(N, device=dev, generator=g) * 1e-3 + 1e-4
    a6, s6 = dptq.rotate_quant_fp6(x, h)
    y6 = dptq.qlinear_fp6(a6, s6, dptq.pack_fp6(w), w_s, M, K, N)
    codes, scales = dptq.rotate_quant(x, h, 4)
    y8 = dptq.qlinear(codes, scales, 4, w, w_s)
    torch.cuda.synchronize()
    assert torch.equal(s6, scales)
    assert torch.equal(dptq.pack_fp6(codes), a6)
    assert torch.equal(y6.view(torch.int16), y8.view(torch.int16))


@pytest.mark.parametrize("name,M,K,N", FULL_SHAPES[:3])
def test_fp6_and_int8_paths_repeatable(dev, name, M, K, N):
    # Both GEMM paths return identical bits on repeated launches (the
    # persistent kernels' ring buffers and shifted edge tiles carry no state
    # between launches).
    g = torch.Generator(device=dev)
    g.manual_seed(M * 3 + N)
    a = torch.randint(0, 256, (M, K // 2), dtype=torch.uint8, device=dev, generator=g)
    w = torch.randint(0, 256, (N, K // 2), dtype=torch.uint8, device=dev, generator=g)
    a_s = torch.rand(M, device=dev, generator=g) * 1e-2 + 1e-3
    w_s = torch.rand(N, device=dev, generator=g) * 1e-3 + 1e-4
    a6, w6 = dptq.pack_fp6(a), dptq.pack_fp6(w)
    y6 = [dptq.qlinear_fp6(a6, a_s, w6, w_s, M, K, N) for _ in range(3)]
    y8 = [dptq.qlinear(a, a_s, 4, w, w_s) for _ in range(3)]
    torch.cuda.synchronize()
    for i in (1, 2):
        assert torch.equal(y6[0].view(torch.int16), y6[i].view(torch.int16)), f"{name}: fp6 run {i} differs"
        assert torch.equal(y8[0].view(torch.int16), y8[i].view(torch.int16)), f"{name}: int8 run {i} differs"
    assert torch.equal(y6[0].view(torch.int16), y8[0].view(torch.int16)), f"{name}: paths differ"
