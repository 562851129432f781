"""GPU parity at the five workloads' full sizes, through the C ABI, in the
launch configuration the benchmark times.

* Codes and scales bit for bit on EVERY token row of the tiny layer, the
  LLaMA-2-7B fused QKV layer (M = 2048) and the LLaMA-3-8B down projection
  (K = 14336, h = 28 x 512; M = 1, 4, 16 and 2048), at 4 and 8 bits, in the
  packed layout and, at 4 bits, in the FP6 block layout (decoded back to
  codes here from the layout's definition).
* For every linear of the LLaMA-2-7B and LLaMA-2-70B stacks: codes and scales
  on >= 256 sampled token rows (row 0 and the last row always included) at a
  layer the default policy runs at 8 bits and one it runs at 4, on the paths
  the benchmark step runs (FP6 at 4 bits, 8-bit-order weights at 8 bits) and
  the canonical int8 path; every row at the M = 8 decode shapes.
* Outputs y on those rows across EVERY output column, for every GEMM path that
  serves the bits, against the oracle's exact GEMM of the oracle's own codes
  with seeded weight codes and weight scales drawn so that no output can leave
  fp16 range (every expected output is asserted finite).
* int32 accumulators in full (every entry) at every full prefill shape, on
  seeded random codes, against the oracle's exact float64 product.
* Offline weight preparation of N(0, 0.02) weights on 256 sampled weight rows
  of every distinct linear.

No expected value comes from the HIP path: inputs are seeded on the host, and
the oracle computes every reference from them.
"""

import numpy as np
import pytest

import workloads
from paritylib import (assert_acc, sample_rows, oracle_rotate, oracle_codes, oracle_acc, oracle_y,
                       oracle_prepare, safe_w_scales, assert_bytes, assert_f16,
                       fp6_layout_decode)
from oracle import unpack_int4

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


def _check_fp6(buf, c_ref_packed, rows, M, K, what):
    """Codes held by an FP6-layout activation buffer on `rows` against the
    oracle's packed 4-bit codes of those rows; padding rows must be zero."""
    codes, pad = fp6_layout_decode(_h(buf), M, K)
    assert (pad == 0).all(), f"{what}: nonzero padding rows"
    ref = unpack_int4(c_ref_packed)
    assert_bytes(codes[rows], ref, what + " FP6 codes")


def _gemm_paths(dev, bits, codes, scales, a6, wq, ws, M, K, N):
    """y [M, N] of every GEMM path that serves `bits`, by name."""
    wqd, wsd = _d(wq, dev), _d(ws, dev)
    out = {"int8": dptq.qlinear(codes, scales, bits, wqd, wsd)}
    if bits == 8:
        w8 = dptq.prepack_weights(wqd, dptq.WEIGHTS_A8_ORDER)
        out["int8_a8order"] = dptq.qlinear_a8(codes, scales, w8.view(N, K // 2), wsd)
    elif a6 is not None:
        w6 = dptq.prepack_weights(wqd, dptq.WEIGHTS_FP6)
        out["fp6"] = dptq.qlinear_fp6(a6, scales, w6, wsd, M, K, N)
    return {k: _h(v) for k, v in out.items()}


# ---------------------------------------------------------------------------
# single linears: every row
# ---------------------------------------------------------------------------
SINGLE = [("tiny", 16), ("llama2_7b_qkv", 2048), ("llama3_8b_down", 1),
          ("llama3_8b_down", 4), ("llama3_8b_down", 16), ("llama3_8b_down", 2048)]


@pytest.mark.parametrize("name,M", SINGLE)
def test_single_linear_every_row(dev, name, M):
    cfg = workloads.CONFIGS[name]
    K, N, h = cfg["K"], cfg["N"], cfg["h"]
    x = workloads.activations_for(name, M=M)
    xd = _d(x, dev)
    y_rot = oracle_rotate(x, h)
    rng = np.random.default_rng([cfg["seed"], M, 99])
    wq = workloads.random_weight_bytes(rng, N, K)
    rows = np.arange(M)
    for bits in (4, 8):
        what = f"{name} M={M} A{bits}"
        c_ref, s_ref = oracle_codes(y_rot, bits)
        codes, scales = dptq.rotate_quant(xd, h, bits)
        assert_bytes(_h(scales), s_ref, what + " scales")
        assert_bytes(_h(codes), c_ref, what + " codes")
        a6 = None
        if bits == 4:
            a6, s6 = dptq.rotate_quant_fp6(xd, h)
            assert_bytes(_h(s6), s_ref, what + " FP6-path scales")
            _check_fp6(a6, c_ref, rows, M, K, what)
        ws = safe_w_scales(rng, N, K, s_ref, bits)
        acc_ref = oracle_acc(c_ref, bits, wq)
        y_ref = oracle_y(acc_ref, s_ref, ws)
        for path, y in _gemm_paths(dev, bits, codes, scales, a6, wq, ws, M, K, N).items():
            assert_f16(y, y_ref, f"{what} y ({path})")
        wqd = _d(wq, dev)
        assert_acc(_h(dptq.qlinear_acc(codes, bits, wqd)), acc_ref, what + " int8")
        if a6 is not None:
            w6 = dptq.prepack_weights(wqd, dptq.WEIGHTS_FP6)
            assert_acc(_h(dptq.qlinear_fp6_acc(a6, w6, M, K, N)), acc_ref, what + " FP6")


# ---------------------------------------------------------------------------
# offline weight preparation, every distinct linear
# ---------------------------------------------------------------------------
WEIGHT_SHAPES = [("tiny", None), ("llama2_7b_qkv", None), ("llama3_8b_down", None)] + \
    [(cfg, lin) for cfg in ("llama2_7b_stack", "llama2_70b_layer")
     for lin, *_ in workloads.CONFIGS[cfg]["linears"]]


@pytest.mark.parametrize("cfg,linear", WEIGHT_SHAPES)
def test_prepare_weights_sampled_rows(dev, cfg, linear):
    c = workloads.CONFIGS[cfg]
    if linear is None:
        K, N, h = c["K"], c["N"], c["h"]
        w = workloads.weights(np.random.default_rng([c["seed"], 1]), N, K)
    else:
        _, K, N, h = next(t for t in c["linears"] if t[0] == linear)
        w = workloads.stack_weights(cfg, 0, linear)
    wp, ws = dptq.prepare_weights(_d(w, dev), h)
    rows = sample_rows(N, 256, seed=N + K)
    wp_ref, ws_ref = oracle_prepare(w[rows], h)
    assert_bytes(_h(ws)[rows], ws_ref, f"{cfg}/{linear} w_scales")
    assert_bytes(_h(wp)[rows], wp_ref, f"{cfg}/{linear} w codes")


# ---------------------------------------------------------------------------
# layer stacks: >= 256 sampled rows, every output column
# ---------------------------------------------------------------------------
STACK = [(cfg, lin) for cfg in ("llama2_7b_stack", "llama2_70b_layer")
         for lin, *_ in workloads.CONFIGS[cfg]["linears"]]


def _policy_layers(cfg):
    """An 8-bit layer of the default policy and a 4-bit one (inside the
    massive-activation phase window of the 7B stack)."""
    L = workloads.CONFIGS[cfg]["L"]
    bits = dptq.layer_policy(L)
    mid = L // 2
    assert bits[0] == 8 and bits[mid] == 4
    return [(0, 8), (mid, 4)]


@pytest.mark.parametrize("cfg,linear", STACK)
def test_stack_linear_prefill(dev, cfg, linear):
    c = workloads.CONFIGS[cfg]
    _, K, N, h = next(t for t in c["linears"] if t[0] == linear)
    M = c["M"]
    rng = np.random.default_rng([c["seed"], K, N, 7])
    wq = workloads.random_weight_bytes(rng, N, K)
    for layer, bits in _policy_layers(cfg):
        what = f"{cfg}/{linear} layer {layer} M={M} A{bits}"
        x = workloads.stack_layer_input(cfg, layer, linear, M=M)
        xd = _d(x, dev)
        rows = sample_rows(M, 256, seed=M + layer + K)
        c_ref, s_ref = oracle_codes(oracle_rotate(x[rows], h), bits)
        codes, scales = dptq.rotate_quant(xd, h, bits)
        assert_bytes(_h(scales)[rows], s_ref, what + " scales")
        assert_bytes(_h(codes)[rows], c_ref, what + " codes")
        a6 = None
        if bits == 4:
            a6, s6 = dptq.rotate_quant_fp6(xd, h)
            assert_bytes(_h(s6)[rows], s_ref, what + " FP6-path scales")
            _check_fp6(a6, c_ref, rows, M, K, what)
        ws = safe_w_scales(rng, N, K, s_ref, bits)
        y_ref = oracle_y(oracle_acc(c_ref, bits, wq), s_ref, ws)
        for path, y in _gemm_paths(dev, bits, codes, scales, a6, wq, ws, M, K, N).items():
            assert_f16(y[rows], y_ref, f"{what} y ({path})")
        del xd, codes, scales, a6
        torch.cuda.empty_cache()


DECODE = [(cfg, lin) for cfg in ("llama2_70b_layer",)
          for lin, *_ in workloads.CONFIGS[cfg]["linears"]]


@pytest.mark.parametrize("cfg,linear", DECODE)
def test_stack_linear_decode(dev, cfg, linear):
    # M = 8 decode of the 70B layer: every row and column, on the decode
    # GEMM and on the decode entry point from fp16 x (its automatic choice of
    # one launch or two, as the benchmark runs it).
    c = workloads.CONFIGS[cfg]
    _, K, N, h = next(t for t in c["linears"] if t[0] == linear)
    M = 8
    rng = np.random.default_rng([c["seed"], K, N, 8])
    wq = workloads.random_weight_bytes(rng, N, K)
    for layer, bits in _policy_layers(cfg):
        what = f"{cfg}/{linear} layer {layer} M={M} A{bits}"
        x = workloads.stack_layer_input(cfg, layer, linear, M=M)
        xd = _d(x, dev)
        c_ref, s_ref = oracle_codes(oracle_rotate(x, h), bits)
        codes, scales = dptq.rotate_quant(xd, h, bits)
        assert_bytes(_h(scales), s_ref, what + " scales")
        assert_bytes(_h(codes), c_ref, what + " codes")
        ws = safe_w_scales(rng, N, K, s_ref, bits)
        y_ref = oracle_y(oracle_acc(c_ref, bits, wq), s_ref, ws)
        wqd, wsd = _d(wq, dev), _d(ws, dev)
        assert_f16(_h(dptq.qlinear(codes, scales, bits, wqd, wsd)), y_ref, what + " y (decode GEMM)")
        y, c2, s2 = dptq.qlinear_decode_fused(xd, h, bits, wqd, wsd, mode=dptq.DECODE_AUTO)
        assert_bytes(_h(c2), c_ref, what + " codes (decode entry point)")
        assert_f16(_h(y), y_ref, what + " y (decode entry point)")


# ---------------------------------------------------------------------------
# int32 accumulators in full at every full prefill shape
# ---------------------------------------------------------------------------
FULL = [("llama2_7b_qkv", 2048, 4096, 12288), ("llama3_8b_down", 2048, 14336, 4096)] + \
    [(f"{cfg}/{lin}", workloads.CONFIGS[cfg]["M"], K, N)
     for cfg in ("llama2_7b_stack", "llama2_70b_layer")
     for lin, K, N, _ in workloads.CONFIGS[cfg]["linears"]]


@pytest.mark.parametrize("bits", [4, 8])
@pytest.mark.parametrize("name,M,K,N", FULL)
def test_full_accumulators(dev, name, M, K, N, bits):
    rng = np.random.default_rng([M, K, N, bits])
    a = workloads.random_code_bytes(rng, M, K, bits)
    wq = workloads.random_weight_bytes(rng, N, K)
    acc_ref = oracle_acc(a, bits, wq)
    ad, wqd = _d(a, dev), _d(wq, dev)
    assert_acc(_h(dptq.qlinear_acc(ad, bits, wqd)), acc_ref, f"{name} A{bits} int8")
    if bits == 4:
        w6 = dptq.prepack_weights(wqd, dptq.WEIGHTS_FP6)
        assert_acc(_h(dptq.qlinear_fp6_acc(dptq.pack_fp6(ad), w6, M, K, N)), acc_ref,
                   f"{name} A4 FP6")
    else:
        a_s = workloads.random_scales(rng, M, 1e-3, 1.0)
        ws = safe_w_scales(rng, N, K, a_s, bits)
        w8 = dptq.prepack_weights(wqd, dptq.WEIGHTS_A8_ORDER)
        y = _h(dptq.qlinear_a8(ad, _d(a_s, dev), w8.view(N, K // 2), _d(ws, dev)))
        assert_f16(y, oracle_y(acc_ref, a_s, ws), f"{name} A8 y (8-bit-order weights)")
    torch.cuda.empty_cache()


def test_prepack_weights_matches_both_packers(dev):
    # dptq_prepack_weights equals the FP6 packer and the 8-bit-order packer,
    # and its output sizes are what the layouts state.
    from oracle import pack_int4_a8order
    from paritylib import fp6_layout_ref
    rng = np.random.default_rng(3)
    for N, K in [(16, 128), (33, 640), (272, 4096)]:
        wq = workloads.random_weight_bytes(rng, N, K)
        wqd = _d(wq, dev)
        w6 = _h(dptq.prepack_weights(wqd, dptq.WEIGHTS_FP6))
        assert w6.shape == (dptq.fp6_bytes(N, K),)
        assert_bytes(w6[None], fp6_layout_ref(wq, K)[None], f"FP6 N={N} K={K}")
        w8 = _h(dptq.prepack_weights(wqd, dptq.WEIGHTS_A8_ORDER))
        assert w8.shape == (N * K // 2,)
        assert_bytes(w8.reshape(N, K // 2), pack_int4_a8order(unpack_int4(wq)), f"A8 order N={N} K={K}")
