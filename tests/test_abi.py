"""Host-side tests of the C ABI (no GPU needed).

The library must load, export every function include/dptq.h declares, run the
host-only policy exactly as the oracle does, and reject every invalid argument
before anything is enqueued (so these calls never touch a GPU).
"""

import ctypes
import os
import re

import pytest

import paper_2606_12487_amd as dptq
from oracle.policy import layer_policy_ref

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dptq.h")

OK, INVALID, UNSUPPORTED, HIPERR = 0, 1, 2, 3
FAKE = ctypes.c_void_p(0x10000)           # aligned, never dereferenced
MISALIGNED = ctypes.c_void_p(0x10004)
NULL = ctypes.c_void_p(0)


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dptq_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(dptq.library_path()):
        import __graft_entry__
        __graft_entry__.build()
    return dptq.lib()


def test_header_and_binding_agree():
    assert _declared_functions() == sorted(dptq.EXPORTED_FUNCTIONS)


def test_every_declared_symbol_is_exported(L):
    for name in _declared_functions():
        assert hasattr(L, name), name


def test_status_strings_and_version(L):
    for st in (OK, INVALID, UNSUPPORTED, HIPERR):
        assert L.dptq_status_string(st)
    assert L.dptq_status_string(99) == b"unknown status"
    assert dptq.version() >= 100


@pytest.mark.parametrize("L_layers", [1, 2, 3, 4, 5, 28, 32, 40, 80])
def test_policy_default_matches_oracle(L, L_layers):
    assert dptq.layer_policy(L_layers) == layer_policy_ref(L_layers)


def test_policy_mask_matches_oracle(L):
    import workloads
    for Ls, seed in ((32, 3), (80, 5)):
        mask = workloads.layer_mask(Ls, 4, seed)
        assert dptq.layer_policy(Ls, mask) == layer_policy_ref(Ls, list(mask))
        assert sum(b == 8 for b in dptq.layer_policy(Ls, mask)) == 4


def test_policy_rejects_bad_args(L):
    out = (ctypes.c_int32 * 4)()
    assert L.dptq_layer_policy(0, NULL, ctypes.cast(out, ctypes.c_void_p)) == INVALID
    assert L.dptq_layer_policy(4, NULL, NULL) == INVALID


def rq(L, x=FAKE, M=4, K=256, h=256, bits=4, codes=FAKE, scales=FAKE):
    return L.dptq_rotate_quant(x, M, K, h, bits, codes, scales, NULL)


def test_rotate_quant_validation(L):
    assert rq(L, bits=5) == INVALID
    assert rq(L, bits=0) == INVALID
    assert rq(L, M=-1) == INVALID
    assert rq(L, K=0) == INVALID
    assert rq(L, h=12) == INVALID            # not 2^j or 28 * 2^j
    assert rq(L, h=0) == INVALID
    assert rq(L, h=65536, K=65536) == INVALID
    assert rq(L, K=384, h=256) == INVALID   # h does not divide K
    assert rq(L, K=28 * 9, h=28) == INVALID  # K not a multiple of 8
    assert rq(L, K=36864 + 256, h=256) == UNSUPPORTED
    assert rq(L, x=NULL) == INVALID
    assert rq(L, codes=NULL) == INVALID
    assert rq(L, scales=NULL) == INVALID
    assert rq(L, x=MISALIGNED) == INVALID
    assert rq(L, codes=MISALIGNED) == INVALID
    # M = 0 is a valid empty call: nothing is enqueued, pointers may be null
    assert rq(L, M=0, x=NULL, codes=NULL, scales=NULL) == OK


def ql(L, codes=FAKE, a_s=FAKE, M=32, K=256, bits=4, w=FAKE, w_s=FAKE, N=64, y=FAKE):
    return L.dptq_qlinear(codes, a_s, M, K, bits, w, w_s, N, y, NULL)


def test_qlinear_validation(L):
    assert ql(L, bits=2) == INVALID
    assert ql(L, M=-3) == INVALID
    assert ql(L, N=0) == INVALID
    assert ql(L, K=0) == INVALID
    assert ql(L, K=192) == UNSUPPORTED       # K % 128
    assert ql(L, K=65536 + 128) == UNSUPPORTED
    assert ql(L, N=72) == UNSUPPORTED        # N % 16
    for name in ("codes", "a_s", "w", "w_s", "y"):
        assert ql(L, **{name: NULL}) == INVALID, name
        assert ql(L, **{name: MISALIGNED}) == INVALID, name
    assert ql(L, M=0, codes=NULL, a_s=NULL, w=NULL, w_s=NULL, y=NULL) == OK


def test_qlinear_acc_validation(L):
    f = L.dptq_qlinear_acc
    assert f(FAKE, 8, 256, 3, FAKE, 64, FAKE, NULL) == INVALID
    assert f(NULL, 8, 256, 4, FAKE, 64, FAKE, NULL) == INVALID
    assert f(FAKE, 8, 256, 4, NULL, 64, FAKE, NULL) == INVALID
    assert f(FAKE, 8, 256, 4, FAKE, 64, NULL, NULL) == INVALID
    assert f(FAKE, 8, 200, 4, FAKE, 64, FAKE, NULL) == UNSUPPORTED
    assert f(FAKE, 0, 256, 8, NULL, 64, NULL, NULL) == OK


def qk(L, codes=FAKE, a_s=FAKE, M=300, K=1024, bits=4, w=FAKE, w_s=FAKE, N=272, y=FAKE,
       acc=NULL, kernel=0):
    return L.dptq_qlinear_kernel(codes, a_s, M, K, bits, w, w_s, N, y, acc, kernel, NULL)


def test_qlinear_kernel_validation(L):
    assert qk(L, kernel=-1) == INVALID
    assert qk(L, kernel=4) == INVALID
    assert qk(L, acc=FAKE) == INVALID                       # both y and acc
    assert qk(L, y=NULL) == INVALID                         # neither
    assert qk(L, kernel=dptq.GEMM_DECODE) == UNSUPPORTED    # M > 16
    assert qk(L, kernel=dptq.GEMM_TILE_192X256, M=255) == UNSUPPORTED
    assert qk(L, kernel=dptq.GEMM_TILE_192X256, N=176) == UNSUPPORTED
    assert qk(L, kernel=dptq.GEMM_TILE_192X256, K=384) == UNSUPPORTED
    assert qk(L, K=200) == UNSUPPORTED
    for name in ("codes", "a_s", "w", "w_s"):
        assert qk(L, **{name: NULL}) == INVALID, name
        assert qk(L, **{name: MISALIGNED}) == INVALID, name
    # the accumulator output ignores the scales
    assert qk(L, M=0, y=NULL, acc=FAKE, a_s=NULL, w_s=NULL, codes=NULL, w=NULL) == OK
    assert qk(L, y=NULL, acc=MISALIGNED, a_s=NULL, w_s=NULL) == INVALID
    assert qk(L, M=0, kernel=dptq.GEMM_DECODE, codes=NULL, a_s=NULL, w=NULL, w_s=NULL) == OK


def rd(L, x=FAKE, dx=FAKE, T=4, K=256, h=256, bits=4, eps=1e-8, jr=FAKE, snr=FAKE, means=FAKE):
    return L.dptq_residual_dynamics(x, dx, T, K, h, bits, eps, jr, snr, means, NULL)


def test_residual_dynamics_validation(L):
    assert rd(L, bits=3) == INVALID
    assert rd(L, h=12) == INVALID
    assert rd(L, K=384) == INVALID               # h does not divide K
    assert rd(L, K=36864 + 256) == UNSUPPORTED
    assert rd(L, eps=-1.0) == INVALID
    assert rd(L, eps=float("nan")) == INVALID
    assert rd(L, eps=float("inf")) == INVALID
    for name in ("x", "dx", "jr", "snr"):
        assert rd(L, **{name: NULL}) == INVALID, name
    assert rd(L, x=MISALIGNED) == INVALID
    assert rd(L, dx=MISALIGNED) == INVALID
    assert rd(L, means=ctypes.c_void_p(0x10004)) == INVALID    # doubles need 8-byte alignment
    assert rd(L, T=0, x=NULL, dx=NULL, jr=NULL, snr=NULL, means=NULL) == OK


def test_select_layers_matches_oracle(L):
    import random
    from oracle.residual import select_sensitive_layers_ref
    rnd = random.Random(7)
    for _ in range(50):
        n = rnd.randint(1, 40)
        jr = [rnd.choice([0.1, 0.5, 0.9, rnd.random()]) for _ in range(n)]
        snr = [rnd.choice([5.0, 15.0, 25.0, 30 * rnd.random()]) for _ in range(n)]
        tj, ts = rnd.choice([0.5, 0.3]), rnd.choice([15.0, 20.0])
        assert dptq.select_layers(jr, snr, tj, ts) == select_sensitive_layers_ref(jr, snr, tj, ts)[1]
    out = (ctypes.c_int32 * 2)()
    assert L.dptq_select_layers(0, FAKE, FAKE, 0.0, 0.0, ctypes.cast(out, ctypes.c_void_p)) == INVALID


def kvq(L, kv=FAKE, T=4, D=256, group=128, codes=FAKE, scales=FAKE, mins=FAKE):
    return L.dptq_kv_quant(kv, T, D, group, codes, scales, mins, NULL)


def kvd(L, codes=FAKE, scales=FAKE, mins=FAKE, T=4, D=256, group=128, out=FAKE):
    return L.dptq_kv_dequant(codes, scales, mins, T, D, group, out, NULL)


def test_kv_codec_validation(L):
    for f in (kvq, kvd):
        assert f(L, group=96) == INVALID                  # not a power of two
        assert f(L, group=8) == INVALID
        assert f(L, group=1024) == INVALID
        assert f(L, D=320) == INVALID                     # not a multiple of the group
        assert f(L, T=-1) == INVALID
        assert f(L, D=0) == INVALID
        assert f(L, T=1 << 30, D=4096) == UNSUPPORTED     # T * D >= 2^40
        assert f(L, scales=NULL) == INVALID
        assert f(L, mins=NULL) == INVALID
        assert f(L, codes=ctypes.c_void_p(0x10002)) == INVALID
        assert f(L, scales=ctypes.c_void_p(0x10002)) == INVALID
        assert f(L, T=0, codes=NULL, scales=NULL, mins=NULL) == OK
    assert kvq(L, kv=NULL) == INVALID
    assert kvq(L, kv=MISALIGNED) == INVALID
    assert kvd(L, out=NULL) == INVALID
    assert kvd(L, out=MISALIGNED) == INVALID


def test_prepare_weights_validation(L):
    f = L.dptq_prepare_weights
    assert f(FAKE, 16, 256, 100, FAKE, FAKE, NULL) == INVALID
    assert f(NULL, 16, 256, 256, FAKE, FAKE, NULL) == INVALID
    assert f(FAKE, 16, 256, 256, MISALIGNED, FAKE, NULL) == INVALID
    assert f(FAKE, -1, 256, 256, FAKE, FAKE, NULL) == INVALID
    assert f(NULL, 0, 256, 256, NULL, NULL, NULL) == OK


def test_python_wrappers_check_tensors():
    torch = pytest.importorskip("torch")
    with pytest.raises(TypeError):
        dptq.rotate_quant(torch.zeros(4, 256, dtype=torch.float32), 256, 4)
    with pytest.raises(ValueError):
        dptq.rotate_quant(torch.zeros(4, 256, dtype=torch.float16), 256, 4)  # not on GPU
    with pytest.raises(ValueError):
        dptq.layer_policy(3, [1, 0])


def test_rotate_quant_ex_validation(L):
    def call(bits=4, layout=0, K=256, h=256, x=FAKE, out=FAKE, sc=FAKE, M=4):
        return L.dptq_rotate_quant_ex(x, M, K, h, bits, NULL, layout, out, sc, NULL)
    assert call(layout=2) == INVALID
    assert call(layout=1, bits=8) == INVALID
    assert call(layout=1, K=64, h=64) == UNSUPPORTED          # FP6 layout needs K % 128 == 0
    assert call(bits=5) == INVALID
    assert call(x=NULL) == INVALID
    assert call(out=MISALIGNED) == INVALID
    assert call(M=0, x=NULL) == OK                            # nothing to do, nothing enqueued
    assert L.dptq_prepare_weights_signed(FAKE, 4, 256, 100, NULL, FAKE, FAKE, NULL) == INVALID
    assert L.dptq_prepare_weights_signed(NULL, 4, 256, 256, NULL, FAKE, FAKE, NULL) == INVALID


def test_fp6_entry_points_validation(L):
    assert L.dptq_fp6_bytes(32, 128) == 3072
    assert L.dptq_fp6_bytes(33, 256) == 2 * 2 * 3072
    assert L.dptq_fp6_bytes(1, 100) == -1
    assert L.dptq_pack_fp6(FAKE, 4, 192, FAKE, NULL) == UNSUPPORTED
    assert L.dptq_pack_fp6(MISALIGNED, 4, 256, FAKE, NULL) == INVALID
    # exactly one of y and acc
    assert L.dptq_qlinear_fp6(FAKE, FAKE, 4, 256, FAKE, FAKE, 32, NULL, NULL, NULL) == INVALID
    assert L.dptq_qlinear_fp6(FAKE, FAKE, 4, 256, FAKE, FAKE, 32, FAKE, FAKE, NULL) == INVALID
    assert L.dptq_qlinear_fp6(FAKE, FAKE, 4, 200, FAKE, FAKE, 32, FAKE, NULL, NULL) == UNSUPPORTED
    assert L.dptq_qlinear_fp6(FAKE, FAKE, 4, 256, FAKE, FAKE, 24, FAKE, NULL, NULL) == UNSUPPORTED
    assert L.dptq_rotate_quant_fp6(FAKE, 4, 192, 64, FAKE, FAKE, NULL) == UNSUPPORTED


def test_prepack_weights_validation(L):
    assert L.dptq_prepacked_bytes(33, 256, 1) == L.dptq_fp6_bytes(33, 256)
    assert L.dptq_prepacked_bytes(33, 256, 2) == 33 * 128
    assert L.dptq_prepacked_bytes(33, 256, 0) == -1            # no such layout
    assert L.dptq_prepacked_bytes(33, 200, 2) == -1            # K % 128 != 0
    assert L.dptq_prepacked_bytes(-1, 256, 1) == -1
    assert L.dptq_prepacked_bytes(32, 256, 3) == 32 * 128       # decode layout
    assert L.dptq_prepacked_bytes(33, 256, 3) == -1            # N % 16 != 0
    for layout in (1, 2, 3):
        assert L.dptq_prepack_weights(FAKE, 16, 192, layout, FAKE, NULL) == UNSUPPORTED
        assert L.dptq_prepack_weights(MISALIGNED, 16, 256, layout, FAKE, NULL) == INVALID
        assert L.dptq_prepack_weights(FAKE, 16, 256, layout, NULL, NULL) == INVALID
        assert L.dptq_prepack_weights(NULL, 0, 256, layout, NULL, NULL) == OK   # nothing to do
    assert L.dptq_prepack_weights(FAKE, 4, 256, 3, FAKE, NULL) == UNSUPPORTED  # N % 16 != 0
    assert L.dptq_prepack_weights(FAKE, 4, 256, 0, FAKE, NULL) == INVALID
    assert L.dptq_prepack_weights(FAKE, 16, 256, 4, FAKE, NULL) == INVALID


def test_decode_native_validation(L):
    def dn(codes=FAKE, a_s=FAKE, M=4, K=1024, bits=4, w=FAKE, w_s=FAKE, N=256, y=FAKE, acc=NULL):
        return L.dptq_qlinear_decode_native(codes, a_s, M, K, bits, w, w_s, N, y, acc, NULL)
    assert dn(M=17) == UNSUPPORTED                 # decode batches only
    assert dn(K=1000) == UNSUPPORTED
    assert dn(N=40) == UNSUPPORTED
    assert dn(bits=6) == INVALID
    assert dn(acc=FAKE) == INVALID                 # both outputs
    assert dn(y=NULL) == INVALID                   # neither output
    assert dn(w=MISALIGNED) == INVALID
    assert dn(a_s=NULL) == INVALID
    assert dn(codes=NULL) == INVALID
    assert dn(M=0) == OK                           # nothing to do


def test_a8order_entry_points_validation(L):
    pk = L.dptq_pack_w4_a8
    assert pk(FAKE, -1, 256, FAKE, NULL) == INVALID
    assert pk(FAKE, 4, 192, FAKE, NULL) == UNSUPPORTED
    assert pk(FAKE, 4, 256, MISALIGNED, NULL) == INVALID
    assert pk(NULL, 4, 256, FAKE, NULL) == INVALID
    assert pk(NULL, 0, 256, NULL, NULL) == OK

    def qa(codes=FAKE, a_s=FAKE, M=300, K=1024, w=FAKE, w_s=FAKE, N=272, y=FAKE, kernel=0):
        return L.dptq_qlinear_a8(codes, a_s, M, K, w, w_s, N, y, kernel, NULL)
    assert qa(kernel=4) == INVALID
    assert qa(kernel=dptq.GEMM_DECODE) == UNSUPPORTED          # M > 16
    assert qa(kernel=dptq.GEMM_TILE_192X256, M=255) == UNSUPPORTED
    assert qa(K=200) == UNSUPPORTED
    assert qa(N=24) == UNSUPPORTED
    for name in ("codes", "a_s", "w", "w_s", "y"):
        assert qa(**{name: NULL}) == INVALID, name
        assert qa(**{name: MISALIGNED}) == INVALID, name
    assert qa(M=0, codes=NULL, a_s=NULL, w=NULL, w_s=NULL, y=NULL) == OK


def test_fused_decode_validation(L):
    def call(M=4, K=4096, h=4096, bits=4, N=64, x=FAKE, y=FAKE, codes=FAKE, scales=FAKE, mode=1):
        return L.dptq_qlinear_decode_fused(x, M, K, h, bits, FAKE, FAKE, N, y, codes, scales, mode,
                                           NULL)
    assert call(M=17) == UNSUPPORTED            # decode shapes only
    assert call(M=17, mode=2) == UNSUPPORTED
    assert call(K=36864, h=4096) == UNSUPPORTED # one row's staging does not fit on chip
    # 16 A8 rows of 14336 codes do not fit on chip for the one launch; the
    # two launches take them (then the null y is the first error)
    assert call(M=16, K=14336, h=28 * 512, bits=8) == UNSUPPORTED
    assert call(M=16, K=14336, h=28 * 512, bits=8, mode=2, y=NULL) == INVALID
    assert call(M=16, K=14336, h=28 * 512, bits=8, mode=0, y=NULL) == INVALID
    assert call(mode=3) == INVALID
    assert call(mode=-1) == INVALID
    assert call(bits=6) == INVALID
    assert call(y=NULL) == INVALID
    assert call(codes=NULL) == INVALID
    assert call(scales=NULL) == INVALID
    assert call(codes=MISALIGNED) == INVALID
    assert call(N=24) == UNSUPPORTED
    assert call(h=3) == INVALID
    assert call(M=0, x=NULL) == OK


def test_range_entry_points_validation(L):
    def rq(M=4, K=4096, h=4096, bits=4, x=FAKE, codes=FAKE, scales=FAKE, zeros=FAKE):
        return L.dptq_rotate_quant_range(x, M, K, h, bits, codes, scales, zeros, NULL)
    assert rq(bits=5) == INVALID
    assert rq(K=4104, h=8) == UNSUPPORTED        # rows must be whole 128-element chunks
    assert rq(h=3) == INVALID
    assert rq(zeros=NULL) == INVALID
    assert rq(codes=MISALIGNED) == INVALID
    assert rq(M=0, x=NULL) == OK
    assert L.dptq_weight_sums(FAKE, 4, 48, FAKE, NULL) == UNSUPPORTED
    assert L.dptq_weight_sums(FAKE, 4, 64, NULL, NULL) == INVALID
    assert L.dptq_weight_sums(MISALIGNED, 4, 64, FAKE, NULL) == INVALID
    assert L.dptq_weight_sums(NULL, 0, 64, NULL, NULL) == OK

    def ql(M=4, K=256, bits=4, N=32, y=FAKE, sums=FAKE, scales=FAKE):
        return L.dptq_qlinear_range(FAKE, scales, FAKE, M, K, bits, FAKE, FAKE, sums, N, y, NULL)
    assert ql(K=200) == UNSUPPORTED
    assert ql(N=24) == UNSUPPORTED
    assert ql(bits=6) == INVALID
    assert ql(sums=NULL) == INVALID
    assert ql(y=MISALIGNED) == INVALID
    assert ql(scales=MISALIGNED) == INVALID
    assert ql(M=0, y=NULL) == OK
