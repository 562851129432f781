"""Python binding of libdptq, the MI355X quantized linear layer of DynamicPTQ.

Thin ctypes marshalling over the C ABI declared in ``include/dptq.h``: the
functions below check tensor dtypes and shapes, allocate outputs with torch
(device memory and streams only) and call the library on the current HIP
stream.  Every arithmetic step runs in the library's kernels; there is no
fallback path, and importing a function whose library is missing raises.

    codes, scales = rotate_quant(x_fp16, had_size=4096, bits=4)
    w_packed, w_scales = prepare_weights(w_fp32, had_size=4096)
    y = qlinear(codes, scales, 4, w_packed, w_scales)
"""

import ctypes
import os

__all__ = ["DptqError", "lib", "library_path", "rotate_quant", "qlinear", "qlinear_acc",
           "layer_policy", "prepare_weights", "residual_dynamics", "select_layers",
           "kv_quant", "kv_dequant", "version", "fp6_bytes", "pack_fp6", "rotate_quant_fp6", "qlinear_fp6",
           "LAYOUT_PACKED", "LAYOUT_FP6", "qlinear_decode_fused", "DECODE_AUTO", "DECODE_ONE_LAUNCH",
           "DECODE_TWO_LAUNCHES", "rotate_quant_range", "weight_sums", "qlinear_range",
           "qlinear_fp6_acc", "pack_w4_a8", "qlinear_a8", "prepacked_bytes", "prepack_weights",
           "WEIGHTS_FP6", "WEIGHTS_A8_ORDER", "WEIGHTS_DECODE", "qlinear_decode_native",
           "qlinear_decode_native_acc",
           "EXPORTED_FUNCTIONS", "GEMM_AUTO",
           "GEMM_DECODE", "GEMM_TILE_256X128", "GEMM_TILE_192X256"]

_PKG_DIR = os.path.dirname(os.path.abspath(__file__))
_LIB_NAME = "libdptq.so"
_lib = None

# Every function the C ABI exports (include/dptq.h).
EXPORTED_FUNCTIONS = ("dptq_status_string", "dptq_version", "dptq_rotate_quant",
                      "dptq_qlinear", "dptq_qlinear_acc", "dptq_qlinear_kernel",
                      "dptq_residual_dynamics", "dptq_select_layers",
                      "dptq_kv_quant", "dptq_kv_dequant",
                      "dptq_layer_policy", "dptq_prepare_weights",
                      "dptq_fp6_bytes", "dptq_pack_fp6", "dptq_rotate_quant_fp6",
                      "dptq_qlinear_fp6", "dptq_rotate_quant_ex", "dptq_prepare_weights_signed",
                      "dptq_qlinear_decode_fused", "dptq_rotate_quant_range",
                      "dptq_weight_sums", "dptq_qlinear_range", "dptq_pack_w4_a8",
                      "dptq_qlinear_a8", "dptq_prepacked_bytes", "dptq_prepack_weights",
                      "dptq_qlinear_decode_native")

# Code layouts of dptq_rotate_quant_ex.
LAYOUT_PACKED, LAYOUT_FP6 = 0, 1

# Device-native weight layouts of dptq_prepack_weights.
WEIGHTS_FP6, WEIGHTS_A8_ORDER, WEIGHTS_DECODE = 1, 2, 3

# GEMM kernels (dptq_gemm_kernel); every kernel returns the same bits.
GEMM_AUTO, GEMM_DECODE, GEMM_TILE_256X128, GEMM_TILE_192X256 = 0, 1, 2, 3


class DptqError(RuntimeError):
    def __init__(self, status, what):
        self.status = status
        super().__init__(f"{what}: {_status_string(status)} (status {status})")


def library_path():
    return os.path.join(_PKG_DIR, _LIB_NAME)


def lib():
    """The loaded libdptq (ctypes.CDLL).  Raises if it has not been built."""
    global _lib
    if _lib is None:
        path = library_path()
        if not os.path.exists(path):
            raise RuntimeError(
                f"{path} is missing: build it with `python -m paper_2606_12487_amd.build` "
                "(the HIP library is required; there is no fallback)")
        L = ctypes.CDLL(path)
        i64, i32, vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p
        L.dptq_status_string.argtypes = [ctypes.c_int]
        L.dptq_status_string.restype = ctypes.c_char_p
        L.dptq_version.argtypes = []
        L.dptq_version.restype = ctypes.c_int
        L.dptq_rotate_quant.argtypes = [vp, i64, i64, i32, i32, vp, vp, vp]
        L.dptq_rotate_quant.restype = ctypes.c_int
        L.dptq_qlinear.argtypes = [vp, vp, i64, i64, i32, vp, vp, i64, vp, vp]
        L.dptq_qlinear.restype = ctypes.c_int
        L.dptq_qlinear_acc.argtypes = [vp, i64, i64, i32, vp, i64, vp, vp]
        L.dptq_qlinear_acc.restype = ctypes.c_int
        L.dptq_qlinear_kernel.argtypes = [vp, vp, i64, i64, i32, vp, vp, i64, vp, vp, i32, vp]
        L.dptq_qlinear_kernel.restype = ctypes.c_int
        L.dptq_qlinear_decode_native.argtypes = [vp, vp, i64, i64, i32, vp, vp, i64, vp, vp, vp]
        L.dptq_qlinear_decode_native.restype = ctypes.c_int
        L.dptq_residual_dynamics.argtypes = [vp, vp, i64, i64, i32, i32, ctypes.c_float,
                                             vp, vp, vp, vp]
        L.dptq_residual_dynamics.restype = ctypes.c_int
        L.dptq_select_layers.argtypes = [i32, vp, vp, ctypes.c_double, ctypes.c_double, vp]
        L.dptq_select_layers.restype = ctypes.c_int
        L.dptq_kv_quant.argtypes = [vp, i64, i64, i32, vp, vp, vp, vp]
        L.dptq_kv_quant.restype = ctypes.c_int
        L.dptq_kv_dequant.argtypes = [vp, vp, vp, i64, i64, i32, vp, vp]
        L.dptq_kv_dequant.restype = ctypes.c_int
        L.dptq_layer_policy.argtypes = [i32, vp, vp]
        L.dptq_layer_policy.restype = ctypes.c_int
        L.dptq_prepare_weights.argtypes = [vp, i64, i64, i32, vp, vp, vp]
        L.dptq_prepare_weights.restype = ctypes.c_int
        L.dptq_fp6_bytes.argtypes = [i64, i64]
        L.dptq_fp6_bytes.restype = ctypes.c_int64
        L.dptq_pack_fp6.argtypes = [vp, i64, i64, vp, vp]
        L.dptq_pack_fp6.restype = ctypes.c_int
        L.dptq_rotate_quant_fp6.argtypes = [vp, i64, i64, i32, vp, vp, vp]
        L.dptq_rotate_quant_fp6.restype = ctypes.c_int
        L.dptq_rotate_quant_ex.argtypes = [vp, i64, i64, i32, i32, vp, i32, vp, vp, vp]
        L.dptq_rotate_quant_ex.restype = ctypes.c_int
        L.dptq_prepare_weights_signed.argtypes = [vp, i64, i64, i32, vp, vp, vp, vp]
        L.dptq_prepare_weights_signed.restype = ctypes.c_int
        L.dptq_qlinear_decode_fused.argtypes = [vp, i64, i64, i32, i32, vp, vp, i64, vp, vp, vp,
                                                 i32, vp]
        L.dptq_qlinear_decode_fused.restype = ctypes.c_int
        L.dptq_rotate_quant_range.argtypes = [vp, i64, i64, i32, i32, vp, vp, vp, vp]
        L.dptq_rotate_quant_range.restype = ctypes.c_int
        L.dptq_weight_sums.argtypes = [vp, i64, i64, vp, vp]
        L.dptq_weight_sums.restype = ctypes.c_int
        L.dptq_qlinear_range.argtypes = [vp, vp, vp, i64, i64, i32, vp, vp, vp, i64, vp, vp]
        L.dptq_qlinear_range.restype = ctypes.c_int
        L.dptq_qlinear_fp6.argtypes = [vp, vp, i64, i64, vp, vp, i64, vp, vp, vp]
        L.dptq_qlinear_fp6.restype = ctypes.c_int
        L.dptq_pack_w4_a8.argtypes = [vp, i64, i64, vp, vp]
        L.dptq_pack_w4_a8.restype = ctypes.c_int
        L.dptq_qlinear_a8.argtypes = [vp, vp, i64, i64, vp, vp, i64, vp, i32, vp]
        L.dptq_qlinear_a8.restype = ctypes.c_int
        L.dptq_prepacked_bytes.argtypes = [i64, i64, i32]
        L.dptq_prepacked_bytes.restype = ctypes.c_int64
        L.dptq_prepack_weights.argtypes = [vp, i64, i64, i32, vp, vp]
        L.dptq_prepack_weights.restype = ctypes.c_int
        _lib = L
    return _lib


def _status_string(status):
    try:
        return lib().dptq_status_string(int(status)).decode()
    except Exception:  # pragma: no cover - library unavailable
        return "unknown"


def version():
    return lib().dptq_version()


def _check(status, what):
    if status != 0:
        raise DptqError(status, what)


def _torch():
    import torch
    return torch


def _stream(t):
    torch = _torch()
    return ctypes.c_void_p(torch.cuda.current_stream(t.device).cuda_stream)


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _require(t, name, dtype, shape=None):
    torch = _torch()
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must have dtype {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")


def code_shape(M, K, bits):
    return (M, K // 2) if bits == 4 else (M, K)


def _signs_arg(signs, K, dev):
    if signs is None:
        return None
    _require(signs, "signs", _torch().uint8, ((K + 7) // 8,))
    if signs.device != dev:
        raise ValueError("signs must be on the same device as x")
    return signs


def rotate_quant(x, had_size, bits, codes=None, scales=None, signs=None):
    """Rotate (I (x) H_h) and quantize fp16 rows x [M, K] -> (codes, fp32 scales [M]).
    signs: optional uint8 bitmask [ceil(K/8)] of randomized signs (bit set = -1)."""
    torch = _torch()
    _require(x, "x", torch.float16)
    if x.dim() != 2:
        raise ValueError("x must be 2-D [M, K]")
    M, K = x.shape
    if bits not in (4, 8):
        raise ValueError("bits must be 4 or 8")
    cdt = torch.uint8 if bits == 4 else torch.int8
    if codes is None:
        codes = torch.empty(code_shape(M, K, bits), dtype=cdt, device=x.device)
    _require(codes, "codes", cdt, code_shape(M, K, bits))
    if scales is None:
        scales = torch.empty((M,), dtype=torch.float32, device=x.device)
    _require(scales, "scales", torch.float32, (M,))
    signs = _signs_arg(signs, K, x.device)
    if signs is None:
        _check(lib().dptq_rotate_quant(_ptr(x), M, K, int(had_size), int(bits), _ptr(codes),
                                       _ptr(scales), _stream(x)), "dptq_rotate_quant")
    else:
        _check(lib().dptq_rotate_quant_ex(_ptr(x), M, K, int(had_size), int(bits), _ptr(signs),
                                          LAYOUT_PACKED, _ptr(codes), _ptr(scales), _stream(x)),
               "dptq_rotate_quant_ex")
    return codes, scales


def _gemm_args(codes, bits, w_packed):
    torch = _torch()
    if bits not in (4, 8):
        raise ValueError("bits must be 4 or 8")
    cdt = torch.uint8 if bits == 4 else torch.int8
    _require(codes, "codes", cdt)
    _require(w_packed, "w_packed", torch.uint8)
    M = codes.shape[0]
    K = codes.shape[1] * (2 if bits == 4 else 1)
    N = w_packed.shape[0]
    if w_packed.shape[1] * 2 != K:
        raise ValueError(f"w_packed must be [N, K/2] with K = {K}")
    return M, K, N


def qlinear(codes, a_scales, bits, w_packed, w_scales, y=None, kernel=GEMM_AUTO):
    """y [M, N] fp16 = dequant(codes . w^T) with per-token x per-channel scales.
    kernel: one of the GEMM_* kernels (default: the library's choice)."""
    torch = _torch()
    M, K, N = _gemm_args(codes, bits, w_packed)
    _require(a_scales, "a_scales", torch.float32, (M,))
    _require(w_scales, "w_scales", torch.float32, (N,))
    if y is None:
        y = torch.empty((M, N), dtype=torch.float16, device=codes.device)
    _require(y, "y", torch.float16, (M, N))
    if kernel == GEMM_AUTO:
        _check(lib().dptq_qlinear(_ptr(codes), _ptr(a_scales), M, K, int(bits), _ptr(w_packed),
                                  _ptr(w_scales), N, _ptr(y), _stream(codes)), "dptq_qlinear")
    else:
        _check(lib().dptq_qlinear_kernel(_ptr(codes), _ptr(a_scales), M, K, int(bits),
                                         _ptr(w_packed), _ptr(w_scales), N, _ptr(y), None,
                                         int(kernel), _stream(codes)), "dptq_qlinear_kernel")
    return y


def qlinear_acc(codes, bits, w_packed, acc=None, kernel=GEMM_AUTO):
    """Raw int32 accumulators acc [M, N] = codes . w^T (exact)."""
    torch = _torch()
    M, K, N = _gemm_args(codes, bits, w_packed)
    if acc is None:
        acc = torch.empty((M, N), dtype=torch.int32, device=codes.device)
    _require(acc, "acc", torch.int32, (M, N))
    if kernel == GEMM_AUTO:
        _check(lib().dptq_qlinear_acc(_ptr(codes), M, K, int(bits), _ptr(w_packed), N, _ptr(acc),
                                      _stream(codes)), "dptq_qlinear_acc")
    else:
        _check(lib().dptq_qlinear_kernel(_ptr(codes), None, M, K, int(bits), _ptr(w_packed), None,
                                         N, None, _ptr(acc), int(kernel), _stream(codes)),
               "dptq_qlinear_kernel")
    return acc


def pack_w4_a8(w_packed, out=None):
    """4-bit weights [N, K/2] in the qlinear layout -> the same codes in the
    8-bit activation order (uint8 [N, K/2]) taken by qlinear_a8."""
    torch = _torch()
    _require(w_packed, "w_packed", torch.uint8)
    if w_packed.dim() != 2:
        raise ValueError("w_packed must be 2-D [N, K/2]")
    N, K = w_packed.shape[0], w_packed.shape[1] * 2
    if out is None:
        out = torch.empty_like(w_packed)
    _require(out, "out", torch.uint8, (N, K // 2))
    _check(lib().dptq_pack_w4_a8(_ptr(w_packed), N, K, _ptr(out), _stream(w_packed)),
           "dptq_pack_w4_a8")
    return out


def prepacked_bytes(N, K, layout):
    """Bytes of the prepack_weights output for [N, K] weights in `layout`."""
    n = lib().dptq_prepacked_bytes(int(N), int(K), int(layout))
    if n < 0:
        raise ValueError(f"no layout {layout} for N={N}, K={K} (K must be a multiple of 128; "
                         "the decode layout also needs N % 16 == 0)")
    return n


def prepack_weights(w_packed, layout, out=None):
    """4-bit weights [N, K/2] in the qlinear layout -> the device-native layout
    of their layer's GEMM (WEIGHTS_FP6 for qlinear_fp6, WEIGHTS_A8_ORDER for
    qlinear_a8, WEIGHTS_DECODE for qlinear_decode_native), uint8
    [prepacked_bytes(N, K, layout)]."""
    torch = _torch()
    _require(w_packed, "w_packed", torch.uint8)
    if w_packed.dim() != 2:
        raise ValueError("w_packed must be 2-D [N, K/2]")
    N, K = w_packed.shape[0], w_packed.shape[1] * 2
    n = prepacked_bytes(N, K, layout)
    if out is None:
        out = torch.empty((n,), dtype=torch.uint8, device=w_packed.device)
    _require(out, "out", torch.uint8, (n,))
    _check(lib().dptq_prepack_weights(_ptr(w_packed), N, K, int(layout), _ptr(out),
                                      _stream(w_packed)), "dptq_prepack_weights")
    return out


def _decode_native_args(codes, bits, w_dec, N):
    torch = _torch()
    if bits not in (4, 8):
        raise ValueError("bits must be 4 or 8")
    cdt = torch.uint8 if bits == 4 else torch.int8
    _require(codes, "codes", cdt)
    M = codes.shape[0]
    K = codes.shape[1] * (2 if bits == 4 else 1)
    _require(w_dec, "w_dec", torch.uint8, (prepacked_bytes(N, K, WEIGHTS_DECODE),))
    return M, K


def qlinear_decode_native(codes, a_scales, bits, w_dec, w_scales, y=None):
    """qlinear for M <= 16 tokens on weights from prepack_weights(w, WEIGHTS_DECODE):
    the same y bit for bit.  N is taken from w_scales."""
    torch = _torch()
    N = w_scales.shape[0]
    M, K = _decode_native_args(codes, bits, w_dec, N)
    _require(a_scales, "a_scales", torch.float32, (M,))
    _require(w_scales, "w_scales", torch.float32, (N,))
    if y is None:
        y = torch.empty((M, N), dtype=torch.float16, device=codes.device)
    _require(y, "y", torch.float16, (M, N))
    _check(lib().dptq_qlinear_decode_native(_ptr(codes), _ptr(a_scales), M, K, int(bits), _ptr(w_dec),
                                            _ptr(w_scales), N, _ptr(y), None, _stream(codes)),
           "dptq_qlinear_decode_native")
    return y


def qlinear_decode_native_acc(codes, bits, w_dec, N, acc=None):
    """The int32 accumulators [M, N] of qlinear_decode_native (exact)."""
    torch = _torch()
    M, K = _decode_native_args(codes, bits, w_dec, N)
    if acc is None:
        acc = torch.empty((M, N), dtype=torch.int32, device=codes.device)
    _require(acc, "acc", torch.int32, (M, N))
    _check(lib().dptq_qlinear_decode_native(_ptr(codes), None, M, K, int(bits), _ptr(w_dec), None, N,
                                            None, _ptr(acc), _stream(codes)),
           "dptq_qlinear_decode_native")
    return acc


def qlinear_a8(codes, a_scales, w_a8, w_scales, y=None, kernel=GEMM_AUTO):
    """The W4A8 linear (qlinear with bits = 8) against weights from pack_w4_a8:
    the same y bit for bit."""
    torch = _torch()
    M, K, N = _gemm_args(codes, 8, w_a8)
    _require(a_scales, "a_scales", torch.float32, (M,))
    _require(w_scales, "w_scales", torch.float32, (N,))
    if y is None:
        y = torch.empty((M, N), dtype=torch.float16, device=codes.device)
    _require(y, "y", torch.float16, (M, N))
    _check(lib().dptq_qlinear_a8(_ptr(codes), _ptr(a_scales), M, K, _ptr(w_a8), _ptr(w_scales), N,
                                 _ptr(y), int(kernel), _stream(codes)), "dptq_qlinear_a8")
    return y


def residual_dynamics(x, dx, had_size, bits=4, eps=1e-8, jr=None, snr=None, means=None):
    """One layer's residual-dynamics statistics (Eq. 8-11): per-token Jump Ratio
    and historical SNR (dB) of the updates dx added to the states x (both fp16
    [T, K]), measured through the rotated `bits`-bit quantizer; returns
    (jr float32 [T], snr float32 [T], means float64 [2] = layer JR, layer SNR)."""
    torch = _torch()
    _require(x, "x", torch.float16)
    if x.dim() != 2:
        raise ValueError("x must be 2-D [T, K]")
    T, K = x.shape
    _require(dx, "dx", torch.float16, (T, K))
    if bits not in (4, 8):
        raise ValueError("bits must be 4 or 8")
    if jr is None:
        jr = torch.empty((T,), dtype=torch.float32, device=x.device)
    if snr is None:
        snr = torch.empty((T,), dtype=torch.float32, device=x.device)
    if means is None:
        means = torch.empty((2,), dtype=torch.float64, device=x.device)
    _require(jr, "jr", torch.float32, (T,))
    _require(snr, "snr", torch.float32, (T,))
    _require(means, "means", torch.float64, (2,))
    _check(lib().dptq_residual_dynamics(_ptr(x), _ptr(dx), T, K, int(had_size), int(bits),
                                        float(eps), _ptr(jr), _ptr(snr), _ptr(means),
                                        _stream(x)), "dptq_residual_dynamics")
    return jr, snr, means


def select_layers(jr_layers, snr_layers, tau_jr, tau_snr):
    """Activation bits per layer by the sensitive-layer rule of Eq. 20."""
    jr = [float(v) for v in jr_layers]
    snr = [float(v) for v in snr_layers]
    if len(jr) != len(snr) or not jr:
        raise ValueError("one JR and one SNR value per layer, at least one layer")
    L = len(jr)
    a = (ctypes.c_double * L)(*jr)
    b = (ctypes.c_double * L)(*snr)
    out = (ctypes.c_int32 * L)()
    _check(lib().dptq_select_layers(L, ctypes.cast(a, ctypes.c_void_p), ctypes.cast(b, ctypes.c_void_p),
                                    float(tau_jr), float(tau_snr), ctypes.cast(out, ctypes.c_void_p)),
           "dptq_select_layers")
    return list(out)


def kv_quant(kv, group=128, codes=None, scales=None, mins=None):
    """Group-wise 4-bit quantization of fp16 KV rows kv [T, D] ->
    (codes uint8 [T, D/2], scales float32 [T, D/group], mins float32 [T, D/group])."""
    torch = _torch()
    _require(kv, "kv", torch.float16)
    if kv.dim() != 2:
        raise ValueError("kv must be 2-D [T, D]")
    T, D = kv.shape
    if group <= 0 or D % group:
        raise ValueError("D must be a multiple of group")
    G = D // group
    if codes is None:
        codes = torch.empty((T, D // 2), dtype=torch.uint8, device=kv.device)
    if scales is None:
        scales = torch.empty((T, G), dtype=torch.float32, device=kv.device)
    if mins is None:
        mins = torch.empty((T, G), dtype=torch.float32, device=kv.device)
    _require(codes, "codes", torch.uint8, (T, D // 2))
    _require(scales, "scales", torch.float32, (T, G))
    _require(mins, "mins", torch.float32, (T, G))
    _check(lib().dptq_kv_quant(_ptr(kv), T, D, int(group), _ptr(codes), _ptr(scales), _ptr(mins),
                               _stream(kv)), "dptq_kv_quant")
    return codes, scales, mins


def kv_dequant(codes, scales, mins, group=128, out=None):
    """Reconstruct fp16 [T, D] from kv_quant's output."""
    torch = _torch()
    _require(codes, "codes", torch.uint8)
    if codes.dim() != 2:
        raise ValueError("codes must be 2-D [T, D/2]")
    T, D = codes.shape[0], 2 * codes.shape[1]
    if group <= 0 or D % group:
        raise ValueError("D must be a multiple of group")
    _require(scales, "scales", torch.float32, (T, D // group))
    _require(mins, "mins", torch.float32, (T, D // group))
    if out is None:
        out = torch.empty((T, D), dtype=torch.float16, device=codes.device)
    _require(out, "out", torch.float16, (T, D))
    _check(lib().dptq_kv_dequant(_ptr(codes), _ptr(scales), _ptr(mins), T, D, int(group),
                                 _ptr(out), _stream(codes)), "dptq_kv_dequant")
    return out


def layer_policy(num_layers, mask=None):
    """Activation bits per layer (Eq. 21 default set, or the layers a mask marks)."""
    L = int(num_layers)
    out = (ctypes.c_int32 * max(L, 1))()
    if mask is None:
        mptr = ctypes.c_void_p(0)
    else:
        m = [1 if v else 0 for v in mask]
        if len(m) != L:
            raise ValueError("mask length must equal num_layers")
        buf = (ctypes.c_uint8 * max(L, 1))(*m)
        mptr = ctypes.cast(buf, ctypes.c_void_p)
    _check(lib().dptq_layer_policy(L, mptr, ctypes.cast(out, ctypes.c_void_p)),
           "dptq_layer_policy")
    return [int(v) for v in out[:L]]


def prepare_weights(w, had_size, w_packed=None, w_scales=None, signs=None):
    """Offline: rotate, quantize to 4 bits per output channel and pack fp32 w [N, K].
    signs: the randomized-sign bitmask of the activations' rotation, if any."""
    torch = _torch()
    _require(w, "w", torch.float32)
    if w.dim() != 2:
        raise ValueError("w must be 2-D [N, K]")
    N, K = w.shape
    if w_packed is None:
        w_packed = torch.empty((N, K // 2), dtype=torch.uint8, device=w.device)
    _require(w_packed, "w_packed", torch.uint8, (N, K // 2))
    if w_scales is None:
        w_scales = torch.empty((N,), dtype=torch.float32, device=w.device)
    _require(w_scales, "w_scales", torch.float32, (N,))
    signs = _signs_arg(signs, K, w.device)
    if signs is None:
        _check(lib().dptq_prepare_weights(_ptr(w), N, K, int(had_size), _ptr(w_packed),
                                          _ptr(w_scales), _stream(w)), "dptq_prepare_weights")
    else:
        _check(lib().dptq_prepare_weights_signed(_ptr(w), N, K, int(had_size), _ptr(signs),
                                                 _ptr(w_packed), _ptr(w_scales), _stream(w)),
               "dptq_prepare_weights_signed")
    return w_packed, w_scales


def fp6_bytes(rows, K):
    """Bytes of the FP6 block layout of a [rows, K] matrix of 4-bit codes."""
    n = lib().dptq_fp6_bytes(int(rows), int(K))
    if n < 0:
        raise ValueError(f"no FP6 layout for rows={rows}, K={K} (K must be a multiple of 128)")
    return n


def pack_fp6(codes, out=None):
    """Packed 4-bit codes [R, K/2] (activations or weights) -> FP6 block layout
    (uint8 [fp6_bytes(R, K)]), the operand format of qlinear_fp6."""
    torch = _torch()
    _require(codes, "codes", torch.uint8)
    if codes.dim() != 2:
        raise ValueError("codes must be 2-D [R, K/2]")
    R, K = codes.shape[0], codes.shape[1] * 2
    n = fp6_bytes(R, K)
    if out is None:
        out = torch.empty((n,), dtype=torch.uint8, device=codes.device)
    _require(out, "out", torch.uint8, (n,))
    _check(lib().dptq_pack_fp6(_ptr(codes), R, K, _ptr(out), _stream(codes)), "dptq_pack_fp6")
    return out


def rotate_quant_fp6(x, had_size, out=None, scales=None, signs=None):
    """Rotate and quantize fp16 rows x [M, K] at 4 bits, codes written in the
    FP6 block layout -> (uint8 [fp6_bytes(M, K)], fp32 scales [M])."""
    torch = _torch()
    _require(x, "x", torch.float16)
    if x.dim() != 2:
        raise ValueError("x must be 2-D [M, K]")
    M, K = x.shape
    n = fp6_bytes(M, K)
    if out is None:
        out = torch.empty((n,), dtype=torch.uint8, device=x.device)
    _require(out, "out", torch.uint8, (n,))
    if scales is None:
        scales = torch.empty((M,), dtype=torch.float32, device=x.device)
    _require(scales, "scales", torch.float32, (M,))
    signs = _signs_arg(signs, K, x.device)
    if signs is None:
        _check(lib().dptq_rotate_quant_fp6(_ptr(x), M, K, int(had_size), _ptr(out), _ptr(scales),
                                           _stream(x)), "dptq_rotate_quant_fp6")
    else:
        _check(lib().dptq_rotate_quant_ex(_ptr(x), M, K, int(had_size), 4, _ptr(signs), LAYOUT_FP6,
                                          _ptr(out), _ptr(scales), _stream(x)),
               "dptq_rotate_quant_ex")
    return out, scales


def _fp6_args(a6, w6, M, K, N):
    torch = _torch()
    _require(a6, "a_fp6", torch.uint8, (fp6_bytes(M, K),))
    _require(w6, "w_fp6", torch.uint8, (fp6_bytes(N, K),))


def qlinear_fp6(a6, a_scales, w6, w_scales, M, K, N, y=None):
    """y [M, N] fp16 = dequant(a . w^T) for 4-bit codes in the FP6 block layout
    (the same bits as qlinear at 4 bits)."""
    torch = _torch()
    _fp6_args(a6, w6, M, K, N)
    _require(a_scales, "a_scales", torch.float32, (M,))
    _require(w_scales, "w_scales", torch.float32, (N,))
    if y is None:
        y = torch.empty((M, N), dtype=torch.float16, device=a6.device)
    _require(y, "y", torch.float16, (M, N))
    _check(lib().dptq_qlinear_fp6(_ptr(a6), _ptr(a_scales), M, K, _ptr(w6), _ptr(w_scales), N,
                                  _ptr(y), None, _stream(a6)), "dptq_qlinear_fp6")
    return y


def qlinear_fp6_acc(a6, w6, M, K, N, acc=None):
    """Raw int32 accumulators [M, N] of the FP6 GEMM (exact)."""
    torch = _torch()
    _fp6_args(a6, w6, M, K, N)
    if acc is None:
        acc = torch.empty((M, N), dtype=torch.int32, device=a6.device)
    _require(acc, "acc", torch.int32, (M, N))
    _check(lib().dptq_qlinear_fp6(_ptr(a6), None, M, K, _ptr(w6), None, N, None, _ptr(acc),
                                  _stream(a6)), "dptq_qlinear_fp6")
    return acc


DECODE_AUTO, DECODE_ONE_LAUNCH, DECODE_TWO_LAUNCHES = 0, 1, 2


def qlinear_decode_fused(x, had_size, bits, w_packed, w_scales, y=None, codes=None,
                         scales=None, mode=DECODE_AUTO):
    """Decode-shape (M <= 16) rotate + quantize + GEMM from fp16 x: one launch
    or two (mode, DECODE_AUTO picks).  Returns (y [M, N] fp16, codes, scales)."""
    torch = _torch()
    _require(x, "x", torch.float16)
    M, K = x.shape
    N = w_packed.shape[0]
    _require(w_packed, "w_packed", torch.uint8, (N, K // 2))
    _require(w_scales, "w_scales", torch.float32, (N,))
    cdt = torch.uint8 if bits == 4 else torch.int8
    if y is None:
        y = torch.empty((M, N), dtype=torch.float16, device=x.device)
    if codes is None:
        codes = torch.empty(code_shape(M, K, bits), dtype=cdt, device=x.device)
    if scales is None:
        scales = torch.empty((M,), dtype=torch.float32, device=x.device)
    _require(y, "y", torch.float16, (M, N))
    _require(codes, "codes", cdt, code_shape(M, K, bits))
    _require(scales, "scales", torch.float32, (M,))
    _check(lib().dptq_qlinear_decode_fused(_ptr(x), M, K, int(had_size), int(bits), _ptr(w_packed),
                                           _ptr(w_scales), N, _ptr(y), _ptr(codes), _ptr(scales),
                                           int(mode), _stream(x)), "dptq_qlinear_decode_fused")
    return y, codes, scales


def rotate_quant_range(x, had_size, bits, codes=None, scales=None, zeros=None):
    """Rotation + per-token range quantization with an integer zero point.
    Returns (codes, scales fp32 [M], zeros int32 [M])."""
    torch = _torch()
    _require(x, "x", torch.float16)
    M, K = x.shape
    cdt = torch.uint8 if bits == 4 else torch.int8
    if codes is None:
        codes = torch.empty(code_shape(M, K, bits), dtype=cdt, device=x.device)
    if scales is None:
        scales = torch.empty((M,), dtype=torch.float32, device=x.device)
    if zeros is None:
        zeros = torch.empty((M,), dtype=torch.int32, device=x.device)
    _require(codes, "codes", cdt, code_shape(M, K, bits))
    _require(scales, "scales", torch.float32, (M,))
    _require(zeros, "zeros", torch.int32, (M,))
    _check(lib().dptq_rotate_quant_range(_ptr(x), M, K, int(had_size), int(bits), _ptr(codes),
                                         _ptr(scales), _ptr(zeros), _stream(x)),
           "dptq_rotate_quant_range")
    return codes, scales, zeros


def weight_sums(w_packed, out=None):
    """int32 [N]: the sum of each packed 4-bit weight row's codes."""
    torch = _torch()
    _require(w_packed, "w_packed", torch.uint8)
    N, K2 = w_packed.shape
    if out is None:
        out = torch.empty((N,), dtype=torch.int32, device=w_packed.device)
    _require(out, "out", torch.int32, (N,))
    _check(lib().dptq_weight_sums(_ptr(w_packed), N, 2 * K2, _ptr(out), _stream(w_packed)),
           "dptq_weight_sums")
    return out


def qlinear_range(codes, scales, zeros, bits, w_packed, w_scales, w_sums, y=None):
    """Quantized linear on range-quantized activations (zero-point corrected
    in the GEMM epilogue).  Returns y [M, N] fp16."""
    torch = _torch()
    M = scales.shape[0]
    N, K2 = w_packed.shape
    K = 2 * K2
    _require(codes, "codes", torch.uint8 if bits == 4 else torch.int8, code_shape(M, K, bits))
    _require(scales, "scales", torch.float32, (M,))
    _require(zeros, "zeros", torch.int32, (M,))
    _require(w_packed, "w_packed", torch.uint8, (N, K2))
    _require(w_scales, "w_scales", torch.float32, (N,))
    _require(w_sums, "w_sums", torch.int32, (N,))
    if y is None:
        y = torch.empty((M, N), dtype=torch.float16, device=codes.device)
    _require(y, "y", torch.float16, (M, N))
    _check(lib().dptq_qlinear_range(_ptr(codes), _ptr(scales), _ptr(zeros), M, K, int(bits),
                                    _ptr(w_packed), _ptr(w_scales), _ptr(w_sums), N, _ptr(y),
                                    _stream(codes)), "dptq_qlinear_range")
    return y
