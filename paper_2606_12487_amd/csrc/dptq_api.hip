// C ABI: argument checks, then dispatch to the gfx950 kernels.
#include "dptq.h"
#include "internal.h"

namespace {

using dptq::HadSplit;

constexpr int kVersion = 100;  // 0.1.0

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// h = 2^j or 28 * 2^j with h <= 32768.
bool split_had(int64_t h, HadSplit* out) {
  if (h < 1 || h > 32768) return false;
  if ((h & (h - 1)) == 0) {
    int j = 0;
    while ((int64_t{1} << j) < h) ++j;
    *out = HadSplit{1, j};
    return true;
  }
  if (h % 28 == 0) {
    const int64_t p = h / 28;
    if ((p & (p - 1)) == 0) {
      int j = 0;
      while ((int64_t{1} << j) < p) ++j;
      *out = HadSplit{28, j};
      return true;
    }
  }
  return false;
}

int check_rotation_shape(int64_t M, int64_t K, int32_t had_size, HadSplit* hs) {
  if (M < 0 || K < 1) return DPTQ_ERR_INVALID_ARG;
  if (!split_had(had_size, hs)) return DPTQ_ERR_INVALID_ARG;
  if (K % had_size != 0 || K % 8 != 0) return DPTQ_ERR_INVALID_ARG;
  if (K > dptq::kMaxRotateK) return DPTQ_ERR_UNSUPPORTED;
  if (M > 0x7FFFFFFF) return DPTQ_ERR_UNSUPPORTED;
  return DPTQ_OK;
}

int check_gemm_shape(int64_t M, int64_t K, int32_t bits, int64_t N) {
  if (M < 0 || K < 1 || N < 1) return DPTQ_ERR_INVALID_ARG;
  if (bits != 4 && bits != 8) return DPTQ_ERR_INVALID_ARG;
  if (K % 128 != 0 || K > DPTQ_MAX_K) return DPTQ_ERR_UNSUPPORTED;
  if (N % 16 != 0 || N > 0x7FFFFFF0) return DPTQ_ERR_UNSUPPORTED;
  if (M > 0x7FFFFFFF) return DPTQ_ERR_UNSUPPORTED;
  if ((M > 16) && ((M + 127) / 128) * ((N + 255) / 256) > 0x7FFFFFFF) return DPTQ_ERR_UNSUPPORTED;
  return DPTQ_OK;
}

int from_hip(hipError_t e) { return e == hipSuccess ? DPTQ_OK : DPTQ_ERR_HIP; }

bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

// KV-cache shapes: group a power of two in [16, 512] dividing D; T * D < 2^40.
int check_kv_shape(int64_t T, int64_t D, int32_t group) {
  if (T < 0 || D < 1) return DPTQ_ERR_INVALID_ARG;
  if (group < 16 || group > 512 || (group & (group - 1)) != 0) return DPTQ_ERR_INVALID_ARG;
  if (D % group != 0) return DPTQ_ERR_INVALID_ARG;
  if (D > (int64_t{1} << 31) || T > (int64_t{1} << 40) / D) return DPTQ_ERR_UNSUPPORTED;
  return DPTQ_OK;
}

}  // namespace

extern "C" {

const char* dptq_status_string(int status) {
  switch (status) {
    case DPTQ_OK: return "ok";
    case DPTQ_ERR_INVALID_ARG: return "invalid argument";
    case DPTQ_ERR_UNSUPPORTED: return "unsupported shape or size";
    case DPTQ_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

int dptq_version(void) { return kVersion; }

int dptq_rotate_quant(const void* x, int64_t M, int64_t K, int32_t had_size, int32_t bits,
                      void* codes, float* a_scales, void* stream) {
  HadSplit hs{};
  int st = check_rotation_shape(M, K, had_size, &hs);
  if (st != DPTQ_OK) return st;
  if (bits != 4 && bits != 8) return DPTQ_ERR_INVALID_ARG;
  if (M == 0) return DPTQ_OK;
  if (!x || !codes || !a_scales) return DPTQ_ERR_INVALID_ARG;
  if (!aligned16(x) || !aligned16(codes) || !aligned16(a_scales)) return DPTQ_ERR_INVALID_ARG;
  return from_hip(dptq::launch_rotate_quant_f16(x, M, (int)K, hs, bits, codes, a_scales,
                                                static_cast<hipStream_t>(stream)));
}

int dptq_qlinear(const void* codes, const float* a_scales, int64_t M, int64_t K, int32_t bits,
                 const uint8_t* w_packed, const float* w_scales, int64_t N, void* y,
                 void* stream) {
  int st = check_gemm_shape(M, K, bits, N);
  if (st != DPTQ_OK) return st;
  if (M == 0) return DPTQ_OK;
  if (!codes || !a_scales || !w_packed || !w_scales || !y) return DPTQ_ERR_INVALID_ARG;
  if (!aligned16(codes) || !aligned16(a_scales) || !aligned16(w_packed) ||
      !aligned16(w_scales) || !aligned16(y))
    return DPTQ_ERR_INVALID_ARG;
  return from_hip(dptq::launch_qlinear(codes, a_scales, M, (int)K, bits, w_packed, w_scales, N,
                                       y, nullptr, dptq::kGemmAuto, static_cast<hipStream_t>(stream)));
}

int dptq_qlinear_acc(const void* codes, int64_t M, int64_t K, int32_t bits,
                     const uint8_t* w_packed, int64_t N, int32_t* acc, void* stream) {
  int st = check_gemm_shape(M, K, bits, N);
  if (st != DPTQ_OK) return st;
  if (M == 0) return DPTQ_OK;
  if (!codes || !w_packed || !acc) return DPTQ_ERR_INVALID_ARG;
  if (!aligned16(codes) || !aligned16(w_packed) || !aligned16(acc)) return DPTQ_ERR_INVALID_ARG;
  return from_hip(dptq::launch_qlinear(codes, nullptr, M, (int)K, bits, w_packed, nullptr, N,
                                       nullptr, acc, dptq::kGemmAuto, static_cast<hipStream_t>(stream)));
}

int dptq_residual_dynamics(const void* x, const void* dx, int64_t T, int64_t K, int32_t had_size,
                           int32_t bits, float eps, float* jr, float* snr, double* layer_means,
                           void* stream) {
  HadSplit hs{};
  int st = check_rotation_shape(T, K, had_size, &hs);
  if (st != DPTQ_OK) return st;
  if (bits != 4 && bits != 8) return DPTQ_ERR_INVALID_ARG;
  if (!(eps >= 0.0f) || eps > 3.0e38f) return DPTQ_ERR_INVALID_ARG;   // also rejects NaN
  if (T == 0) return DPTQ_OK;
  if (!x || !dx || !jr || !snr) return DPTQ_ERR_INVALID_ARG;
  if (!aligned16(x) || !aligned16(dx)) return DPTQ_ERR_INVALID_ARG;
  if ((reinterpret_cast<uintptr_t>(jr) & 3u) || (reinterpret_cast<uintptr_t>(snr) & 3u) ||
      (reinterpret_cast<uintptr_t>(layer_means) & 7u))
    return DPTQ_ERR_INVALID_ARG;
  return from_hip(dptq::launch_residual_stats(x, dx, T, (int)K, hs, bits, eps, jr, snr,
                                              layer_means, static_cast<hipStream_t>(stream)));
}

int dptq_select_layers(int32_t num_layers, const double* jr, const double* snr, double tau_jr,
                       double tau_snr, int32_t* bits_out) {
  if (num_layers < 1 || !jr || !snr || !bits_out) return DPTQ_ERR_INVALID_ARG;
  for (int32_t l = 0; l < num_layers; ++l)
    bits_out[l] = (jr[l] > tau_jr && snr[l] < tau_snr) ? 8 : 4;
  return DPTQ_OK;
}

int dptq_kv_quant(const void* kv, int64_t T, int64_t D, int32_t group, uint8_t* codes,
                  float* scales, float* mins, void* stream) {
  const int st = check_kv_shape(T, D, group);
  if (st != DPTQ_OK) return st;
  if (T == 0) return DPTQ_OK;
  if (!kv || !codes || !scales || !mins) return DPTQ_ERR_INVALID_ARG;
  if (!aligned16(kv) || !aligned4(codes) || !aligned4(scales) || !aligned4(mins))
    return DPTQ_ERR_INVALID_ARG;
  return from_hip(dptq::launch_kv_quant(kv, T, D, group, codes, scales, mins,
                                        static_cast<hipStream_t>(stream)));
}

int dptq_kv_dequant(const uint8_t* codes, const float* scales, const float* mins, int64_t T,
                    int64_t D, int32_t group, void* kv_out, void* stream) {
  const int st = check_kv_shape(T, D, group);
  if (st != DPTQ_OK) return st;
  if (T == 0) return DPTQ_OK;
  if (!kv_out || !codes || !scales || !mins) return DPTQ_ERR_INVALID_ARG;
  if (!aligned16(kv_out) || !aligned4(codes) || !aligned4(scales) || !aligned4(mins))
    return DPTQ_ERR_INVALID_ARG;
  return from_hip(dptq::launch_kv_dequant(codes, scales, mins, T, D, group, kv_out,
                                          static_cast<hipStream_t>(stream)));
}

int dptq_qlinear_kernel(const void* codes, const float* a_scales, int64_t M, int64_t K,
                        int32_t bits, const uint8_t* w_packed, const float* w_scales,
                        int64_t N, void* y, int32_t* acc, int32_t kernel, void* stream) {
  int st = check_gemm_shape(M, K, bits, N);
  if (st != DPTQ_OK) return st;
  if (kernel < DPTQ_GEMM_AUTO || kernel > DPTQ_GEMM_TILE_192X256) return DPTQ_ERR_INVALID_ARG;
  if ((y == nullptr) == (acc == nullptr)) return DPTQ_ERR_INVALID_ARG;
  if (!dptq::gemm_kernel_fits(kernel, M, N, (int)K, bits)) return DPTQ_ERR_UNSUPPORTED;
  if (M == 0) return DPTQ_OK;
  if (!codes || !w_packed) return DPTQ_ERR_INVALID_ARG;
  if (!aligned16(codes) || !aligned16(w_packed)) return DPTQ_ERR_INVALID_ARG;
  if (y) {
    if (!a_scales || !w_scales) return DPTQ_ERR_INVALID_ARG;
    if (!aligned16(a_scales) || !aligned16(w_scales) || !aligned16(y)) return DPTQ_ERR_INVALID_ARG;
    return from_hip(dptq::launch_qlinear(codes, a_scales, M, (int)K, bits, w_packed, w_scales, N,
                                         y, nullptr, kernel, static_cast<hipStream_t>(stream)));
  }
  if (!aligned16(acc)) return DPTQ_ERR_INVALID_ARG;
  return from_hip(dptq::launch_qlinear(codes, nullptr, M, (int)K, bits, w_packed, nullptr, N,
                                       nullptr, acc, kernel, static_cast<hipStream_t>(stream)));
}

int dptq_pack_w4_a8(const uint8_t* w_packed, int64_t N, int64_t K, uint8_t* out, void* stream) {
  if (N < 0 || K < 1) return DPTQ_ERR_INVALID_ARG;
  if (K % 128 != 0 || K > DPTQ_MAX_K || N > 0x7FFFFFF0) return DPTQ_ERR_UNSUPPORTED;
  if (N == 0) return DPTQ_OK;
  if (!w_packed || !out) return DPTQ_ERR_INVALID_ARG;
  if (!aligned16(w_packed) || !aligned16(out)) return DPTQ_ERR_INVALID_ARG;
  return from_hip(dptq::launch_pack_w4_a8(w_packed, N, (int)K, out, static_cast<hipStream_t>(stream)));
}

int dptq_qlinear_a8(const void* codes, const float* a_scales, int64_t M, int64_t K,
                    const uint8_t* w_a8, const float* w_scales, int64_t N, void* y, int32_t kernel,
                    void* stream) {
  int st = check_gemm_shape(M, K, 8, N);
  if (st != DPTQ_OK) return st;
  if (kernel < DPTQ_GEMM_AUTO || kernel > DPTQ_GEMM_TILE_192X256) return DPTQ_ERR_INVALID_ARG;
  if (!dptq::gemm_kernel_fits(kernel, M, N, (int)K, 8)) return DPTQ_ERR_UNSUPPORTED;
  if (M == 0) return DPTQ_OK;
  if (!codes || !a_scales || !w_a8 || !w_scales || !y) return DPTQ_ERR_INVALID_ARG;
  if (!aligned16(codes) || !aligned16(a_scales) || !aligned16(w_a8) || !aligned16(w_scales) ||
      !aligned16(y))
    return DPTQ_ERR_INVALID_ARG;
  return from_hip(dptq::launch_qlinear_a8(codes, a_scales, M, (int)K, w_a8, w_scales, N, y, kernel,
                                          static_cast<hipStream_t>(stream)));
}

int64_t dptq_fp6_bytes(int64_t rows, int64_t K) {
  if (rows < 0 || K < 128 || K % 128 != 0 || K > DPTQ_MAX_K || rows > 0x7FFFFFFF) return -1;
  return dptq::fp6_bytes(rows, K);
}

int dptq_pack_fp6(const uint8_t* codes, int64_t rows, int64_t K, uint8_t* out, void* stream) {
  if (rows < 0 || K < 1) return DPTQ_ERR_INVALID_ARG;
  if (K % 128 != 0 || K > DPTQ_MAX_K || rows > 0x7FFFFFFF) return DPTQ_ERR_UNSUPPORTED;
  if (rows == 0) return DPTQ_OK;
  if (!codes || !out) return DPTQ_ERR_INVALID_ARG;
  if (!aligned16(codes) || !aligned16(out)) return DPTQ_ERR_INVALID_ARG;
  return from_hip(dptq::launch_pack_fp6(codes, rows, (int)K, out, static_cast<hipStream_t>(stream)));
}

int64_t dptq_prepacked_bytes(int64_t N, int64_t K, int32_t layout) {
  if (N < 0 || K < 128 || K % 128 != 0 || K > DPTQ_MAX_K) return -1;
  if (layout == DPTQ_WEIGHTS_FP6) return dptq_fp6_bytes(N, K);
  if (layout == DPTQ_WEIGHTS_A8_ORDER) return N > 0x7FFFFFF0 ? -1 : N * (K / 2);
  if (layout == DPTQ_WEIGHTS_DECODE) return (N > 0x7FFFFFF0 || N % 16 != 0) ? -1 : N * (K / 2);
  return -1;
}

int dptq_prepack_weights(const uint8_t* w_packed, int64_t N, int64_t K, int32_t layout,
                         uint8_t* w_native, void* stream) {
  if (layout == DPTQ_WEIGHTS_FP6) return dptq_pack_fp6(w_packed, N, K, w_native, stream);
  if (layout == DPTQ_WEIGHTS_A8_ORDER) return dptq_pack_w4_a8(w_packed, N, K, w_native, stream);
  if (layout == DPTQ_WEIGHTS_DECODE) {
    if (N < 0 || K < 1) return DPTQ_ERR_INVALID_ARG;
    if (K % 128 != 0 || K > DPTQ_MAX_K || N > 0x7FFFFFF0 || N % 16 != 0) return DPTQ_ERR_UNSUPPORTED;
    if (N == 0) return DPTQ_OK;
    if (!w_packed || !w_native) return DPTQ_ERR_INVALID_ARG;
    if (!aligned16(w_packed) || !aligned16(w_native)) return DPTQ_ERR_INVALID_ARG;
    return from_hip(dptq::launch_pack_decode(w_packed, N, (int)K, w_native,
                                             static_cast<hipStream_t>(stream)));
  }
  return DPTQ_ERR_INVALID_ARG;
}

int dptq_qlinear_decode_native(const void* codes, const float* a_scales, int64_t M, int64_t K,
                               int32_t bits, const uint8_t* w_dec, const float* w_scales,
                               int64_t N, void* y, int32_t* acc, void* stream) {
  int st = check_gemm_shape(M, K, bits, N);
  if (st != DPTQ_OK) return st;
  if (M > 16) return DPTQ_ERR_UNSUPPORTED;
  if ((y == nullptr) == (acc == nullptr)) return DPTQ_ERR_INVALID_ARG;
  if (M == 0) return DPTQ_OK;
  if (!codes || !w_dec) return DPTQ_ERR_INVALID_ARG;
  if (!aligned16(codes) || !aligned16(w_dec)) return DPTQ_ERR_INVALID_ARG;
  if (y) {
    if (!a_scales || !w_scales) return DPTQ_ERR_INVALID_ARG;
    if (!aligned16(a_scales) || !aligned16(w_scales) || !aligned16(y)) return DPTQ_ERR_INVALID_ARG;
  } else if (!aligned16(acc)) {
    return DPTQ_ERR_INVALID_ARG;
  }
  return from_hip(dptq::launch_qlinear_decode_native(codes, y ? a_scales : nullptr, M, (int)K, bits,
                                                     w_dec, y ? w_scales : nullptr, N, y,
                                                     y ? nullptr : acc,
                                                     static_cast<hipStream_t>(stream)));
}

int dptq_rotate_quant_fp6(const void* x, int64_t M, int64_t K, int32_t had_size, uint8_t* out,
                          float* a_scales, void* stream) {
  HadSplit hs{};
  int st = check_rotation_shape(M, K, had_size, &hs);
  if (st != DPTQ_OK) return st;
  if (K % 128 != 0) return DPTQ_ERR_UNSUPPORTED;
  if (M == 0) return DPTQ_OK;
  if (!x || !out || !a_scales) return DPTQ_ERR_INVALID_ARG;
  if (!aligned16(x) || !aligned16(out) || !aligned16(a_scales)) return DPTQ_ERR_INVALID_ARG;
  return from_hip(dptq::launch_rotate_quant_fp6(x, M, (int)K, hs, out, a_scales,
                                                static_cast<hipStream_t>(stream)));
}

int dptq_rotate_quant_ex(const void* x, int64_t M, int64_t K, int32_t had_size, int32_t bits,
                         const uint8_t* signs, int32_t layout, void* out, float* a_scales,
                         void* stream) {
  HadSplit hs{};
  int st = check_rotation_shape(M, K, had_size, &hs);
  if (st != DPTQ_OK) return st;
  if (bits != 4 && bits != 8) return DPTQ_ERR_INVALID_ARG;
  if (layout != DPTQ_LAYOUT_PACKED && layout != DPTQ_LAYOUT_FP6) return DPTQ_ERR_INVALID_ARG;
  if (layout == DPTQ_LAYOUT_FP6 && bits != 4) return DPTQ_ERR_INVALID_ARG;
  if (layout == DPTQ_LAYOUT_FP6 && K % 128 != 0) return DPTQ_ERR_UNSUPPORTED;
  if (M == 0) return DPTQ_OK;
  if (!x || !out || !a_scales) return DPTQ_ERR_INVALID_ARG;
  if (!aligned16(x) || !aligned16(out) || !aligned16(a_scales)) return DPTQ_ERR_INVALID_ARG;
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (layout == DPTQ_LAYOUT_FP6)
    return from_hip(dptq::launch_rotate_quant_fp6(x, M, (int)K, hs, static_cast<uint8_t*>(out),
                                                  a_scales, s, signs));
  return from_hip(dptq::launch_rotate_quant_signed(x, M, (int)K, hs, bits, signs, out, a_scales, s));
}

int dptq_prepare_weights_signed(const float* w, int64_t N, int64_t K, int32_t had_size,
                                const uint8_t* signs, uint8_t* w_packed, float* w_scales,
                                void* stream) {
  HadSplit hs{};
  int st = check_rotation_shape(N, K, had_size, &hs);
  if (st != DPTQ_OK) return st;
  if (N == 0) return DPTQ_OK;
  if (!w || !w_packed || !w_scales) return DPTQ_ERR_INVALID_ARG;
  if (!aligned16(w) || !aligned16(w_packed) || !aligned16(w_scales)) return DPTQ_ERR_INVALID_ARG;
  return from_hip(dptq::launch_prepare_weights(w, N, (int)K, hs, w_packed, w_scales,
                                               static_cast<hipStream_t>(stream), signs));
}

int dptq_qlinear_fp6(const uint8_t* a_fp6, const float* a_scales, int64_t M, int64_t K,
                     const uint8_t* w_fp6, const float* w_scales, int64_t N, void* y,
                     int32_t* acc, void* stream) {
  int st = check_gemm_shape(M, K, 4, N);
  if (st != DPTQ_OK) return st;
  if ((y == nullptr) == (acc == nullptr)) return DPTQ_ERR_INVALID_ARG;
  if (((M + 255) / 256) * ((N + 191) / 192) > 0x7FFFFFFF) return DPTQ_ERR_UNSUPPORTED;
  if (M == 0) return DPTQ_OK;
  if (!a_fp6 || !w_fp6) return DPTQ_ERR_INVALID_ARG;
  if (!aligned16(a_fp6) || !aligned16(w_fp6)) return DPTQ_ERR_INVALID_ARG;
  if (y) {
    if (!a_scales || !w_scales) return DPTQ_ERR_INVALID_ARG;
    if (!aligned4(a_scales) || !aligned4(w_scales) || !aligned16(y)) return DPTQ_ERR_INVALID_ARG;
  } else if (!aligned16(acc)) {
    return DPTQ_ERR_INVALID_ARG;
  }
  return from_hip(dptq::launch_qlinear_fp6(a_fp6, y ? a_scales : nullptr, M, (int)K, w_fp6,
                                           y ? w_scales : nullptr, N, y, y ? nullptr : acc,
                                           static_cast<hipStream_t>(stream)));
}

int dptq_qlinear_decode_fused(const void* x, int64_t M, int64_t K, int32_t had_size,
                              int32_t bits, const uint8_t* w_packed, const float* w_scales,
                              int64_t N, void* y, void* codes, float* a_scales, int32_t mode,
                              void* stream) {
  HadSplit hs{};
  int st = check_rotation_shape(M, K, had_size, &hs);
  if (st != DPTQ_OK) return st;
  st = check_gemm_shape(M, K, bits, N);
  if (st != DPTQ_OK) return st;
  if (mode < DPTQ_DECODE_AUTO || mode > DPTQ_DECODE_TWO_LAUNCHES) return DPTQ_ERR_INVALID_ARG;
  if (M > 16) return DPTQ_ERR_UNSUPPORTED;
  if (mode == DPTQ_DECODE_ONE_LAUNCH && dptq::decode_fused_lds(M, (int)K, hs, bits) > dptq::kFusedLdsMax)
    return DPTQ_ERR_UNSUPPORTED;
  if (M == 0) return DPTQ_OK;
  if (!x || !w_packed || !w_scales || !y || !codes || !a_scales) return DPTQ_ERR_INVALID_ARG;
  if (!aligned16(x) || !aligned16(w_packed) || !aligned16(w_scales) || !aligned16(y) ||
      !aligned16(codes) || !aligned16(a_scales))
    return DPTQ_ERR_INVALID_ARG;
  return from_hip(dptq::launch_decode_fused(x, M, (int)K, hs, bits, w_packed, w_scales, N, y, codes,
                                            a_scales, mode, static_cast<hipStream_t>(stream)));
}

int dptq_rotate_quant_range(const void* x, int64_t M, int64_t K, int32_t had_size, int32_t bits,
                            void* codes, float* a_scales, int32_t* a_zeros, void* stream) {
  HadSplit hs{};
  int st = check_rotation_shape(M, K, had_size, &hs);
  if (st != DPTQ_OK) return st;
  if (bits != 4 && bits != 8) return DPTQ_ERR_INVALID_ARG;
  if (K % 128 != 0) return DPTQ_ERR_UNSUPPORTED;
  if (M == 0) return DPTQ_OK;
  if (!x || !codes || !a_scales || !a_zeros) return DPTQ_ERR_INVALID_ARG;
  if (!aligned16(x) || !aligned16(codes) || !aligned4(a_scales) || !aligned4(a_zeros))
    return DPTQ_ERR_INVALID_ARG;
  return from_hip(dptq::launch_rotate_quant_range(x, M, (int)K, hs, bits, codes, a_scales, a_zeros,
                                                  static_cast<hipStream_t>(stream)));
}

int dptq_weight_sums(const uint8_t* w_packed, int64_t N, int64_t K, int32_t* w_sums, void* stream) {
  if (N < 0 || K < 1) return DPTQ_ERR_INVALID_ARG;
  if (K % 32 != 0 || K > DPTQ_MAX_K || N > 0x7FFFFFF0) return DPTQ_ERR_UNSUPPORTED;
  if (N == 0) return DPTQ_OK;
  if (!w_packed || !w_sums || !aligned16(w_packed) || !aligned4(w_sums)) return DPTQ_ERR_INVALID_ARG;
  return from_hip(dptq::launch_weight_sums(w_packed, N, (int)K, w_sums,
                                           static_cast<hipStream_t>(stream)));
}

int dptq_qlinear_range(const void* codes, const float* a_scales, const int32_t* a_zeros, int64_t M,
                       int64_t K, int32_t bits, const uint8_t* w_packed, const float* w_scales,
                       const int32_t* w_sums, int64_t N, void* y, void* stream) {
  int st = check_gemm_shape(M, K, bits, N);
  if (st != DPTQ_OK) return st;
  if (M == 0) return DPTQ_OK;
  if (!codes || !a_scales || !a_zeros || !w_packed || !w_scales || !w_sums || !y)
    return DPTQ_ERR_INVALID_ARG;
  if (!aligned16(codes) || !aligned16(a_scales) || !aligned4(a_zeros) || !aligned16(w_packed) ||
      !aligned16(w_scales) || !aligned16(w_sums) || !aligned16(y))
    return DPTQ_ERR_INVALID_ARG;
  return from_hip(dptq::launch_qlinear_zp(codes, a_scales, a_zeros, M, (int)K, bits, w_packed, w_scales,
                                          w_sums, N, y, static_cast<hipStream_t>(stream)));
}

int dptq_layer_policy(int32_t num_layers, const uint8_t* mask, int32_t* bits_out) {
  if (num_layers < 1 || !bits_out) return DPTQ_ERR_INVALID_ARG;
  for (int32_t l = 0; l < num_layers; ++l) {
    bool sensitive;
    if (mask) {
      sensitive = mask[l] != 0;
    } else {
      // Eq. 21: S = {1, 2, 3, L} counted from 1, i.e. {0, 1, 2, L-1}.
      sensitive = l <= 2 || l == num_layers - 1;
    }
    bits_out[l] = sensitive ? 8 : 4;
  }
  return DPTQ_OK;
}

int dptq_prepare_weights(const float* w, int64_t N, int64_t K, int32_t had_size,
                         uint8_t* w_packed, float* w_scales, void* stream) {
  HadSplit hs{};
  int st = check_rotation_shape(N, K, had_size, &hs);
  if (st != DPTQ_OK) return st;
  if (N == 0) return DPTQ_OK;
  if (!w || !w_packed || !w_scales) return DPTQ_ERR_INVALID_ARG;
  if (!aligned16(w) || !aligned16(w_packed) || !aligned16(w_scales)) return DPTQ_ERR_INVALID_ARG;
  return from_hip(dptq::launch_prepare_weights(w, N, (int)K, hs, w_packed, w_scales,
                                               static_cast<hipStream_t>(stream)));
}

}  // extern "C"
