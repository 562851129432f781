// Internal declarations shared by the C-ABI layer and the kernel sources.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
#include <stdint.h>

namespace dptq {

// Hadamard size h = f * 2^j with f in {1, 28}.
struct HadSplit {
  int f;      // 1 or 28
  int j;      // log2 of the power-of-two factor
};

// Largest row the rotate-quant kernel stages on chip (fp32 + padding < 160 KiB).
constexpr int kMaxRotateK = 36864;

// Launchers return hipSuccess or the launch error; arguments are already valid.
hipError_t launch_rotate_quant_f16(const void* x, int64_t M, int K, HadSplit hs,
                                   int bits, void* codes, float* scales,
                                   hipStream_t stream);
// Rotate + quantize at 4 bits writing the codes in the FP6 block layout
// (padding rows of the last 32-row block are written as zero codes).
hipError_t launch_rotate_quant_fp6(const void* x, int64_t M, int K, HadSplit hs, uint8_t* out,
                                   float* scales, hipStream_t stream,
                                   const uint8_t* signs = nullptr);
// signs (optional, nullptr = none): randomized-sign bitmask over K, bit
// (k & 7) of byte k >> 3 set = negate element k before the rotation.
hipError_t launch_prepare_weights(const float* w, int64_t N, int K, HadSplit hs,
                                  uint8_t* w_packed, float* w_scales,
                                  hipStream_t stream, const uint8_t* signs = nullptr);
hipError_t launch_rotate_quant_signed(const void* x, int64_t M, int K, HadSplit hs, int bits,
                                      const uint8_t* signs, void* codes, float* scales,
                                      hipStream_t stream);
// Residual-dynamics statistics of x + dx (statistics mode of the rotate+quantize
// kernels): per-row Jump Ratio and historical SNR (dB), and their means when
// means != nullptr.
hipError_t launch_residual_stats(const void* x, const void* dx, int64_t T, int K, HadSplit hs,
                                 int bits, float eps, float* jr, float* snr, double* means,
                                 hipStream_t stream);

// Group-wise 4-bit KV-cache codec over fp16 [T, D]; group in {16, ..., 512}
// (a power of two dividing D).
hipError_t launch_kv_quant(const void* kv, int64_t T, int64_t D, int group, uint8_t* codes,
                           float* scales, float* mins, hipStream_t stream);
hipError_t launch_kv_dequant(const uint8_t* codes, const float* scales, const float* mins,
                             int64_t T, int64_t D, int group, void* out, hipStream_t stream);

// GEMM kernels (values of dptq_gemm_kernel).
constexpr int kGemmAuto = 0, kGemmDecode = 1, kGemmTile = 2, kGemmWide = 3;

// Whether a kernel covers the shape (kGemmAuto and kGemmTile cover all).
bool gemm_kernel_fits(int kernel, int64_t M, int64_t N, int K, int bits);

// out_acc != nullptr selects the raw int32 accumulator output.
hipError_t launch_qlinear(const void* codes, const float* a_scales, int64_t M,
                          int K, int bits, const uint8_t* w_packed,
                          const float* w_scales, int64_t N, void* y,
                          int32_t* out_acc, int kernel, hipStream_t stream);

// 4-bit weights [N, K/2] in the canonical nibble order -> the 8-bit
// activation order (per dword: k0..k3 in the low nibbles, k4..k7 in the high
// ones; K % 8 == 0).
hipError_t launch_pack_w4_a8(const uint8_t* w_packed, int64_t N, int K, uint8_t* out,
                             hipStream_t stream);
// 4-bit weights [N, K/2] (canonical order, N % 16 == 0, K % 128 == 0) -> the
// decode layout of the M <= 16 GEMM (same size): per 16-row block and 128-k
// chunk, 1 KiB holding piece g (bytes 16 g .. 16 g + 15 of the chunk) of
// row r at position g * 16 + r, in units of 16 bytes.
hipError_t launch_pack_decode(const uint8_t* w_packed, int64_t N, int K, uint8_t* out,
                              hipStream_t stream);
// The decode GEMM (1 <= M <= 16) + epilogue, or the int32 accumulators when
// out_acc != nullptr, against weights in the decode layout.
hipError_t launch_qlinear_decode_native(const void* codes, const float* a_scales, int64_t M, int K,
                                        int bits, const uint8_t* w_dec, const float* w_scales,
                                        int64_t N, void* y, int32_t* out_acc, hipStream_t stream);
// W4A8 GEMM + epilogue against weights in the 8-bit activation order; the
// kernel choice as for launch_qlinear.
hipError_t launch_qlinear_a8(const void* codes, const float* a_scales, int64_t M, int K,
                             const uint8_t* w_a8, const float* w_scales, int64_t N, void* y,
                             int kernel, hipStream_t stream);

// Dynamic LDS available to the fused decode kernel (160 KiB less its 8.1 KiB
// of static arrays, rounded down).
constexpr int64_t kFusedLdsMax = 151 * 1024;
// Dynamic LDS the fused decode kernel needs for M rows of K at had split hs
// and activation bits (with one row in flight; two when that also fits).
int64_t decode_fused_lds(int64_t M, int K, HadSplit hs, int bits);
// Decode-shape (M <= 16) rotate + quantize + GEMM + epilogue.  mode 1: one
// launch, every workgroup rotating the M rows itself (requires
// decode_fused_lds(M, K, hs, bits) <= kFusedLdsMax); mode 2: the
// rotate+quantize kernel then the decode GEMM; mode 0: the one launch where
// it is the faster (decode_one_launch_wins).  codes / a_scales receive the
// activation codes and scales (both always written).
constexpr int kDecodeAuto = 0, kDecodeOneLaunch = 1, kDecodeTwoLaunches = 2;
bool decode_one_launch_wins(int64_t M, int K, HadSplit hs, int bits, int64_t N);
hipError_t launch_decode_fused(const void* x, int64_t M, int K, HadSplit hs, int bits,
                               const uint8_t* w_packed, const float* w_scales, int64_t N, void* y,
                               void* codes, float* a_scales, int mode, hipStream_t stream);

// Range-based quantizer with an integer zero point (rows of K % 128 == 0):
// codes (q - 2^(b-1), the symmetric path's packing), scales, zeros [M].
hipError_t launch_rotate_quant_range(const void* x, int64_t M, int K, HadSplit hs, int bits,
                                     void* codes, float* scales, int32_t* zeros,
                                     hipStream_t stream);
// sums[n] = sum of weight row n's 4-bit codes (K % 32 == 0).
hipError_t launch_weight_sums(const uint8_t* w_packed, int64_t N, int K, int32_t* sums,
                              hipStream_t stream);
// The quantized linear with the zero-point correction in the GEMM epilogue
// (any M; the kernel choice of launch_qlinear).
hipError_t launch_qlinear_zp(const void* codes, const float* a_scales, const int32_t* a_zeros,
                             int64_t M, int K, int bits, const uint8_t* w_packed,
                             const float* w_scales, const int32_t* w_sums, int64_t N, void* y,
                             hipStream_t stream);

// Compute units of the current device (cached per device).
int device_cus();

// FP6 block layout of 4-bit codes (e2m3(c / 2), 32-row x 128-k blocks of
// 3072 bytes; see qgemm_fp6.hip): bytes for a [rows, K] code matrix.
int64_t fp6_bytes(int64_t rows, int64_t K);
// Canonical packed 4-bit codes [R, K/2] -> FP6 block layout (K % 128 == 0).
hipError_t launch_pack_fp6(const uint8_t* codes, int64_t R, int K, uint8_t* out,
                           hipStream_t stream);
// W4A4 GEMM on the FP6 matrix cores; operands in the FP6 block layout.
// out_acc != nullptr selects the raw int32 accumulator output.
hipError_t launch_qlinear_fp6(const uint8_t* a6, const float* a_scales, int64_t M, int K,
                              const uint8_t* w6, const float* w_scales, int64_t N, void* y,
                              int32_t* out_acc, hipStream_t stream);

}  // namespace dptq
