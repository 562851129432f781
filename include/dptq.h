/*
 * dptq.h - C ABI of the DynamicPTQ quantized linear layer for AMD MI355X (gfx950).
 *
 * The library computes the inference hot path of a W4A4 / W4A8 linear layer as
 * described by DynamicPTQ (arXiv 2606.12487):
 *
 *   1. an online Hadamard rotation of the fp16 activations (Section 2, Eq. 4),
 *   2. per-token symmetric quantization to 4 bits, or to 8 bits on the layers
 *      the phase-aware policy marks sensitive (Section 4.2; Algorithm 1 step 2;
 *      Eq. 21),
 *   3. an exact integer GEMM against packed 4-bit per-output-channel weights
 *      (Y = X W^T, Section 2; weights pre-rotated offline, Eq. 5), followed by
 *      a per-token x per-channel dequant epilogue.
 *
 * Around it: the residual-dynamics calibration statistics and the layer rule
 * of Section 3 (Eq. 8-11, 20), the group-wise 4-bit KV-cache codec
 * (Section 4.2), the same 4-bit x 4-bit product on the FP6 matrix cores,
 * and variants of the path: randomized-sign (QuaRot-style) rotation, decode
 * from fp16 activations in one launch, and the range quantizer of Eq. 1 with
 * a zero point.
 *
 * Conventions shared by every entry point
 *   - Every pointer named "device" is GPU memory owned by the caller; the
 *     library never allocates, frees or retains memory and keeps no state
 *     between calls.
 *   - GPU work is enqueued asynchronously on `stream` (a hipStream_t; NULL is
 *     the null stream).  Nothing synchronises the host.
 *   - Arguments are checked before anything is enqueued.  On an error the
 *     call returns a nonzero dptq_status and enqueues nothing.  A failed
 *     kernel launch returns DPTQ_ERR_HIP.
 *   - Device pointers must be 16-byte aligned.  Matrices are row-major and
 *     dense (row stride = row length).
 *   - Rotation B_h = I_{K/h} (x) H_h is unnormalised (+-1 entries).  H_h is
 *     Sylvester's natural-order matrix for h = 2^j and H_28 (x) H_{2^j}
 *     (Paley construction II, q = 13, on the slow index) for h = 28 * 2^j.
 *     The 1/h that makes (xB)(WB)^T = h X W^T is folded into the weight
 *     scales by dptq_prepare_weights.
 *   - Inputs must be finite; codes for rows holding Inf or NaN are
 *     unspecified.
 */
#ifndef DPTQ_H
#define DPTQ_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DPTQ_OK = 0,
  DPTQ_ERR_INVALID_ARG = 1, /* null pointer, negative size, bad bits, ... */
  DPTQ_ERR_UNSUPPORTED = 2, /* well-formed but outside what the kernels cover */
  DPTQ_ERR_HIP = 3          /* the HIP runtime reported an error */
} dptq_status;

/* Largest supported reduction length K (bounds the int32 accumulator). */
#define DPTQ_MAX_K 65536

/* Static description of a status code (never NULL). */
const char* dptq_status_string(int status);

/* Library version as MAJOR*10000 + MINOR*100 + PATCH. */
int dptq_version(void);

/*
 * dptq_rotate_quant - online rotation + per-token symmetric quantization.
 * Section 2 Eq. 4 (quantize X R), Eq. 1-2 in symmetric form (Section 4.2).
 *
 * For each token row m of x:
 *   y      = x_m . B_h                  in fp32, pinned order: radix-2
 *            butterflies over index bit 0, 1, 2, ... of the 2^j factor, then
 *            (for 28 * 2^j) a sequential sum over the 28-point index a = 0..27
 *   s_m    = fl32(max_k |y_k| / qmax),  qmax = 7 (bits 4) or 127 (bits 8)
 *   code_k = clamp(rne(fl32(y_k / s_m)), -2^(bits-1), 2^(bits-1) - 1)
 *   (s_m = 0 and all codes 0 when the row is all zero)
 *
 *   x        device, fp16 [M, K]
 *   M        tokens, >= 0 (M = 0 enqueues nothing and returns DPTQ_OK)
 *   K        features, 1 <= K <= DPTQ_MAX_K, multiple of 8 and of had_size;
 *            K <= 36864 (the row is staged in on-chip memory)
 *   had_size h in {2^j : 1 <= 2^j <= 32768} or {28 * 2^j : 28*2^j <= 32768}
 *   bits     4 or 8
 *   codes    device: bits 4 -> uint8 [M, K/2], byte j = code[2j] (low nibble)
 *            | code[2j+1] << 4 (4-bit two's complement);
 *            bits 8 -> int8 [M, K]
 *   a_scales device, float [M] (s_m)
 */
int dptq_rotate_quant(const void* x, int64_t M, int64_t K, int32_t had_size,
                      int32_t bits, void* codes, float* a_scales, void* stream);

/*
 * dptq_qlinear - quantized linear: exact integer GEMM + dequant epilogue.
 * Section 2 (Y = X W^T with W [out, in]), Eq. 5 (pre-rotated weights),
 * Section 4.2 (per-token activation and per-channel weight scales).
 *
 *   acc[m,n] = sum_k a_code[m,k] * w_code[n,k]          (exact, int32)
 *   y[m,n]   = fl16(fl32(fl32(fl32(acc) * a_scales[m]) * w_scales[n]))
 *
 *   codes    device, activation codes in the dptq_rotate_quant layout
 *   a_scales device, float [M]
 *   M        tokens >= 0; M <= 16 runs the weight-streaming decode kernel,
 *            larger M one of two MFMA tile kernels, whichever the shape
 *            keeps busier (same results bit for bit; see dptq_qlinear_kernel)
 *   K        multiple of 128, 128 <= K <= DPTQ_MAX_K
 *   bits     activation bits, 4 or 8
 *   w_packed device, uint8 [N, K/2]: 4-bit weight codes, same nibble layout as
 *            4-bit activation codes (as written by dptq_prepare_weights)
 *   w_scales device, float [N]
 *   N        output features, multiple of 16, >= 16
 *   y        device, fp16 [M, N]
 */
int dptq_qlinear(const void* codes, const float* a_scales, int64_t M, int64_t K,
                 int32_t bits, const uint8_t* w_packed, const float* w_scales,
                 int64_t N, void* y, void* stream);

/*
 * dptq_qlinear_acc - the same GEMM as dptq_qlinear, writing the raw int32
 * accumulators acc[m,n] (device, int32 [M, N]) instead of y.  Exposes the
 * exact integer result for verification; same argument rules.
 */
int dptq_qlinear_acc(const void* codes, int64_t M, int64_t K, int32_t bits,
                     const uint8_t* w_packed, int64_t N, int32_t* acc,
                     void* stream);

/* GEMM kernels of dptq_qlinear_kernel.  All return the same bits. */
typedef enum {
  DPTQ_GEMM_AUTO = 0,          /* the choice dptq_qlinear makes */
  DPTQ_GEMM_DECODE = 1,        /* weight streaming; M <= 16 */
  DPTQ_GEMM_TILE_256X128 = 2,  /* 256 (n) x 128 (m) output tiles; any M */
  DPTQ_GEMM_TILE_192X256 = 3   /* 192 (n) x 256 (m) tiles, persistent;
                                  M >= 256, N >= 192, K >= 512 */
} dptq_gemm_kernel;

/*
 * dptq_qlinear_kernel - dptq_qlinear (y != NULL; a_scales and w_scales
 * required, acc NULL) or dptq_qlinear_acc (acc != NULL; scales ignored, y
 * NULL) on a chosen kernel, for verification, benchmarks and tuning: every
 * kernel returns the same bits and the choice only changes speed.  Same
 * argument rules as dptq_qlinear; DPTQ_ERR_UNSUPPORTED when the shape is
 * outside the kernel's range, DPTQ_ERR_INVALID_ARG for an unknown kernel or
 * when not exactly one of y and acc is given.
 */
int dptq_qlinear_kernel(const void* codes, const float* a_scales, int64_t M, int64_t K,
                        int32_t bits, const uint8_t* w_packed, const float* w_scales,
                        int64_t N, void* y, int32_t* acc, int32_t kernel, void* stream);

/*
 * dptq_pack_w4_a8 - reorders 4-bit weights for W4A8 layers (the Eq. 5 weights
 * of the layers that Algorithm 1 step 2 / Eq. 21 run at 8 bits).  The layout is the same
 * size as w_packed; within each 4-byte group of a row (k = 8g .. 8g+7) byte
 * j holds k = 8g + j in its low nibble and k = 8g + j + 4 in its high nibble
 * (4-bit two's complement).  With this order the int8 matrix cores take the
 * 8-bit activation codes as they are stored, with no byte regrouping in the
 * GEMM's inner loop.  Offline, once per weight matrix.
 *
 *   w_packed device, uint8 [N, K/2] in the dptq_qlinear layout
 *   N        rows >= 0 (N = 0 enqueues nothing)
 *   K        multiple of 128, 128 <= K <= DPTQ_MAX_K
 *   out      device, uint8 [N, K/2]; must not overlap w_packed
 */
int dptq_pack_w4_a8(const uint8_t* w_packed, int64_t N, int64_t K, uint8_t* out, void* stream);

/*
 * dptq_qlinear_a8 - the W4A8 linear of dptq_qlinear (bits = 8) against
 * weights in the dptq_pack_w4_a8 order: the same accumulators and outputs
 * bit for bit.  Section 2, Eq. 5, Section 4.2.
 *
 *   codes    device, int8 [M, K] (dptq_rotate_quant, bits 8)
 *   a_scales device, float [M]
 *   w_a8     device, uint8 [N, K/2] from dptq_pack_w4_a8
 *   w_scales device, float [N]
 *   y        device, fp16 [M, N]
 *   kernel   a dptq_gemm_kernel value; DPTQ_ERR_UNSUPPORTED when it does not
 *            cover the shape; shapes and alignment as for dptq_qlinear
 */
int dptq_qlinear_a8(const void* codes, const float* a_scales, int64_t M, int64_t K,
                    const uint8_t* w_a8, const float* w_scales, int64_t N, void* y, int32_t kernel,
                    void* stream);

/* Paths of dptq_qlinear_decode_fused. */
typedef enum {
  DPTQ_DECODE_AUTO = 0,          /* the one launch where it is the faster path */
  DPTQ_DECODE_ONE_LAUNCH = 1,    /* rotation repeated in every workgroup */
  DPTQ_DECODE_TWO_LAUNCHES = 2   /* dptq_rotate_quant, then the decode GEMM */
} dptq_decode_mode;

/*
 * dptq_qlinear_decode_fused - a decode-shape quantized linear from the fp16
 * activations: dptq_rotate_quant followed by dptq_qlinear for M <= 16 tokens
 * (Eq. 4, Eq. 2, Section 2 Y = X W^T, Section 4.2 scales; the decode stage of
 * Section 4.9), with the same results bit for bit on every path.
 *
 * DPTQ_DECODE_ONE_LAUNCH runs a single kernel in which every workgroup
 * rotates and quantizes the M rows into on-chip memory while its first weight
 * loads are in flight, then streams its weight slice against them: no second
 * launch, and the GEMM never reads the codes back from HBM (workgroup 0 still
 * stores them).  The rotation is repeated in every workgroup, so this path
 * wins only for one or two rows of moderate K; DPTQ_DECODE_AUTO takes it for
 * N <= 16384 and either M = 1 with K <= 16384 and had_size a power of two
 * <= 8192, or M = 2 with K <= 12288 and had_size a power of two <= 4096; and
 * the two launches otherwise (had_size = 28 * 2^j included).
 *
 *   x, M, K, had_size, bits   as for dptq_rotate_quant; 1 <= M <= 16 (M = 0
 *            enqueues nothing), K a multiple of 128
 *   w_packed, w_scales, N, y  as for dptq_qlinear
 *   codes    device, the activation codes (dptq_rotate_quant layout), written
 *   a_scales device, float [M], written (16-byte aligned)
 *   mode     a dptq_decode_mode
 *
 * DPTQ_DECODE_ONE_LAUNCH needs the rows on chip: M * (K * bits / 8 + 16)
 * bytes of codes plus the fp32 staging of one row (17408 bytes per 4096
 * elements of K, rounded up) at most 151 KiB, else DPTQ_ERR_UNSUPPORTED.
 */
int dptq_qlinear_decode_fused(const void* x, int64_t M, int64_t K, int32_t had_size,
                              int32_t bits, const uint8_t* w_packed, const float* w_scales,
                              int64_t N, void* y, void* codes, float* a_scales, int32_t mode,
                              void* stream);

/*
 * dptq_rotate_quant_range - dptq_rotate_quant with the range-based quantizer
 * of Eq. 1 and an integer zero point instead of the symmetric one (Eq. 4 and
 * Eq. 1-2; Algorithm 1 lists zero points among the quantizer parameters).
 * Per token row y of x B_h (rotated exactly as dptq_rotate_quant rotates):
 *
 *   mx = max(max y, 0), mn = min(min y, 0)    (the range covers 0: zero is a level)
 *   s  = fl32(fl32(mx - mn) / (2^bits - 1))   one IEEE division per row
 *   z  = clamp(RNE(fl32(-mn / s)), 0, 2^bits - 1)
 *   q  = clamp(RNE(fl32(y / s)) + z, 0, 2^bits - 1),   Q(y) = s (q - z)
 *
 * and the stored code is q - 2^(bits-1), packed as dptq_rotate_quant packs
 * (4-bit two's complement nibbles, or int8).  A row of zeros gets s = 0,
 * z = 0 and q = 0.
 *
 *   x, M, K, had_size, bits   as for dptq_rotate_quant, K a multiple of 128
 *                             (else DPTQ_ERR_UNSUPPORTED)
 *   codes     device, output, dptq_rotate_quant's layout
 *   a_scales  device, float [M] output (s)
 *   a_zeros   device, int32 [M] output (z)
 */
int dptq_rotate_quant_range(const void* x, int64_t M, int64_t K, int32_t had_size, int32_t bits,
                            void* codes, float* a_scales, int32_t* a_zeros, void* stream);

/*
 * dptq_weight_sums - w_sums[n] = sum over k of weight row n's 4-bit codes (the
 * per-channel term of the zero-point correction in dptq_qlinear_range).
 *
 *   w_packed  device, uint8 [N, K/2] (dptq_prepare_weights layout), 16-byte aligned
 *   N, K      N >= 0, K a multiple of 32 (else DPTQ_ERR_UNSUPPORTED)
 *   w_sums    device, int32 [N] output
 */
int dptq_weight_sums(const uint8_t* w_packed, int64_t N, int64_t K, int32_t* w_sums, void* stream);

/*
 * dptq_qlinear_range - the quantized linear on range-quantized activations
 * (Section 2 Y = X W^T with Q(y) = s (q - z)): the exact integer GEMM of the
 * stored codes, corrected by the zero point,
 *
 *   acc'[m, n] = acc[m, n] + (2^(bits-1) - a_zeros[m]) w_sums[n]
 *             = sum_k (q[m, k] - a_zeros[m]) w[n, k]            (exact int32)
 *   y[m, n]    = fl16(fl32(fl32(fl32(acc'[m, n]) * a_scales[m]) * w_scales[n]))
 *
 * One launch on the kernel dptq_qlinear chooses for the shape, the
 * correction applied in the GEMM's epilogue; no workspace.
 *
 *   codes, a_scales, a_zeros  dptq_rotate_quant_range's outputs for M rows
 *                             (a_scales 16-byte aligned, a_zeros 4-byte)
 *   M, K, bits, w_packed, w_scales, N   as for dptq_qlinear
 *   w_sums    device, int32 [N] (dptq_weight_sums), 16-byte aligned
 *   y         device, fp16 [M, N] output, 16-byte aligned
 */
int dptq_qlinear_range(const void* codes, const float* a_scales, const int32_t* a_zeros, int64_t M,
                       int64_t K, int32_t bits, const uint8_t* w_packed, const float* w_scales,
                       const int32_t* w_sums, int64_t N, void* y, void* stream);

/*
 * dptq_residual_dynamics - residual-dynamics calibration statistics of one
 * layer (Section 3.1 Eq. 8-11; quantization in the rotated space, Section 3.2
 * Eq. 14-16).  For every token row t of the residual state x entering the
 * layer and the update dx the layer adds:
 *
 *   jr[t]  = ||dx_t||_2 / (||x_t||_2 + eps)                       (Eq. 8)
 *   snr[t] = 10 log10(||x_t||^2 / (||xhat_t - x_t||^2 + eps))      (Eq. 11)
 *
 * with xhat_t = Q_b(x_t + dx_t) - dx_t (Eq. 10), where Q_b is the path's own
 * quantizer: u = fl32(x + dx) rotated by I (x) H_h exactly as
 * dptq_rotate_quant rotates, quantized per token at `bits`, and mapped back by
 * the inverse rotation.  The error energy is taken in the rotated space and
 * divided by h, which equals ||Q_b(u) - u||^2 for the unnormalized H_h.
 * Norms and error energy accumulate in fp32 (any order), the final
 * arithmetic is fp64; results agree with an fp64 evaluation within 2e-5
 * relative (JR) and 1e-3 dB (SNR).
 *
 *   x, dx       device, fp16 [T, K], row-major, 16-byte aligned
 *   T, K, had_size   as for dptq_rotate_quant
 *   bits        4 or 8: the activation precision whose damage is measured
 *   eps         >= 0, finite (the eps of Eq. 8 and 11; the paper gives no value)
 *   jr, snr     device, float [T] outputs
 *   layer_means device, double [2] output {mean jr, mean snr} (Eq. 9 and the
 *               layer value of Eq. 11), or NULL to skip
 *
 * T = 0 enqueues nothing.
 */
int dptq_residual_dynamics(const void* x, const void* dx, int64_t T, int64_t K, int32_t had_size,
                           int32_t bits, float eps, float* jr, float* snr, double* layer_means,
                           void* stream);

/*
 * dptq_select_layers - the sensitive-layer rule of Eq. 20 (host only):
 * bits_out[l] = 8 if jr[l] > tau_jr and snr[l] < tau_snr, else 4, for the
 * layer statistics jr[l], snr[l] (host arrays [num_layers], e.g. the layer
 * means of dptq_residual_dynamics).  The paper gives no threshold values.
 */
int dptq_select_layers(int32_t num_layers, const double* jr, const double* snr, double tau_jr,
                       double tau_snr, int32_t* bits_out);

/*
 * dptq_kv_quant - group-wise 4-bit KV-cache quantization (Section 4.2: KV cache
 * at 4 bits with groups of 128; Eq. 1 range step, Eq. 2 rounding).
 *
 * Each row of kv is split into groups of `group` consecutive elements (with
 * head_dim 128 and group 128, one head of one token).  Per group, with m the
 * minimum and M the maximum:
 *
 *   s = fl32(fl32(M - m) / 15)                     (2^4 - 1 intervals, Eq. 1)
 *   code = min(15, RNE(fl32(fl32(x - m) / s)))     (Eq. 2 on the offset; 0 if s = 0)
 *
 * IEEE fp32 arithmetic, round half to even.
 *
 *   kv      device, fp16 [T, D], row-major, 16-byte aligned (K or V rows of T tokens)
 *   T       tokens, >= 0
 *   D       row length; a multiple of group, <= 2^31, T * D < 2^40
 *   group   power of two in [16, 512]
 *   codes   device, uint8 [T, D/2] output, 4-byte aligned: byte j of a row holds
 *           code[2j] in its low nibble and code[2j+1] in its high nibble
 *   scales  device, float [T, D/group] output (s per group), 4-byte aligned
 *   mins    device, float [T, D/group] output (m per group), 4-byte aligned
 *
 * To append tokens to a cache, pass pointers offset to the first new row.
 * Non-finite inputs give unspecified codes.  T = 0 enqueues nothing.
 */
int dptq_kv_quant(const void* kv, int64_t T, int64_t D, int32_t group, uint8_t* codes,
                  float* scales, float* mins, void* stream);

/*
 * dptq_kv_dequant - reconstruct the fp16 cache from dptq_kv_quant's output:
 * kv_out = fl16(fl32(fl32(code * s) + m)), two fp32 roundings then one fp16.
 * Arguments as for dptq_kv_quant; kv_out is device fp16 [T, D], 16-byte aligned.
 */
int dptq_kv_dequant(const uint8_t* codes, const float* scales, const float* mins, int64_t T,
                    int64_t D, int32_t group, void* kv_out, void* stream);

/*
 * dptq_layer_policy - phase-aware activation precision (host only).
 * Algorithm 1 step 2 with the sensitive set of Eq. 21.
 *
 *   bits_out[l] = 8 if layer l is sensitive else 4, for l = 0 .. num_layers-1.
 *   mask == NULL: the paper's default S = {1, 2, 3, L} (1-indexed), i.e.
 *                 {0, 1, 2, L-1} 0-indexed.
 *   mask != NULL: host uint8 [num_layers]; mask[l] != 0 marks layer l.
 *   num_layers >= 1; bits_out host int32 [num_layers].
 */
int dptq_layer_policy(int32_t num_layers, const uint8_t* mask, int32_t* bits_out);

/*
 * dptq_prepare_weights - offline weight preparation (Eq. 5 absorption,
 * per-output-channel symmetric round-to-nearest at 4 bits, Section 4.2).
 *
 * For each output row n of w: z = w_n . B_h (same rotation and order as
 * dptq_rotate_quant, on fp32 input), s = fl32(max|z| / 7), codes as in
 * dptq_rotate_quant at 4 bits, and w_scales[n] = fl32(s / h).
 *
 *   w        device, float [N, K]
 *   N        >= 0; K, had_size as for dptq_rotate_quant
 *   w_packed device, uint8 [N, K/2]
 *   w_scales device, float [N]
 */
int dptq_prepare_weights(const float* w, int64_t N, int64_t K, int32_t had_size,
                         uint8_t* w_packed, float* w_scales, void* stream);

/* Code layouts of dptq_rotate_quant_ex. */
typedef enum {
  DPTQ_LAYOUT_PACKED = 0, /* the dptq_rotate_quant layout: 4-bit nibbles or int8 */
  DPTQ_LAYOUT_FP6 = 1     /* 4-bit codes in the FP6 block layout (below) */
} dptq_code_layout;

/*
 * dptq_rotate_quant_ex - dptq_rotate_quant with the options of the path's
 * variants: a randomized-sign rotation and the output layout.
 *
 * Randomized signs (the QuaRot-style online Hadamard of Section 4.2): the
 * rotation becomes y = (x_m * d) . B_h, the signs d_k = +-1 applied to the
 * fp16 input before the first butterfly (exact).  Weights must be prepared
 * with the same signs (dptq_prepare_weights_signed), which cancel in the
 * product (Eq. 5).
 *
 *   signs    device, uint8 [ceil(K/8)], bit (k & 7) of byte k >> 3 set means
 *            d_k = -1; NULL for the plain rotation (then the call equals
 *            dptq_rotate_quant or dptq_rotate_quant_fp6)
 *   layout   DPTQ_LAYOUT_PACKED (bits 4 or 8; out as the codes of
 *            dptq_rotate_quant) or DPTQ_LAYOUT_FP6 (bits 4, K % 128 == 0; out
 *            as dptq_rotate_quant_fp6, dptq_fp6_bytes(M, K) bytes)
 *   other arguments as for dptq_rotate_quant
 */
int dptq_rotate_quant_ex(const void* x, int64_t M, int64_t K, int32_t had_size, int32_t bits,
                         const uint8_t* signs, int32_t layout, void* out, float* a_scales,
                         void* stream);

/*
 * dptq_prepare_weights_signed - dptq_prepare_weights for the randomized-sign
 * rotation: each weight row is multiplied by the same signs d (the signs
 * argument of dptq_rotate_quant_ex) before the rotation, so that
 * (x D B)(W D B)^T = h X W^T (Eq. 5).  signs NULL equals dptq_prepare_weights.
 */
int dptq_prepare_weights_signed(const float* w, int64_t N, int64_t K, int32_t had_size,
                                const uint8_t* signs, uint8_t* w_packed, float* w_scales,
                                void* stream);

/*
 * FP6 operand path of the 4-bit x 4-bit GEMM.  The same integer product as
 * dptq_qlinear at bits 4 (Section 2, Y = X W^T; Section 4.2 scales) computed
 * on the FP6 matrix cores: every 4-bit code c in [-8, 7] is stored as the
 * e2m3 value c / 2 (exact) and multiplied with a block scale of 2 per
 * operand, so each product is the exact integer a * w and the fp32
 * accumulation is exact (|partial sums| <= 64 K <= 2^22).  Results equal
 * dptq_qlinear's bit for bit.
 *
 * FP6 block layout of a [rows, K] code matrix (K % 128 == 0): rows padded to
 * Rp = 32 * ceil(rows / 32) with zero codes; blocks of 32 rows x 128 k, block
 * (rb, kb) at byte offset (kb * Rp/32 + rb) * 3072.  A block is two halves of
 * 1536 bytes, s = 0, 1.  In half s, lane l = 0..63 owns row 32 rb + (l & 31)
 * and codes k = 128 kb + 64 (l >> 5) + 32 s + j, j = 0..31, as a 192-bit
 * little-endian value whose bits 6 j .. 6 j + 5 hold the e2m3 field of code
 * j; its bytes 8 c .. 8 c + 7 (c = 0, 1, 2) sit at byte 1536 s + 512 c + 8 l.
 */

/* Bytes of the FP6 block layout of a [rows, K] code matrix; -1 when rows < 0
   or K is not a multiple of 128 in [128, DPTQ_MAX_K]. */
int64_t dptq_fp6_bytes(int64_t rows, int64_t K);

/*
 * dptq_pack_fp6 - canonical packed 4-bit codes -> FP6 block layout.  Serves
 * weights (once, offline) and activation codes (per call, after
 * dptq_rotate_quant at bits 4).
 *
 *   codes  device, uint8 [rows, K/2] in the dptq_rotate_quant 4-bit layout
 *   rows   >= 0 (0 enqueues nothing); K multiple of 128, <= DPTQ_MAX_K
 *   out    device, dptq_fp6_bytes(rows, K) bytes, 16-byte aligned; padding
 *          rows are written as zero codes
 */
int dptq_pack_fp6(const uint8_t* codes, int64_t rows, int64_t K, uint8_t* out, void* stream);

/*
 * dptq_rotate_quant_fp6 - dptq_rotate_quant at bits 4 (same rotation, scales
 * and codes, Section 2 Eq. 4, Section 4.2) writing the codes straight into
 * the FP6 block layout, so that no packing pass sits between the rotation
 * and dptq_qlinear_fp6.
 *
 *   x, M, had_size   as for dptq_rotate_quant; K also a multiple of 128
 *   out      device, dptq_fp6_bytes(M, K) bytes, 16-byte aligned; padding rows
 *            of the last 32-row block are written as zero codes
 *   a_scales device, float [M]
 */
int dptq_rotate_quant_fp6(const void* x, int64_t M, int64_t K, int32_t had_size, uint8_t* out,
                          float* a_scales, void* stream);

/*
 * dptq_qlinear_fp6 - dptq_qlinear at bits 4 on FP6 operands: y (fp16 [M, N])
 * from the dequant epilogue when y != NULL (a_scales, w_scales required), or
 * the raw int32 accumulators when acc != NULL (device int32 [M, N]; scales
 * ignored).  Exactly one of y and acc.
 *
 *   a_fp6    device, FP6 block layout of the [M, K] activation codes
 *   w_fp6    device, FP6 block layout of the [N, K] weight codes
 *   a_scales device, float [M]; w_scales device, float [N] (4-byte aligned)
 *   M >= 0, K multiple of 128 in [128, DPTQ_MAX_K], N multiple of 16
 *
 * Any M runs (the kernel tiles 256 tokens x 192 channels; it pays off for
 * prefill shapes, M in the hundreds and above).
 */
int dptq_qlinear_fp6(const uint8_t* a_fp6, const float* a_scales, int64_t M, int64_t K,
                     const uint8_t* w_fp6, const float* w_scales, int64_t N, void* y,
                     int32_t* acc, void* stream);

/* Device-native weight layouts of dptq_prepack_weights. */
typedef enum {
  DPTQ_WEIGHTS_FP6 = 1,     /* FP6 block layout: the 4-bit layers on dptq_qlinear_fp6 */
  DPTQ_WEIGHTS_A8_ORDER = 2, /* 8-bit activation order: the 8-bit layers on dptq_qlinear_a8 */
  DPTQ_WEIGHTS_DECODE = 3    /* decode layout: any layer's M <= 16 GEMM on
                                dptq_qlinear_decode_native */
} dptq_weight_layout;

/*
 * dptq_prepacked_bytes - bytes of the dptq_prepack_weights output for an
 * [N, K] weight matrix: dptq_fp6_bytes(N, K) for DPTQ_WEIGHTS_FP6 (rows padded
 * to a multiple of 32), N * K / 2 for DPTQ_WEIGHTS_A8_ORDER.  -1 for an
 * unknown layout, N < 0, or K not a multiple of 128 in [128, DPTQ_MAX_K];
 * N * K / 2 for DPTQ_WEIGHTS_DECODE, which also needs N % 16 == 0 (-1
 * otherwise).
 */
int64_t dptq_prepacked_bytes(int64_t N, int64_t K, int32_t layout);

/*
 * dptq_prepack_weights - the offline weights of Eq. 5 (rotated, quantized per
 * output channel at 4 bits, Section 4.2; dptq_prepare_weights output) moved
 * into the layout the GEMM of their layer reads natively.  The policy of
 * Algorithm 1 step 2 / Eq. 21 fixes one activation width per layer, so each
 * weight matrix needs one prefill layout: DPTQ_WEIGHTS_FP6 for a 4-bit layer
 * (dptq_qlinear_fp6), DPTQ_WEIGHTS_A8_ORDER for an 8-bit layer
 * (dptq_qlinear_a8); the call then equals dptq_pack_fp6 or dptq_pack_w4_a8 on
 * the same arguments.  DPTQ_WEIGHTS_DECODE (N % 16 == 0) is the layout of the
 * decode GEMM at either activation width (dptq_qlinear_decode_native): per
 * block of 16 rows and chunk of 128 k, the 64 bytes of each row's chunk as
 * four 16-byte pieces, the 1 KiB in the order (piece, row), so that the
 * decode GEMM streams each chunk as one contiguous KiB.  The codes are
 * unchanged and so is every product.  Run once per weight matrix, offline.
 *
 *   w_packed device, uint8 [N, K/2] in the dptq_qlinear layout (low nibble =
 *            even k), 16-byte aligned
 *   N        rows >= 0 (0 enqueues nothing)
 *   K        multiple of 128, 128 <= K <= DPTQ_MAX_K
 *   layout   a dptq_weight_layout value, else DPTQ_ERR_INVALID_ARG
 *   w_native device, dptq_prepacked_bytes(N, K, layout) bytes, 16-byte
 *            aligned, must not overlap w_packed; the caller owns it
 */
int dptq_prepack_weights(const uint8_t* w_packed, int64_t N, int64_t K, int32_t layout,
                         uint8_t* w_native, void* stream);

/*
 * dptq_qlinear_decode_native - dptq_qlinear (y != NULL; a_scales and
 * w_scales required, acc NULL) or dptq_qlinear_acc (acc != NULL; scales
 * ignored, y NULL) for decode batches, 0 <= M <= 16 tokens (Section 2
 * Y = X W^T, Section 4.2 scales; the decode stage of Section 4.9), on weights
 * in DPTQ_WEIGHTS_DECODE: the same results bit for bit as dptq_qlinear on the
 * canonical weights.  codes, a_scales, bits, K, N, y and acc as for
 * dptq_qlinear / dptq_qlinear_acc; w_dec device, dptq_prepacked_bytes(N, K,
 * DPTQ_WEIGHTS_DECODE) bytes, 16-byte aligned.  DPTQ_ERR_UNSUPPORTED for
 * M > 16 or a shape outside dptq_qlinear's range, DPTQ_ERR_INVALID_ARG when
 * not exactly one of y and acc is given.
 */
int dptq_qlinear_decode_native(const void* codes, const float* a_scales, int64_t M, int64_t K,
                               int32_t bits, const uint8_t* w_dec, const float* w_scales,
                               int64_t N, void* y, int32_t* acc, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* DPTQ_H */
