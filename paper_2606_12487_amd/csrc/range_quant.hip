// Range-based activation quantizer with an integer zero point (Eq. 1 with the
// zero point of asymmetric quantization) and the zero-point correction of the
// integer GEMM.
//
// Quantizer, per token row y (the rotated activations, Eq. 4): the range is
// taken over the row and 0, mx = max(max y, 0) and mn = min(min y, 0), so that
// zero is a level; s = fl32(fl32(mx - mn) / (2^b - 1)) (Eq. 1, one IEEE
// division per row); z = clamp(RNE(fl32(-mn / s)), 0, 2^b - 1); the level of
// each element is q = clamp(RNE(fl32(y / s)) + z, 0, 2^b - 1) (Eq. 2) and the
// stored code is q - 2^(b-1), packed like the symmetric path's codes.  A row
// of zeros gets s = 0, z = 0, q = 0.
//
// GEMM: sum_k (q_k - z) w_k = acc + (2^(b-1) - z) wsum[n], with acc the exact
// accumulator of the stored codes and wsum[n] the sum of weight row n's
// codes; the corrected sum is exact in int32, and the epilogue is the
// symmetric path's, fl16(fl32(fl32(fl32(acc') * s_m) * w_s[n])).  The
// correction runs in the GEMM kernels' epilogues (qgemm.hip); this file
// holds the quantizer and the weight sums.

#include "internal.h"
#include "quant_device.h"

namespace dptq {
namespace {

using namespace qd;

constexpr int kRT = 256;   // threads per row

// One row per workgroup: rotate (rotate_row_segments), reduce the two row
// maxima, then the scale, zero point and codes.
template <int BITS, int JP, bool F28>
__global__ void __launch_bounds__(kRT)
rq_range_kernel(const __half* __restrict__ x, int K, int J, uint8_t* __restrict__ codes,
                float* __restrict__ scales, int32_t* __restrict__ zeros) {
  extern __shared__ float lds[];
  __shared__ float red[2][kRT / 64];
  const int row = blockIdx.x, r = threadIdx.x;
  const uint4 none[2] = {make_uint4(0, 0, 0, 0), make_uint4(0, 0, 0, 0)};
  float hi = 0.0f, neg = 0.0f;
  rotate_row_segments<JP, F28, true, 1>(x + (size_t)row * K, K, J, true, r, RowSplit{0, 1, r, kRT},
                                        false, none, lds, hi, neg);
  hi = wave_max_nonneg(hi);
  neg = wave_max_nonneg(neg);
  if ((r & 63) == 0) {
    red[0][r >> 6] = hi;
    red[1][r >> 6] = neg;
  }
  __syncthreads();
  hi = fmaxf(fmaxf(red[0][0], red[0][1]), fmaxf(red[0][2], red[0][3]));
  neg = fmaxf(fmaxf(red[1][0], red[1][1]), fmaxf(red[1][2], red[1][3]));

  constexpr int kLevels = (1 << BITS) - 1;
  constexpr int kHalf = 1 << (BITS - 1);
  const float width = hi + neg;                  // fl32(mx - mn), mn = -neg
  const float sc = width / (float)kLevels;       // IEEE division
  const float rc = sc != 0.0f ? 1.0f / sc : 0.0f;
  const int zp = sc != 0.0f ? min(max((int)rintf(neg / sc), 0), kLevels) : 0;
  if (r == 0) {
    scales[row] = sc;
    zeros[row] = zp;
  }
  const int nseg = (K + kSeg - 1) / kSeg;
  const int b1 = seg_off(16 * r);
  for (int sg = 0; sg < nseg; ++sg) {
    const int e = sg * kSeg + 16 * r;
    if (e >= K) continue;
    const float* sl = lds + sg * kSegFloats + b1;
    uint32_t bt[16];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 w4 = *reinterpret_cast<const float4*>(sl + 4 * q);
      const float w[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        // round_bits leaves RNE(y / s) + 0x4B400000 in the word.
        const int it = (int)(round_bits(w[u], sc, rc) - 0x4B400000u);
        const int lv = min(max(it + zp, 0), kLevels);
        bt[4 * q + u] = (uint32_t)(lv - kHalf);
      }
    }
    if (BITS == 4) {
      *reinterpret_cast<uint2*>(codes + (size_t)row * (K / 2) + e / 2) =
          make_uint2(pack_nibbles(bt), pack_nibbles(bt + 8));
    } else {
      *reinterpret_cast<uint4*>(codes + (size_t)row * K + e) =
          make_uint4(low_bytes(bt[0], bt[1], bt[2], bt[3]), low_bytes(bt[4], bt[5], bt[6], bt[7]),
                     low_bytes(bt[8], bt[9], bt[10], bt[11]), low_bytes(bt[12], bt[13], bt[14], bt[15]));
    }
  }
}

// Sum of the eight signed nibbles of a word.
__device__ __forceinline__ int nibble_sum(uint32_t w) {
  int s = 0;
#pragma unroll
  for (int k = 0; k < 8; ++k) s += ((int)(w << (28 - 4 * k))) >> 28;
  return s;
}

// wsum[n] = sum of weight row n's 4-bit codes: one wavefront per row.
__global__ void __launch_bounds__(256)
weight_sums_kernel(const uint8_t* __restrict__ w, int N, int K, int32_t* __restrict__ out) {
  const int n = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (n >= N) return;
  const uint8_t* row = w + (size_t)n * (K / 2);
  int s = 0;
  for (int b = 16 * lane; b < K / 2; b += 16 * 64) {
    const uint4 u = *reinterpret_cast<const uint4*>(row + b);
    s += nibble_sum(u.x) + nibble_sum(u.y) + nibble_sum(u.z) + nibble_sum(u.w);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
  if (lane == 0) out[n] = s;
}

size_t range_lds_bytes(int K) { return (size_t)((K + kSeg - 1) / kSeg) * kSegFloats * sizeof(float); }

template <int BITS, int JP, bool F28>
hipError_t launch_range_t(const void* x, int64_t M, int K, HadSplit hs, uint8_t* codes,
                          float* scales, int32_t* zeros, hipStream_t stream) {
  auto kern = rq_range_kernel<BITS, JP, F28>;
  static bool attr_set = false;
  if (!attr_set) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                              hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)range_lds_bytes(kMaxRotateK));
    (void)hipGetLastError();
    attr_set = true;
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)M), dim3(kRT), range_lds_bytes(K), stream,
                     static_cast<const __half*>(x), K, hs.j, codes, scales, zeros);
  return hipGetLastError();
}

// h = 28 * 2^j has j <= 10; h = 2^j goes to JP = min(j, 12).
template <int BITS, int JP = 0>
hipError_t dispatch_range(const void* x, int64_t M, int K, HadSplit hs, uint8_t* codes,
                          float* scales, int32_t* zeros, hipStream_t stream) {
  if constexpr (JP == 12) {
    return launch_range_t<BITS, 12, false>(x, M, K, hs, codes, scales, zeros, stream);
  } else {
    if (hs.j == JP) {
      if constexpr (JP <= 10) {
        if (hs.f == 28) return launch_range_t<BITS, JP, true>(x, M, K, hs, codes, scales, zeros, stream);
      }
      return launch_range_t<BITS, JP, false>(x, M, K, hs, codes, scales, zeros, stream);
    }
    return dispatch_range<BITS, JP + 1>(x, M, K, hs, codes, scales, zeros, stream);
  }
}

}  // namespace

hipError_t launch_rotate_quant_range(const void* x, int64_t M, int K, HadSplit hs, int bits,
                                     void* codes, float* scales, int32_t* zeros,
                                     hipStream_t stream) {
  if (M == 0) return hipSuccess;
  uint8_t* c = static_cast<uint8_t*>(codes);
  if (bits == 4) return dispatch_range<4>(x, M, K, hs, c, scales, zeros, stream);
  return dispatch_range<8>(x, M, K, hs, c, scales, zeros, stream);
}

hipError_t launch_weight_sums(const uint8_t* w_packed, int64_t N, int K, int32_t* sums,
                              hipStream_t stream) {
  if (N == 0) return hipSuccess;
  hipLaunchKernelGGL(weight_sums_kernel, dim3((unsigned)((N + 3) / 4)), dim3(256), 0, stream,
                     w_packed, (int)N, K, sums);
  return hipGetLastError();
}

}  // namespace dptq
