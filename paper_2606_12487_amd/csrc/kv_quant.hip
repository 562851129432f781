// Group-wise 4-bit KV-cache codec (Section 4.2: KV cache at 4 bits, group 128;
// Eq. 1 range step over 2^4 - 1 intervals; Eq. 2 rounding).
//
// The cache is a row-major fp16 [T, D] matrix whose rows are split into groups
// of G consecutive elements (G = 128: one head of one token).  Per group:
//   m = min, s = fl32(fl32(max - m) / 15),
//   code = min(15, RNE(fl32(fl32(x - m) / s)))   (0 when s = 0),
// packed two per byte, the even element in the low nibble; s and m are fp32.
// Reconstruction: fl16(fl32(fl32(code * s) + m)).
//
// Both kernels are HBM-bound streams.  Each lane owns 8 consecutive elements
// (one 16-byte load of halves, one 4-byte store of codes); the G / 8 lanes of
// a group are consecutive lanes of one wavefront, so the group's min and max
// are butterfly reductions over those lanes.  Groups never straddle a
// wavefront because G / 8 divides 64.
#include "internal.h"

namespace dptq {
namespace {

constexpr int kKvThreads = 256;

__device__ __forceinline__ void halves8(const uint4 raw, float v[8]) {
  const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __half2float(__ushort_as_half((unsigned short)(w[i] & 0xFFFFu)));
    v[2 * i + 1] = __half2float(__ushort_as_half((unsigned short)(w[i] >> 16)));
  }
}

// Correctly rounded fl32(d / s) from rc = fl32(1 / s) (Markstein's final
// correction: the residual d - q s is exact under an FMA), then round half to
// even by the fp32 adder: adding 1.5 * 2^23 leaves RNE(t) in the low mantissa
// bits for 0 <= t < 2^22.
__device__ __forceinline__ uint32_t level(float d, float s, float rc) {
  const float q = d * rc;
  const float e = fmaf(-q, s, d);
  const float t = fmaf(e, rc, q);
  const float r = t + 12582912.0f;
  const uint32_t c = __float_as_uint(r) - 0x4B400000u;
  return c < 15u ? c : 15u;
}

template <int LPG>
__global__ void __launch_bounds__(kKvThreads)
kv_quant_kernel(const uint4* __restrict__ kv, int64_t n_lanes, uint32_t* __restrict__ codes,
                float* __restrict__ scales, float* __restrict__ mins) {
  const int64_t lane = (int64_t)blockIdx.x * kKvThreads + threadIdx.x;
  const bool live = lane < n_lanes;
  float v[8];
  halves8(live ? kv[lane] : make_uint4(0, 0, 0, 0), v);
  float lo = v[0], hi = v[0];
#pragma unroll
  for (int k = 1; k < 8; ++k) {
    lo = fminf(lo, v[k]);
    hi = fmaxf(hi, v[k]);
  }
#pragma unroll
  for (int off = LPG / 2; off > 0; off >>= 1) {
    lo = fminf(lo, __shfl_xor(lo, off));
    hi = fmaxf(hi, __shfl_xor(hi, off));
  }
  const float s = (hi - lo) / 15.0f;           // IEEE subtraction and division
  uint32_t packed = 0;
  if (s != 0.0f) {
    const float rc = 1.0f / s;
#pragma unroll
    for (int k = 0; k < 8; ++k) packed |= level(v[k] - lo, s, rc) << (4 * k);
  }
  if (!live) return;
  codes[lane] = packed;
  if ((lane & (LPG - 1)) == 0) {
    scales[lane / LPG] = s;
    mins[lane / LPG] = lo;
  }
}

// fl16(fl32(fl32(code * s) + m)).  The empty asm statements keep each fp32
// rounding: without them the backend may fuse the multiply, the add and the
// fp16 conversion into mixed-precision FMAs with fewer roundings.
__device__ __forceinline__ uint32_t rebuild(uint32_t c, float s, float m) {
  float t = (float)c * s;
  asm("" : "+v"(t));
  float u = t + m;
  asm("" : "+v"(u));
  return (uint32_t)__half_as_ushort(__float2half_rn(u));
}

template <int LPG>
__global__ void __launch_bounds__(kKvThreads)
kv_dequant_kernel(const uint32_t* __restrict__ codes, const float* __restrict__ scales,
                  const float* __restrict__ mins, int64_t n_lanes, uint4* __restrict__ out) {
  const int64_t lane = (int64_t)blockIdx.x * kKvThreads + threadIdx.x;
  if (lane >= n_lanes) return;
  const uint32_t c = codes[lane];
  const float s = scales[lane / LPG];
  const float m = mins[lane / LPG];
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
    w[i] = rebuild((c >> (8 * i)) & 0xFu, s, m) | (rebuild((c >> (8 * i + 4)) & 0xFu, s, m) << 16);
  out[lane] = make_uint4(w[0], w[1], w[2], w[3]);
}

template <int LPG>
hipError_t launch_lpg(bool quant, const void* kv, int64_t n_lanes, void* codes, float* scales,
                      float* mins, void* out, hipStream_t stream) {
  const unsigned blocks = (unsigned)((n_lanes + kKvThreads - 1) / kKvThreads);
  if (quant) {
    kv_quant_kernel<LPG><<<blocks, kKvThreads, 0, stream>>>(
        static_cast<const uint4*>(kv), n_lanes, static_cast<uint32_t*>(codes), scales, mins);
  } else {
    kv_dequant_kernel<LPG><<<blocks, kKvThreads, 0, stream>>>(
        static_cast<const uint32_t*>(codes), scales, mins, n_lanes, static_cast<uint4*>(out));
  }
  return hipGetLastError();
}

hipError_t launch_kv(bool quant, const void* kv, int64_t T, int64_t D, int group, void* codes,
                     float* scales, float* mins, void* out, hipStream_t stream) {
  const int64_t n_lanes = T * D / 8;
  switch (group) {
    case 16: return launch_lpg<2>(quant, kv, n_lanes, codes, scales, mins, out, stream);
    case 32: return launch_lpg<4>(quant, kv, n_lanes, codes, scales, mins, out, stream);
    case 64: return launch_lpg<8>(quant, kv, n_lanes, codes, scales, mins, out, stream);
    case 128: return launch_lpg<16>(quant, kv, n_lanes, codes, scales, mins, out, stream);
    case 256: return launch_lpg<32>(quant, kv, n_lanes, codes, scales, mins, out, stream);
    case 512: return launch_lpg<64>(quant, kv, n_lanes, codes, scales, mins, out, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_kv_quant(const void* kv, int64_t T, int64_t D, int group, uint8_t* codes,
                           float* scales, float* mins, hipStream_t stream) {
  return launch_kv(true, kv, T, D, group, codes, scales, mins, nullptr, stream);
}

hipError_t launch_kv_dequant(const uint8_t* codes, const float* scales, const float* mins,
                             int64_t T, int64_t D, int group, void* out, hipStream_t stream) {
  return launch_kv(false, nullptr, T, D, group, const_cast<uint8_t*>(codes),
                   const_cast<float*>(scales), const_cast<float*>(mins), out, stream);
}

}  // namespace dptq
