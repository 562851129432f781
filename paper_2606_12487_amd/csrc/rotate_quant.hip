// Online Hadamard rotation + per-token symmetric quantization (gfx950).
//
// One workgroup owns one row (token, or weight output channel for the offline
// weight preparation).  The row is widened to fp32 and staged in LDS; the
// rotation B_h = I (x) H_h runs as radix-2 butterflies in registers, a group of
// index bits per pass, strictly in the order bit 0, bit 1, ... (the summation
// order the rotation is defined with), followed for h = 28 * 2^j by the dense
// 28-point stage summed sequentially over the slow index.  The row absmax is
// reduced across the workgroup, and the final pass divides, rounds to nearest
// even, packs and stores the codes with coalesced writes.
//
// Quotient: t = fl32(y / s) is formed as q = y * r, e = fma(-q, s, y),
// t = fma(e, r, q) with r = fl32(1 / s) (Markstein's correction, one
// correctly rounded reciprocal per row), which returns the correctly rounded
// quotient for every input reachable here.

#include "internal.h"

namespace dptq {
namespace {

constexpr int kThreads = 256;

// Paley construction II for q = 13: H28 = C (x) [[1,1],[1,-1]] + I (x) [[1,-1],[-1,-1]]
// with the conference matrix C = [[0, 1^T], [1, Q]], Q_ij = chi(j - i).
constexpr int chi13(int a) {
  a = ((a % 13) + 13) % 13;
  if (a == 0) return 0;
  for (int v = 1; v < 13; ++v)
    if ((v * v) % 13 == a) return 1;
  return -1;
}
constexpr int conference14(int p, int q) {
  if (p == 0 && q == 0) return 0;
  if (p == 0 || q == 0) return 1;
  return chi13((q - 1) - (p - 1));
}
constexpr int paley28_entry(int i, int j) {
  const int p = i >> 1, s = i & 1, q = j >> 1, t = j & 1;
  const int h2 = (s & t) ? -1 : 1;
  int v = conference14(p, q) * h2;
  if (p == q) v += (s == 0 && t == 0) ? 1 : -1;
  return v;
}
struct Paley28 {
  signed char e[28][28];
  constexpr Paley28() : e{} {
    for (int i = 0; i < 28; ++i)
      for (int j = 0; j < 28; ++j) e[i][j] = (signed char)paley28_entry(i, j);
  }
};
constexpr Paley28 kH28{};

// LDS index of row element i: 8 floats of padding after every 256.
__device__ __forceinline__ int lidx(int i) { return i + ((i >> 8) << 3); }

// Radix-2 butterflies on v[0..2^G) over local bits lo .. lo+nb-1, low bit first.
template <int G>
__device__ __forceinline__ void butterflies(float* v, int lo, int nb) {
#pragma unroll
  for (int b = 0; b < G; ++b) {
    if (b < lo || b >= lo + nb) continue;
#pragma unroll
    for (int k = 0; k < (1 << G); ++k) {
      if (k & (1 << b)) continue;
      const float a = v[k], c = v[k | (1 << b)];
      v[k] = a + c;
      v[k | (1 << b)] = a - c;
    }
  }
}

__device__ __forceinline__ void load8(const __half* p, float* v) {
  const uint4 u = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    v[2 * k] = __half2float(__ushort_as_half((unsigned short)(w[k] & 0xFFFFu)));
    v[2 * k + 1] = __half2float(__ushort_as_half((unsigned short)(w[k] >> 16)));
  }
}

__device__ __forceinline__ void load8(const float* p, float* v) {
  const float4 a = *reinterpret_cast<const float4*>(p);
  const float4 b = *reinterpret_cast<const float4*>(p + 4);
  v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

__device__ __forceinline__ float absmax8(const float* v, float m) {
#pragma unroll
  for (int k = 0; k < 8; ++k) m = fmaxf(m, fabsf(v[k]));
  return m;
}

// One pass over index bits [s, s+G): each work item gathers the 2^G elements
// that differ only in those bits, applies the butterflies, and writes back.
template <int G>
__device__ __forceinline__ float pass_bits(float* lds, int K, int s, bool last, float tmax) {
  const int groups = K >> G;
  const int low_mask = (1 << s) - 1;
  for (int g = threadIdx.x; g < groups; g += kThreads) {
    const int base = (g & low_mask) | ((g >> s) << (s + G));
    float v[1 << G];
#pragma unroll
    for (int k = 0; k < (1 << G); ++k) v[k] = lds[lidx(base + (k << s))];
    butterflies<G>(v, 0, G);
#pragma unroll
    for (int k = 0; k < (1 << G); ++k) {
      lds[lidx(base + (k << s))] = v[k];
      if (last) tmax = fmaxf(tmax, fabsf(v[k]));
    }
  }
  return tmax;
}

// Dense 28-point stage: y[b*p + c] = sum over a = 0..27 (in order) of
// H28[a][b] * z[a*p + c], per block and fast index c.
__device__ __forceinline__ float pass_28(float* lds, int K, int j, float tmax) {
  const int p = 1 << j;
  const int cols = K / 28;
  for (int col = threadIdx.x; col < cols; col += kThreads) {
    const int blk = col >> j, c = col & (p - 1);
    const int base = blk * 28 * p + c;
    float z[28];
#pragma unroll
    for (int a = 0; a < 28; ++a) z[a] = lds[lidx(base + a * p)];
#pragma unroll
    for (int b = 0; b < 28; ++b) {
      float acc = kH28.e[0][b] > 0 ? z[0] : -z[0];
#pragma unroll
      for (int a = 1; a < 28; ++a) acc = kH28.e[a][b] > 0 ? acc + z[a] : acc - z[a];
      lds[lidx(base + b * p)] = acc;
      tmax = fmaxf(tmax, fabsf(acc));
    }
  }
  return tmax;
}

template <int BITS>
__device__ __forceinline__ int quantize_one(float y, float s, float r) {
  constexpr int lo = -(1 << (BITS - 1)), hi = (1 << (BITS - 1)) - 1;
  const float q = y * r;
  const float e = __builtin_fmaf(-q, s, y);
  const float t = __builtin_fmaf(e, r, q);
  int c = (int)__builtin_rintf(t);
  c = c < lo ? lo : c;
  c = c > hi ? hi : c;
  return c;
}

// Compile-time pass plan for h = F * 2^J: the load pass covers index bits
// 0 .. min(J, 3) - 1, the remaining power-of-two bits are split as evenly as
// possible into at most three passes of at most 5 bits.
template <int J>
struct Plan {
  static constexpr int j0 = J < 3 ? J : 3;
  static constexpr int np = (J - j0 + 4) / 5;
  static constexpr int start(int i) {
    int s = j0;
    for (int k = 0; k < i; ++k) s += width_from(s, np - k);
    return s;
  }
  static constexpr int width(int i) { return width_from(start(i), np - i); }
  static constexpr int width_from(int s, int left) { return (J - s + left - 1) / left; }
};

template <typename Tin, int BITS, bool WEIGHT, int F, int J>
__global__ void __launch_bounds__(kThreads)
rotate_quant_kernel(const Tin* __restrict__ x, int K, uint8_t* __restrict__ codes,
                    float* __restrict__ scales) {
  extern __shared__ float lds[];
  __shared__ float red[kThreads / 64];
  using P = Plan<J>;
  static_assert(P::np <= 3, "pass plan too long");
  const int row = blockIdx.x;
  const Tin* xr = x + (size_t)row * K;
  const int nchunk = K >> 3;
  constexpr bool load_last = (P::np == 0 && F == 1);

  float tmax = 0.0f;
  for (int q = threadIdx.x; q < nchunk; q += kThreads) {
    float v[8];
    load8(xr + (size_t)q * 8, v);
    butterflies<3>(v, 0, P::j0);
    if (load_last) tmax = absmax8(v, tmax);
    float4* d = reinterpret_cast<float4*>(lds + lidx(q * 8));
    d[0] = make_float4(v[0], v[1], v[2], v[3]);
    d[1] = make_float4(v[4], v[5], v[6], v[7]);
  }
  __syncthreads();

  if constexpr (P::np > 0) {
    tmax = pass_bits<P::width(0)>(lds, K, P::start(0), P::np == 1 && F == 1, tmax);
    __syncthreads();
  }
  if constexpr (P::np > 1) {
    tmax = pass_bits<P::width(1)>(lds, K, P::start(1), P::np == 2 && F == 1, tmax);
    __syncthreads();
  }
  if constexpr (P::np > 2) {
    tmax = pass_bits<P::width(2)>(lds, K, P::start(2), F == 1, tmax);
    __syncthreads();
  }
  if constexpr (F == 28) {
    tmax = pass_28(lds, K, J, tmax);
    __syncthreads();
  }

  // Row absmax: wavefront reduction, then across the 4 wavefronts.
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) tmax = fmaxf(tmax, __shfl_xor(tmax, off));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = tmax;
  __syncthreads();
  float amax = red[0];
#pragma unroll
  for (int w = 1; w < kThreads / 64; ++w) amax = fmaxf(amax, red[w]);

  constexpr float qmax = (float)((1 << (BITS - 1)) - 1);
  const float sc = amax / qmax;                 // IEEE division
  const float rc = sc != 0.0f ? 1.0f / sc : 0.0f;
  if (threadIdx.x == 0) {
    if (WEIGHT) {
      constexpr int h = F << J;
      scales[row] = sc / (float)h;              // fold the 1/h of the rotation
    } else {
      scales[row] = sc;
    }
  }

  for (int q = threadIdx.x; q < nchunk; q += kThreads) {
    const float4* src = reinterpret_cast<const float4*>(lds + lidx(q * 8));
    const float4 a = src[0], b = src[1];
    const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    if (BITS == 4) {
      uint32_t packed = 0;
#pragma unroll
      for (int k = 0; k < 8; ++k)
        packed |= (uint32_t)(quantize_one<4>(v[k], sc, rc) & 0xF) << (4 * k);
      reinterpret_cast<uint32_t*>(codes + (size_t)row * (K / 2))[q] = packed;
    } else {
      uint32_t lo = 0, hi = 0;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        lo |= (uint32_t)(quantize_one<8>(v[k], sc, rc) & 0xFF) << (8 * k);
        hi |= (uint32_t)(quantize_one<8>(v[k + 4], sc, rc) & 0xFF) << (8 * k);
      }
      reinterpret_cast<uint2*>(codes + (size_t)row * K)[q] = make_uint2(lo, hi);
    }
  }
}

size_t lds_bytes(int K) {
  return (size_t)(K + ((K + 255) >> 8) * 8) * sizeof(float);
}

template <typename Tin, int BITS, bool WEIGHT, int F, int J>
hipError_t launch_one(const Tin* x, int64_t M, int K, uint8_t* codes, float* scales,
                      hipStream_t stream) {
  auto kern = rotate_quant_kernel<Tin, BITS, WEIGHT, F, J>;
  static bool attr_set = false;
  if (!attr_set) {
    // Rows above 64 KiB of LDS need the larger dynamic allocation enabled.
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                              hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)lds_bytes(kMaxRotateK));
    (void)hipGetLastError();
    attr_set = true;
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)M), dim3(kThreads), lds_bytes(K), stream, x, K,
                     codes, scales);
  return hipGetLastError();
}

template <typename Tin, int BITS, bool WEIGHT, int F, int J = 0>
hipError_t dispatch_j(int j, const Tin* x, int64_t M, int K, uint8_t* codes, float* scales,
                      hipStream_t stream) {
  constexpr int kMaxJ = F == 1 ? 15 : 10;   // h <= 32768
  if constexpr (J > kMaxJ) {
    return hipErrorInvalidValue;
  } else {
    if (j == J) return launch_one<Tin, BITS, WEIGHT, F, J>(x, M, K, codes, scales, stream);
    return dispatch_j<Tin, BITS, WEIGHT, F, J + 1>(j, x, M, K, codes, scales, stream);
  }
}

template <typename Tin, int BITS, bool WEIGHT>
hipError_t launch_rq(const Tin* x, int64_t M, int K, HadSplit hs, uint8_t* codes,
                     float* scales, hipStream_t stream) {
  if (M == 0) return hipSuccess;
  if (hs.f == 28) return dispatch_j<Tin, BITS, WEIGHT, 28>(hs.j, x, M, K, codes, scales, stream);
  return dispatch_j<Tin, BITS, WEIGHT, 1>(hs.j, x, M, K, codes, scales, stream);
}

}  // namespace

hipError_t launch_rotate_quant_f16(const void* x, int64_t M, int K, HadSplit hs,
                                   int bits, void* codes, float* scales,
                                   hipStream_t stream) {
  const __half* xh = static_cast<const __half*>(x);
  uint8_t* c = static_cast<uint8_t*>(codes);
  if (bits == 4) return launch_rq<__half, 4, false>(xh, M, K, hs, c, scales, stream);
  return launch_rq<__half, 8, false>(xh, M, K, hs, c, scales, stream);
}

hipError_t launch_prepare_weights(const float* w, int64_t N, int K, HadSplit hs,
                                  uint8_t* w_packed, float* w_scales,
                                  hipStream_t stream) {
  return launch_rq<float, 4, true>(w, N, K, hs, w_packed, w_scales, stream);
}

}  // namespace dptq
