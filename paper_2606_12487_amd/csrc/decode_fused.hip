// Decode-shape quantized linear in one launch: rotate + quantize the M <= 16
// token rows and the weight-streaming GEMM with its dequant epilogue.
//
// The grid is the decode GEMM's (one workgroup of 512 threads per 16 output
// channels).  Workgroup b first rotates and quantizes rows m = b, b + G, ...
// (< M) exactly as the rotate+quantize kernels do: the row is widened to fp32
// in LDS, the butterflies run one index bit per pass in the order bit 0, 1,
// 2, ..., then for h = 28 * 2^j the dense 28-point stage summed sequentially
// over the slow index; the scale is fl32(absmax / qmax) and the codes are the
// correctly rounded quotients rounded half to even.  It writes the codes and
// scale of its rows to the caller's buffers, makes them visible device-wide
// and counts them in sync[0].  Every workgroup then loads the first batch of
// its weight slice, waits until sync[0] = M (a bounded spin: past the limit
// it sets sync[2] and carries on, so the grid always drains), reads the codes
// and runs the decode GEMM.  The last workgroup to finish resets sync[0] and
// sync[1], so the caller's zero-initialised sync words are zero again after
// every call.  Producers never wait for a workgroup of higher index, so in
// the in-order dispatch of workgroups no wait can block the producer it waits
// for.

#include "internal.h"
#include "quant_device.h"

namespace dptq {
namespace {

using namespace qd;

typedef int v4i_t __attribute__((ext_vector_type(4)));

constexpr int kFT = 512;          // threads per workgroup
constexpr int kFWaves = kFT / 64;
constexpr int kFBatch = 4;        // 128-k chunks in flight per wavefront
constexpr int kSpinLimit = 1 << 22;

__device__ __forceinline__ int f_lidx(int i) { return i + ((i >> 8) << 3); }

__device__ __forceinline__ uint32_t f_nib_lo(uint32_t v) { return (v << 4) & 0xF0F0F0F0u; }
__device__ __forceinline__ uint32_t f_nib_hi(uint32_t v) { return v & 0xF0F0F0F0u; }
__device__ __forceinline__ v4i_t f_op_nibbles(uint32_t v0, uint32_t v1) {
  v4i_t r;
  r.x = (int)f_nib_lo(v0);
  r.y = (int)f_nib_hi(v0);
  r.z = (int)f_nib_lo(v1);
  r.w = (int)f_nib_hi(v1);
  return r;
}
__device__ __forceinline__ v4i_t f_op_bytes(uint32_t d0, uint32_t d1, uint32_t d2, uint32_t d3) {
  v4i_t r;
  r.x = (int)__builtin_amdgcn_perm(d1, d0, 0x06040200u);
  r.y = (int)__builtin_amdgcn_perm(d1, d0, 0x07050301u);
  r.z = (int)__builtin_amdgcn_perm(d3, d2, 0x06040200u);
  r.w = (int)__builtin_amdgcn_perm(d3, d2, 0x07050301u);
  return r;
}
template <int BITS>
__device__ __forceinline__ int f_unscale(int v) { return BITS == 4 ? (v >> 8) : (v >> 4); }

__device__ __forceinline__ __half f_dequant(int acc, float as, float ws) {
  const float t1 = (float)acc * as;
  float t2 = t1 * ws;
  asm("" : "+v"(t2));
  return __float2half_rn(t2);
}

// Rotate + quantize one row into codes / scale (all 512 threads).
template <int BITS>
__device__ void produce_row(const __half* __restrict__ xr, int K, int F, int J, float* lds,
                            float* red, uint8_t* __restrict__ crow, float* __restrict__ srow) {
  const int t = threadIdx.x;
  for (int q = t; q < K / 8; q += kFT) {
    const uint4 u = *reinterpret_cast<const uint4*>(xr + 8 * q);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
    float* d = lds + f_lidx(8 * q);
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      d[2 * k] = __half2float(__ushort_as_half((unsigned short)(w[k] & 0xFFFFu)));
      d[2 * k + 1] = __half2float(__ushort_as_half((unsigned short)(w[k] >> 16)));
    }
  }
  __syncthreads();
  // Power-of-two factor: one index bit per pass, bit 0 first.  Pairs never
  // cross a Hadamard block (its offset is a multiple of 2^J).
  for (int b = 0; b < J; ++b) {
    const int lo = (1 << b) - 1;
    for (int u = t; u < K / 2; u += kFT) {
      const int i = ((u >> b) << (b + 1)) | (u & lo);
      const float a = lds[f_lidx(i)], c = lds[f_lidx(i + (1 << b))];
      lds[f_lidx(i)] = a + c;
      lds[f_lidx(i + (1 << b))] = a - c;
    }
    __syncthreads();
  }
  if (F == 28) {
    // y[b p + c] = sum over a = 0..27, in order, of H28[a][b] z[a p + c].
    const int p = 1 << J;
    for (int col = t; col < K / 28; col += kFT) {
      const int base = (col >> J) * 28 * p + (col & (p - 1));
      float z[28];
#pragma unroll
      for (int a = 0; a < 28; ++a) z[a] = lds[f_lidx(base + a * p)];
#pragma unroll
      for (int bb = 0; bb < 28; ++bb) {
        float acc = kH28.e[0][bb] > 0 ? z[0] : -z[0];
#pragma unroll
        for (int a = 1; a < 28; ++a) acc = kH28.e[a][bb] > 0 ? acc + z[a] : acc - z[a];
        lds[f_lidx(base + bb * p)] = acc;
      }
    }
    __syncthreads();
  }
  float m = 0.0f;
  for (int i = t; i < K; i += kFT) m = fmaxf(m, fabsf(lds[f_lidx(i)]));
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) m = fmaxf(m, __shfl_xor(m, off));
  if ((t & 63) == 0) red[t >> 6] = m;
  __syncthreads();
  float amax = red[0];
#pragma unroll
  for (int w = 1; w < kFWaves; ++w) amax = fmaxf(amax, red[w]);
  constexpr float qmax = (float)((1 << (BITS - 1)) - 1);
  const float sc = amax / qmax;                 // IEEE division
  const float rc = sc != 0.0f ? 1.0f / sc : 0.0f;
  if (t == 0) *srow = sc;
  for (int q = t; q < K / 8; q += kFT) {
    const float* src = lds + f_lidx(8 * q);
    uint32_t bt[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) bt[k] = round_bits(src[k], sc, rc);
    if (BITS == 4) {
      reinterpret_cast<uint32_t*>(crow)[q] = pack_nibbles(bt);
    } else {
      reinterpret_cast<uint2*>(crow)[q] =
          make_uint2(low_bytes(bt[0], bt[1], bt[2], bt[3]), low_bytes(bt[4], bt[5], bt[6], bt[7]));
    }
  }
  __syncthreads();   // the row's LDS is reused by the next row
}

// Rotate + quantize one row for h = 2^J <= 4096 with the register-phase
// rotation of the rotate+quantize kernel (threads 0..255 hold 16 elements of
// a 4096-element segment in each of three phases covering index bits 0-3,
// 4-7 and 8-11, in that order); the other 256 threads only join the
// barriers.  K is a multiple of 128, so a thread's 16 elements are all in
// the row or all past it.
template <int BITS, int J>
__device__ void produce_row_pow2(const __half* __restrict__ xr, int K, float* lds, float* red,
                                 uint8_t* __restrict__ crow, float* __restrict__ srow) {
  const int t = threadIdx.x;
  const bool act = t < 256;
  const int nseg = (K + kSeg - 1) / kSeg;
  const int b1 = seg_off(16 * (t & 255));
  const int b2 = seg_off(256 * ((t & 255) >> 4) + (t & 15));
  const int b3 = seg_off(t & 255);
  float tmax = 0.0f;
  if (act) {
    for (int sg = 0; sg < nseg; ++sg) {
      // Past the row end (the last segment of a K that is not a multiple of
      // 4096) the segment is zero: whole Hadamard blocks of zeros.
      const int e = sg * kSeg + 16 * t;
      float v[16];
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) {
        const uint4 u = e < K ? *reinterpret_cast<const uint4*>(xr + e + 8 * h2) : make_uint4(0, 0, 0, 0);
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          v[8 * h2 + 2 * k] = __half2float(__ushort_as_half((unsigned short)(w[k] & 0xFFFFu)));
          v[8 * h2 + 2 * k + 1] = __half2float(__ushort_as_half((unsigned short)(w[k] >> 16)));
        }
      }
      stages16<0, (J < 4 ? J : 4)>(v);
      if (J <= 4) tmax = absmax16(v, tmax);
      float* sl = lds + sg * kSegFloats + b1;
#pragma unroll
      for (int q = 0; q < 4; ++q)
        *reinterpret_cast<float4*>(sl + 4 * q) = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
    }
  }
  if constexpr (J > 4) {
    __syncthreads();
    if (act) {
      for (int sg = 0; sg < nseg; ++sg) {
        if (sg * kSeg >= K) continue;
        float* sl = lds + sg * kSegFloats + b2;
        float v[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) v[r] = sl[16 * r + 4 * (r >> 2)];
        stages16<0, (J < 8 ? J : 8) - 4>(v);
        if (J <= 8) tmax = absmax16(v, tmax);
#pragma unroll
        for (int r = 0; r < 16; ++r) sl[16 * r + 4 * (r >> 2)] = v[r];
      }
    }
  }
  if constexpr (J > 8) {
    __syncthreads();
    if (act) {
      for (int sg = 0; sg < nseg; ++sg) {
        if (sg * kSeg >= K) continue;
        float* sl = lds + sg * kSegFloats + b3;
        float v[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) v[r] = sl[272 * r];
        stages16<0, J - 8>(v);
        tmax = absmax16(v, tmax);
#pragma unroll
        for (int r = 0; r < 16; ++r) sl[272 * r] = v[r];
      }
    }
  }
  tmax = wave_max_nonneg(tmax);
  if ((t & 63) == 0) red[t >> 6] = tmax;
  __syncthreads();
  float amax = red[0];
#pragma unroll
  for (int w = 1; w < kFWaves; ++w) amax = fmaxf(amax, red[w]);
  constexpr float qmax = (float)((1 << (BITS - 1)) - 1);
  const float sc = amax / qmax;                 // IEEE division
  const float rc = sc != 0.0f ? 1.0f / sc : 0.0f;
  if (t == 0) *srow = sc;
  if (act) {
    for (int sg = 0; sg < nseg; ++sg) {
      const int e = sg * kSeg + 16 * t;
      if (e >= K) continue;
      const float* sl = lds + sg * kSegFloats + b1;
      uint32_t bt[16];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 w4 = *reinterpret_cast<const float4*>(sl + 4 * q);
        bt[4 * q] = round_bits(w4.x, sc, rc);
        bt[4 * q + 1] = round_bits(w4.y, sc, rc);
        bt[4 * q + 2] = round_bits(w4.z, sc, rc);
        bt[4 * q + 3] = round_bits(w4.w, sc, rc);
      }
      if (BITS == 4) {
        *reinterpret_cast<uint2*>(crow + e / 2) = make_uint2(pack_nibbles(bt), pack_nibbles(bt + 8));
      } else {
        *reinterpret_cast<uint4*>(crow + e) =
            make_uint4(low_bytes(bt[0], bt[1], bt[2], bt[3]), low_bytes(bt[4], bt[5], bt[6], bt[7]),
                       low_bytes(bt[8], bt[9], bt[10], bt[11]), low_bytes(bt[12], bt[13], bt[14], bt[15]));
      }
    }
  }
  __syncthreads();   // the row's LDS is reused by the next row
}

// JP >= 0: h = 2^JP <= 4096 (register-phase producer); JP < 0: any h, with
// the generic one-bit passes.
template <int BITS, int JP>
__global__ void __launch_bounds__(kFT)
qdecode_fused(const __half* __restrict__ x, int M, int K, int F, int J,
              const uint8_t* __restrict__ w_packed, const float* __restrict__ w_scales, int N,
              __half* __restrict__ y, uint8_t* __restrict__ codes, float* __restrict__ a_scales,
              int32_t* __restrict__ sync) {
  extern __shared__ float lds[];
  __shared__ float red[kFWaves];
  __shared__ v4i_t part[kFWaves][64];
  const int G = gridDim.x, b = blockIdx.x, t = threadIdx.x;
  const size_t arow = BITS == 4 ? (size_t)K / 2 : (size_t)K;

  // Producer rows of this workgroup.
  for (int m = b; m < M; m += G) {
    if constexpr (JP >= 0)
      produce_row_pow2<BITS, JP>(x + (size_t)m * K, K, lds, red, codes + (size_t)m * arow, a_scales + m);
    else
      produce_row<BITS>(x + (size_t)m * K, K, F, J, lds, red, codes + (size_t)m * arow, a_scales + m);
  }
  if (b < M) {
    // Every thread's code stores precede the barrier; thread 0 then publishes
    // them device-wide and counts its rows.
    __syncthreads();
    if (t == 0) {
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
      int mine = 0;
      for (int m = b; m < M; m += G) ++mine;
      atomicAdd(&sync[0], mine);
    }
  }

  // Consumer: the weight slice of 16 output channels, K split over the
  // wavefronts in 128-k chunks.
  const int lane = t & 63, wave = t >> 6;
  const int n0 = b * 16;
  const int fr = lane & 15, fg = lane >> 4;
  const int nck = K / 128;
  const int c_begin = (int)((long)nck * wave / kFWaves);
  const int c_end = (int)((long)nck * (wave + 1) / kFWaves);
  const bool mvalid = fr < M;
  const uint8_t* wp = w_packed + (size_t)(n0 + fr) * (K / 2) + fg * 16;
  const uint8_t* ap = codes + (size_t)(mvalid ? fr : 0) * arow + (BITS == 4 ? fg * 16 : fg * 32);

  // First batch of weights while the producers finish.
  uint4 wv[kFBatch];
#pragma unroll
  for (int k = 0; k < kFBatch; ++k) {
    const int ck = c_begin + k;
    wv[k] = ck < c_end ? *reinterpret_cast<const uint4*>(wp + (size_t)ck * 64) : make_uint4(0, 0, 0, 0);
  }
  if (t == 0) {
    int spins = 0;
    while (__hip_atomic_load(&sync[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < M) {
      if (++spins > kSpinLimit) {
        atomicOr(&sync[2], 1);
        break;
      }
      __builtin_amdgcn_s_sleep(2);
    }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  }
  __syncthreads();

  v4i_t acc = v4i_t{0, 0, 0, 0};
  for (int c = c_begin; c < c_end; c += kFBatch) {
    uint4 av[kFBatch], av2[kFBatch];
    if (c != c_begin) {
#pragma unroll
      for (int k = 0; k < kFBatch; ++k) {
        const int ck = c + k;
        wv[k] = ck < c_end ? *reinterpret_cast<const uint4*>(wp + (size_t)ck * 64) : make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int k = 0; k < kFBatch; ++k) {
      const int ck = c + k;
      const bool ok = ck < c_end && mvalid;
      if (BITS == 4) {
        av[k] = ok ? *reinterpret_cast<const uint4*>(ap + (size_t)ck * 64) : make_uint4(0, 0, 0, 0);
      } else {
        av[k] = ok ? *reinterpret_cast<const uint4*>(ap + (size_t)ck * 128) : make_uint4(0, 0, 0, 0);
        av2[k] = ok ? *reinterpret_cast<const uint4*>(ap + (size_t)ck * 128 + 16) : make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int k = 0; k < kFBatch; ++k) {
      v4i_t b0, b1;
      if (BITS == 4) {
        b0 = f_op_nibbles(av[k].x, av[k].y);
        b1 = f_op_nibbles(av[k].z, av[k].w);
      } else {
        b0 = f_op_bytes(av[k].x, av[k].y, av[k].z, av[k].w);
        b1 = f_op_bytes(av2[k].x, av2[k].y, av2[k].z, av2[k].w);
      }
      acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(f_op_nibbles(wv[k].x, wv[k].y), b0, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(f_op_nibbles(wv[k].z, wv[k].w), b1, acc, 0, 0, 0);
    }
  }
  part[wave][lane] = acc;
  __syncthreads();
  if (wave == 0) {
    v4i_t tot = part[0][lane];
#pragma unroll
    for (int w = 1; w < kFWaves; ++w) {
      const v4i_t p = part[w][lane];
      tot.x += p.x; tot.y += p.y; tot.z += p.z; tot.w += p.w;
    }
    if (mvalid) {
      const int m = fr, n = n0 + fg * 4;
      const float as = a_scales[m];
      const float4 wsv = *reinterpret_cast<const float4*>(w_scales + n);
      const __half h0 = f_dequant(f_unscale<BITS>(tot.x), as, wsv.x);
      const __half h1 = f_dequant(f_unscale<BITS>(tot.y), as, wsv.y);
      const __half h2 = f_dequant(f_unscale<BITS>(tot.z), as, wsv.z);
      const __half h3 = f_dequant(f_unscale<BITS>(tot.w), as, wsv.w);
      uint2 pk;
      pk.x = (uint32_t)__half_as_ushort(h0) | ((uint32_t)__half_as_ushort(h1) << 16);
      pk.y = (uint32_t)__half_as_ushort(h2) | ((uint32_t)__half_as_ushort(h3) << 16);
      *reinterpret_cast<uint2*>(y + (size_t)m * N + n) = pk;
    }
  }
  // The last workgroup past its wait resets the counters.
  if (t == 0) {
    if (atomicAdd(&sync[1], 1) == G - 1) {
      atomicExch(&sync[0], 0);
      atomicExch(&sync[1], 0);
    }
  }
}

template <int BITS, int JP>
hipError_t launch_fused_t(const void* x, int64_t M, int K, HadSplit hs, const uint8_t* w,
                          const float* ws, int64_t N, void* y, void* codes, float* as,
                          int32_t* sync, hipStream_t stream) {
  auto kern = qdecode_fused<BITS, JP>;
  const size_t lds = JP >= 0 ? (size_t)((K + kSeg - 1) / kSeg) * kSegFloats * sizeof(float)
                             : (size_t)(K + ((K + 255) >> 8) * 8) * sizeof(float);
  static bool attr_set = false;
  if (!attr_set) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                              hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)((kMaxFusedK + (kMaxFusedK >> 8) * 8) * sizeof(float)));
    (void)hipGetLastError();
    attr_set = true;
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)(N / 16)), dim3(kFT), lds, stream,
                     static_cast<const __half*>(x), (int)M, K, hs.f, hs.j, w, ws, (int)N,
                     static_cast<__half*>(y), static_cast<uint8_t*>(codes), as, sync);
  return hipGetLastError();
}

template <int BITS, int J = 0>
hipError_t dispatch_fused(const void* x, int64_t M, int K, HadSplit hs, const uint8_t* w,
                          const float* ws, int64_t N, void* y, void* codes, float* as,
                          int32_t* sync, hipStream_t stream) {
  if constexpr (J > 12) {
    return launch_fused_t<BITS, -1>(x, M, K, hs, w, ws, N, y, codes, as, sync, stream);
  } else {
    if (hs.f == 1 && hs.j == J)
      return launch_fused_t<BITS, J>(x, M, K, hs, w, ws, N, y, codes, as, sync, stream);
    return dispatch_fused<BITS, J + 1>(x, M, K, hs, w, ws, N, y, codes, as, sync, stream);
  }
}

}  // namespace

hipError_t launch_decode_fused(const void* x, int64_t M, int K, HadSplit hs, int bits,
                               const uint8_t* w_packed, const float* w_scales, int64_t N, void* y,
                               void* codes, float* a_scales, int32_t* sync, hipStream_t stream) {
  if (M == 0) return hipSuccess;
  if (bits == 4)
    return dispatch_fused<4>(x, M, K, hs, w_packed, w_scales, N, y, codes, a_scales, sync, stream);
  return dispatch_fused<8>(x, M, K, hs, w_packed, w_scales, N, y, codes, a_scales, sync, stream);
}

}  // namespace dptq
