// W4A4 / W4A8 GEMM with exact int32 accumulation and the dequant epilogue (gfx950).
//
//   acc[m,n] = sum_k a[m,k] * w[n,k]
//   y[m,n]   = fl16(fl32(fl32(fl32(acc) * a_s[m]) * w_s[n]))
//
// gfx950 has no 4-bit integer MFMA, so 4-bit codes are widened to int8 in
// registers: a packed dword v holding eight nibbles becomes
//   lo = (v << 4) & 0xF0F0F0F0   (the even-k nibbles, each times 16)
//   hi =  v       & 0xF0F0F0F0   (the odd-k nibbles, each times 16)
// i.e. every code lands in the high half of its byte as 16 * code (exact two's
// complement).  The MFMA therefore accumulates 256 * acc (4-bit x 4-bit) or
// 16 * acc (8-bit x 4-bit); |256 * acc| <= 256 * 64 * K < 2^31 for K <= 2^17,
// and an arithmetic shift recovers acc exactly.  The even/odd k permutation
// is applied identically to both operands (8-bit activations are permuted
// with v_perm), so the dot product is unchanged.
//
// The MFMA's A operand is the weight tile (rows = output channels n) and its
// B operand the activation tile (columns = tokens m).  Each lane then holds
// four consecutive n of one m, i.e. 8 contiguous bytes of a row of y.

#include "internal.h"

namespace dptq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t nib_lo(uint32_t v) { return (v << 4) & 0xF0F0F0F0u; }
__device__ __forceinline__ uint32_t nib_hi(uint32_t v) { return v & 0xF0F0F0F0u; }

// Even-k bytes of an 8-byte run (d0 = k0..3, d1 = k4..7): [k0, k2, k4, k6].
__device__ __forceinline__ uint32_t even_bytes(uint32_t d0, uint32_t d1) {
  return __builtin_amdgcn_perm(d1, d0, 0x06040200u);
}
// Odd-k bytes: [k1, k3, k5, k7].
__device__ __forceinline__ uint32_t odd_bytes(uint32_t d0, uint32_t d1) {
  return __builtin_amdgcn_perm(d1, d0, 0x07050301u);
}

// MFMA operand for one 64-k step from two packed 4-bit dwords (k 0..7, 8..15
// of this lane's 16-k slice).
__device__ __forceinline__ v4i op_from_nibbles(uint32_t v0, uint32_t v1) {
  v4i r;
  r.x = (int)nib_lo(v0);
  r.y = (int)nib_hi(v0);
  r.z = (int)nib_lo(v1);
  r.w = (int)nib_hi(v1);
  return r;
}
// Same k order from 16 int8 codes d0..d3 (k 0..15).
__device__ __forceinline__ v4i op_from_bytes(uint32_t d0, uint32_t d1, uint32_t d2, uint32_t d3) {
  v4i r;
  r.x = (int)even_bytes(d0, d1);
  r.y = (int)odd_bytes(d0, d1);
  r.z = (int)even_bytes(d2, d3);
  r.w = (int)odd_bytes(d2, d3);
  return r;
}

__device__ __forceinline__ v4i mfma(v4i a, v4i b, v4i c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

template <int BITS>
__device__ __forceinline__ int unscale(int v) { return BITS == 4 ? (v >> 8) : (v >> 4); }

// fl16(fl32(fl32(fl32(acc) * as) * ws)).  The empty asm pins t2 as an fp32
// value: without it the backend folds the last multiply and the fp16
// conversion into one mixed-precision FMA (a single rounding to fp16), which
// differs from the two roundings the epilogue is defined with.
__device__ __forceinline__ __half dequant(int acc, float as, float ws) {
  const float t0 = (float)acc;
  const float t1 = t0 * as;
  float t2 = t1 * ws;
  asm("" : "+v"(t2));
  return __float2half_rn(t2);
}

// ---------------------------------------------------------------------------
// Prefill: 256 (n) x 128 (m) tiles, 4 wavefronts of 128 (n) x 64 (m), K steps
// of 128 staged in double-buffered LDS.
// ---------------------------------------------------------------------------
constexpr int kBN = 256, kBM = 128, kBK = 128, kThreads = 256;

template <int BITS>
struct TileLds {
  static constexpr int kW = kBN * (kBK / 2);                     // bytes per W stage
  static constexpr int kA = kBM * (BITS == 4 ? kBK / 2 : kBK);   // bytes per A stage
  static constexpr int kStage = kW + kA;
};

__device__ __forceinline__ int xcd_remap(int bid, int total) {
  const int per = total >> 3, rem = total & 7;
  const int x = bid & 7, idx = bid >> 3;
  return x * per + (x < rem ? x : rem) + idx;
}

template <int BITS, bool ACC_OUT>
__global__ void __launch_bounds__(kThreads)
qgemm_prefill(const uint8_t* __restrict__ a_codes, const float* __restrict__ a_scales,
              const uint8_t* __restrict__ w_packed, const float* __restrict__ w_scales,
              int M, int N, int K, __half* __restrict__ y, int32_t* __restrict__ acc_out) {
  using L = TileLds<BITS>;
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * L::kStage];

  const int tiles_m = (M + kBM - 1) / kBM;
  const int tiles_n = N / kBN + (N % kBN ? 1 : 0);
  const int logical = xcd_remap(blockIdx.x, tiles_m * tiles_n);
  const int tm = logical % tiles_m, tn = logical / tiles_m;
  const int m0 = tm * kBM, n0 = tn * kBN;

  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int wn = wave & 1, wm = wave >> 1;
  const size_t wrow = (size_t)K / 2;
  const size_t arow = BITS == 4 ? (size_t)K / 2 : (size_t)K;

  constexpr int kWChunks = L::kW / 16 / kThreads;   // 4
  constexpr int kAChunks = L::kA / 16 / kThreads;   // 2 (A4) or 4 (A8)
  uint4 wreg[kWChunks], areg[kAChunks];

  auto gload = [&](int kk) {
#pragma unroll
    for (int i = 0; i < kWChunks; ++i) {
      const int q = t + kThreads * i, r = q >> 2, c = q & 3;
      const int n = n0 + r;
      wreg[i] = n < N ? *reinterpret_cast<const uint4*>(w_packed + (size_t)n * wrow + kk / 2 + c * 16)
                      : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < kAChunks; ++i) {
      const int q = t + kThreads * i;
      const int r = BITS == 4 ? (q >> 2) : (q >> 3);
      const int c = BITS == 4 ? (q & 3) : (q & 7);
      const int m = m0 + r;
      const size_t off = BITS == 4 ? (size_t)kk / 2 + c * 16 : (size_t)kk + c * 16;
      areg[i] = m < M ? *reinterpret_cast<const uint4*>(a_codes + (size_t)m * arow + off)
                      : make_uint4(0, 0, 0, 0);
    }
  };
  auto sstore = [&](int buf) {
    uint8_t* ws = smem + buf * L::kStage;
    uint8_t* as = ws + L::kW;
#pragma unroll
    for (int i = 0; i < kWChunks; ++i)
      *reinterpret_cast<uint4*>(ws + (t + kThreads * i) * 16) = wreg[i];
#pragma unroll
    for (int i = 0; i < kAChunks; ++i) {
      const int q = t + kThreads * i;
      int off;
      if (BITS == 4) {
        off = q * 16;
      } else {
        // [k half][row][16-byte column]: row r, chunk c -> half c & 1
        const int r = q >> 3, c = q & 7;
        off = (c & 1) * (kBM * 64) + r * 64 + (c >> 1) * 16;
      }
      *reinterpret_cast<uint4*>(as + off) = areg[i];
    }
  };

  v4i acc[8][4];
#pragma unroll
  for (int i = 0; i < 8; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = v4i{0, 0, 0, 0};

  const int steps = K / kBK;
  gload(0);
  sstore(0);
  __syncthreads();

  const int fr = lane & 15, fg = lane >> 4;
  for (int s = 0; s < steps; ++s) {
    const int buf = s & 1;
    if (s + 1 < steps) gload((s + 1) * kBK);
    const uint8_t* ws = smem + buf * L::kStage;
    const uint8_t* as = ws + L::kW;

    uint4 af[4];
    uint4 af2[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = wm * 64 + j * 16 + fr;
      if (BITS == 4) {
        af[j] = *reinterpret_cast<const uint4*>(as + r * 64 + fg * 16);
      } else {
        af[j] = *reinterpret_cast<const uint4*>(as + r * 64 + fg * 16);
        af2[j] = *reinterpret_cast<const uint4*>(as + kBM * 64 + r * 64 + fg * 16);
      }
    }
    uint4 wf[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int r = wn * 128 + i * 16 + fr;
      wf[i] = *reinterpret_cast<const uint4*>(ws + r * 64 + fg * 16);
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      v4i bop[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (BITS == 4) {
          bop[j] = ks == 0 ? op_from_nibbles(af[j].x, af[j].y) : op_from_nibbles(af[j].z, af[j].w);
        } else {
          bop[j] = ks == 0 ? op_from_bytes(af[j].x, af[j].y, af[j].z, af[j].w)
                           : op_from_bytes(af2[j].x, af2[j].y, af2[j].z, af2[j].w);
        }
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const v4i aop = ks == 0 ? op_from_nibbles(wf[i].x, wf[i].y) : op_from_nibbles(wf[i].z, wf[i].w);
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma(aop, bop[j], acc[i][j]);
      }
    }
    if (s + 1 < steps) sstore(buf ^ 1);
    __syncthreads();
  }

  // Epilogue: lane holds rows n = base + 4*fg + r (r = 0..3) of column m.
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int m = m0 + wm * 64 + j * 16 + fr;
    if (m >= M) continue;
    const float as = ACC_OUT ? 0.0f : a_scales[m];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int n = n0 + wn * 128 + i * 16 + fg * 4;
      if (n >= N) continue;
      const int c0 = unscale<BITS>(acc[i][j].x), c1 = unscale<BITS>(acc[i][j].y);
      const int c2 = unscale<BITS>(acc[i][j].z), c3 = unscale<BITS>(acc[i][j].w);
      if (ACC_OUT) {
        *reinterpret_cast<int4*>(acc_out + (size_t)m * N + n) = make_int4(c0, c1, c2, c3);
      } else {
        const float4 wsv = *reinterpret_cast<const float4*>(w_scales + n);
        const __half h0 = dequant(c0, as, wsv.x), h1 = dequant(c1, as, wsv.y);
        const __half h2 = dequant(c2, as, wsv.z), h3 = dequant(c3, as, wsv.w);
        uint2 pk;
        pk.x = (uint32_t)__half_as_ushort(h0) | ((uint32_t)__half_as_ushort(h1) << 16);
        pk.y = (uint32_t)__half_as_ushort(h2) | ((uint32_t)__half_as_ushort(h3) << 16);
        *reinterpret_cast<uint2*>(y + (size_t)m * N + n) = pk;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Decode (M <= 16): one workgroup per 16 output channels; its 8 wavefronts
// split K, stream the weight rows once with 16-byte loads, and the int32
// partial tiles are summed exactly in LDS.
// ---------------------------------------------------------------------------
constexpr int kDecWaves = 8;
constexpr int kDecBatch = 4;

template <int BITS, bool ACC_OUT>
__global__ void __launch_bounds__(kDecWaves * 64)
qgemm_decode(const uint8_t* __restrict__ a_codes, const float* __restrict__ a_scales,
             const uint8_t* __restrict__ w_packed, const float* __restrict__ w_scales,
             int M, int N, int K, __half* __restrict__ y, int32_t* __restrict__ acc_out) {
  __shared__ v4i part[kDecWaves][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n0 = blockIdx.x * 16;
  const int fr = lane & 15, fg = lane >> 4;
  const int nck = K / 128;
  const int c_begin = (int)((long)nck * wave / kDecWaves);
  const int c_end = (int)((long)nck * (wave + 1) / kDecWaves);
  const bool mvalid = fr < M;

  const uint8_t* wp = w_packed + (size_t)(n0 + fr) * (K / 2) + fg * 16;
  const size_t arow = BITS == 4 ? (size_t)K / 2 : (size_t)K;
  const uint8_t* ap = a_codes + (size_t)(mvalid ? fr : 0) * arow + (BITS == 4 ? fg * 16 : fg * 32);

  v4i acc = v4i{0, 0, 0, 0};
  for (int c = c_begin; c < c_end; c += kDecBatch) {
    uint4 wv[kDecBatch], av[kDecBatch], av2[kDecBatch];
#pragma unroll
    for (int b = 0; b < kDecBatch; ++b) {
      const int ck = c + b;
      const bool ok = ck < c_end;
      wv[b] = ok ? *reinterpret_cast<const uint4*>(wp + (size_t)ck * 64) : make_uint4(0, 0, 0, 0);
      if (BITS == 4) {
        av[b] = (ok && mvalid) ? *reinterpret_cast<const uint4*>(ap + (size_t)ck * 64)
                               : make_uint4(0, 0, 0, 0);
      } else {
        av[b] = (ok && mvalid) ? *reinterpret_cast<const uint4*>(ap + (size_t)ck * 128)
                               : make_uint4(0, 0, 0, 0);
        av2[b] = (ok && mvalid) ? *reinterpret_cast<const uint4*>(ap + (size_t)ck * 128 + 16)
                                : make_uint4(0, 0, 0, 0);
      }
    }
#pragma unroll
    for (int b = 0; b < kDecBatch; ++b) {
      v4i b0, b1;
      if (BITS == 4) {
        b0 = op_from_nibbles(av[b].x, av[b].y);
        b1 = op_from_nibbles(av[b].z, av[b].w);
      } else {
        b0 = op_from_bytes(av[b].x, av[b].y, av[b].z, av[b].w);
        b1 = op_from_bytes(av2[b].x, av2[b].y, av2[b].z, av2[b].w);
      }
      acc = mfma(op_from_nibbles(wv[b].x, wv[b].y), b0, acc);
      acc = mfma(op_from_nibbles(wv[b].z, wv[b].w), b1, acc);
    }
  }
  part[wave][lane] = acc;
  __syncthreads();
  if (wave != 0) return;
  v4i tot = part[0][lane];
#pragma unroll
  for (int w = 1; w < kDecWaves; ++w) {
    const v4i p = part[w][lane];
    tot.x += p.x; tot.y += p.y; tot.z += p.z; tot.w += p.w;
  }
  if (!mvalid) return;
  const int m = fr, n = n0 + fg * 4;
  const int c0 = unscale<BITS>(tot.x), c1 = unscale<BITS>(tot.y);
  const int c2 = unscale<BITS>(tot.z), c3 = unscale<BITS>(tot.w);
  if (ACC_OUT) {
    *reinterpret_cast<int4*>(acc_out + (size_t)m * N + n) = make_int4(c0, c1, c2, c3);
  } else {
    const float as = a_scales[m];
    const float4 wsv = *reinterpret_cast<const float4*>(w_scales + n);
    const __half h0 = dequant(c0, as, wsv.x), h1 = dequant(c1, as, wsv.y);
    const __half h2 = dequant(c2, as, wsv.z), h3 = dequant(c3, as, wsv.w);
    uint2 pk;
    pk.x = (uint32_t)__half_as_ushort(h0) | ((uint32_t)__half_as_ushort(h1) << 16);
    pk.y = (uint32_t)__half_as_ushort(h2) | ((uint32_t)__half_as_ushort(h3) << 16);
    *reinterpret_cast<uint2*>(y + (size_t)m * N + n) = pk;
  }
}

template <int BITS, bool ACC_OUT>
hipError_t launch_t(const uint8_t* a, const float* as, int64_t M, int K,
                    const uint8_t* w, const float* ws, int64_t N, __half* y,
                    int32_t* acc, hipStream_t stream) {
  if (M == 0) return hipSuccess;
  if (M <= 16) {
    hipLaunchKernelGGL((qgemm_decode<BITS, ACC_OUT>), dim3((unsigned)(N / 16)),
                       dim3(kDecWaves * 64), 0, stream, a, as, w, ws, (int)M, (int)N, K, y, acc);
  } else {
    const int64_t tiles = ((M + kBM - 1) / kBM) * ((N + kBN - 1) / kBN);
    hipLaunchKernelGGL((qgemm_prefill<BITS, ACC_OUT>), dim3((unsigned)tiles), dim3(kThreads), 0,
                       stream, a, as, w, ws, (int)M, (int)N, K, y, acc);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_qlinear(const void* codes, const float* a_scales, int64_t M, int K,
                          int bits, const uint8_t* w_packed, const float* w_scales,
                          int64_t N, void* y, int32_t* out_acc, hipStream_t stream) {
  const uint8_t* a = static_cast<const uint8_t*>(codes);
  __half* yh = static_cast<__half*>(y);
  if (out_acc) {
    if (bits == 4)
      return launch_t<4, true>(a, a_scales, M, K, w_packed, w_scales, N, yh, out_acc, stream);
    return launch_t<8, true>(a, a_scales, M, K, w_packed, w_scales, N, yh, out_acc, stream);
  }
  if (bits == 4)
    return launch_t<4, false>(a, a_scales, M, K, w_packed, w_scales, N, yh, nullptr, stream);
  return launch_t<8, false>(a, a_scales, M, K, w_packed, w_scales, N, yh, nullptr, stream);
}

}  // namespace dptq
