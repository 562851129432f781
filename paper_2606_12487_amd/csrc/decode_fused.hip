// Decode-shape quantized linear in one launch: rotate + quantize the M <= 16
// token rows and the weight-streaming GEMM with its dequant epilogue.
//
// The grid is the decode GEMM's: one workgroup of 512 threads per 16 output
// channels, whose 8 wavefronts split K.  Each workgroup starts the loads of
// its first weight chunks, rotates and quantizes all M rows itself into LDS,
// and runs the GEMM with the codes read from LDS.  The rotation is the
// rotate+quantize kernels' arithmetic: the row widened to fp32, butterflies
// over index bits 0, 1, 2, ... in that order, then for h = 28 * 2^j the dense
// 28-point stage summed sequentially over the slow index; the scale is
// fl32(absmax / qmax) and the codes are the correctly rounded quotients
// rounded half to even.  Every workgroup repeats the rotation of the few
// decode rows; that costs less than a second launch and a round trip of the
// codes through HBM, and no workgroup ever waits for another.  Workgroup 0
// also stores the codes and scales when the caller asks for them.

#include "internal.h"
#include "quant_device.h"

namespace dptq {
namespace {

using namespace qd;

typedef int v4i_t __attribute__((ext_vector_type(4)));

constexpr int kFT = 512;          // threads per workgroup
constexpr int kFWaves = kFT / 64;
constexpr int kFBatch = 4;        // 128-k chunks in flight per wavefront

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

// Codes of 8 consecutive elements stored at element e of a row: to the LDS
// row, and to the global row when there is one.
template <int BITS>
__device__ __forceinline__ void f_store8(const uint32_t* bt, int e, uint8_t* cl, uint8_t* cg) {
  if (BITS == 4) {
    const uint32_t v = pack_nibbles(bt);
    *reinterpret_cast<uint32_t*>(cl + e / 2) = v;
    if (cg) *reinterpret_cast<uint32_t*>(cg + e / 2) = v;
  } else {
    const uint2 v = make_uint2(low_bytes(bt[0], bt[1], bt[2], bt[3]), low_bytes(bt[4], bt[5], bt[6], bt[7]));
    *reinterpret_cast<uint2*>(cl + e) = v;
    if (cg) *reinterpret_cast<uint2*>(cg + e) = v;
  }
}

// Rotate + quantize row m0 and, with two rows in flight (!SPLIT), m0 + 1.
// Two rows: threads 256 * half + r (r < 256) rotate row m0 + half in its own
// staging.  One row (SPLIT): both groups of 256 work on it, splitting its
// segments by parity and its 28-point columns.  The row is then quantized
// into the LDS code rows (and the caller's buffers when given).  pre with
// use_pre: this thread's first NPRE segments of its work, loaded by the
// caller.
template <int BITS, int JP, bool F28, bool SPLIT, int NPRE>
__device__ __forceinline__ void rows_fast(const __half* __restrict__ x, int M, int K, int J,
                                          int m0, bool use_pre, const uint4 (&pre)[2 * NPRE],
                                          float* rot, float* red, uint8_t* cl, int cstride,
                                          float* as_lds, uint8_t* __restrict__ codes_out,
                                          float* __restrict__ scales_out) {
  const int t = threadIdx.x, half = t >> 8, r = t & 255;
  constexpr bool split = SPLIT;
  const int m = split ? m0 : m0 + half;
  const bool act = m < M;
  const int nseg = (K + kSeg - 1) / kSeg;
  float* rh = split ? rot : rot + half * nseg * kSegFloats;
  const RowSplit sp = split ? RowSplit{half, 2, t, kFT} : RowSplit{0, 1, r, 256};
  const int b1 = seg_off(16 * r);
  const __half* xr = x + (size_t)m * K;
  float tmax = 0.0f, unused = 0.0f;
  rotate_row_segments<JP, F28, false, NPRE>(xr, K, J, act, r, sp, use_pre, pre, rh, tmax, unused);
  // Row maximum: waves 0-3 hold row m0, waves 4-7 row m0 + 1 (or row m0 too).
  tmax = wave_max_nonneg(tmax);
  if ((t & 63) == 0) red[t >> 6] = tmax;
  __syncthreads();
  const float* rr = red + (split ? 0 : 4 * half);
  float amax = fmaxf(fmaxf(rr[0], rr[1]), fmaxf(rr[2], rr[3]));
  if (split) amax = fmaxf(amax, fmaxf(fmaxf(red[4], red[5]), fmaxf(red[6], red[7])));
  constexpr float qmax = (float)((1 << (BITS - 1)) - 1);
  const float sc = amax / qmax;                 // IEEE division
  const float rc = sc != 0.0f ? 1.0f / sc : 0.0f;
  if (act) {
    if (t == 0 || (!split && r == 0)) {
      as_lds[m] = sc;
      if (scales_out) scales_out[m] = sc;
    }
    uint8_t* crow = cl + (size_t)m * cstride;
    uint8_t* grow = codes_out ? codes_out + (size_t)m * (BITS == 4 ? K / 2 : K) : nullptr;
    for (int sg = sp.sg0; sg < nseg; sg += sp.sgstep) {
      const int e = sg * kSeg + 16 * r;
      if (e >= K) continue;
      const float* sl = rh + sg * kSegFloats + b1;
      uint32_t bt[16];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 w4 = *reinterpret_cast<const float4*>(sl + 4 * q);
        bt[4 * q] = round_bits(w4.x, sc, rc);
        bt[4 * q + 1] = round_bits(w4.y, sc, rc);
        bt[4 * q + 2] = round_bits(w4.z, sc, rc);
        bt[4 * q + 3] = round_bits(w4.w, sc, rc);
      }
      f_store8<BITS>(bt, e, crow, grow);
      f_store8<BITS>(bt + 8, e + 8, crow, grow);
    }
  }
  __syncthreads();   // the staging and red[] are reused by the next rows
}

// h = F * 2^J with JP = min(J, 12), F28 = (F == 28); SPLIT: one row at a time
// on all 512 threads, else two rows in flight.  Dynamic LDS: the M code rows
// (row stride cstride = K * BITS / 8 + 16 bytes), then the fp32 staging of one
// row (SPLIT) or two.
template <int BITS, int JP, bool F28, bool SPLIT>
__global__ void __launch_bounds__(kFT) __attribute__((amdgpu_waves_per_eu(F28 ? 2 : 6)))
qdecode_fused(const __half* __restrict__ x, int M, int K, int J,
              const uint8_t* __restrict__ w_packed, const float* __restrict__ w_scales, int N,
              __half* __restrict__ y, uint8_t* __restrict__ codes_out, float* __restrict__ scales_out) {
  extern __shared__ __align__(16) uint8_t dyn[];
  __shared__ float red[kFWaves];
  __shared__ float as_lds[16];
  __shared__ v4i_t part[kFWaves][64];
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);   // uniform: scalar chunk bounds
  __builtin_assume(M >= 1 && M <= 16);   // the launcher's range
  const int cstride = K * BITS / 8 + 16;
  uint8_t* cl = dyn;
  float* rot = reinterpret_cast<float*>(dyn + (size_t)M * cstride);
  uint8_t* cg = blockIdx.x == 0 ? codes_out : nullptr;
  float* sgl = blockIdx.x == 0 ? scales_out : nullptr;

  // The GEMM's geometry: the weight slice of 16 output channels, K split
  // over the wavefronts in 128-k chunks.
  const int n0 = blockIdx.x * 16;
  const int fr = lane & 15, fg = lane >> 4;
  const int nck = K / 128;
  const int c_begin = (int)((long)nck * wave / kFWaves);
  const int c_end = (int)((long)nck * (wave + 1) / kFWaves);
  const bool mvalid = fr < M;
  const uint8_t* wp = w_packed + (size_t)(n0 + fr) * (K / 2) + fg * 16;

  // This thread's activation segments (the first kPreSeg of its first row),
  // then its first weights: the rotation waits for the activations alone while
  // the weights stay in flight.  Loads are unconditional (addresses clamped
  // into the buffers, values past the range zeroed at use), so no branch
  // around a load forces an early wait.  The 28-point instances, whose rows
  // are long, preload four segments.
  constexpr int kPreSeg = F28 ? 4 : 1;
  uint4 pre[2 * kPreSeg];
  {
    // The segments rows_fast gives this thread in its first call: row half
    // from segment 0 (two rows in flight), or row 0 from segment half in
    // steps of two (one row, both groups on it).
    const int half = t >> 8, r = t & 255;
    const int row = SPLIT ? 0 : half, sg0 = SPLIT ? half : 0, sgstep = SPLIT ? 2 : 1;
    const bool ok = row < M;
#pragma unroll
    for (int i = 0; i < kPreSeg; ++i) {
      const int e = (sg0 + i * sgstep) * kSeg + 16 * r;
      const __half* xp = ok && e < K ? x + (size_t)row * K + e : x;
#pragma unroll
      for (int h2 = 0; h2 < 2; ++h2) pre[2 * i + h2] = *reinterpret_cast<const uint4*>(xp + 8 * h2);
    }
    __builtin_amdgcn_sched_barrier(0);   // the activation loads go out first
  }
  const int last = nck - 1;
  // Weights prefetched before the rotation: one batch, or for the 28-point
  // stage (whose rotation takes longest) up to 16 chunks, the whole slice of
  // a wavefront at K <= 16384.  Raw loads; values past the wavefront's
  // chunks are zeroed at use.
  constexpr int kPF = F28 ? 16 : kFBatch;
  uint4 wpre[kPF];
#pragma unroll
  for (int k = 0; k < kPF; ++k)
    wpre[k] = *reinterpret_cast<const uint4*>(wp + (size_t)min(c_begin + k, last) * 64);
  __builtin_amdgcn_sched_barrier(0);     // ... then the weights, then the rotation

  for (int m0 = 0; m0 < M; m0 += SPLIT ? 1 : 2)
    rows_fast<BITS, JP, F28, SPLIT, kPreSeg>(x, M, K, J, m0, m0 == 0, pre, rot, red, cl, cstride,
                                             as_lds, cg, sgl);

  const uint8_t* ap = cl + (size_t)(mvalid ? fr : 0) * cstride + (BITS == 4 ? fg * 16 : fg * 32);
  v4i_t acc = v4i_t{0, 0, 0, 0};
  // Chunk ck (c_begin <= ck, and some chunk of this wavefront exists) with
  // its weights w; the codes come from LDS chunk by chunk.
  auto consume = [&](int ck, uint4 w) __attribute__((always_inline)) {
    const bool in = ck < c_end;
    const bool ok = in && mvalid;
    const int cc = min(ck, c_end - 1);
    w = keep_or_zero(in, w);
    v4i_t b0, b1;
    if (BITS == 4) {
      const uint4 u = keep_or_zero(ok, *reinterpret_cast<const uint4*>(ap + (size_t)cc * 64));
      b0 = f_op_nibbles(u.x, u.y);
      b1 = f_op_nibbles(u.z, u.w);
    } else {
      const uint4 u = keep_or_zero(ok, *reinterpret_cast<const uint4*>(ap + (size_t)cc * 128));
      const uint4 u2 = keep_or_zero(ok, *reinterpret_cast<const uint4*>(ap + (size_t)cc * 128 + 16));
      b0 = f_op_bytes(u.x, u.y, u.z, u.w);
      b1 = f_op_bytes(u2.x, u2.y, u2.z, u2.w);
    }
    acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(f_op_nibbles(w.x, w.y), b0, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(f_op_nibbles(w.z, w.w), b1, acc, 0, 0, 0);
  };
  if (c_begin < c_end) {
#pragma unroll
    for (int k = 0; k < kPF; ++k) consume(c_begin + k, wpre[k]);
  }
  for (int c = c_begin + kPF; c < c_end; c += kFBatch) {
    uint4 wv[kFBatch];
#pragma unroll
    for (int k = 0; k < kFBatch; ++k)
      wv[k] = *reinterpret_cast<const uint4*>(wp + (size_t)min(c + k, last) * 64);
#pragma unroll
    for (int k = 0; k < kFBatch; ++k) consume(c + k, wv[k]);
  }
  part[wave][lane] = acc;
  __syncthreads();
  if (wave != 0) return;
  v4i_t tot = part[0][lane];
#pragma unroll
  for (int w = 1; w < kFWaves; ++w) {
    const v4i_t p = part[w][lane];
    tot.x += p.x; tot.y += p.y; tot.z += p.z; tot.w += p.w;
  }
  if (!mvalid) return;
  const int m = fr, n = n0 + fg * 4;
  const float as = as_lds[m];
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

// Staging of one row: whole 4096-element segments.
int64_t staging_bytes(int K) { return (int64_t)((K + kSeg - 1) / kSeg) * kSegFloats * 4; }

int64_t code_rows_bytes(int64_t M, int K, int bits) { return M * ((int64_t)K * bits / 8 + 16); }

template <int BITS, int JP, bool F28, bool SPLIT>
hipError_t launch_fused_split(const void* x, int64_t M, int K, HadSplit hs, const uint8_t* w,
                              const float* ws, int64_t N, void* y, void* codes, float* as,
                              size_t lds, hipStream_t stream) {
  auto kern = qdecode_fused<BITS, JP, F28, SPLIT>;
  static bool attr_set = false;
  if (!attr_set) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                              hipFuncAttributeMaxDynamicSharedMemorySize, (int)kFusedLdsMax);
    (void)hipGetLastError();
    attr_set = true;
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)(N / 16)), dim3(kFT), lds, stream,
                     static_cast<const __half*>(x), (int)M, K, hs.j, w, ws, (int)N,
                     static_cast<__half*>(y), static_cast<uint8_t*>(codes), as);
  return hipGetLastError();
}

// Two rows in flight when M >= 2 and both stagings fit; else one row at a
// time on all threads.
template <int BITS, int JP, bool F28>
hipError_t launch_fused_t(const void* x, int64_t M, int K, HadSplit hs, const uint8_t* w,
                          const float* ws, int64_t N, void* y, void* codes, float* as,
                          hipStream_t stream) {
  const int64_t rows = code_rows_bytes(M, K, BITS), stage = staging_bytes(K);
  if (M >= 2 && rows + 2 * stage <= kFusedLdsMax)
    return launch_fused_split<BITS, JP, F28, false>(x, M, K, hs, w, ws, N, y, codes, as,
                                                    (size_t)(rows + 2 * stage), stream);
  return launch_fused_split<BITS, JP, F28, true>(x, M, K, hs, w, ws, N, y, codes, as,
                                                 (size_t)(rows + stage), stream);
}

// h = 28 * 2^j has j <= 10 (h <= the longest row); h = 2^j goes to JP = min(j, 12).
template <int BITS, int JP = 0>
hipError_t dispatch_fused(const void* x, int64_t M, int K, HadSplit hs, const uint8_t* w,
                          const float* ws, int64_t N, void* y, void* codes, float* as,
                          hipStream_t stream) {
  if constexpr (JP == 12) {
    return launch_fused_t<BITS, 12, false>(x, M, K, hs, w, ws, N, y, codes, as, stream);
  } else {
    if (hs.j == JP) {
      if constexpr (JP <= 10) {
        if (hs.f == 28) return launch_fused_t<BITS, JP, true>(x, M, K, hs, w, ws, N, y, codes, as, stream);
      }
      return launch_fused_t<BITS, JP, false>(x, M, K, hs, w, ws, N, y, codes, as, stream);
    }
    return dispatch_fused<BITS, JP + 1>(x, M, K, hs, w, ws, N, y, codes, as, stream);
  }
}

}  // namespace

int64_t decode_fused_lds(int64_t M, int K, HadSplit hs, int bits) {
  (void)hs;
  return code_rows_bytes(M, K, bits) + staging_bytes(K);
}

// Measured on decode shapes: the repeated rotation costs less than the
// second launch for one row of K <= 16384 with h = 2^j <= 8192, and for two
// rows of K <= 12288 with h = 2^j <= 4096; in every case for at most 1024
// workgroups (about three per compute unit, so each rotates once).  More
// rows, longer rows or more workgroups make it the slower path, and so does
// h = 28 * 2^j since the two-launch rotation got faster (15.1 against
// 15.7 us for one row of 14336, h = 28 x 512, N = 4096).
bool decode_one_launch_wins(int64_t M, int K, HadSplit hs, int bits, int64_t N) {
  if (N > 16384 || decode_fused_lds(M, K, hs, bits) > kFusedLdsMax) return false;
  if (M == 1) return hs.f == 1 && hs.j <= 13 && K <= 16384;
  return M == 2 && hs.f == 1 && hs.j <= 12 && K <= 12288;
}

hipError_t launch_decode_fused(const void* x, int64_t M, int K, HadSplit hs, int bits,
                               const uint8_t* w_packed, const float* w_scales, int64_t N, void* y,
                               void* codes, float* a_scales, int mode, hipStream_t stream) {
  if (M == 0) return hipSuccess;
  if (mode == kDecodeAuto)
    mode = decode_one_launch_wins(M, K, hs, bits, N) ? kDecodeOneLaunch : kDecodeTwoLaunches;
  if (mode == kDecodeTwoLaunches) {
    hipError_t e = launch_rotate_quant_f16(x, M, K, hs, bits, codes, a_scales, stream);
    if (e != hipSuccess) return e;
    return launch_qlinear(codes, a_scales, M, K, bits, w_packed, w_scales, N, y, nullptr, kGemmDecode,
                          stream);
  }
  if (bits == 4)
    return dispatch_fused<4>(x, M, K, hs, w_packed, w_scales, N, y, codes, a_scales, stream);
  return dispatch_fused<8>(x, M, K, hs, w_packed, w_scales, N, y, codes, a_scales, stream);
}

}  // namespace dptq
