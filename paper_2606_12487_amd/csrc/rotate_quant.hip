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
// Two kernels: a register-phase kernel for power-of-two sizes up to 4096 (the
// sizes of every LLaMA projection except the largest ones), and a general
// kernel for the others (28 * 2^j, and 2^j above 4096).  Both are limited by
// vector ALU issue, not by memory: the fp32 butterflies alone are log2(h)
// instructions per element, and packed fp32 arithmetic is not used.
//
// Quotient: t = fl32(y / s) is formed as q = y * r, e = fma(-q, s, y),
// t = fma(e, r, q) with r = fl32(1 / s) (Markstein's correction, one
// correctly rounded reciprocal per row), which returns the correctly rounded
// quotient for every input reachable here.

#include "internal.h"
#include "quant_device.h"

namespace dptq {
namespace {

using namespace qd;

constexpr int kThreads = 256;
// Batches above this many rows take the segmented kernel for large and
// 28 * 2^j Hadamard sizes (0: never).
constexpr int64_t kSegRows = 64;

// LDS index of row element i in the general kernel: PD = 0 pads 8 floats
// after every 256, PD = 1 pads 4 after every 32 (more room, fewer bank
// conflicts for the 28 * 2^j passes at j = 9 and 10, where rows are at most
// 28672 long).
template <int PD>
__host__ __device__ constexpr int lidx(int i) {
  return PD == 0 ? i + ((i >> 8) << 3) : i + ((i >> 5) << 2);
}
template <int F, int J>
constexpr int pad_of() {
  return (F == 28 && (J == 9 || J == 10)) ? 1 : 0;
}

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

// Randomized signs (bit set = negate) of N consecutive elements, from their
// bitmask bits m (bit r for element r): a sign-bit flip, exact.
template <int N>
__device__ __forceinline__ void apply_sign_bits(float* v, uint32_t m) {
#pragma unroll
  for (int r = 0; r < N; ++r) v[r] = __uint_as_float(__float_as_uint(v[r]) ^ (((m >> r) & 1u) << 31));
}

__device__ __forceinline__ float absmax8(const float* v, float m) {
#pragma unroll
  for (int k = 0; k < 8; ++k) m = fmaxf(m, fabsf(v[k]));
  return m;
}


// lidx(b | o) = lidx(b) + lidx(o) whenever b and o share no set bit (the
// shift that forms the padding distributes over a disjoint OR), so an element
// at a constant bit pattern o from a base b is a constant offset from lidx(b)
// in LDS, which the LDS instructions take as an immediate.

// One pass over index bits [S, S+G): each work item gathers the 2^G elements
// that differ only in those bits (base with those bits clear, plus k << S),
// applies the butterflies, and writes back.
template <int G, int S, int T, int PD>
__device__ __forceinline__ float pass_bits(float* lds, int K, bool last, float tmax) {
  const int groups = K >> G;
  constexpr int low_mask = (1 << S) - 1;
  for (int g = threadIdx.x; g < groups; g += T) {
    const int base = (g & low_mask) | ((g >> S) << (S + G));
    const float* src = lds + lidx<PD>(base);
    float v[1 << G];
#pragma unroll
    for (int k = 0; k < (1 << G); ++k) v[k] = src[lidx<PD>(k << S)];
    butterflies<G>(v, 0, G);
    float* dst = lds + lidx<PD>(base);
#pragma unroll
    for (int k = 0; k < (1 << G); ++k) {
      dst[lidx<PD>(k << S)] = v[k];
      if (last) tmax = fmaxf(tmax, fabsf(v[k]));
    }
  }
  return tmax;
}

// Element a (slow index) of a 28-point column at base: lidx(base + a p).
// With p = 2^J at least the padding period (256 or 32) the padding splits
// (base's fast part lies below bit J, and a p adds whole periods), so it is
// lidx(base) plus the constant a lidx(p); the column then reads from two
// bases, 14 rows apart, so that every offset fits the LDS instructions'
// immediate.  Below that it is computed per element.
template <int J, int PD>
struct Col28 {
  static constexpr int kP = 1 << J;
  static constexpr bool kSplit = J >= (PD == 0 ? 8 : 5);
  static constexpr int kStep = lidx<PD>(kP);
  float* b0;
  float* b1;
  int base;
  __device__ __forceinline__ Col28(float* lds, int base_) : base(base_) {
    if constexpr (kSplit) {
      b0 = lds + lidx<PD>(base_);
      b1 = b0 + 14 * kStep;
    } else {
      b0 = lds;
      b1 = lds;
    }
  }
  __device__ __forceinline__ float& at(int a) const {
    if constexpr (kSplit) return a < 14 ? b0[a * kStep] : b1[(a - 14) * kStep];
    else return b0[lidx<PD>(base + a * kP)];
  }
};

// Dense 28-point stage: y[b*p + c] = sum over a = 0..27 (in order) of
// H28[a][b] * z[a*p + c], per block and fast index c.  Outputs B0 .. B0+NB-1
// of one column from its 28 inputs z (shared partial sums, h28_column).
template <int NB, int B0, int J, int PD>
__device__ __forceinline__ float dense28(const Col28<J, PD>& col, const float* z, float tmax) {
  h28_column<B0, NB>(z, [&](int b, float acc) __attribute__((always_inline)) {
    col.at(B0 + b) = acc;
    tmax = fmaxf(tmax, fabsf(acc));
  });
  return tmax;
}

template <int T, int J, int PD>
__device__ __forceinline__ float pass_28(float* lds, int K, float tmax) {
  constexpr int p = 1 << J;
  const int cols = K / 28;
  if (2 * cols <= T && cols % 64 == 0) {
    // Two threads per column (wavefront-uniform halves), each writing 14 of
    // its outputs; every input is read before any output is written.
    const int t = threadIdx.x;
    const bool active = t < 2 * cols;
    const int c = t % cols, half = t / cols;
    const Col28<J, PD> col(lds, (c >> J) * 28 * p + (c & (p - 1)));
    float z[28];
    if (active) {
#pragma unroll
      for (int a = 0; a < 28; ++a) z[a] = col.at(a);
    }
    __syncthreads();
    if (active) {
      if (half == 0) tmax = dense28<14, 0, J, PD>(col, z, tmax);
      else tmax = dense28<14, 14, J, PD>(col, z, tmax);
    }
    return tmax;
  }
  for (int c = threadIdx.x; c < cols; c += T) {
    const Col28<J, PD> col(lds, (c >> J) * 28 * p + (c & (p - 1)));
    float z[28];
#pragma unroll
    for (int a = 0; a < 28; ++a) z[a] = col.at(a);
    tmax = dense28<28, 0, J, PD>(col, z, tmax);
  }
  return tmax;
}

// FP6 block-layout output (4-bit codes as e2m3 values c / 2; the layout is
// described with the FP6 GEMM).  Row m's codes k = 128 kb + 64 g + 32 s + j
// are field j of the MFMA operand of lane 32 g + (m & 31) in half s of block
// (kb, m / 32); its 8-byte plane c lies at byte 512 c + 8 lane of the half.
typedef _Float16 f6_v32h __attribute__((ext_vector_type(32)));
typedef int f6_v6i __attribute__((ext_vector_type(6)));

// Byte offset of the half-block slot (plane 0) holding code k of row m.
__device__ __forceinline__ size_t fp6_slot(int m, int k, int mblk) {
  const int kb = k >> 7, g = (k >> 6) & 1, s = (k >> 5) & 1;
  return ((size_t)kb * mblk + (m >> 5)) * 3072 + 1536 * s + 8 * (32 * g + (m & 31));
}
// c / 2 from round_bits' output word (c = the code in its low mantissa
// bits): exact, (t + 1.5 * 2^23) / 2 - 0.75 * 2^23.
__device__ __forceinline__ float half_code(uint32_t bits) {
  return __builtin_fmaf(__uint_as_float(bits), 0.5f, -6291456.0f);
}
// Fields 0 .. N-1 of an operand from N codes (N = 16 or 32); the hardware
// conversion packs field i at bit 6 i, exactly the layout's order, and the
// values c / 2 are exact in e2m3.
template <int N>
__device__ __forceinline__ f6_v6i fp6_fields(const uint32_t* bt) {
  f6_v32h h = {};
#pragma unroll
  for (int i = 0; i < N; ++i) h[i] = (_Float16)half_code(bt[i]);
  return __builtin_amdgcn_cvt_scalef32_pk32_fp6_f16(h, 1.0f);
}
// Workgroup b's row when the output is the FP6 block layout: the rows of the
// eight XCDs are contiguous ranges, so the rows of one 32-row block (whose
// operands share cache lines) are written through one L2.
__device__ __forceinline__ int fp6_row(int b, int mp) {
  const int per = mp >> 3;   // mp is a multiple of 32
  return (b & 7) * per + (b >> 3);
}

// Statistics mode (residual-dynamics calibration, Section 3.1): the kernels
// rotate and quantize u = fl32(x + dx) and, instead of codes, write per row
// the Jump Ratio ||dx|| / (||x|| + eps) and the historical SNR
// 10 log10(||x||^2 / (||Q(u) - u||^2 + eps)), where ||Q(u) - u||^2 is the
// rotated-space error energy over h (Eq. 16 with the unnormalized B_h).
struct StatsArgs {
  const __half* dx;   // [M, K] updates (nullptr in codes mode)
  float* jr;          // [M]
  float* snr;         // [M], dB
  float eps;
};

// Eight elements of x and dx: v = fl32(x + dx), and the squared norms.
__device__ __forceinline__ void load8_sum(const __half* x, const __half* d, float* v,
                                          float& sx, float& sd) {
  float b[8];
  load8(x, v);
  load8(d, b);
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    sx = __builtin_fmaf(v[k], v[k], sx);
    sd = __builtin_fmaf(b[k], b[k], sd);
    v[k] = v[k] + b[k];
  }
}

// Sum over the workgroup, in a fixed order (wavefront butterflies, then the
// wavefronts in order); every thread gets the result.
template <int T>
__device__ __forceinline__ float3 block_sum3(float3 a, float (*red)[3]) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    a.x += __shfl_xor(a.x, off);
    a.y += __shfl_xor(a.y, off);
    a.z += __shfl_xor(a.z, off);
  }
  __syncthreads();
  if ((threadIdx.x & 63) == 0) {
    red[threadIdx.x >> 6][0] = a.x;
    red[threadIdx.x >> 6][1] = a.y;
    red[threadIdx.x >> 6][2] = a.z;
  }
  __syncthreads();
  float3 r = make_float3(red[0][0], red[0][1], red[0][2]);
#pragma unroll
  for (int w = 1; w < T / 64; ++w) {
    r.x += red[w][0];
    r.y += red[w][1];
    r.z += red[w][2];
  }
  return r;
}

// Error energy of quantizing v[0..n) with scale s (reciprocal r).
template <int N>
__device__ __forceinline__ float quant_error_energy(const float* v, float s, float r, float ee) {
#pragma unroll
  for (int k = 0; k < N; ++k) {
    const int code = (int)(round_bits(v[k], s, r) - 0x4B400000u);
    const float e = __builtin_fmaf((float)code, s, -v[k]);
    ee = __builtin_fmaf(e, e, ee);
  }
  return ee;
}

// JR and SNR of one row from ||x||^2, ||dx||^2 and the rotated error energy.
__device__ __forceinline__ void write_stats(const StatsArgs& st, int row, float3 sums, int h) {
  const double sx = sums.x, sd = sums.y, ee = sums.z;
  st.jr[row] = (float)(sqrt(sd) / (sqrt(sx) + (double)st.eps));
  st.snr[row] = (float)(10.0 * log10(sx / (ee / h + (double)st.eps)));
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

template <typename Tin, int BITS, bool WEIGHT, int F, int J, int T, bool STATS, bool FP6>
__global__ void __launch_bounds__(T)
rotate_quant_kernel(const Tin* __restrict__ x, int M, int K, const uint8_t* __restrict__ signs,
                    uint8_t* __restrict__ codes, float* __restrict__ scales, StatsArgs st,
                    int touch_stride) {
  extern __shared__ float lds[];
  __shared__ float red[T / 64];
  __shared__ float red3[T / 64][3];
  float3 sums = make_float3(0.0f, 0.0f, 0.0f);
  using P = Plan<J>;
  constexpr int PD = pad_of<F, J>();
  static_assert(P::np <= 3, "pass plan too long");
  static_assert(!FP6 || BITS == 4, "FP6 output holds 4-bit codes");
  const int mblk = (M + 31) >> 5;
  const int row = FP6 ? fp6_row(blockIdx.x, mblk * 32) : (int)blockIdx.x;
  // The row of workgroup blockIdx.x + touch_stride (0: none), which the
  // dispatcher, dealing workgroups to the eight XCDs in turn, sends to this
  // XCD once a compute unit frees up.
  int next_row = -1;
  if (touch_stride > 0) {
    const int nb = (int)blockIdx.x + touch_stride;
    if (nb < (int)gridDim.x) {
      const int nr = FP6 ? fp6_row(nb, mblk * 32) : nb;
      next_row = nr < M ? nr : -1;
    }
  }
  if constexpr (FP6) {
    if (row >= M) {   // padding row of the last block: zero codes
      for (int q = threadIdx.x; q < K / 32; q += T) {
        uint8_t* d = codes + fp6_slot(row, 32 * q, mblk);
#pragma unroll
        for (int c = 0; c < 3; ++c) *reinterpret_cast<uint2*>(d + 512 * c) = make_uint2(0, 0);
      }
      return;
    }
  }
  const Tin* xr = x + (size_t)row * K;
  const int nchunk = K >> 3;
  constexpr bool load_last = (P::np == 0 && F == 1);

  float tmax = 0.0f;
  for (int q = threadIdx.x; q < nchunk; q += T) {
    float v[8];
    if constexpr (STATS) {
      load8_sum(xr + (size_t)q * 8, st.dx + (size_t)row * K + (size_t)q * 8, v, sums.x, sums.y);
    } else {
      load8(xr + (size_t)q * 8, v);
      if (signs) apply_sign_bits<8>(v, signs[q]);
    }
    butterflies<3>(v, 0, P::j0);
    if (load_last) tmax = absmax8(v, tmax);
    float4* d = reinterpret_cast<float4*>(lds + lidx<PD>(q * 8));
    d[0] = make_float4(v[0], v[1], v[2], v[3]);
    d[1] = make_float4(v[4], v[5], v[6], v[7]);
  }
  __syncthreads();
  // With one workgroup per compute unit the rows of a round load together
  // and nothing hides that burst.  So, once this row is staged, touch one
  // dword in every 64 bytes of the next row this XCD will take: it is in the
  // L2 when its workgroup starts.  The value is only consumed (by an empty
  // asm) when the row is done, so the load never stalls this row.
  uint32_t touch = 0;
  if (next_row >= 0) {
    constexpr int kStep = 64 / (int)sizeof(Tin);
    const Tin* xn = x + (size_t)next_row * K;
    for (int e = threadIdx.x * kStep; e < K; e += T * kStep)
      touch ^= *reinterpret_cast<const uint32_t*>(xn + e);
  }

  if constexpr (P::np > 0) {
    tmax = pass_bits<P::width(0), P::start(0), T, PD>(lds, K, P::np == 1 && F == 1, tmax);
    __syncthreads();
  }
  if constexpr (P::np > 1) {
    tmax = pass_bits<P::width(1), P::start(1), T, PD>(lds, K, P::np == 2 && F == 1, tmax);
    __syncthreads();
  }
  if constexpr (P::np > 2) {
    tmax = pass_bits<P::width(2), P::start(2), T, PD>(lds, K, F == 1, tmax);
    __syncthreads();
  }
  if constexpr (F == 28) {
    tmax = pass_28<T, J, PD>(lds, K, tmax);
    __syncthreads();
  }

  // Row absmax: wavefront reduction, then across the 4 wavefronts.
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) tmax = fmaxf(tmax, __shfl_xor(tmax, off));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = tmax;
  __syncthreads();
  float amax = red[0];
#pragma unroll
  for (int w = 1; w < T / 64; ++w) amax = fmaxf(amax, red[w]);

  constexpr float qmax = (float)((1 << (BITS - 1)) - 1);
  const float sc = amax / qmax;                 // IEEE division
  const float rc = sc != 0.0f ? 1.0f / sc : 0.0f;
  if (!STATS && threadIdx.x == 0) {
    if (WEIGHT) {
      constexpr int h = F << J;
      scales[row] = sc / (float)h;              // fold the 1/h of the rotation
    } else {
      scales[row] = sc;
    }
  }

  if constexpr (FP6) {
    // Each thread quantizes 8 consecutive elements (the read pattern of the
    // 4- and 8-bit outputs); the four threads of a lane quad hold one
    // operand's 32 codes, gather them with DPP, convert, and store one 8-byte
    // plane each (the fourth thread has none).  K % 128 == 0 and T % 4 == 0,
    // so quads stay together and every quad's items exist or none do.
    for (int q0 = threadIdx.x & ~3; q0 < nchunk; q0 += T) {
      const int q = q0 + (threadIdx.x & 3);
      const float4* src = reinterpret_cast<const float4*>(lds + lidx<PD>(q * 8));
      const float4 a = src[0], b = src[1];
      const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
      uint32_t hw[4];   // the 8 values c / 2 as packed fp16 pairs
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const _Float16 lo = (_Float16)half_code(round_bits(v[2 * k], sc, rc));
        const _Float16 hi = (_Float16)half_code(round_bits(v[2 * k + 1], sc, rc));
        hw[k] = (uint32_t)__builtin_bit_cast(unsigned short, lo) |
                ((uint32_t)__builtin_bit_cast(unsigned short, hi) << 16);
      }
      typedef unsigned int f6_v16u __attribute__((ext_vector_type(16)));
      f6_v16u all;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        all[k] = (uint32_t)__builtin_amdgcn_mov_dpp((int)hw[k], 0x00, 0xF, 0xF, false);       // quad lane 0
        all[4 + k] = (uint32_t)__builtin_amdgcn_mov_dpp((int)hw[k], 0x55, 0xF, 0xF, false);   // lane 1
        all[8 + k] = (uint32_t)__builtin_amdgcn_mov_dpp((int)hw[k], 0xAA, 0xF, 0xF, false);   // lane 2
        all[12 + k] = (uint32_t)__builtin_amdgcn_mov_dpp((int)hw[k], 0xFF, 0xF, 0xF, false);  // lane 3
      }
      const f6_v6i f = __builtin_amdgcn_cvt_scalef32_pk32_fp6_f16(__builtin_bit_cast(f6_v32h, all), 1.0f);
      const int c = threadIdx.x & 3;
      if (c < 3) {
        uint8_t* d = codes + fp6_slot(row, 8 * q0, mblk) + 512 * c;
        const uint32_t lo = c == 0 ? (uint32_t)f[0] : c == 1 ? (uint32_t)f[2] : (uint32_t)f[4];
        const uint32_t hi = c == 0 ? (uint32_t)f[1] : c == 1 ? (uint32_t)f[3] : (uint32_t)f[5];
        *reinterpret_cast<uint2*>(d) = make_uint2(lo, hi);
      }
    }
    asm volatile("" : : "v"(touch));
    return;
  }
  for (int q = threadIdx.x; q < nchunk; q += T) {
    const float4* src = reinterpret_cast<const float4*>(lds + lidx<PD>(q * 8));
    const float4 a = src[0], b = src[1];
    const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
    if constexpr (STATS) {
      sums.z = quant_error_energy<8>(v, sc, rc, sums.z);
      continue;
    }
    uint32_t bt[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) bt[k] = round_bits(v[k], sc, rc);
    if (BITS == 4) {
      reinterpret_cast<uint32_t*>(codes + (size_t)row * (K / 2))[q] = pack_nibbles(bt);
    } else {
      reinterpret_cast<uint2*>(codes + (size_t)row * K)[q] =
          make_uint2(low_bytes(bt[0], bt[1], bt[2], bt[3]), low_bytes(bt[4], bt[5], bt[6], bt[7]));
    }
  }
  if constexpr (STATS) {
    sums = block_sum3<T>(sums, red3);
    if (threadIdx.x == 0) write_stats(st, row, sums, F << J);
  }
  asm volatile("" : : "v"(touch));
}

size_t lds_bytes(int K, int pd) {
  return (size_t)(K + (pd == 0 ? ((K + 255) >> 8) * 8 : ((K + 31) >> 5) * 4)) * sizeof(float);
}
constexpr size_t kLdsMax = 160 * 1024;

template <typename Tin, int BITS, bool WEIGHT, int F, int J, int T, bool STATS, bool FP6>
hipError_t launch_one_t(const Tin* x, int64_t M, int K, const uint8_t* signs, uint8_t* codes,
                        float* scales, StatsArgs st, int touch_stride, hipStream_t stream) {
  auto kern = rotate_quant_kernel<Tin, BITS, WEIGHT, F, J, T, STATS, FP6>;
  constexpr int PD = pad_of<F, J>();
  static bool attr_set = false;
  if (!attr_set) {
    // Rows above 64 KiB of LDS need the larger dynamic allocation enabled.
    const size_t most = lds_bytes(kMaxRotateK, PD);
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                              hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)(most < kLdsMax - 4096 ? most : kLdsMax - 4096));
    (void)hipGetLastError();
    attr_set = true;
  }
  const int64_t grid = FP6 ? (M + 31) / 32 * 32 : M;
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(T), lds_bytes(K, PD), stream, x, (int)M, K,
                     signs, codes, scales, st, touch_stride);
  return hipGetLastError();
}

// Few rows (decode), or rows so long that one compute unit's LDS holds only
// one of them: 1024 threads per row shorten each row's latency and keep 16
// wavefronts per compute unit.  Many shorter rows: 256 threads, several rows
// per compute unit.
constexpr int64_t kFewRows = 64;
constexpr size_t kOneRowLds = 80 * 1024;

template <typename Tin, int BITS, bool WEIGHT, int F, int J, bool STATS, bool FP6>
hipError_t launch_one(const Tin* x, int64_t M, int K, const uint8_t* signs, uint8_t* codes,
                      float* scales, StatsArgs st, hipStream_t stream) {
  // Rows past the first round of resident workgroups get their next row
  // touched into the L2: the row of the workgroup one round later, which the
  // dispatcher sends to the same XCD (decode batches have no next round).
  const int cus = device_cus();
  if (M <= kFewRows || lds_bytes(K, pad_of<F, J>()) > kOneRowLds) {
    // one 1024-thread workgroup per compute unit
    const int touch = lds_bytes(K, pad_of<F, J>()) > kOneRowLds && M > cus ? cus : 0;
    return launch_one_t<Tin, BITS, WEIGHT, F, J, 1024, STATS, FP6>(x, M, K, signs, codes, scales, st,
                                                                  touch, stream);
  }
  // several 256-thread workgroups per compute unit, as many as their LDS
  // allows (at most eight)
  const size_t per = kLdsMax / (lds_bytes(K, pad_of<F, J>()) + 1024);
  const int resident = cus * (int)(per < 8 ? per : 8);
  return launch_one_t<Tin, BITS, WEIGHT, F, J, kThreads, STATS, FP6>(x, M, K, signs, codes, scales,
                                                                    st, M > resident ? resident : 0,
                                                                    stream);
}

template <typename Tin, int BITS, bool WEIGHT, int F, bool STATS, bool FP6, int J = 0>
hipError_t dispatch_j(int j, const Tin* x, int64_t M, int K, const uint8_t* signs, uint8_t* codes,
                      float* scales, StatsArgs st, hipStream_t stream) {
  constexpr int kMaxJ = F == 1 ? 15 : 10;   // h <= 32768
  if constexpr (J > kMaxJ) {
    return hipErrorInvalidValue;
  } else {
    if (j == J)
      return launch_one<Tin, BITS, WEIGHT, F, J, STATS, FP6>(x, M, K, signs, codes, scales, st, stream);
    return dispatch_j<Tin, BITS, WEIGHT, F, STATS, FP6, J + 1>(j, x, M, K, signs, codes, scales, st,
                                                               stream);
  }
}

// ---------------------------------------------------------------------------
// Power-of-two Hadamard sizes up to 4096.  The row sits in LDS as 4096-element
// segments (the last one zero-padded); in every phase each of the 256 threads
// holds 16 elements of a segment in registers, so the 12 index bits of a
// segment are covered by three register phases of 4 bits each:
//   phase 1: thread t holds i = 16 t + r        (register bits = index bits 0-3)
//   phase 2: thread t holds i = 256 (t >> 4) + 16 r + (t & 15)   (bits 4-7)
//   phase 3: thread t holds i = 256 r + t                        (bits 8-11)
// and the stages run in the order bit 0, 1, 2, ...  Element i of a segment
// sits at float offset i + 4 (i >> 6): every phase's accesses are then free
// of bank conflicts and their addresses are a per-thread base plus
// compile-time offsets.  Phase 1 loads from global memory and the final pass
// re-reads the phase-1 layout to quantize 16 consecutive elements per thread.
// ---------------------------------------------------------------------------
template <typename Tin, int BITS, bool WEIGHT, int J, bool STATS, bool FP6>
__global__ void __launch_bounds__(kThreads)
rq_pow2_kernel(const Tin* __restrict__ x, int M, int K, const uint8_t* __restrict__ signs,
               uint8_t* __restrict__ codes, float* __restrict__ scales, StatsArgs st) {
  static_assert(J <= 12, "segments hold 4096 elements");
  static_assert(!FP6 || BITS == 4, "FP6 output holds 4-bit codes");
  extern __shared__ float lds[];
  __shared__ float red[kThreads / 64];
  __shared__ float red3[kThreads / 64][3];
  float3 sums = make_float3(0.0f, 0.0f, 0.0f);
  const int mblk = (M + 31) >> 5;
  const int row = FP6 ? fp6_row(blockIdx.x, mblk * 32) : (int)blockIdx.x;
  const int t = threadIdx.x;
  const int nseg = (K + kSeg - 1) / kSeg;
  if constexpr (FP6) {
    if (row >= M) {   // padding row of the last block: zero codes
      for (int q = t; q < K / 32; q += kThreads) {
        uint8_t* d = codes + fp6_slot(row, 32 * q, mblk);
#pragma unroll
        for (int c = 0; c < 3; ++c) *reinterpret_cast<uint2*>(d + 512 * c) = make_uint2(0, 0);
      }
      return;
    }
  }
  const Tin* xr = x + (size_t)row * K;
  constexpr int kLast = J <= 4 ? 1 : (J <= 8 ? 2 : 3);   // last phase with stages
  // Per-thread LDS bases of the three layouts (segment offset added per use).
  const int b1 = seg_off(16 * t);
  const int b2 = seg_off(256 * (t >> 4) + (t & 15));
  const int b3 = seg_off(t);
  float tmax = 0.0f;

  for (int sg = 0; sg < nseg; ++sg) {
    float v[16];
    const int e = sg * kSeg + 16 * t;
    // K is a multiple of 8: a thread's second 8 elements may lie past the
    // row end (then h <= 8 and they form blocks of their own).
    const __half* dr = STATS ? st.dx + (size_t)row * K : nullptr;
    if (e < K) {
      if constexpr (STATS) load8_sum(xr + e, dr + e, v, sums.x, sums.y);
      else load8(xr + e, v);
    } else {
#pragma unroll
      for (int r = 0; r < 8; ++r) v[r] = 0.0f;
    }
    if (e + 8 < K) {
      if constexpr (STATS) load8_sum(xr + e + 8, dr + e + 8, v + 8, sums.x, sums.y);
      else load8(xr + e + 8, v + 8);
    } else {
#pragma unroll
      for (int r = 8; r < 16; ++r) v[r] = 0.0f;
    }
    if (!STATS && signs) {
      const uint32_t m = (e < K ? (uint32_t)signs[e / 8] : 0u) |
                         (e + 8 < K ? (uint32_t)signs[e / 8 + 1] << 8 : 0u);
      apply_sign_bits<16>(v, m);
    }
    stages16<0, (J < 4 ? J : 4)>(v);
    if (kLast == 1) tmax = absmax16(v, tmax);
    float* sl = lds + sg * kSegFloats + b1;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      *reinterpret_cast<float4*>(sl + 4 * q) = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
  }
  if constexpr (J > 4) {
    __syncthreads();
    for (int sg = 0; sg < nseg; ++sg) {
      float* sl = lds + sg * kSegFloats + b2;
      float v[16];
      // i = 256 (t >> 4) + 16 r + (t & 15): offset 16 r + 4 (r >> 2) from b2.
#pragma unroll
      for (int r = 0; r < 16; ++r) v[r] = sl[16 * r + 4 * (r >> 2)];
      stages16<0, (J < 8 ? J : 8) - 4>(v);
      if (kLast == 2) tmax = absmax16(v, tmax);
#pragma unroll
      for (int r = 0; r < 16; ++r) sl[16 * r + 4 * (r >> 2)] = v[r];
    }
  }
  if constexpr (J > 8) {
    __syncthreads();
    for (int sg = 0; sg < nseg; ++sg) {
      float* sl = lds + sg * kSegFloats + b3;
      float v[16];
      // i = 256 r + t: offset 272 r from b3.
#pragma unroll
      for (int r = 0; r < 16; ++r) v[r] = sl[272 * r];
      stages16<0, J - 8>(v);
      tmax = absmax16(v, tmax);
#pragma unroll
      for (int r = 0; r < 16; ++r) sl[272 * r] = v[r];
    }
  }

  // Row absmax (padding elements are zero): wavefronts, then the workgroup.
  tmax = wave_max_nonneg(tmax);
  if ((t & 63) == 0) red[t >> 6] = tmax;
  __syncthreads();
  float amax = red[0];
#pragma unroll
  for (int w = 1; w < kThreads / 64; ++w) amax = fmaxf(amax, red[w]);

  constexpr float qmax = (float)((1 << (BITS - 1)) - 1);
  const float sc = amax / qmax;                 // IEEE division
  const float rc = sc != 0.0f ? 1.0f / sc : 0.0f;
  if (!STATS && t == 0) scales[row] = WEIGHT ? sc / (float)(1 << J) : sc;

  if constexpr (STATS) {
    // Padding elements are zero and quantize to zero without error.
    for (int sg = 0; sg < nseg; ++sg) {
      const float* sl = lds + sg * kSegFloats + b1;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 w4 = *reinterpret_cast<const float4*>(sl + 4 * q);
        const float w[4] = {w4.x, w4.y, w4.z, w4.w};
        sums.z = quant_error_energy<4>(w, sc, rc, sums.z);
      }
    }
    sums = block_sum3<kThreads>(sums, red3);
    if (t == 0) write_stats(st, row, sums, 1 << J);
    return;
  }

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
    const bool full = e + 8 < K;   // else only the first 8 elements are in the row
    if constexpr (FP6) {
      // 16 codes = fields 0..15 (t even) or 16..31 (t odd) of an operand:
      // planes 0 and the low half of 1, or the high half of 1 and plane 2.
      const f6_v6i f = fp6_fields<16>(bt);
      uint8_t* d = codes + fp6_slot(row, e, mblk);
      if ((e & 16) == 0) {
        *reinterpret_cast<uint2*>(d) = make_uint2((uint32_t)f[0], (uint32_t)f[1]);
        *reinterpret_cast<uint32_t*>(d + 512) = (uint32_t)f[2];
      } else {
        *reinterpret_cast<uint32_t*>(d + 516) = (uint32_t)f[0];
        *reinterpret_cast<uint2*>(d + 1024) = make_uint2((uint32_t)f[1], (uint32_t)f[2]);
      }
    } else if (BITS == 4) {
      const uint32_t w[2] = {pack_nibbles(bt), pack_nibbles(bt + 8)};
      // Rows start 8-byte aligned when K % 32 == 0; otherwise word stores.
      uint32_t* dst = reinterpret_cast<uint32_t*>(codes + (size_t)row * (K / 2) + e / 2);
      if (full && K % 32 == 0) {
        *reinterpret_cast<uint2*>(dst) = make_uint2(w[0], w[1]);
      } else {
        dst[0] = w[0];
        if (full) dst[1] = w[1];
      }
    } else {
      uint32_t d[4];
      d[0] = low_bytes(bt[0], bt[1], bt[2], bt[3]);
      d[1] = low_bytes(bt[4], bt[5], bt[6], bt[7]);
      d[2] = low_bytes(bt[8], bt[9], bt[10], bt[11]);
      d[3] = low_bytes(bt[12], bt[13], bt[14], bt[15]);
      // Rows start 16-byte aligned when K % 16 == 0, else 8-byte aligned.
      uint8_t* dst = codes + (size_t)row * K + e;
      if (full && K % 16 == 0) {
        *reinterpret_cast<uint4*>(dst) = make_uint4(d[0], d[1], d[2], d[3]);
      } else {
        reinterpret_cast<uint2*>(dst)[0] = make_uint2(d[0], d[1]);
        if (full) reinterpret_cast<uint2*>(dst)[1] = make_uint2(d[2], d[3]);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Many rows (prefill) of h = 2^j, j >= 14, at 4 or 8 bits: the segmented
// rotation of quant_device.h (three register phases over 4096-element
// segments with compile-time LDS offsets, one LDS pass per index bit above 11
// pairing whole segments, in the pinned order), one row per 256-thread
// workgroup, then the quantizer and the nibble or byte output of
// rq_pow2_kernel on the phase-1 layout.  K % 128 == 0.
// ---------------------------------------------------------------------------
template <int BITS>
__global__ void __launch_bounds__(kThreads)
rq_seg_kernel(const __half* __restrict__ x, int M, int K, int J, uint8_t* __restrict__ codes,
              float* __restrict__ scales) {
  extern __shared__ float lds[];
  __shared__ float red[kThreads / 64];
  const int row = (int)blockIdx.x;
  const int t = threadIdx.x;
  const uint4 none[2] = {make_uint4(0, 0, 0, 0), make_uint4(0, 0, 0, 0)};
  float ma = 0.0f, mb = 0.0f;
  rotate_row_segments<12, false, false, 1>(x + (size_t)row * K, K, J, true, t,
                                           RowSplit{0, 1, t, kThreads}, false, none, lds, ma, mb);
  ma = wave_max_nonneg(ma);
  if ((t & 63) == 0) red[t >> 6] = ma;
  __syncthreads();
  float amax = red[0];
#pragma unroll
  for (int w = 1; w < kThreads / 64; ++w) amax = fmaxf(amax, red[w]);

  constexpr float qmax = (float)((1 << (BITS - 1)) - 1);
  const float sc = amax / qmax;                 // IEEE division
  const float rc = sc != 0.0f ? 1.0f / sc : 0.0f;
  if (t == 0) scales[row] = sc;

  const int nseg = (K + kSeg - 1) / kSeg;
  const int b1 = seg_off(16 * t);
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
    if constexpr (BITS == 4) {
      *reinterpret_cast<uint2*>(codes + (size_t)row * (K / 2) + e / 2) =
          make_uint2(pack_nibbles(bt), pack_nibbles(bt + 8));
    } else {
      *reinterpret_cast<uint4*>(codes + (size_t)row * K + e) =
          make_uint4(low_bytes(bt[0], bt[1], bt[2], bt[3]), low_bytes(bt[4], bt[5], bt[6], bt[7]),
                     low_bytes(bt[8], bt[9], bt[10], bt[11]), low_bytes(bt[12], bt[13], bt[14], bt[15]));
    }
  }
}

size_t pow2_lds_bytes(int K) { return (size_t)((K + kSeg - 1) / kSeg) * kSegFloats * sizeof(float); }

template <typename Tin, int BITS, bool WEIGHT, int J, bool STATS, bool FP6>
hipError_t launch_pow2(const Tin* x, int64_t M, int K, const uint8_t* signs, uint8_t* codes,
                       float* scales, StatsArgs st, hipStream_t stream) {
  auto kern = rq_pow2_kernel<Tin, BITS, WEIGHT, J, STATS, FP6>;
  static bool attr_set = false;
  if (!attr_set) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                              hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)pow2_lds_bytes(kMaxRotateK));
    (void)hipGetLastError();
    attr_set = true;
  }
  const int64_t grid = FP6 ? (M + 31) / 32 * 32 : M;
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(kThreads), pow2_lds_bytes(K), stream, x,
                     (int)M, K, signs, codes, scales, st);
  return hipGetLastError();
}

template <typename Tin, int BITS, bool WEIGHT, bool STATS, bool FP6, int J = 0>
hipError_t dispatch_pow2(int j, const Tin* x, int64_t M, int K, const uint8_t* signs,
                         uint8_t* codes, float* scales, StatsArgs st, hipStream_t stream) {
  if constexpr (J > 12) {
    return hipErrorInvalidValue;
  } else {
    if (j == J)
      return launch_pow2<Tin, BITS, WEIGHT, J, STATS, FP6>(x, M, K, signs, codes, scales, st, stream);
    return dispatch_pow2<Tin, BITS, WEIGHT, STATS, FP6, J + 1>(j, x, M, K, signs, codes, scales, st,
                                                               stream);
  }
}

size_t seg_lds_bytes(int K) { return (size_t)((K + kSeg - 1) / kSeg) * kSegFloats * sizeof(float); }

template <int BITS>
hipError_t launch_seg(const __half* x, int64_t M, int K, int J, uint8_t* codes, float* scales,
                      hipStream_t stream) {
  auto kern = rq_seg_kernel<BITS>;
  static bool attr_set = false;
  if (!attr_set) {
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                              hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)seg_lds_bytes(kMaxRotateK));
    (void)hipGetLastError();
    attr_set = true;
  }
  hipLaunchKernelGGL(kern, dim3((unsigned)M), dim3(kThreads), seg_lds_bytes(K), stream, x, (int)M,
                     K, J, codes, scales);
  return hipGetLastError();
}

// Plain fp16 rotation of many rows at h = 2^j, j >= 14, with nibble or byte
// output goes to the segmented kernel while its staging leaves room for two
// rows per compute unit (K <= 16384): 85.5 / 86.6 us against 90.0 / 94.1 us
// for the general kernel at 4096 x 16384 (A4 / A8).  Everywhere else the
// general kernel, with its constant-offset LDS addressing, was as fast or
// faster: at 28 * 2^j by 4-12%, at 8192 by 1-4%.
bool use_seg(int64_t M, int K, HadSplit hs, bool fp6) {
  return kSegRows > 0 && M > kSegRows && K % 128 == 0 && hs.f == 1 && hs.j >= 14 && !fp6 &&
         seg_lds_bytes(K) <= kOneRowLds;
}

// signs: optional randomized-sign bitmask (bit set = negate the element
// before the rotation); nullptr for the plain rotation.
template <typename Tin, int BITS, bool WEIGHT, bool STATS = false, bool FP6 = false>
hipError_t launch_rq(const Tin* x, int64_t M, int K, HadSplit hs, uint8_t* codes,
                     float* scales, hipStream_t stream, StatsArgs st = StatsArgs{},
                     const uint8_t* signs = nullptr) {
  if (M == 0) return hipSuccess;
  if constexpr (!WEIGHT && !STATS && sizeof(Tin) == 2) {
    if constexpr (!FP6) {
      if (signs == nullptr && use_seg(M, K, hs, FP6))
        return launch_seg<BITS>(reinterpret_cast<const __half*>(x), M, K, hs.j, codes, scales,
                                stream);
    }
  }
  if (hs.f == 28)
    return dispatch_j<Tin, BITS, WEIGHT, 28, STATS, FP6>(hs.j, x, M, K, signs, codes, scales, st,
                                                          stream);
  // Up to 4096 the register-phase kernel; larger sizes the general one.
  if (hs.j <= 12)
    return dispatch_pow2<Tin, BITS, WEIGHT, STATS, FP6>(hs.j, x, M, K, signs, codes, scales, st,
                                                        stream);
  return dispatch_j<Tin, BITS, WEIGHT, 1, STATS, FP6>(hs.j, x, M, K, signs, codes, scales, st,
                                                       stream);
}

// Layer means of the per-token statistics (Eq. 9 and Eq. 11): one workgroup
// sums in fp64 in a fixed order.
__global__ void __launch_bounds__(256)
layer_means_kernel(const float* __restrict__ jr, const float* __restrict__ snr, int64_t T,
                   double* __restrict__ out) {
  __shared__ double red[2][256];
  double a = 0.0, b = 0.0;
  for (int64_t i = threadIdx.x; i < T; i += 256) {
    a += (double)jr[i];
    b += (double)snr[i];
  }
  red[0][threadIdx.x] = a;
  red[1][threadIdx.x] = b;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if ((int)threadIdx.x < w) {
      red[0][threadIdx.x] += red[0][threadIdx.x + w];
      red[1][threadIdx.x] += red[1][threadIdx.x + w];
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    out[0] = red[0][0] / (double)T;
    out[1] = red[1][0] / (double)T;
  }
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

hipError_t launch_rotate_quant_fp6(const void* x, int64_t M, int K, HadSplit hs, uint8_t* out,
                                   float* scales, hipStream_t stream, const uint8_t* signs) {
  return launch_rq<__half, 4, false, false, true>(static_cast<const __half*>(x), M, K, hs, out,
                                                  scales, stream, StatsArgs{}, signs);
}

hipError_t launch_rotate_quant_signed(const void* x, int64_t M, int K, HadSplit hs, int bits,
                                      const uint8_t* signs, void* codes, float* scales,
                                      hipStream_t stream) {
  const __half* xh = static_cast<const __half*>(x);
  uint8_t* c = static_cast<uint8_t*>(codes);
  if (bits == 4) return launch_rq<__half, 4, false>(xh, M, K, hs, c, scales, stream, StatsArgs{}, signs);
  return launch_rq<__half, 8, false>(xh, M, K, hs, c, scales, stream, StatsArgs{}, signs);
}

hipError_t launch_prepare_weights(const float* w, int64_t N, int K, HadSplit hs,
                                  uint8_t* w_packed, float* w_scales,
                                  hipStream_t stream, const uint8_t* signs) {
  return launch_rq<float, 4, true>(w, N, K, hs, w_packed, w_scales, stream, StatsArgs{}, signs);
}

hipError_t launch_residual_stats(const void* x, const void* dx, int64_t T, int K, HadSplit hs,
                                 int bits, float eps, float* jr, float* snr, double* means,
                                 hipStream_t stream) {
  if (T == 0) return hipSuccess;
  const __half* xh = static_cast<const __half*>(x);
  const StatsArgs st{static_cast<const __half*>(dx), jr, snr, eps};
  const hipError_t e =
      bits == 4 ? launch_rq<__half, 4, false, true>(xh, T, K, hs, nullptr, nullptr, stream, st)
                : launch_rq<__half, 8, false, true>(xh, T, K, hs, nullptr, nullptr, stream, st);
  if (e != hipSuccess || means == nullptr) return e;
  hipLaunchKernelGGL(layer_means_kernel, dim3(1), dim3(256), 0, stream, jr, snr, T, means);
  return hipGetLastError();
}

}  // namespace dptq
