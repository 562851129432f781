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

#include <utility>

#include "dptq.h"
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

// 8-bit activation operand of one 32-k step.  Against weights in the
// canonical nibble order the activation bytes are regrouped like the nibble
// unpack (even k, then odd k).  Weights in the 8-bit order (each dword holds
// k0..k3 in its low nibbles and k4..k7 in its high ones, pack_w4_a8_kernel)
// unpack to natural k order, so the activation dwords are the operand as
// they stand.
template <bool WA8>
__device__ __forceinline__ v4i op_a8(uint32_t d0, uint32_t d1, uint32_t d2, uint32_t d3) {
  if constexpr (WA8) {
    v4i r;
    r.x = (int)d0;
    r.y = (int)d1;
    r.z = (int)d2;
    r.w = (int)d3;
    return r;
  } else {
    return op_from_bytes(d0, d1, d2, d3);
  }
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

// Four accumulators of one lane (rows n .. n+3 of one column m), unscaled,
// with the zero-point correction off * wz when ZP, dequantized and packed as
// fp16.
template <int BITS, bool ZP>
__device__ __forceinline__ uint2 dequant4z(int a0, int a1, int a2, int a3, float as, float4 ws,
                                           int off, int4 wz) {
  int c0 = unscale<BITS>(a0), c1 = unscale<BITS>(a1), c2 = unscale<BITS>(a2), c3 = unscale<BITS>(a3);
  if constexpr (ZP) {
    c0 += off * wz.x;
    c1 += off * wz.y;
    c2 += off * wz.z;
    c3 += off * wz.w;
  }
  const __half h0 = dequant(c0, as, ws.x), h1 = dequant(c1, as, ws.y);
  const __half h2 = dequant(c2, as, ws.z), h3 = dequant(c3, as, ws.w);
  uint2 pk;
  pk.x = (uint32_t)__half_as_ushort(h0) | ((uint32_t)__half_as_ushort(h1) << 16);
  pk.y = (uint32_t)__half_as_ushort(h2) | ((uint32_t)__half_as_ushort(h3) << 16);
  return pk;
}

// ---------------------------------------------------------------------------
// Prefill.  An output tile of BN (n) x BM (m) is computed by WN x WM
// wavefronts, each owning a TI x TJ grid of 32 x 32 x 32 int8 MFMAs.  K is
// consumed in stages of 256 (128-byte row slices for 4-bit operands, so every
// global request is a full cache line) through a ring of LDS buffers filled
// by direct global->LDS 16-byte loads issued ahead of use.  The fp16 tile is
// staged through LDS so output rows are written with coalesced stores.
//
// The instantiated shape is 256 x 128 on eight wavefronts of 64 x 64, two
// per SIMD: one wavefront's unpack and LDS reads co-execute with the other's
// MFMAs.  Large problems use the wide-tile kernel further below instead.
// ---------------------------------------------------------------------------
constexpr int kBK = 256;

typedef __attribute__((address_space(3))) uint8_t* lds_ptr;
typedef int v16i __attribute__((ext_vector_type(16)));

// One wavefront-wide 16-byte-per-lane direct load from global memory into LDS
// at byte offset lds_off (+ 16 * lane).  Issued as asm so that the compiler's
// conservative wait (it cannot tell the ring buffers apart) does not drain
// the loads before every LDS read; completion is tracked with wait_vmcnt.
// Address = wavefront-uniform base + 32-bit per-lane offset.
__device__ __forceinline__ void dma16(const void* sbase, uint32_t voff, uint32_t lds_off) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(sbase), "s"(lds_off)
               : "memory", "m0");
}

// The same with the LDS destination given as a wavefront-uniform base plus a
// compile-time offset, formed in M0 by one scalar add (the global address is
// sbase + voff, the per-lane offset carrying the row).
template <uint32_t OFF>
__device__ __forceinline__ void dma16_at(const void* sbase, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_add_u32 m0, %2, %3\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(sbase), "s"(lds_base), "i"(OFF)
               : "memory", "m0", "scc");
}

// The same with 4 bytes per lane (LDS byte offset lds_off + 4 * lane).
__device__ __forceinline__ void dma4(const void* sbase, uint32_t voff, uint32_t lds_off) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dword %0, %1"
               :
               : "v"(voff), "s"(sbase), "s"(lds_off)
               : "memory", "m0");
}

// Workgroup barrier without the release/acquire fences of __syncthreads(): the
// fences would drain every outstanding direct-to-LDS load.  Callers wait for
// exactly the loads they need with wait_vmcnt first; the asm clobber keeps LDS
// accesses on their side.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_barrier" ::: "memory"); }

// s_waitcnt vmcnt(N) (gfx9 encoding), leaving the other counters untouched.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

__device__ __forceinline__ v16i mfma32(v4i a, v4i b, v16i c) {
  return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
}

// XOR swizzle of the 16-byte chunks of an LDS tile row so that the fragment
// reads (consecutive rows, one logical chunk per 8- or 16-lane group) hit
// distinct banks: rows of 8 chunks (128 B) and of 16 chunks (256 B).
__device__ __forceinline__ int swz8(int r) { return (r ^ (r >> 3)) & 7; }
__device__ __forceinline__ int swz16(int r) { return r & 15; }

__device__ __forceinline__ int xcd_remap(int bid, int total) {
  const int per = total >> 3, rem = total & 7;
  const int x = bid & 7, idx = bid >> 3;
  return x * per + (x < rem ? x : rem) + idx;
}

// Tile (tm, tn) of logical tile `logical`: logical tiles run in groups of
// kGroupM tile rows, m fastest within a group, so that the tiles an XCD works
// on at one time form a compact block whose operands share its L2.
__device__ __forceinline__ void grouped_tile(int logical, int tiles_m, int tiles_n, int& tm, int& tn) {
  constexpr int kGroupM = 4;
  const int per_group = kGroupM * tiles_n;
  const int g = logical / per_group, t = logical - g * per_group;
  const int gm = min(kGroupM, tiles_m - g * kGroupM);
  tn = t / gm;
  tm = g * kGroupM + (t - tn * gm);
}

template <int BITS, int BN, int BM, int WN, int WM>
struct Cfg {
  static constexpr int kBits = BITS, kBN = BN, kBM = BM, kWN = WN, kWM = WM;
  static constexpr int kWaves = WN * WM, kThreads = kWaves * 64;
  static constexpr int kTI = BN / WN / 32, kTJ = BM / WM / 32;
  static constexpr int kWRow = kBK / 2;                        // 128 B
  static constexpr int kARow = BITS == 4 ? kBK / 2 : kBK;      // 128 or 256 B
  static constexpr int kW = BN * kWRow;
  static constexpr int kA = BM * kARow;
  static constexpr int kStage = kW + kA;
  // Load buffers: as many as fit in 160 KiB, at most 3 (loads issued up to
  // two stages ahead).
  static constexpr int kBufs = (160 * 1024) / kStage >= 3 ? 3 : 2;
  static constexpr int kOutStride = BN * 2 + 16;               // fp16 output row in LDS
  static constexpr int kLds = kBufs * kStage > BM * kOutStride ? kBufs * kStage : BM * kOutStride;
  static constexpr int kWLoads = kW / 1024 / kWaves;           // per wavefront
  static constexpr int kALoads = kA / 1024 / kWaves;
  static constexpr int kLoads = kWLoads + kALoads;
  static_assert(kW % (1024 * kWaves) == 0 && kA % (1024 * kWaves) == 0, "load split");
  static_assert(kWaves == 4 || kWaves == 8, "load swizzle assumes 4 or 8 wavefronts");
  static_assert(kLds <= 160 * 1024, "LDS budget");
  static_assert(BN % (WN * 32) == 0 && BM % (WM * 32) == 0, "wave tiles");
};

template <int BITS> using PrefillCfg = Cfg<BITS, 256, 128, 4, 2>;

// ZP (the prefill kernels and the decode kernel alike): the range quantizer's
// zero-point correction acc + (2^(BITS-1) - a_zeros[m]) * w_sums[n], exact in
// int32, before the dequantization.
template <class C, bool ACC_OUT, bool WA8 = false, bool ZP = false>
__global__ void __launch_bounds__(C::kThreads)
qgemm_prefill(const uint8_t* __restrict__ a_codes, const float* __restrict__ a_scales,
              const uint8_t* __restrict__ w_packed, const float* __restrict__ w_scales,
              int M, int N, int K, __half* __restrict__ y, int32_t* __restrict__ acc_out,
              const int32_t* __restrict__ a_zeros = nullptr,
              const int32_t* __restrict__ w_sums = nullptr) {
  constexpr int BITS = C::kBits, kBN = C::kBN, kBM = C::kBM, kWN = C::kWN;
  constexpr int kTI = C::kTI, kTJ = C::kTJ, kWaves = C::kWaves, kThreads = C::kThreads;
  __shared__ __attribute__((aligned(1024))) uint8_t smem[C::kLds];

  const int tiles_m = (M + kBM - 1) / kBM;
  const int tiles_n = (N + kBN - 1) / kBN;
  const int logical = xcd_remap(blockIdx.x, tiles_m * tiles_n);
  int tm, tn;
  grouped_tile(logical, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * kBM, n0 = tn * kBN;

  const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const int wn = wave % kWN, wm = wave / kWN;
  const int wrow = K / 2;
  const int arow = BITS == 4 ? K / 2 : K;
  const int nst = (K + kBK - 1) / kBK;
  const bool half_tail = (K % kBK) != 0;   // last stage holds only 128 k

  // Direct loads.  One load instruction fills 1 KiB of LDS: 8 rows of 128 B
  // (4-bit operands) or 4 rows of 256 B (8-bit activations); lane l writes
  // physical chunk p of its row, which holds logical chunk p ^ swizzle(row).
  // Load i of wavefront w fills LDS block j = i * kWaves + w, rows j * 8 +
  // (l >> 3) (resp. j * 4 + (l >> 4)).  The swizzle's row term is (j & 7)
  // (resp. 4 (j & 3) + (l >> 4)), which depends on i at most through i & 1,
  // so the row part of the address is a wavefront-uniform base and the lane
  // part one of two offsets.  Tiles that overhang the matrix clamp rows to
  // the last one, and a half tail stage (K % 256 == 128) maps chunks past K
  // onto their first-half twins; both only feed results that are never stored.
  constexpr int kARows = BITS == 4 ? 8 : 4;   // rows per A load instruction
  const bool w_full = n0 + kBN <= N;
  const bool a_full = m0 + kBM <= M;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);   // known wavefront-uniform
  uint32_t wlane[2], alane[2];
#pragma unroll
  for (int x = 0; x < 2; ++x) {
    const int rl = lane >> 3;
    const int jlow = (x * kWaves + wave) & 7;        // (i * kWaves + w) & 7 for i & 1 == x
    const int c = ((lane & 7) ^ rl ^ jlow) & 7;
    wlane[x] = (uint32_t)(rl * wrow + c * 16);
    if (BITS == 4) {
      alane[x] = (uint32_t)(rl * arow + c * 16);
    } else {
      const int r16 = ((x * kWaves + wave) & 3) * 4 + (lane >> 4);
      alane[x] = (uint32_t)((lane >> 4) * arow + ((lane & 15) ^ r16) * 16);
    }
  }
  const uint32_t smem_base = (uint32_t)(uintptr_t)(lds_ptr)smem;
  const uint32_t wave_off = (uint32_t)wave_u * 1024;
  // A stage's weight loads and its activation loads, issued separately so
  // that they can be spread over the stage.
  auto issue_w = [&](int st, int buf) __attribute__((always_inline)) {
    const uint32_t base = smem_base + buf * C::kStage + wave_off;
    const bool tail = half_tail && st == nst - 1;
    const uint8_t* wt = w_packed + (size_t)n0 * wrow + (size_t)st * C::kWRow;   // uniform
    if (w_full && !tail) {
#pragma unroll
      for (int i = 0; i < C::kWLoads; ++i)
        dma16(wt + (size_t)((i * kWaves + wave_u) * 8) * wrow, wlane[i & 1], base + i * kWaves * 1024);
    } else {
#pragma unroll
      for (int i = 0; i < C::kWLoads; ++i) {
        const int r = (i * kWaves + wave) * 8 + (lane >> 3);
        int c = (lane & 7) ^ swz8(r);
        if (tail) c &= 3;
        const int rc = min(r, N - 1 - n0);
        dma16(wt, (uint32_t)(rc * wrow + c * 16), base + i * kWaves * 1024);
      }
    }
  };
  auto issue_a = [&](int st, int buf) __attribute__((always_inline)) {
    const uint32_t base = smem_base + buf * C::kStage + wave_off;
    const bool tail = half_tail && st == nst - 1;
    const uint8_t* at = a_codes + (size_t)m0 * arow + (size_t)st * C::kARow;    // uniform
    if (a_full && !tail) {
#pragma unroll
      for (int i = 0; i < C::kALoads; ++i)
        dma16(at + (size_t)((i * kWaves + wave_u) * kARows) * arow, alane[i & 1],
              base + C::kW + i * kWaves * 1024);
    } else {
#pragma unroll
      for (int i = 0; i < C::kALoads; ++i) {
        int r, c;
        if (BITS == 4) {
          r = (i * kWaves + wave) * 8 + (lane >> 3);
          c = (lane & 7) ^ swz8(r);
          if (tail) c &= 3;
        } else {
          r = (i * kWaves + wave) * 4 + (lane >> 4);
          c = (lane & 15) ^ swz16(r);
          if (tail) c &= 7;
        }
        const int rc = min(r, M - 1 - m0);
        dma16(at, (uint32_t)(rc * arow + c * 16), base + C::kW + i * kWaves * 1024);
      }
    }
  };
  auto issue = [&](int st, int buf) __attribute__((always_inline)) {
    issue_w(st, buf);
    issue_a(st, buf);
  };

  // Fragment addresses.  In half h (128 k) of a stage, lane l reads row l & 31
  // of its 32-row tiles, k range [128 h + 64 g, +64), g = l >> 5: two 16-byte
  // chunks of a 4-bit row, four of an 8-bit row.  The tile index enters as an
  // immediate offset.  For 4-bit rows the swizzle's row term for tile i is
  // 4 ((t0 + i) & 1) ^ s0, t0 = the wavefront's first tile index, so the
  // precomputed variants are indexed by h ^ (i & 1) with t0's parity folded in.
  const int fr = lane & 31, fg = lane >> 5;
  const int s0 = (fr & 7) ^ (fr >> 3);
  const int pw = (wn * kTI) & 1, pa = (wm * kTJ) & 1;
  uint32_t wv[2][2];
  uint32_t av[2][4];
#pragma unroll
  for (int z = 0; z < 2; ++z)
#pragma unroll
    for (int e = 0; e < 2; ++e)
      wv[z][e] = (uint32_t)((wn * kTI * 32 + fr) * C::kWRow +
                            (((2 * fg) ^ s0 ^ (4 * (z ^ pw) + e)) & 7) * 16);
#pragma unroll
  for (int z = 0; z < 2; ++z)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (BITS == 4)
        av[z][e] = e < 2 ? (uint32_t)((wm * kTJ * 32 + fr) * C::kARow +
                                      (((2 * fg) ^ s0 ^ (4 * (z ^ pa) + e)) & 7) * 16)
                         : 0u;
      else
        av[z][e] = (uint32_t)((wm * kTJ * 32 + fr) * C::kARow + (((8 * z + 4 * fg + e) ^ (fr & 15)) & 15) * 16);
    }

  // A stage is consumed as four chunk pairs p = 2 h + e: the 16-byte chunk e
  // of half h of every fragment row, i.e. two 32-k MFMA steps.  The packed
  // fragments of the next pair are read from LDS while the current one is
  // unpacked and multiplied.
  constexpr int kAD = BITS == 4 ? 4 : 8;
  struct Frags {
    uint32_t w[kTI][4];
    uint32_t a[kTJ][kAD];
  };
  auto read_pair = [&](const uint8_t* buf, int h, int e, Frags& f) __attribute__((always_inline)) {
    const uint8_t* ws = buf;
    const uint8_t* as = buf + C::kW;
#pragma unroll
    for (int i = 0; i < kTI; ++i) {
      const uint4 v = *reinterpret_cast<const uint4*>(ws + wv[h ^ (i & 1)][e] + i * 32 * C::kWRow);
      f.w[i][0] = v.x; f.w[i][1] = v.y; f.w[i][2] = v.z; f.w[i][3] = v.w;
    }
#pragma unroll
    for (int j = 0; j < kTJ; ++j) {
      if (BITS == 4) {
        const uint4 v = *reinterpret_cast<const uint4*>(as + av[h ^ (j & 1)][e] + j * 32 * C::kARow);
        f.a[j][0] = v.x; f.a[j][1] = v.y; f.a[j][2] = v.z; f.a[j][3] = v.w;
      } else {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const uint4 v = *reinterpret_cast<const uint4*>(as + av[h][2 * e + q] + j * 32 * C::kARow);
          f.a[j][4 * q] = v.x; f.a[j][4 * q + 1] = v.y; f.a[j][4 * q + 2] = v.z; f.a[j][4 * q + 3] = v.w;
        }
      }
    }
  };

  v16i acc[kTI][kTJ];
#pragma unroll
  for (int i = 0; i < kTI; ++i)
#pragma unroll
    for (int j = 0; j < kTJ; ++j) acc[i][j] = v16i{};

  // Two 32-k MFMA steps from one chunk pair.
  auto compute_pair = [&](const Frags& f) __attribute__((always_inline)) {
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      v4i aop[kTJ];
#pragma unroll
      for (int j = 0; j < kTJ; ++j) {
        if (BITS == 4) aop[j] = op_from_nibbles(f.a[j][2 * kk], f.a[j][2 * kk + 1]);
        else aop[j] = op_a8<WA8>(f.a[j][4 * kk], f.a[j][4 * kk + 1], f.a[j][4 * kk + 2], f.a[j][4 * kk + 3]);
      }
#pragma unroll
      for (int i = 0; i < kTI; ++i) {
        const v4i wop = op_from_nibbles(f.w[i][2 * kk], f.w[i][2 * kk + 1]);
#pragma unroll
        for (int j = 0; j < kTJ; ++j) acc[i][j] = mfma32(wop, aop[j], acc[i][j]);
      }
    }
  };

  // Ring of kBufs load buffers, loads issued kBufs-1 stages ahead.  Every
  // iteration issues exactly one stage (past the end the last stage again,
  // L2-resident, into a buffer nobody reads any more), so the number of load
  // instructions in flight is uniform: stage s has landed once only the
  // kBufs-2 stages after it are outstanding.  The barrier also guarantees
  // every wavefront is done with stage s-1, whose buffer the issue refills.
  constexpr int kB = C::kBufs;
  Frags fa, fb;
  int cur = 0;   // buffer of stage s
  auto begin_stage = [&](int s) __attribute__((always_inline)) -> const uint8_t* {
    wait_vmcnt<(kB - 2) * C::kLoads>();
    lds_barrier();
    const int nb = cur == 0 ? kB - 1 : cur - 1;   // (s + kB - 1) % kB
    issue(min(s + kB - 1, nst - 1), nb);
    const uint8_t* buf = smem + cur * C::kStage;
    cur = cur + 1 == kB ? 0 : cur + 1;
    return buf;
  };
#pragma unroll
  for (int st = 0; st < kB - 1; ++st) issue(min(st, nst - 1), st);
  // The loop body is branch-free; the last stage (possibly holding only
  // 128 k) is peeled off.
  // In the loop a stage's weight loads leave at its barrier; at 8 bits its
  // (twice as many) activation loads leave after the first MFMA pair, so
  // they do not leave in one burst (measured 1-3% faster at 8 bits, no gain
  // at 4).  Both are issued before the next wait, so the counts hold.
  for (int s = 0; s < nst - 1; ++s) {
    wait_vmcnt<(kB - 2) * C::kLoads>();
    lds_barrier();
    const int nb = cur == 0 ? kB - 1 : cur - 1;   // (s + kB - 1) % kB
    const int ist = min(s + kB - 1, nst - 1);
    issue_w(ist, nb);
    if constexpr (BITS == 4) issue_a(ist, nb);
    const uint8_t* buf = smem + cur * C::kStage;
    cur = cur + 1 == kB ? 0 : cur + 1;
    read_pair(buf, 0, 0, fa);
    read_pair(buf, 0, 1, fb);
    compute_pair(fa);
    if constexpr (BITS == 8) issue_a(ist, nb);
    read_pair(buf, 1, 0, fa);
    compute_pair(fb);
    read_pair(buf, 1, 1, fb);
    compute_pair(fa);
    compute_pair(fb);
  }
  {
    const uint8_t* buf = begin_stage(nst - 1);
    read_pair(buf, 0, 0, fa);
    read_pair(buf, 0, 1, fb);
    compute_pair(fa);
    if (!half_tail) {
      read_pair(buf, 1, 0, fa);
      compute_pair(fb);
      read_pair(buf, 1, 1, fb);
      compute_pair(fa);
      compute_pair(fb);
    } else {
      compute_pair(fb);
    }
  }
  wait_vmcnt<0>();   // the re-issued tail loads must land before LDS is reused

  if (ACC_OUT) {
    // Raw accumulators (verification path): direct 16-byte stores.
#pragma unroll
    for (int j = 0; j < kTJ; ++j) {
      const int m = m0 + wm * kTJ * 32 + j * 32 + fr;
      if (m >= M) continue;
#pragma unroll
      for (int i = 0; i < kTI; ++i)
#pragma unroll
        for (int b = 0; b < 4; ++b) {
          const int n = n0 + wn * kTI * 32 + i * 32 + 8 * b + 4 * fg;
          if (n >= N) continue;
          *reinterpret_cast<int4*>(acc_out + (size_t)m * N + n) =
              make_int4(unscale<BITS>(acc[i][j][4 * b]), unscale<BITS>(acc[i][j][4 * b + 1]),
                        unscale<BITS>(acc[i][j][4 * b + 2]), unscale<BITS>(acc[i][j][4 * b + 3]));
        }
    }
    return;
  }

  // Dequantize into an LDS copy of the fp16 tile (rows m, BN n + padding),
  // then write whole rows.  32 x 32 accumulator layout: lane l holds column
  // m = l & 31 and, in registers 4b .. 4b+3, rows n = 8 b + 4 (l >> 5) + 0..3.
  lds_barrier();   // every wavefront is done reading the last stage
#pragma unroll
  for (int j = 0; j < kTJ; ++j) {
    const int ml = wm * kTJ * 32 + j * 32 + fr;
    const float as = a_scales[min(m0 + ml, M - 1)];
    const int off = ZP ? (1 << (BITS - 1)) - a_zeros[min(m0 + ml, M - 1)] : 0;
#pragma unroll
    for (int i = 0; i < kTI; ++i) {
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int nl = wn * kTI * 32 + i * 32 + 8 * b + 4 * fg;
        const float4 wsv = *reinterpret_cast<const float4*>(w_scales + min(n0 + nl, N - 4));
        const int4 wz = ZP ? *reinterpret_cast<const int4*>(w_sums + min(n0 + nl, N - 4)) : make_int4(0, 0, 0, 0);
        *reinterpret_cast<uint2*>(smem + ml * C::kOutStride + nl * 2) =
            dequant4z<BITS, ZP>(acc[i][j][4 * b], acc[i][j][4 * b + 1], acc[i][j][4 * b + 2],
                                acc[i][j][4 * b + 3], as, wsv, off, wz);
      }
    }
  }
  lds_barrier();
  // Rows of BN halves = BN / 8 16-byte chunks.
  constexpr int kRowChunks = kBN / 8;
  for (int idx = t; idx < kBM * kRowChunks; idx += kThreads) {
    const int ml = idx / kRowChunks, cc = idx - ml * kRowChunks;
    const int m = m0 + ml, n = n0 + cc * 8;
    if (m >= M || n >= N) continue;
    const uint4 v = *reinterpret_cast<const uint4*>(smem + ml * C::kOutStride + cc * 16);
    *reinterpret_cast<uint4*>(y + (size_t)m * N + n) = v;
  }
}

// ---------------------------------------------------------------------------
// Prefill, wide wavefront tiles: 192 (n) x 256 (m) output tiles on four
// wavefronts, one per SIMD, each owning 96 x 128 = 3 x 4 MFMAs of 32 x 32 x
// 32.  Every unpacked fragment feeds three or four MFMAs, so unpacking costs
// 3.5 VALU instructions per MFMA with 4-bit activations (6 with 64 x 64
// wavefront tiles) and the VALU work fits beside the matrix pipe.
//
// The kernel is persistent: one workgroup per compute unit walks its tiles,
// and the load ring runs on across tile boundaries, so the first stages of
// the next tile are in flight while a tile's epilogue runs.  Output rows
// leave straight from registers (two lanes' halves of a row are joined with
// a cross-lane swap), which keeps LDS free for the ring.  The activation and
// weight scales of a tile arrive in LDS by the same direct loads.
//
// With one wavefront per SIMD nothing else hides latency, so the k loop is
// pipelined explicitly, one 32-k MFMA step at a time: a step's LDS reads are
// issued two steps before its MFMAs, its unpack one step before, and the
// MFMAs of a step are interleaved one by one with the next step's unpack.
// Stages are 128 k (64-byte slices of 4-bit rows) in a ring of four load
// buffers (three for 8-bit activations); the barrier that opens stage g + 1
// sits in the middle of stage g, once every LDS read of stage g has
// returned.  Tiles at the matrix edge are shifted inward to end at the edge
// (they recompute, and rewrite with identical values, a strip of their
// neighbour), so every tile is full and the loads need no clamping.
// ---------------------------------------------------------------------------
template <int BITS>
struct Wide {
  static constexpr int kBN = 192, kBM = 256, kTI = 3, kTJ = 4;
  static constexpr int kWaves = 4, kThreads = 256, kBK = 128;
  static constexpr int kWRow = kBK / 2;                      // 64 B
  static constexpr int kARow = BITS == 4 ? kBK / 2 : kBK;    // 64 or 128 B
  static constexpr int kW = kBN * kWRow;
  static constexpr int kA = kBM * kARow;
  static constexpr int kStage = kW + kA;
  static constexpr int kBufs = BITS == 4 ? 4 : 3;
  static constexpr int kRing = kBufs * kStage;
  // Two slots (tile parity) of scales: a_s [256] at +0, w_s [192] at +1024.
  static constexpr int kScaleSlot = 2048;
  static_assert(kBM % 64 == 0 && kBN % 64 == 0 && kBM * 4 <= 1024 && kBN * 4 <= kScaleSlot - 1024,
                "scale slots");
  static constexpr int kLds = kRing + 2 * kScaleSlot;
  static constexpr int kWLoads = kW / 1024 / kWaves;         // per wavefront and stage
  static constexpr int kALoads = kA / 1024 / kWaves;
  static constexpr int kLoads = kWLoads + kALoads;
  static constexpr int kAReads = BITS == 4 ? 1 : 2;          // 16-byte reads per A fragment per chunk
  static constexpr int kReads = kTI + kTJ * kAReads;         // per chunk
  // VALU instructions of one step's unpack: 6 per 4-bit fragment, 4 per
  // 8-bit one, spread over the step's 12 MFMAs as kVHi after each of the
  // first kNHi and kVHi - 1 after the rest.
  static constexpr int kValu = 6 * kTI + (BITS == 4 ? 6 : 4) * kTJ;
  static constexpr int kMfma = kTI * kTJ;
  static constexpr int kVHi = (kValu + kMfma - 1) / kMfma;
  static constexpr int kNHi = kValu - (kVHi - 1) * kMfma;
  // The ring holds stages of at most two consecutive tiles: K >= kBufs stages.
  static constexpr int kMinK = kBufs * kBK;
  static_assert(kLds <= 160 * 1024, "LDS budget");
  static_assert(kW % (1024 * kWaves) == 0 && kA % (1024 * kWaves) == 0, "load split");
};

// Scheduling groups for one step: MFMA q, then kVHi (q < kNHi) or kVHi - 1
// VALU instructions, then one LDS read while reads remain.
template <int Q, int NM, int VHI, int NHI, int NR>
__device__ __forceinline__ void sched_step() {
  if constexpr (Q < NM) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x002, Q < NHI ? VHI : VHI - 1, 0);
    if constexpr (Q < NR) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    sched_step<Q + 1, NM, VHI, NHI, NR>();
  }
}

template <int BITS, bool ACC_OUT, bool WA8 = false, bool ZP = false>
__global__ void __launch_bounds__(256)
qgemm_prefill_wide(const uint8_t* __restrict__ a_codes, const float* __restrict__ a_scales,
                   const uint8_t* __restrict__ w_packed, const float* __restrict__ w_scales,
                   int M, int N, int K, __half* __restrict__ y, int32_t* __restrict__ acc_out,
                   const int32_t* __restrict__ a_zeros = nullptr,
                   const int32_t* __restrict__ w_sums = nullptr) {
  using C = Wide<BITS>;
  constexpr int kTI = C::kTI, kTJ = C::kTJ, kB = C::kBufs;
  __shared__ __attribute__((aligned(1024))) uint8_t smem[C::kLds];

  const int tiles_m = (M + C::kBM - 1) / C::kBM;
  const int tiles_n = (N + C::kBN - 1) / C::kBN;
  const int total = tiles_m * tiles_n;
  const int G = gridDim.x;                                       // <= total
  const int ntile = (total - (int)blockIdx.x + G - 1) / G;       // tiles of this workgroup, >= 1
  const int t = threadIdx.x, lane = t & 63;
  const int wave = __builtin_amdgcn_readfirstlane(t >> 6);
  const int wn = wave & 1, wm = wave >> 1;
  const int wrow = K / 2;
  const int arow = BITS == 4 ? K / 2 : K;
  const int nst = K / C::kBK;

  // Row origins of this workgroup's tile r.  The workgroups of one XCD take
  // consecutive logical tiles, in groups of tile rows (grouped_tile), so the
  // tiles in flight on an XCD share their operands in its L2.
  auto origin = [&](int r, int& m0, int& n0) __attribute__((always_inline)) {
    const int logical = xcd_remap((int)blockIdx.x + r * G, total);
    int tm, tn;
    grouped_tile(logical, tiles_m, tiles_n, tm, tn);
    m0 = min(tm * C::kBM, M - C::kBM);
    n0 = min(tn * C::kBN, N - C::kBN);
  };

  // Direct loads.  One load instruction fills 1 KiB of LDS: 16 rows of 64 B
  // (4-bit operands) or 8 rows of 128 B (8-bit activations).  Lane l writes
  // physical chunk p of its row r, which holds logical chunk p ^ sw(r), with
  // sw(r) = (r >> 2) & 3 for 64-byte rows and (r >> 1) & 7 for 128-byte
  // rows.  Load i of wavefront w fills LDS block j = 4 i + w, rows 16 j +
  // (l >> 2) (resp. 8 j + (l >> 3)), so sw depends on the lane (and on w & 1)
  // only and the row part of the address is wavefront-uniform.
  constexpr int kARows = BITS == 4 ? 16 : 8;
  const uint32_t wlane = (uint32_t)((lane >> 2) * wrow + (((lane & 3) ^ ((lane >> 4) & 3)) * 16));
  const uint32_t alane =
      BITS == 4 ? (uint32_t)((lane >> 2) * arow + (((lane & 3) ^ ((lane >> 4) & 3)) * 16))
                : (uint32_t)((lane >> 3) * arow + (((lane & 7) ^ ((4 * (wave & 1) + (lane >> 4)) & 7)) * 16));
  // The row part of each load's address is loop-invariant and lives in the
  // per-lane offset (below 2^32: 256 rows of at most DPTQ_MAX_K bytes), so one
  // stage's loads share one scalar base per operand and each costs a single
  // scalar add (its M0).
  static_assert((uint64_t)C::kBM * DPTQ_MAX_K < (1ull << 32), "32-bit load offsets");
  uint32_t wofs[C::kWLoads], aofs[C::kALoads];
#pragma unroll
  for (int i = 0; i < C::kWLoads; ++i) wofs[i] = wlane + (uint32_t)((4 * i + wave) * 16) * (uint32_t)wrow;
#pragma unroll
  for (int i = 0; i < C::kALoads; ++i) aofs[i] = alane + (uint32_t)((4 * i + wave) * kARows) * (uint32_t)arow;
  const uint32_t smem_base = (uint32_t)(uintptr_t)(lds_ptr)smem;
  // wtile, atile: the tile's first weight and activation rows (uniform).
  auto issue = [&](const uint8_t* wtile, const uint8_t* atile, int st, int buf) __attribute__((always_inline)) {
    const uint32_t base = smem_base + buf * C::kStage + wave * 1024;
    const uint8_t* wt = wtile + (size_t)st * C::kWRow;
    const uint8_t* at = atile + (size_t)st * C::kARow;
    [&]<int... I>(std::integer_sequence<int, I...>) {
      (dma16_at<(uint32_t)(I * 4096)>(wt, wofs[I], base), ...);
    }(std::make_integer_sequence<int, C::kWLoads>{});
    [&]<int... I>(std::integer_sequence<int, I...>) {
      (dma16_at<(uint32_t)(C::kW + I * 4096)>(at, aofs[I], base), ...);
    }(std::make_integer_sequence<int, C::kALoads>{});
  };
  // Loads [I0, I1) of one stage (weights first, then activations), so that a
  // stage's loads can be spread between its MFMAs instead of leaving in one
  // burst.
  auto issue_part = [&](auto i0c, auto i1c, const uint8_t* wtile, const uint8_t* atile, int st, int buf)
      __attribute__((always_inline)) {
    constexpr int I0 = decltype(i0c)::value, I1 = decltype(i1c)::value;
    const uint32_t base = smem_base + buf * C::kStage + wave * 1024;
    const uint8_t* wt = wtile + (size_t)st * C::kWRow;
    const uint8_t* at = atile + (size_t)st * C::kARow;
    [&]<int... I>(std::integer_sequence<int, I...>) {
      (
          [&] {
            if constexpr (I >= I0 && I < I1) {
              if constexpr (I < C::kWLoads)
                dma16_at<(uint32_t)(I * 4096)>(wt, wofs[I], base);
              else
                dma16_at<(uint32_t)(C::kW + (I - C::kWLoads) * 4096)>(at, aofs[I - C::kWLoads], base);
            }
          }(),
          ...);
    }(std::make_integer_sequence<int, C::kLoads>{});
  };
  auto wtile_of = [&](int n0) __attribute__((always_inline)) { return w_packed + (size_t)n0 * wrow; };
  auto atile_of = [&](int m0) __attribute__((always_inline)) { return a_codes + (size_t)m0 * arow; };
  // Scales of a tile into slot q (only when producing y; the accumulator
  // output has none): wavefront 0 loads a_s [256] in four 4-byte-per-lane
  // loads (a shifted tile's m0 need not be 16-byte aligned), wavefront 1
  // w_s [192] in three.  Extra loads only make the other wavefronts' waits
  // stricter, never weaker.
  auto issue_scales = [&](int m0, int n0, int q) __attribute__((always_inline)) {
    if constexpr (!ACC_OUT) {
      const uint32_t base = smem_base + C::kRing + q * C::kScaleSlot;
      if (wave == 0) {
#pragma unroll
        for (int i = 0; i < C::kBM / 64; ++i) dma4(a_scales + m0 + 64 * i, (uint32_t)lane * 4, base + 256 * i);
      } else if (wave == 1) {
#pragma unroll
        for (int i = 0; i < C::kBN / 64; ++i)
          dma4(w_scales + n0 + 64 * i, (uint32_t)lane * 4, base + 1024 + 256 * i);
      }
    }
  };

  // Fragment reads.  In chunk e (64 k) of a stage, lane l reads row l & 31 of
  // each 32-row tile, logical 16-byte chunk 2 g + e of a 64-byte row (g = l >>
  // 5), or chunks 4 g + 2 e and 4 g + 2 e + 1 of a 128-byte row: 32 k per
  // lane, two MFMA steps.  Fragment rows are 32 t + (l & 31) plus a multiple of
  // 32, so sw(row) depends on the lane only and the tile enters as an
  // immediate offset.
  const int fr = lane & 31, fg = lane >> 5;
  const int sw4 = (fr >> 2) & 3, sw8 = (fr >> 1) & 7;
  uint32_t wv[2], av[4];
#pragma unroll
  for (int e = 0; e < 2; ++e) {
    wv[e] = (uint32_t)((wn * kTI * 32 + fr) * C::kWRow + (((2 * fg + e) ^ sw4) * 16));
    if (BITS == 4) av[e] = (uint32_t)(C::kW + (wm * kTJ * 32 + fr) * C::kARow + (((2 * fg + e) ^ sw4) * 16));
  }
  if (BITS == 8) {
#pragma unroll
    for (int c = 0; c < 4; ++c)
      av[c] = (uint32_t)(C::kW + (wm * kTJ * 32 + fr) * C::kARow + (((4 * fg + c) ^ sw8) * 16));
  }

  struct Packed {
    uint32_t w[kTI][4];
    uint32_t a[kTJ][4 * C::kAReads];
  };
  struct Ops {
    v4i w[kTI];
    v4i a[kTJ];
  };
  auto read_chunk = [&](int buf, int e, Packed& p) __attribute__((always_inline)) {
    const uint8_t* s = smem + buf * C::kStage;
#pragma unroll
    for (int i = 0; i < kTI; ++i) {
      const uint4 v = *reinterpret_cast<const uint4*>(s + wv[e] + i * 32 * C::kWRow);
      p.w[i][0] = v.x; p.w[i][1] = v.y; p.w[i][2] = v.z; p.w[i][3] = v.w;
    }
#pragma unroll
    for (int j = 0; j < kTJ; ++j) {
#pragma unroll
      for (int q = 0; q < C::kAReads; ++q) {
        const uint32_t off = BITS == 4 ? av[e] : av[2 * e + q];
        const uint4 v = *reinterpret_cast<const uint4*>(s + off + j * 32 * C::kARow);
        p.a[j][4 * q] = v.x; p.a[j][4 * q + 1] = v.y; p.a[j][4 * q + 2] = v.z; p.a[j][4 * q + 3] = v.w;
      }
    }
  };
  // Read r of read_chunk's sequence (weight fragments, then activation
  // reads), so that other work can be placed between the reads.
  auto read_one = [&](auto rc, int buf, int e, Packed& p) __attribute__((always_inline)) {
    constexpr int r = decltype(rc)::value;
    const uint8_t* s = smem + buf * C::kStage;
    if constexpr (r < kTI) {
      const uint4 v = *reinterpret_cast<const uint4*>(s + wv[e] + r * 32 * C::kWRow);
      p.w[r][0] = v.x; p.w[r][1] = v.y; p.w[r][2] = v.z; p.w[r][3] = v.w;
    } else {
      constexpr int j = (r - kTI) / C::kAReads, q = (r - kTI) % C::kAReads;
      const uint32_t off = BITS == 4 ? av[e] : av[2 * e + q];
      const uint4 v = *reinterpret_cast<const uint4*>(s + off + j * 32 * C::kARow);
      p.a[j][4 * q] = v.x; p.a[j][4 * q + 1] = v.y; p.a[j][4 * q + 2] = v.z; p.a[j][4 * q + 3] = v.w;
    }
  };
  // MFMA operands of step kk (32 k) of a chunk.
  auto unpack = [&](const Packed& p, int kk, Ops& o) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < kTI; ++i) o.w[i] = op_from_nibbles(p.w[i][2 * kk], p.w[i][2 * kk + 1]);
#pragma unroll
    for (int j = 0; j < kTJ; ++j) {
      if (BITS == 4) o.a[j] = op_from_nibbles(p.a[j][2 * kk], p.a[j][2 * kk + 1]);
      else o.a[j] = op_a8<WA8>(p.a[j][4 * kk], p.a[j][4 * kk + 1], p.a[j][4 * kk + 2], p.a[j][4 * kk + 3]);
    }
  };
  v16i acc[kTI][kTJ];
  auto mfmas = [&](const Ops& o) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < kTI; ++i)
#pragma unroll
      for (int j = 0; j < kTJ; ++j) acc[i][j] = mfma32(o.w[i], o.a[j], acc[i][j]);
  };
  constexpr int kNM = C::kMfma, kVH = C::kVHi, kNH = C::kNHi, kNR = C::kReads;

  // Epilogue of the tile at (m0, n0) with its scales in slot q.  Lane l holds
  // column m = l & 31 of each 32 x 32 accumulator and, in registers 4b ..
  // 4b+3, rows n = 8 b + 4 g + 0..3.  For b = 2p, 2p + 1 a swap of the upper
  // half-wavefront's first value with the lower half's second gives lane l <
  // 32 the halves n = 16 p + 0..7 and lane l + 32 the halves 16 p + 8..15 of
  // row m: one 16-byte store each.
  auto epilogue = [&](int m0, int n0, int q) __attribute__((always_inline)) {
    const float* sc = reinterpret_cast<const float*>(smem + C::kRing + q * C::kScaleSlot);
    const int mbase = wm * kTJ * 32 + fr, nbase = wn * kTI * 32;
    if (ACC_OUT) {
#pragma unroll
      for (int j = 0; j < kTJ; ++j) {
        const int m = m0 + mbase + j * 32;
#pragma unroll
        for (int i = 0; i < kTI; ++i)
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            const int n = n0 + nbase + i * 32 + 8 * b + 4 * fg;
            *reinterpret_cast<int4*>(acc_out + (size_t)m * N + n) =
                make_int4(unscale<BITS>(acc[i][j][4 * b]), unscale<BITS>(acc[i][j][4 * b + 1]),
                          unscale<BITS>(acc[i][j][4 * b + 2]), unscale<BITS>(acc[i][j][4 * b + 3]));
          }
      }
      return;
    }
#pragma unroll
    for (int j = 0; j < kTJ; ++j) {
      const float as = sc[mbase + j * 32];
      const int m = m0 + mbase + j * 32;
      const int off = ZP ? (1 << (BITS - 1)) - a_zeros[m] : 0;
#pragma unroll
      for (int i = 0; i < kTI; ++i) {
#pragma unroll
        for (int p = 0; p < 2; ++p) {
          const int nl = nbase + i * 32 + 16 * p + 4 * fg;
          const float4 ws0 = *reinterpret_cast<const float4*>(sc + 256 + nl);
          const float4 ws1 = *reinterpret_cast<const float4*>(sc + 256 + nl + 8);
          int4 wz0 = make_int4(0, 0, 0, 0), wz1 = make_int4(0, 0, 0, 0);
          if constexpr (ZP) {
            wz0 = *reinterpret_cast<const int4*>(w_sums + n0 + nl);
            wz1 = *reinterpret_cast<const int4*>(w_sums + n0 + nl + 8);
          }
          const uint2 x0 = dequant4z<BITS, ZP>(acc[i][j][8 * p], acc[i][j][8 * p + 1], acc[i][j][8 * p + 2],
                                               acc[i][j][8 * p + 3], as, ws0, off, wz0);
          const uint2 x1 = dequant4z<BITS, ZP>(acc[i][j][8 * p + 4], acc[i][j][8 * p + 5],
                                               acc[i][j][8 * p + 6], acc[i][j][8 * p + 7], as, ws1, off, wz1);
          const auto s0 = __builtin_amdgcn_permlane32_swap(x0.x, x1.x, false, false);
          const auto s1 = __builtin_amdgcn_permlane32_swap(x0.y, x1.y, false, false);
          const int n = n0 + nbase + i * 32 + 16 * p + 8 * fg;
          *reinterpret_cast<uint4*>(y + (size_t)m * N + n) = make_uint4(s0[0], s1[0], s0[1], s1[1]);
        }
        // One accumulator at a time: keeps the scheduler from reading all of
        // them out of the accumulator registers at once.
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  };

  // Ring: global stage g (stage g mod nst of tile g / nst) lives in buffer
  // g mod kB.  The loads of stage g + kB - 1 are issued at the barrier that
  // opens stage g, into the buffer of stage g - 1 (every wavefront has waited
  // for all its reads of it by then).  Every barrier issues exactly one stage
  // (after the last tile's end the last stage again, into a buffer nobody
  // reads any more), so at the barrier opening stage g the kB - 2 stages
  // after it are exactly the loads allowed in flight.
  Packed p0, p1;
  Ops u0, u1;
  int m0, n0;
  origin(0, m0, n0);
  issue_scales(m0, n0, 0);
  const uint8_t* wt0 = wtile_of(n0);
  const uint8_t* at0 = atile_of(m0);
#pragma unroll
  for (int st = 0; st < kB - 1; ++st) issue(wt0, at0, st, st);
  wait_vmcnt<(kB - 2) * C::kLoads>();
  lds_barrier();
  issue(wt0, at0, kB - 1, kB - 1);
  read_chunk(0, 0, p0);
  unpack(p0, 0, u0);
  int cur = 0;   // buffer of the current stage
  for (int r = 0; r < ntile; ++r) {
    const bool has_next = r + 1 < ntile;
    int m1 = m0, n1 = n0;
    if (has_next) origin(r + 1, m1, n1);
    const uint8_t* wt1 = wtile_of(n1);
    const uint8_t* at1 = atile_of(m1);
#pragma unroll
    for (int i = 0; i < kTI; ++i)
#pragma unroll
      for (int j = 0; j < kTJ; ++j) acc[i][j] = v16i{};
    for (int s = 0; s < nst - 1; ++s) {
      const int nxt = cur + 1 == kB ? 0 : cur + 1;
      read_chunk(cur, 1, p1);
      mfmas(u0);
      unpack(p0, 1, u1);
      sched_step<0, kNM, kVH, kNH, kNR>();
      mfmas(u1);
      unpack(p1, 0, u0);
      sched_step<0, kNM, kVH, kNH, 0>();
      wait_vmcnt<(kB - 2) * C::kLoads>();
      lds_barrier();
      // Stage s + kB of this tile, or of the next one (after the last tile:
      // this tile's last stage again).
      // Its loads leave in five parts spread over the rest of this stage:
      // after the barrier, between the reads of the next chunk (which the
      // scheduling groups spread over the MFMAs), and after each group of
      // 12 MFMAs.  All of them are issued before the next wait, so the
      // counts hold.
      const int si = s + kB;
      const bool in_next = si >= nst;
      const uint8_t* iw = in_next ? wt1 : wt0;
      const uint8_t* ia = in_next ? at1 : at0;
      const int ist = in_next ? (has_next ? si - nst : nst - 1) : si;
      constexpr int L = C::kLoads;
      issue_part(std::integral_constant<int, 0>{}, std::integral_constant<int, L / 5>{}, iw, ia, ist, cur);
      [&]<int... R>(std::integer_sequence<int, R...>) __attribute__((always_inline)) {
        (
            [&] {
              read_one(std::integral_constant<int, R>{}, nxt, 0, p0);
              if constexpr (R == kNR / 3)
                issue_part(std::integral_constant<int, L / 5>{}, std::integral_constant<int, 2 * L / 5>{}, iw,
                           ia, ist, cur);
              if constexpr (R == 2 * kNR / 3)
                issue_part(std::integral_constant<int, 2 * L / 5>{}, std::integral_constant<int, 3 * L / 5>{},
                           iw, ia, ist, cur);
            }(),
            ...);
      }(std::make_integer_sequence<int, kNR>{});
      mfmas(u0);
      unpack(p1, 1, u1);
      sched_step<0, kNM, kVH, kNH, kNR>();
      __builtin_amdgcn_sched_barrier(0);
      issue_part(std::integral_constant<int, 3 * L / 5>{}, std::integral_constant<int, 4 * L / 5>{}, iw, ia, ist,
                 cur);
      __builtin_amdgcn_sched_barrier(0);
      mfmas(u1);
      unpack(p0, 0, u0);
      sched_step<0, kNM, kVH, kNH, 0>();
      __builtin_amdgcn_sched_barrier(0);
      issue_part(std::integral_constant<int, 4 * L / 5>{}, std::integral_constant<int, L>{}, iw, ia, ist, cur);
      __builtin_amdgcn_sched_barrier(0);
      cur = nxt;
    }
    {
      // Last stage: the next tile's first chunk is read only after the
      // epilogue, so that no operand registers are held across it.
      read_chunk(cur, 1, p1);
      mfmas(u0);
      unpack(p0, 1, u1);
      sched_step<0, kNM, kVH, kNH, kNR>();
      mfmas(u1);
      unpack(p1, 0, u0);
      sched_step<0, kNM, kVH, kNH, 0>();
      if (has_next) {
        wait_vmcnt<(kB - 2) * C::kLoads>();
        lds_barrier();
        issue(wt1, at1, kB - 1, cur);
        issue_scales(m1, n1, (r + 1) & 1);
      }
      mfmas(u0);
      unpack(p1, 1, u1);
      sched_step<0, kNM, kVH, kNH, 0>();
      mfmas(u1);
      cur = cur + 1 == kB ? 0 : cur + 1;
    }
    epilogue(m0, n0, r & 1);
    if (has_next) {
      read_chunk(cur, 0, p0);
      unpack(p0, 0, u0);
    }
    m0 = m1;
    n0 = n1;
    wt0 = wt1;
    at0 = at1;
  }
  wait_vmcnt<0>();   // the re-issued tail loads land before the workgroup's LDS is released
}

// ---------------------------------------------------------------------------
// Decode (M <= 16): one workgroup per NB blocks of 16 output channels; its 8
// wavefronts split K, stream the weight rows once with 16-byte loads, and
// the int32 partial tiles are summed exactly in LDS.  Every workgroup reads
// all M activation rows of its K range, so when those rows are as many bytes
// as its weights two blocks share them (NB = 2).
// ---------------------------------------------------------------------------
constexpr int kDecWaves = 8;
constexpr int kDecBatch = 4;

// ZP: the range quantizer's zero-point correction in the epilogue,
// acc + (2^(BITS-1) - a_zeros[m]) * w_sums[n] (exact int32), before the
// dequantization.  WDEC: weights in the decode layout (below), where the
// 16 rows x 64 bytes of a block's 128-k chunk are one contiguous KiB in lane
// order, so each load instruction streams 1 KiB instead of 16 runs of 64
// bytes 8 K bytes apart.
// BATCH: chunks per wavefront in flight (kDecBatch, or 8 where a wavefront
// streams many chunks and the grid is at most one workgroup per compute
// unit: decode_batch).
template <int BITS, bool ACC_OUT, bool ZP = false, bool WA8 = false, int NB = 1, bool WDEC = false,
          int BATCH = kDecBatch>
__global__ void __launch_bounds__(kDecWaves * 64)
qgemm_decode(const uint8_t* __restrict__ a_codes, const float* __restrict__ a_scales,
             const uint8_t* __restrict__ w_packed, const float* __restrict__ w_scales,
             int M, int N, int K, __half* __restrict__ y, int32_t* __restrict__ acc_out,
             const int32_t* __restrict__ a_zeros = nullptr,
             const int32_t* __restrict__ w_sums = nullptr) {
  static_assert(NB == 1 || NB == 2, "blocks per workgroup");
  __shared__ v4i part[NB][kDecWaves][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n0 = blockIdx.x * 16 * NB;
  const int fr = lane & 15, fg = lane >> 4;
  const int nck = K / 128;
  const int c_begin = (int)((long)nck * wave / kDecWaves);
  const int c_end = (int)((long)nck * (wave + 1) / kDecWaves);
  const bool mvalid = fr < M;

  const size_t wrow = (size_t)K / 2;
  // Chunk ck of weight block nb (16 rows) at wp + nb * 16 * wrow + ck * kChunk.
  constexpr size_t kChunk = WDEC ? 1024 : 64;
  const uint8_t* wp = WDEC ? w_packed + (size_t)n0 * wrow + lane * 16
                           : w_packed + (size_t)(n0 + fr) * wrow + fg * 16;
  const size_t arow = BITS == 4 ? (size_t)K / 2 : (size_t)K;
  const uint8_t* ap = a_codes + (size_t)(mvalid ? fr : 0) * arow + (BITS == 4 ? fg * 16 : fg * 32);

  v4i acc[NB];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) acc[nb] = v4i{0, 0, 0, 0};
  for (int c = c_begin; c < c_end; c += BATCH) {
    uint4 wv[NB][BATCH], av[BATCH], av2[BATCH];
#pragma unroll
    for (int b = 0; b < BATCH; ++b) {
      const int ck = c + b;
      const bool ok = ck < c_end;
#pragma unroll
      for (int nb = 0; nb < NB; ++nb)
        wv[nb][b] = ok ? *reinterpret_cast<const uint4*>(wp + (size_t)nb * 16 * wrow + (size_t)ck * kChunk)
                       : make_uint4(0, 0, 0, 0);
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
    for (int b = 0; b < BATCH; ++b) {
      v4i b0, b1;
      if (BITS == 4) {
        b0 = op_from_nibbles(av[b].x, av[b].y);
        b1 = op_from_nibbles(av[b].z, av[b].w);
      } else {
        b0 = op_a8<WA8>(av[b].x, av[b].y, av[b].z, av[b].w);
        b1 = op_a8<WA8>(av2[b].x, av2[b].y, av2[b].z, av2[b].w);
      }
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        acc[nb] = mfma(op_from_nibbles(wv[nb][b].x, wv[nb][b].y), b0, acc[nb]);
        acc[nb] = mfma(op_from_nibbles(wv[nb][b].z, wv[nb][b].w), b1, acc[nb]);
      }
    }
  }
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) part[nb][wave][lane] = acc[nb];
  __syncthreads();
  // Wavefront nb < NB sums and writes block nb.
  if (wave >= NB) return;
  v4i tot = part[wave][0][lane];
#pragma unroll
  for (int w = 1; w < kDecWaves; ++w) {
    const v4i p = part[wave][w][lane];
    tot.x += p.x; tot.y += p.y; tot.z += p.z; tot.w += p.w;
  }
  if (!mvalid) return;
  const int m = fr, n = n0 + wave * 16 + fg * 4;
  int c0 = unscale<BITS>(tot.x), c1 = unscale<BITS>(tot.y);
  int c2 = unscale<BITS>(tot.z), c3 = unscale<BITS>(tot.w);
  if constexpr (ZP) {
    const int off = (1 << (BITS - 1)) - a_zeros[m];
    const int4 ws = *reinterpret_cast<const int4*>(w_sums + n);
    c0 += off * ws.x;
    c1 += off * ws.y;
    c2 += off * ws.z;
    c3 += off * ws.w;
  }
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

// Blocks of 16 output channels per decode workgroup.  A one-block workgroup
// reads M * K * bits / 8 activation bytes beside 8 K weight bytes; once the
// activations are as large (M * bits >= 64) two blocks share them, provided
// N still gives two workgroups per compute unit.  (Four blocks were slower
// at 8 tokens and 4 bits on the 57344-channel shape: measured.)
int decode_blocks(int64_t M, int64_t N, int bits, int cus) {
  if (M * bits >= 64 && N % 32 == 0 && N / 32 >= 2 * (int64_t)cus) return 2;
  return 1;
}

// Eight chunks in flight instead of four: measured faster (graph-replayed,
// decode layout) where a wavefront streams at least 12 chunks, the grid is at
// most one workgroup per compute unit and M <= 4 (LLaMA-3-8B down, K = 14336,
// N = 4096: M = 1 A4 7.90 -> 7.25 us, M = 4 A4 8.30 -> 7.40 us, M = 1 A8
// 8.60 -> 8.35 us), and slower with fewer chunks or more workgroups (K = 4096,
// N = 12288, M = 1: 6.53 -> 8.25 us; K = 8192, N = 57344, M = 8: 43.4 ->
// 48.0 us at A8).
bool decode_batch8(int64_t M, int K, int64_t N, int cus) {
  return M <= 4 && K / 128 >= 12 * kDecWaves && N / 16 <= cus;
}

template <int BITS, bool ACC_OUT, bool WA8, bool ZP, bool WDEC = false>
void launch_decode(const uint8_t* a, const float* as, int64_t M, int K, const uint8_t* w,
                   const float* ws, int64_t N, __half* y, int32_t* acc, const int32_t* az,
                   const int32_t* wsum, hipStream_t stream) {
  const int cus = device_cus();
  const int nb = decode_blocks(M, N, BITS, cus);
  if (nb == 1 && decode_batch8(M, K, N, cus)) {
    hipLaunchKernelGGL((qgemm_decode<BITS, ACC_OUT, ZP, WA8, 1, WDEC, 8>), dim3((unsigned)(N / 16)),
                       dim3(kDecWaves * 64), 0, stream, a, as, w, ws, (int)M, (int)N, K, y, acc, az,
                       wsum);
    return;
  }
  switch (nb) {
    case 2:
      hipLaunchKernelGGL((qgemm_decode<BITS, ACC_OUT, ZP, WA8, 2, WDEC>), dim3((unsigned)(N / 32)),
                         dim3(kDecWaves * 64), 0, stream, a, as, w, ws, (int)M, (int)N, K, y, acc,
                         az, wsum);
      break;
    default:
      hipLaunchKernelGGL((qgemm_decode<BITS, ACC_OUT, ZP, WA8, 1, WDEC>), dim3((unsigned)(N / 16)),
                         dim3(kDecWaves * 64), 0, stream, a, as, w, ws, (int)M, (int)N, K, y, acc,
                         az, wsum);
      break;
  }
}

// Canonical 4-bit weights [N, K/2] -> the decode layout: block b of 16 rows,
// chunk c of 128 k, piece g of 16 bytes, row r of the block -> the 16 bytes
// at ((b * (K / 128) + c) * 4 + g) * 256 + r * 16, copied from row 16 b + r,
// bytes 64 c + 16 g .. 64 c + 16 g + 15.  One 16-byte piece per thread.
__global__ void __launch_bounds__(256)
pack_decode_kernel(const uint4* __restrict__ w, int64_t npieces, int K, uint4* __restrict__ out) {
  const int64_t o = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (o >= npieces) return;
  const int64_t per_block = (int64_t)(K / 128) * 64;     // 16-byte pieces per 16-row block
  const int64_t b = o / per_block;
  const int rem = (int)(o - b * per_block);
  const int c = rem >> 6, l = rem & 63;
  const int r = l & 15, g = l >> 4;
  const int64_t row_pieces = K / 32;                     // 16-byte pieces per row
  out[o] = w[(16 * b + r) * row_pieces + 4 * c + g];
}

// Weights in the 8-bit activation order: dword g of a row holds k = 8g ..
// 8g + 7; canonical nibble i (bits 4i..4i+3) is k = 8g + i, and the packed
// byte j holds k = 8g + j in its low nibble and k = 8g + j + 4 in its high
// one.  One dword per thread.
__global__ void __launch_bounds__(256)
pack_w4_a8_kernel(const uint32_t* __restrict__ w, int64_t ndw, uint32_t* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= ndw) return;
  const uint32_t v = w[i];
  uint32_t o = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    o |= ((v >> (4 * j)) & 0xFu) << (8 * j);
    o |= ((v >> (4 * (j + 4))) & 0xFu) << (8 * j + 4);
  }
  out[i] = o;
}

template <class C, bool ACC_OUT, bool WA8, bool ZP>
void launch_prefill(const uint8_t* a, const float* as, int64_t M, int K, const uint8_t* w,
                    const float* ws, int64_t N, __half* y, int32_t* acc, const int32_t* az,
                    const int32_t* wsum, hipStream_t stream) {
  const int64_t tiles = ((M + C::kBM - 1) / C::kBM) * ((N + C::kBN - 1) / C::kBN);
  hipLaunchKernelGGL((qgemm_prefill<C, ACC_OUT, WA8, ZP>), dim3((unsigned)tiles), dim3(C::kThreads), 0,
                     stream, a, as, w, ws, (int)M, (int)N, K, y, acc, az, wsum);
}

template <int BITS, bool ACC_OUT, bool WA8, bool ZP>
void launch_wide(const uint8_t* a, const float* as, int64_t M, int K, const uint8_t* w,
                 const float* ws, int64_t N, __half* y, int32_t* acc, const int32_t* az,
                 const int32_t* wsum, int cus, hipStream_t stream) {
  using C = Wide<BITS>;
  const int64_t tiles = ((M + C::kBM - 1) / C::kBM) * ((N + C::kBN - 1) / C::kBN);
  const int64_t grid = tiles < cus ? tiles : cus;
  hipLaunchKernelGGL((qgemm_prefill_wide<BITS, ACC_OUT, WA8, ZP>), dim3((unsigned)grid), dim3(C::kThreads),
                     0, stream, a, as, w, ws, (int)M, (int)N, K, y, acc, az, wsum);
}

// Relative time of a launch: rounds of one tile per compute unit, times the
// tile's area over the measured throughput of the tile shape.
double launch_cost(int64_t M, int64_t N, int bm, int bn, double speed, int cus) {
  const int64_t tiles = ((M + bm - 1) / bm) * ((N + bn - 1) / bn);
  return (double)((tiles + cus - 1) / cus) * (double)bm * (double)bn / speed;
}

// Throughput of the wide tiles per unit of tile area relative to the
// 256 x 128 tiles (measured on large prefill shapes).
constexpr double kWideSpeed = 1.3;

template <int BITS>
bool wide_fits(int64_t M, int64_t N, int K) {
  using W = Wide<BITS>;
  return M >= W::kBM && N >= W::kBN && K >= W::kMinK;
}

// Kernel for a shape: M <= 16 streams the weights; otherwise the tile shape
// with the smaller estimated time (the wide tiles need at least one full
// tile and a ring's worth of k).
template <int BITS>
int auto_kernel(int64_t M, int64_t N, int K) {
  if (M <= 16) return kGemmDecode;
  using S = PrefillCfg<BITS>;
  using W = Wide<BITS>;
  const int cus = device_cus();
  if (wide_fits<BITS>(M, N, K) &&
      launch_cost(M, N, W::kBM, W::kBN, kWideSpeed, cus) <= launch_cost(M, N, S::kBM, S::kBN, 1.0, cus))
    return kGemmWide;
  return kGemmTile;
}

template <int BITS, bool ACC_OUT, bool WA8 = false, bool ZP = false>
hipError_t launch_t(const uint8_t* a, const float* as, int64_t M, int K,
                    const uint8_t* w, const float* ws, int64_t N, __half* y,
                    int32_t* acc, int kernel, hipStream_t stream,
                    const int32_t* az = nullptr, const int32_t* wsum = nullptr) {
  if (M == 0) return hipSuccess;
  if (kernel == kGemmAuto) kernel = auto_kernel<BITS>(M, N, K);
  switch (kernel) {
    case kGemmDecode:
      launch_decode<BITS, ACC_OUT, WA8, ZP>(a, as, M, K, w, ws, N, y, acc, az, wsum, stream);
      break;
    case kGemmWide:
      launch_wide<BITS, ACC_OUT, WA8, ZP>(a, as, M, K, w, ws, N, y, acc, az, wsum, device_cus(), stream);
      break;
    default:
      launch_prefill<PrefillCfg<BITS>, ACC_OUT, WA8, ZP>(a, as, M, K, w, ws, N, y, acc, az, wsum, stream);
      break;
  }
  return hipGetLastError();
}

}  // namespace

// Compute units of the current device (cached per device).
int device_cus() {
  static int cache[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cache[dev] == 0) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0)
      v = 256;
    cache[dev] = v;
  }
  return cache[dev];
}

bool gemm_kernel_fits(int kernel, int64_t M, int64_t N, int K, int bits) {
  switch (kernel) {
    case kGemmAuto:
    case kGemmTile:
      return true;
    case kGemmDecode:
      return M <= 16;
    case kGemmWide:
      return bits == 4 ? wide_fits<4>(M, N, K) : wide_fits<8>(M, N, K);
    default:
      return false;
  }
}

hipError_t launch_qlinear_zp(const void* codes, const float* a_scales, const int32_t* a_zeros,
                             int64_t M, int K, int bits, const uint8_t* w_packed,
                             const float* w_scales, const int32_t* w_sums, int64_t N, void* y,
                             hipStream_t stream) {
  const uint8_t* a = static_cast<const uint8_t*>(codes);
  __half* yh = static_cast<__half*>(y);
  if (bits == 4)
    return launch_t<4, false, false, true>(a, a_scales, M, K, w_packed, w_scales, N, yh, nullptr,
                                           kGemmAuto, stream, a_zeros, w_sums);
  return launch_t<8, false, false, true>(a, a_scales, M, K, w_packed, w_scales, N, yh, nullptr,
                                         kGemmAuto, stream, a_zeros, w_sums);
}

hipError_t launch_qlinear(const void* codes, const float* a_scales, int64_t M, int K,
                          int bits, const uint8_t* w_packed, const float* w_scales,
                          int64_t N, void* y, int32_t* out_acc, int kernel, hipStream_t stream) {
  const uint8_t* a = static_cast<const uint8_t*>(codes);
  __half* yh = static_cast<__half*>(y);
  if (out_acc) {
    if (bits == 4)
      return launch_t<4, true>(a, a_scales, M, K, w_packed, w_scales, N, yh, out_acc, kernel, stream);
    return launch_t<8, true>(a, a_scales, M, K, w_packed, w_scales, N, yh, out_acc, kernel, stream);
  }
  if (bits == 4)
    return launch_t<4, false>(a, a_scales, M, K, w_packed, w_scales, N, yh, nullptr, kernel, stream);
  return launch_t<8, false>(a, a_scales, M, K, w_packed, w_scales, N, yh, nullptr, kernel, stream);
}

hipError_t launch_pack_w4_a8(const uint8_t* w_packed, int64_t N, int K, uint8_t* out,
                             hipStream_t stream) {
  const int64_t ndw = N * (K / 8);
  if (ndw == 0) return hipSuccess;
  hipLaunchKernelGGL(pack_w4_a8_kernel, dim3((unsigned)((ndw + 255) / 256)), dim3(256), 0, stream,
                     reinterpret_cast<const uint32_t*>(w_packed), ndw, reinterpret_cast<uint32_t*>(out));
  return hipGetLastError();
}

hipError_t launch_pack_decode(const uint8_t* w_packed, int64_t N, int K, uint8_t* out,
                              hipStream_t stream) {
  const int64_t npieces = N * (K / 32);
  if (npieces == 0) return hipSuccess;
  hipLaunchKernelGGL(pack_decode_kernel, dim3((unsigned)((npieces + 255) / 256)), dim3(256), 0,
                     stream, reinterpret_cast<const uint4*>(w_packed), npieces, K,
                     reinterpret_cast<uint4*>(out));
  return hipGetLastError();
}

hipError_t launch_qlinear_decode_native(const void* codes, const float* a_scales, int64_t M, int K,
                                        int bits, const uint8_t* w_dec, const float* w_scales,
                                        int64_t N, void* y, int32_t* out_acc, hipStream_t stream) {
  if (M == 0) return hipSuccess;
  const uint8_t* a = static_cast<const uint8_t*>(codes);
  __half* yh = static_cast<__half*>(y);
  if (out_acc) {
    if (bits == 4)
      launch_decode<4, true, false, false, true>(a, nullptr, M, K, w_dec, nullptr, N, nullptr,
                                                 out_acc, nullptr, nullptr, stream);
    else
      launch_decode<8, true, false, false, true>(a, nullptr, M, K, w_dec, nullptr, N, nullptr,
                                                 out_acc, nullptr, nullptr, stream);
  } else if (bits == 4) {
    launch_decode<4, false, false, false, true>(a, a_scales, M, K, w_dec, w_scales, N, yh, nullptr,
                                                nullptr, nullptr, stream);
  } else {
    launch_decode<8, false, false, false, true>(a, a_scales, M, K, w_dec, w_scales, N, yh, nullptr,
                                                nullptr, nullptr, stream);
  }
  return hipGetLastError();
}

hipError_t launch_qlinear_a8(const void* codes, const float* a_scales, int64_t M, int K,
                             const uint8_t* w_a8, const float* w_scales, int64_t N, void* y,
                             int kernel, hipStream_t stream) {
  return launch_t<8, false, true>(static_cast<const uint8_t*>(codes), a_scales, M, K, w_a8, w_scales,
                                  N, static_cast<__half*>(y), nullptr, kernel, stream);
}

}  // namespace dptq
