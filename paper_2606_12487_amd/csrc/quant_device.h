// Device helpers of the quantizer shared by the rotate+quantize kernels and
// the fused decode kernel: the H28 table, the rounding of y / s to a code, and
// code packing.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dptq {
namespace qd {

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

// Code bits of y / s rounded to nearest, ties to even: t + 1.5 * 2^23 leaves
// round(t) in the low mantissa bits (two's complement), from which nibbles
// and bytes are packed.  |code| <= qmax holds without a clamp: |t| <=
// fl32(amax / s) with s = fl32(amax / qmax) rounds to at most qmax.
__device__ __forceinline__ uint32_t round_bits(float y, float s, float r) {
  const float q = y * r;
  const float e = __builtin_fmaf(-q, s, y);
  const float t = __builtin_fmaf(e, r, q);
  return __float_as_uint(t + 12582912.0f);          // 1.5 * 2^23
}
// Low bytes of four words: [b0, b1, b2, b3].
__device__ __forceinline__ uint32_t low_bytes(uint32_t b0, uint32_t b1, uint32_t b2, uint32_t b3) {
  const uint32_t x01 = __builtin_amdgcn_perm(b1, b0, 0x0c0c0400u);
  const uint32_t x23 = __builtin_amdgcn_perm(b3, b2, 0x0c0c0400u);
  return __builtin_amdgcn_perm(x23, x01, 0x05040100u);
}
// Eight codes as packed nibbles (element 2j in the low nibble of byte j).
__device__ __forceinline__ uint32_t pack_nibbles(const uint32_t* b) {
  const uint32_t ev = low_bytes(b[0], b[2], b[4], b[6]);
  const uint32_t od = low_bytes(b[1], b[3], b[5], b[7]);
  return (ev & 0x0F0F0F0Fu) | ((od << 4) & 0xF0F0F0F0u);
}

// Rows in LDS as 4096-element segments (register-phase rotation): element i
// of a segment at float offset i + 4 (i >> 6), free of bank conflicts in
// every phase.
constexpr int kSeg = 4096;
constexpr int kSegFloats = kSeg + kSeg / 16;        // 4 floats of padding per 64
__device__ __forceinline__ int seg_off(int i) { return i + 4 * (i >> 6); }

// Butterflies over bit B of the register index of v[16] (stride 2^B).
template <int B>
__device__ __forceinline__ void stage16(float* v) {
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    if (r & (1 << B)) continue;
    const float a = v[r], c = v[r | (1 << B)];
    v[r] = a + c;
    v[r | (1 << B)] = a - c;
  }
}
// Register bits [LO, HI) in order.
template <int LO, int HI>
__device__ __forceinline__ void stages16(float* v) {
  if constexpr (LO < HI) {
    stage16<LO>(v);
    stages16<LO + 1, HI>(v);
  }
}


__device__ __forceinline__ float absmax16(const float* v, float m) {
#pragma unroll
  for (int r = 0; r < 16; r += 2) m = fmaxf(fmaxf(fabsf(v[r]), fabsf(v[r + 1])), m);
  return m;
}

// Maximum over the wavefront of a non-negative float (compared as integer
// bits, which order non-negative floats): four DPP steps give every lane its
// 16-lane row maximum, then the four rows are combined as scalars.
__device__ __forceinline__ float wave_max_nonneg(float m) {
  int v = __float_as_int(m);
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, false));    // quad_perm [1,0,3,2]
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, false));    // quad_perm [2,3,0,1]
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0x141, 0xF, 0xF, false));   // row_half_mirror
  v = max(v, __builtin_amdgcn_mov_dpp(v, 0x140, 0xF, 0xF, false));   // row_mirror
  const int r0 = __builtin_amdgcn_readlane(v, 0), r1 = __builtin_amdgcn_readlane(v, 16);
  const int r2 = __builtin_amdgcn_readlane(v, 32), r3 = __builtin_amdgcn_readlane(v, 48);
  return __int_as_float(max(max(r0, r1), max(r2, r3)));
}

}  // namespace qd
}  // namespace dptq
