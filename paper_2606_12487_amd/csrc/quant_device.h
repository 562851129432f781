// Device helpers of the quantizer shared by the rotate+quantize kernels, the
// range quantizer and the fused decode kernel: the H28 table, the rounding of
// y / s to a code, code packing, and the segmented row rotation.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_fp16.h>
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

// The dense 28-point stage sums column b as acc = +-z[0], then acc +-= z[a]
// for a = 1 .. 27 in order, signs from H28[a][b].  Two columns whose signs
// agree on rows 0 .. a, up to one common sign flip, hold partial sums that
// are equal or exact negatives of each other (fp32 negation is exact and
// round-to-nearest-even is symmetric), so one value serves both; 634 adds
// instead of 756 give the 28 outputs bit for bit.  H28Trie<B0, NB> is that
// sharing plan for columns B0 .. B0 + NB - 1: at depth a, node n continues
// node par[a][n] of depth a - 1, negated when psg < 0, with +-z[a] by zsg;
// the node of the first (lowest) column in a class holds that column's own
// sum, so at depth 27, where every column has a node of its own, fin[b] is
// the node holding output B0 + b.
template <int B0, int NB>
struct H28Trie {
  int cnt[28];
  signed char par[28][28], psg[28][28], zsg[28][28], fin[28];
  constexpr H28Trie() : cnt{}, par{}, psg{}, zsg{}, fin{} {
    int rep[28][NB] = {}, node_of[28][NB] = {}, sig[28][NB] = {};
    for (int a = 0; a < 28; ++a) {
      int reps = 0;
      for (int i = 0; i < NB; ++i) {
        const int b = B0 + i;
        rep[a][i] = -1;
        for (int k = 0; k < i && rep[a][i] < 0; ++k) {
          const int c = B0 + k;
          if (rep[a][k] != k) continue;            // compare with class leaders only
          const int f = kH28.e[0][b] * kH28.e[0][c];
          bool same = true;
          for (int r = 0; r <= a; ++r) same = same && kH28.e[r][b] == f * kH28.e[r][c];
          if (same) {
            rep[a][i] = k;
            sig[a][i] = f;
            node_of[a][i] = node_of[a][k];
          }
        }
        if (rep[a][i] < 0) {
          rep[a][i] = i;
          sig[a][i] = 1;
          node_of[a][i] = reps++;
        }
      }
      cnt[a] = reps;
      if (a > 0) {
        for (int i = 0; i < NB; ++i) {
          if (rep[a][i] != i) continue;
          const int n = node_of[a][i];
          par[a][n] = (signed char)node_of[a - 1][i];
          psg[a][n] = (signed char)sig[a - 1][i];
          zsg[a][n] = kH28.e[a][B0 + i];
        }
      } else {
        zsg[0][0] = kH28.e[0][B0];
      }
    }
    for (int i = 0; i < NB; ++i) fin[i] = (signed char)(sig[27][i] == 1 ? node_of[27][i] : -1);
  }
};

// Outputs B0 .. B0 + NB - 1 of one column of the 28-point stage from its 28
// inputs z: out(b, value) for each, b counted from 0.
template <int B0, int NB>
constexpr bool h28_trie_complete(const H28Trie<B0, NB>& t) {
  if (t.cnt[27] != NB) return false;
  for (int b = 0; b < NB; ++b)
    if (t.fin[b] < 0) return false;
  return true;
}

template <int B0, int NB, typename Out>
__host__ __device__ __forceinline__ void h28_column(const float* z, Out out) {
  constexpr H28Trie<B0, NB> t{};
  static_assert(h28_trie_complete(t), "every column ends on a node of its own, unnegated");
  float nd[NB];
  nd[0] = t.zsg[0][0] > 0 ? z[0] : -z[0];
#pragma unroll
  for (int a = 1; a < 28; ++a) {
    float nn[NB];
#pragma unroll
    for (int n = 0; n < NB; ++n) {
      if (n < t.cnt[a]) {
        const float pv = t.psg[a][n] > 0 ? nd[t.par[a][n]] : -nd[t.par[a][n]];
        nn[n] = t.zsg[a][n] > 0 ? pv + z[a] : pv - z[a];
      }
    }
#pragma unroll
    for (int n = 0; n < NB; ++n)
      if (n < t.cnt[a]) nd[n] = nn[n];
  }
#pragma unroll
  for (int b = 0; b < NB; ++b) out(b, nd[t.fin[b]]);
}

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

// ---------------------------------------------------------------------------
// One row rotated by 256 threads (r = 0..255) in 4096-element LDS segments,
// for h = F * 2^J with F = 28 when F28, else 1, and JP = min(J, 12).  Each
// thread holds 16 elements of a segment in each of three register phases
// covering index bits 0-3, 4-7 and 8-11, in that order; bits 12 and up pair
// whole segments, one LDS pass per bit; for F = 28 a last pass gives each
// thread whole columns of the dense 28-point stage, summed in order over the
// slow index.  K is a multiple of 128, so a thread's 16 elements are all in
// the row or all past it; past the row end the segment is zero (whole
// Hadamard blocks of zeros).  The rotated row is left in rh (element i at
// seg_index(i)).  r is the thread's place in its group of 256 (its part of a
// segment), sp how the row's work is shared.  Every thread of the workgroup
// calls this (it holds barriers); act = false threads only join them.  With use_pre, pre[2 sg] and
// pre[2 sg + 1] are this thread's 16 elements of segment sg < NPRE, loaded by
// the caller (any values where they lie past the row end).
//
// Row maxima, each starting at 0: RANGE = false keeps the absolute maximum
// in ma; RANGE = true keeps max(0, max v) in ma and max(0, max -v) in mb.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int seg_index(int i) { return (i >> 12) * kSegFloats + seg_off(i & (kSeg - 1)); }

// u where ok, else zero (component-wise selects).
__device__ __forceinline__ uint4 keep_or_zero(bool ok, uint4 u) {
  return make_uint4(ok ? u.x : 0u, ok ? u.y : 0u, ok ? u.z : 0u, ok ? u.w : 0u);
}

// Eight fp16 values (one 16-byte load) widened to fp32.
__device__ __forceinline__ void widen8(uint4 u, float* d) {
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    d[2 * k] = __half2float(__ushort_as_half((unsigned short)(w[k] & 0xFFFFu)));
    d[2 * k + 1] = __half2float(__ushort_as_half((unsigned short)(w[k] >> 16)));
  }
}

template <bool RANGE>
__device__ __forceinline__ void row_max1(float v, float& ma, float& mb) {
  if constexpr (RANGE) {
    ma = fmaxf(ma, v);
    mb = fmaxf(mb, -v);
  } else {
    ma = fmaxf(ma, fabsf(v));
  }
}

template <bool RANGE>
__device__ __forceinline__ void row_max16(const float* v, float& ma, float& mb) {
  if constexpr (RANGE) {
#pragma unroll
    for (int q = 0; q < 16; ++q) row_max1<true>(v[q], ma, mb);
  } else {
    ma = absmax16(v, ma);
  }
}

// How the threads of a row share its work: segments sg0, sg0 + sgstep, ... in
// the register phases and the passes across segments, and columns tid,
// tid + nthr, ... in the 28-point pass.  One group of 256 threads per row is
// {0, 1, r, 256}; two groups on one row split the segments by parity.
struct RowSplit {
  int sg0, sgstep, tid, nthr;
};

template <int JP, bool F28, bool RANGE, int NPRE>
__device__ __forceinline__ void rotate_row_segments(const __half* __restrict__ xr, int K, int J,
                                                    bool act, int r, RowSplit sp, bool use_pre,
                                                    const uint4 (&pre)[2 * NPRE], float* rh,
                                                    float& ma, float& mb) {
  const int nseg = (K + kSeg - 1) / kSeg;
  const int b1 = seg_off(16 * r);
  const int b2 = seg_off(256 * (r >> 4) + (r & 15));
  const int b3 = seg_off(r);
  // Phase 1 of segment sg from its 16 fp16 values (zero past the row end).
  auto phase1 = [&](int sg, uint4 u0, uint4 u1) __attribute__((always_inline)) {
    const bool in = sg * kSeg + 16 * r < K;
    float v[16];
    widen8(keep_or_zero(in, u0), v);
    widen8(keep_or_zero(in, u1), v + 8);
    stages16<0, (JP < 4 ? JP : 4)>(v);
    if (JP <= 4) row_max16<RANGE>(v, ma, mb);
    float* sl = rh + sg * kSegFloats + b1;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      *reinterpret_cast<float4*>(sl + 4 * q) = make_float4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3]);
  };
  auto load16 = [&](int sg, int h2) __attribute__((always_inline)) {
    const int e = sg * kSeg + 16 * r;
    return e < K ? *reinterpret_cast<const uint4*>(xr + e + 8 * h2) : make_uint4(0, 0, 0, 0);
  };
  if (act) {
    // The first NPRE segments may come preloaded (the caller issued those
    // loads before others it wants to stay in flight).
    if constexpr (NPRE == 1) {
      for (int sg = sp.sg0; sg < nseg; sg += sp.sgstep) {
        if (use_pre && sg == sp.sg0) phase1(sg, pre[0], pre[1]);
        else phase1(sg, load16(sg, 0), load16(sg, 1));
      }
    } else {
#pragma unroll
      for (int i = 0; i < NPRE; ++i) {
        const int sg = sp.sg0 + i * sp.sgstep;
        if (sg < nseg) {
          if (use_pre) phase1(sg, pre[2 * i], pre[2 * i + 1]);
          else phase1(sg, load16(sg, 0), load16(sg, 1));
        }
      }
      for (int sg = sp.sg0 + NPRE * sp.sgstep; sg < nseg; sg += sp.sgstep)
        phase1(sg, load16(sg, 0), load16(sg, 1));
    }
  }
  if constexpr (JP > 4) {
    __syncthreads();
    if (act) {
      for (int sg = sp.sg0; sg < nseg; sg += sp.sgstep) {
        if (sg * kSeg >= K) continue;
        float* sl = rh + sg * kSegFloats + b2;
        float v[16];
#pragma unroll
        for (int q = 0; q < 16; ++q) v[q] = sl[16 * q + 4 * (q >> 2)];
        stages16<0, (JP < 8 ? JP : 8) - 4>(v);
        if (JP <= 8) row_max16<RANGE>(v, ma, mb);
#pragma unroll
        for (int q = 0; q < 16; ++q) sl[16 * q + 4 * (q >> 2)] = v[q];
      }
    }
  }
  if constexpr (JP > 8) {
    __syncthreads();
    if (act) {
      for (int sg = sp.sg0; sg < nseg; sg += sp.sgstep) {
        if (sg * kSeg >= K) continue;
        float* sl = rh + sg * kSegFloats + b3;
        float v[16];
#pragma unroll
        for (int q = 0; q < 16; ++q) v[q] = sl[272 * q];
        stages16<0, JP - 8>(v);
        row_max16<RANGE>(v, ma, mb);
#pragma unroll
        for (int q = 0; q < 16; ++q) sl[272 * q] = v[q];
      }
    }
  }
  if (F28 || (JP == 12 && J > 12)) {
    // The row maxima are taken in the last pass instead.
    ma = 0.0f;
    mb = 0.0f;
    for (int b = 12; JP == 12 && b < J; ++b) {
      // Bit b: segments s and s + 2^(b - 12), s with that bit clear.
      __syncthreads();
      if (act) {
        const int S = 1 << (b - 12);
        const bool last_pass = b == J - 1 && !F28;
        // Pair p: the segment with bit b - 12 inserted as 0, and its partner.
        for (int p = sp.sg0; p < nseg / 2; p += sp.sgstep) {
          const int sg = ((p >> (b - 12)) << (b - 11)) | (p & (S - 1));
          float* lo = rh + sg * kSegFloats + b1;
          float* hi = lo + S * kSegFloats;
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const float4 a = *reinterpret_cast<const float4*>(lo + 4 * q);
            const float4 c = *reinterpret_cast<const float4*>(hi + 4 * q);
            const float4 s4 = make_float4(a.x + c.x, a.y + c.y, a.z + c.z, a.w + c.w);
            const float4 d4 = make_float4(a.x - c.x, a.y - c.y, a.z - c.z, a.w - c.w);
            *reinterpret_cast<float4*>(lo + 4 * q) = s4;
            *reinterpret_cast<float4*>(hi + 4 * q) = d4;
            if (last_pass) {
              const float o[8] = {s4.x, s4.y, s4.z, s4.w, d4.x, d4.y, d4.z, d4.w};
#pragma unroll
              for (int u = 0; u < 8; ++u) row_max1<RANGE>(o[u], ma, mb);
            }
          }
        }
      }
    }
    if constexpr (F28) {
      // y[b p + c] = sum over a = 0..27, in order, of H28[a][b] z[a p + c],
      // one column (block, c) per thread at a time.
      __syncthreads();
      if (act) {
        const int p = 1 << J;
        for (int col = sp.tid; col < K / 28; col += sp.nthr) {
          const int base = (col >> J) * 28 * p + (col & (p - 1));
          float z[28];
#pragma unroll
          for (int a = 0; a < 28; ++a) z[a] = rh[seg_index(base + a * p)];
          h28_column<0, 28>(z, [&](int bb, float acc) __attribute__((always_inline)) {
            rh[seg_index(base + bb * p)] = acc;
            row_max1<RANGE>(acc, ma, mb);
          });
        }
      }
    }
  }
}

}  // namespace qd
}  // namespace dptq
