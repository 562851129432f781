// W4A4 GEMM on the gfx950 FP6 matrix cores, exact, with the dequant epilogue.
//
//   acc[m,n] = sum_k a[m,k] * w[n,k]                 (4-bit codes, exact)
//   y[m,n]   = fl16(fl32(fl32(fl32(acc) * a_s[m]) * w_s[n]))
//
// The same operation as the int8-MFMA kernels, computed on the block-scaled
// f8f6f4 MFMA, which runs at twice the int8 rate per cycle.  Every 4-bit code
// c in [-8, 7] is exactly representable as the e2m3 value c / 2 (sign, two
// exponent bits with bias 1, three mantissa bits): 0, +-0.5 (subnormal),
// +-1, +-1.5, +-2, +-2.5, +-3, +-3.5 and -4.  With an E8M0 block scale of 2 on
// both operands each product is the exact integer a * w.  The MFMA
// accumulates in fp32; every partial sum is an integer of magnitude at most
// 64 * K <= 2^22 for K <= 65536, so fp32 holds it exactly and the accumulator
// equals the int32 one bit for bit (fl32(acc) in the epilogue is exact too).
//
// FP6 block layout of a [R, K] code matrix (K % 128 == 0): rows are padded
// to Rp = 32 * ceil(R / 32) with zero codes, and the matrix is cut into
// blocks of 32 rows x 128 k, block (rb, kb) at byte offset
// (kb * Rp / 32 + rb) * 3072 (the row blocks of one k block are adjacent, so
// a tile's rows at one k block are one contiguous run).  A block is two halves of 1536 bytes, one per
// 64-k MFMA step s = 0, 1.  In half s, lane l (row 32 rb + (l & 31),
// g = l >> 5) owns the 32 codes k = 128 kb + 64 g + 32 s + j, j = 0..31,
// as a 192-bit value whose six-bit field j (bits 6 j .. 6 j + 5) encodes
// code j; its bytes 8 c .. 8 c + 7 (c = 0, 1, 2) are at 1536 s + 512 c + 8 l.
// A half is thus one MFMA operand for all 64 lanes, laid out so that a block
// moves from memory to LDS as three 1 KiB direct loads and an operand from
// LDS into six consecutive registers as three 8-byte reads per lane, free of
// bank conflicts.

#include "internal.h"

#include <utility>

namespace dptq {
namespace {

typedef int v8i_t __attribute__((ext_vector_type(8)));
typedef float v16f_t __attribute__((ext_vector_type(16)));
typedef __attribute__((address_space(3))) uint8_t* lds_ptr_t;

constexpr int kF6Block = 3072;   // bytes of one 32-row x 128-k block

// e2m3 encoding of c / 2 for the 4-bit two's complement nibble n (c = n for
// n < 8, n - 16 otherwise): byte n & 3 of one of four dwords (c = 0..3, 4..7,
// -8..-5, -4..-1).  Only 32-bit operations: the data path of this file uses
// no 64-bit shifts.
__device__ __forceinline__ uint32_t e2m3_half(uint32_t n) {
  const uint32_t lo = (n & 8u) ? 0x32343638u : 0x0C080400u;
  const uint32_t hi = (n & 8u) ? 0x24282C30u : 0x16141210u;
  return (((n & 4u) ? hi : lo) >> ((n & 3u) * 8u)) & 0x3Fu;
}

// ---------------------------------------------------------------------------
// Canonical packed 4-bit codes [R, K/2] -> FP6 block layout.  One thread per
// (block, lane): it reads the lane's 32 code bytes (64 codes), encodes two
// 192-bit operands and writes them to the two halves of the block.
// ---------------------------------------------------------------------------
__global__ void __launch_bounds__(256)
pack_fp6_kernel(const uint8_t* __restrict__ codes, int R, int K, uint8_t* __restrict__ out,
                int64_t nslots) {
  const int64_t slot = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (slot >= nslots) return;
  const int64_t nrb = (R + 31) / 32;
  const int64_t blk = slot >> 6;
  const int l = (int)(slot & 63);
  const int kb = (int)(blk / nrb);
  const int64_t rb = blk - kb * nrb;
  const int64_t r = rb * 32 + (l & 31);
  uint4 in0 = make_uint4(0, 0, 0, 0), in1 = make_uint4(0, 0, 0, 0);
  if (r < R) {
    const uint8_t* src = codes + r * (int64_t)(K / 2) + kb * 64 + (l >> 5) * 32;
    in0 = *reinterpret_cast<const uint4*>(src);
    in1 = *reinterpret_cast<const uint4*>(src + 16);
  }
  const uint32_t w[8] = {in0.x, in0.y, in0.z, in0.w, in1.x, in1.y, in1.z, in1.w};
  uint8_t* base = out + blk * kF6Block;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    // Codes 32 h .. 32 h + 31 of the lane's 64 (input dwords 4 h .. 4 h + 3):
    // field j occupies bits 6 j .. 6 j + 5 of the six output dwords.
    uint32_t o[6] = {0u, 0u, 0u, 0u, 0u, 0u};
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      const uint32_t f = e2m3_half((w[4 * h + j / 8] >> (4 * (j % 8))) & 15u);
      const int d = (6 * j) / 32, off = (6 * j) % 32;
      o[d] |= f << off;
      if (off > 26) o[d + 1] |= f >> (32 - off);
    }
#pragma unroll
    for (int c = 0; c < 3; ++c)
      *reinterpret_cast<uint2*>(base + 1536 * h + 512 * c + 8 * l) = make_uint2(o[2 * c], o[2 * c + 1]);
  }
}

// ---------------------------------------------------------------------------
// GEMM.  192 (n) x 256 (m) output tiles on four wavefronts, one per SIMD,
// each 96 x 128 = 3 x 4 MFMAs of 32 x 32 x 64 per 64-k step.  Persistent:
// one workgroup per compute unit walks its tiles.  K is consumed in stages
// of 128 (one block column) through a ring of three LDS stage buffers
// filled by direct global->LDS loads.  Operands are read into registers one
// 64-k step ahead of their MFMAs.  The barrier that lets stage g + 3 into
// stage g's buffer sits between the two steps of stage g, once every read of
// stage g has returned, so a stage's loads have two stages of MFMA time to
// land.  The ring runs on across tile boundaries.  Tiles that overhang the padded matrix
// clamp their block rows (the duplicate rows feed only discarded results).
// ---------------------------------------------------------------------------
struct F6 {
  static constexpr int kBN = 192, kBM = 256, kTI = 3, kTJ = 4;
  static constexpr int kWBlk = kBN / 32, kABlk = kBM / 32;      // 6, 8
  static constexpr int kW = kWBlk * kF6Block;                   // 18 KiB
  static constexpr int kA = kABlk * kF6Block;                   // 24 KiB
  static constexpr int kStage = kW + kA;                        // 42 KiB
  static constexpr int kBufs = 3;
  static constexpr int kRing = kBufs * kStage;
  static constexpr int kScaleSlot = 2048;                       // a_s [256] + w_s [192]
  static constexpr int kLds = kRing + 2 * kScaleSlot;
  static constexpr int kLoads = kStage / 1024;                  // 42 per stage
  static constexpr int kWLoads = kW / 1024;                     // the first 18 are weights
  static_assert(kLds <= 160 * 1024, "LDS budget");
  static_assert(kLoads == 42, "load split");
  // Wavefront w issues loads Q0(w) .. Q0(w) + NL(w) - 1 of a stage.
  static constexpr int q0(int w) { return w < 2 ? 11 * w : 22 + 10 * (w - 2); }
  static constexpr int nl(int w) { return w < 2 ? 11 : 10; }
};

__device__ __forceinline__ void f6_dma16(const void* sbase, uint32_t voff, uint32_t lds_off) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(sbase), "s"(lds_off)
               : "memory", "m0");
}
// The same with the LDS destination a wavefront-uniform base plus a
// compile-time offset, formed in M0 by one scalar add; the global address is
// sbase + voff.
template <uint32_t OFF>
__device__ __forceinline__ void f6_dma16_at(const void* sbase, uint32_t voff, uint32_t lds_base) {
  asm volatile("s_add_u32 m0, %2, %3\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(sbase), "s"(lds_base), "i"(OFF)
               : "memory", "m0", "scc");
}
__device__ __forceinline__ void f6_dma4(const void* sbase, uint32_t voff, uint32_t lds_off) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dword %0, %1"
               :
               : "v"(voff), "s"(sbase), "s"(lds_off)
               : "memory", "m0");
}
__device__ __forceinline__ void f6_barrier() { asm volatile("s_barrier" ::: "memory"); }

template <int N>
__device__ __forceinline__ void f6_wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
__device__ __forceinline__ void f6_wait_lgkm0() {
  __builtin_amdgcn_s_waitcnt((15) | (3 << 14) | (7 << 4) | (0 << 8));
}

__device__ __forceinline__ int f6_xcd_remap(int bid, int total) {
  const int per = total >> 3, rem = total & 7;
  const int x = bid & 7, idx = bid >> 3;
  return x * per + (x < rem ? x : rem) + idx;
}

// Scheduling groups: NM MFMAs, each followed by two LDS reads for the first
// ND of them and one after the rest.
template <int Q, int NM, int ND>
__device__ __forceinline__ void f6_sched() {
  if constexpr (Q < NM) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, Q < ND ? 2 : 1, 0);
    f6_sched<Q + 1, NM, ND>();
  }
}

// Scheduling groups of a stage: NM MFMAs with the stage's LDS reads spread
// between them (one after each, two after the first few).
template <int Q, int NM, int NLD>
__device__ __forceinline__ void f6_sched_mixed() {
  if constexpr (Q < NM) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x100, Q < 4 ? 2 : 1, 0);
    f6_sched_mixed<Q + 1, NM, NLD>();
  }
}

// The part of a stage's loads issued after operand read f when a stage's
// frags reads carry its loads in parts (part k after read k * frags / parts
// - 1), or 0 when none follows read f.
constexpr int f6_part_after(int f, int frags, int parts) {
  for (int k = 1; k < parts; ++k)
    if (f == k * frags / parts - 1) return k;
  return 0;
}

// One MFMA step: fp6 x fp6, E8M0 scale 128 (= 2) on both operands.
__device__ __forceinline__ v16f_t mfma_f6(const uint32_t* w, const uint32_t* a, v16f_t c) {
  const v8i_t wa = {(int)w[0], (int)w[1], (int)w[2], (int)w[3], (int)w[4], (int)w[5], 0, 0};
  const v8i_t ab = {(int)a[0], (int)a[1], (int)a[2], (int)a[3], (int)a[4], (int)a[5], 0, 0};
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(wa, ab, c, 2, 2, 0, 128, 0, 128);
}

// fl16(fl32(fl32(acc) * as) * ws); acc is an exact integer held in fp32.  The
// empty asm keeps the second product an fp32 value (see the int8 kernels).
__device__ __forceinline__ __half f6_dequant(float acc, float as, float ws) {
  const float t1 = acc * as;
  float t2 = t1 * ws;
  asm("" : "+v"(t2));
  return __float2half_rn(t2);
}

__device__ __forceinline__ uint2 f6_dequant4(float a0, float a1, float a2, float a3, float as,
                                             float4 ws) {
  const __half h0 = f6_dequant(a0, as, ws.x), h1 = f6_dequant(a1, as, ws.y);
  const __half h2 = f6_dequant(a2, as, ws.z), h3 = f6_dequant(a3, as, ws.w);
  uint2 pk;
  pk.x = (uint32_t)__half_as_ushort(h0) | ((uint32_t)__half_as_ushort(h1) << 16);
  pk.y = (uint32_t)__half_as_ushort(h2) | ((uint32_t)__half_as_ushort(h3) << 16);
  return pk;
}

// Body of the GEMM for wavefront WV of a workgroup.  Fast shapes (at least
// one full tile of padded rows each way and three stages per tile) shift edge
// tiles inward so every load is a base plus a constant; the CLAMP variant
// (small shapes) clamps each block row instead.
template <int WV, bool ACC_OUT, bool CLAMP>
__device__ __forceinline__ void qgemm_fp6_body(const uint8_t* __restrict__ a6,
                                               const float* __restrict__ a_scales,
                                               const uint8_t* __restrict__ w6,
                                               const float* __restrict__ w_scales, int M, int N,
                                               int K, __half* __restrict__ y,
                                               int32_t* __restrict__ acc_out, uint8_t* smem) {
  using C = F6;
  constexpr int kTI = C::kTI, kTJ = C::kTJ;
  constexpr int WN = WV & 1, WM = WV >> 1;
  constexpr int Q0 = C::q0(WV), NL = C::nl(WV);

  const int tiles_m = (M + C::kBM - 1) / C::kBM;
  const int tiles_n = (N + C::kBN - 1) / C::kBN;
  const int total = tiles_m * tiles_n;
  const int G = gridDim.x;                                       // <= total
  const int ntile = (total - (int)blockIdx.x + G - 1) / G;       // >= 1
  const int nkb = K / 128;                                       // stages per tile
  const int mblk = (M + 31) / 32, nblk = (N + 31) / 32;
  const int lane = threadIdx.x & 63;

  // Row origins of this workgroup's tile r (r clamped to its last tile).
  // The workgroups of one XCD take consecutive logical tiles, and logical
  // tiles run in groups of kGroupM tile rows, m fastest within a group: a
  // round of 32 tiles on one XCD is a 4 (m) x 8 (n) block, whose operands
  // (4 activation and 8 weight tiles) share that XCD's L2.
  auto origin = [&](int r, int& m0, int& n0) __attribute__((always_inline)) {
    r = min(r, ntile - 1);
    const int logical = f6_xcd_remap((int)blockIdx.x + r * G, total);
    constexpr int kGroupM = 4;
    const int per_group = kGroupM * tiles_n;
    const int g = logical / per_group, t = logical - g * per_group;
    const int gm = min(kGroupM, tiles_m - g * kGroupM);
    const int tn = t / gm, tm = g * kGroupM + (t - tn * gm);
    m0 = tm * C::kBM;
    n0 = tn * C::kBN;
    if constexpr (!CLAMP) {
      m0 = min(m0, mblk * 32 - C::kBM);
      n0 = min(n0, nblk * 32 - C::kBN);
    }
  };

  const uint32_t smem_base = (uint32_t)(uintptr_t)(lds_ptr_t)smem;
  const uint32_t lane16 = (uint32_t)lane * 16;
  const size_t wstride = (size_t)nblk * kF6Block, astride = (size_t)mblk * kF6Block;

  // Loads of one stage: kb of the tile whose first blocks are at wt / at,
  // into ring buffer buf.  Load q < 18 is part q % 3 of weight block q / 3,
  // load q >= 18 part of activation block (q - 18) / 3; it lands at q KiB.
  // Loads P0 .. P1 - 1 of this wavefront's NL.
  auto issue_part = [&](const uint8_t* wt, const uint8_t* at, int rbw, int rba, int kb, int buf, auto p0c,
                        auto p1c) __attribute__((always_inline)) {
    constexpr int P0 = decltype(p0c)::value, P1 = decltype(p1c)::value;
    const uint8_t* wst = wt + (size_t)kb * wstride;
    const uint8_t* ast = at + (size_t)kb * astride;
    const uint32_t base = smem_base + buf * C::kStage;
    if constexpr (!CLAMP) {
      // Contiguous: load q reads 1 KiB at a constant offset from the stage base.
      auto one = [&](auto qc) __attribute__((always_inline)) {
        constexpr int q = decltype(qc)::value;
        constexpr int rel = q < C::kWLoads ? q : q - C::kWLoads;
        // The block offset travels in the per-lane offset (one vector
        // instruction) and the LDS offset in M0's add, so a load costs one
        // scalar instruction beside it.
        f6_dma16_at<(uint32_t)(q * 1024)>(q < C::kWLoads ? wst : ast, lane16 + (uint32_t)(rel * 1024), base);
      };
      [&]<int... I>(std::integer_sequence<int, I...>) __attribute__((always_inline)) {
        (one(std::integral_constant<int, Q0 + P0 + I>{}), ...);
      }(std::make_integer_sequence<int, P1 - P0>{});
    } else {
#pragma unroll
      for (int i = P0; i < P1; ++i) {
        const int q = Q0 + i;
        const bool isa = q >= C::kWLoads;
        const int qq = isa ? q - C::kWLoads : q;
        const int b = qq / 3;
        const int rb = isa ? min(rba + b, mblk - 1) : min(rbw + b, nblk - 1);
        const uint8_t* src = (isa ? a6 + (size_t)kb * astride : w6 + (size_t)kb * wstride) +
                             (uint32_t)(rb * kF6Block + (qq - 3 * b) * 1024);
        f6_dma16(src, lane16, base + q * 1024);
      }
    }
  };
  auto issue = [&](const uint8_t* wt, const uint8_t* at, int rbw, int rba, int kb, int buf)
      __attribute__((always_inline)) {
    issue_part(wt, at, rbw, rba, kb, buf, std::integral_constant<int, 0>{}, std::integral_constant<int, NL>{});
  };
  // Scales of tile r into slot r & 1 (only when producing y): wavefront 0
  // loads a_s [256], wavefront 1 w_s [192], 4 bytes per lane, rows clamped.
  auto issue_scales = [&](int r) __attribute__((always_inline)) {
    if constexpr (!ACC_OUT && WV < 2) {
      if (r >= ntile) return;
      int m0, n0;
      origin(r, m0, n0);
      const uint32_t base = smem_base + C::kRing + (r & 1) * C::kScaleSlot;
      if constexpr (WV == 0) {
#pragma unroll
        for (int i = 0; i < C::kBM / 64; ++i) {
          const int m = min(m0 + 64 * i + lane, M - 1);
          f6_dma4(a_scales, (uint32_t)m * 4, base + 256 * i);
        }
      } else {
#pragma unroll
        for (int i = 0; i < C::kBN / 64; ++i) {
          const int n = min(n0 + 64 * i + lane, N - 1);
          f6_dma4(w_scales, (uint32_t)n * 4, base + 1024 + 256 * i);
        }
      }
    }
  };

  // Operands of one stage: 3 weight and 4 activation fragments per 64-k
  // step, six dwords each (three 8-byte planes).
  struct Frag {
    uint32_t w[2][kTI][6];
    uint32_t a[2][kTJ][6];
  };
  constexpr uint32_t kWOff = (uint32_t)(WN * kTI) * kF6Block;
  constexpr uint32_t kAOff = (uint32_t)C::kW + (uint32_t)(WM * kTJ) * kF6Block;
  const uint32_t lane8 = (uint32_t)lane * 8;
  // Planes 0 and 1 of an operand are one paired read.  The address of plane 2
  // is hidden from the compiler so that it is not paired with a plane of a
  // different operand, which would need register moves.
  auto read_frag = [&](const uint8_t* s, uint32_t* d) __attribute__((always_inline)) {
    typedef unsigned int v2u __attribute__((ext_vector_type(2)));
    const v2u p0 = *reinterpret_cast<const v2u*>(s + lane8);
    const v2u p1 = *reinterpret_cast<const v2u*>(s + 512 + lane8);
    uint32_t a2 = (uint32_t)(uintptr_t)(lds_ptr_t)(s + 1024) + lane8;
    asm volatile("" : "+v"(a2));
    typedef const __attribute__((address_space(3))) v2u* lds_v2u;
    const v2u p2 = *(lds_v2u)(uintptr_t)a2;
    d[0] = p0.x; d[1] = p0.y; d[2] = p1.x; d[3] = p1.y; d[4] = p2.x; d[5] = p2.y;
  };

  v16f_t acc[kTI][kTJ];

  // One stage: its operands are in cur.  At its top every read of this stage
  // has returned and the next stage has landed (only the stage after it may
  // be in flight), so after the barrier the stage three ahead is issued into
  // this stage's buffer and the next stage is read into nxt, all between
  // this stage's 24 MFMAs.  The scheduling fences keep that order.
  constexpr int kParts = 5;   // parts a stage's loads are issued in
  auto stage = [&](const Frag& cur, Frag& nxt, int buf, const uint8_t* wt, const uint8_t* at,
                   int rbw, int rba, int kbi) __attribute__((always_inline)) {
    const int nbuf = buf == 2 ? 0 : buf + 1;
    f6_wait_lgkm0();
    f6_wait_vmcnt<NL>();
    f6_barrier();
    __builtin_amdgcn_sched_barrier(0);
    // The stage's loads leave in kParts parts between the operand reads; the
    // reads are spread over the MFMAs, so the loads are too, instead of
    // leaving in one burst ahead of them.  Part k holds loads
    // [k NL / kParts, (k + 1) NL / kParts) and follows read k * kFrags / kParts - 1.
    constexpr int kFrags = 2 * (kTI + kTJ);
    const uint8_t* s = smem + nbuf * C::kStage;
    issue_part(wt, at, rbw, rba, kbi, buf, std::integral_constant<int, 0>{},
               std::integral_constant<int, NL / kParts>{});
    [&]<int... F>(std::integer_sequence<int, F...>) __attribute__((always_inline)) {
      (
          [&] {
            constexpr int st = F / (kTI + kTJ), x = F % (kTI + kTJ);
            if constexpr (x < kTI)
              read_frag(s + st * 1536 + kWOff + x * kF6Block, nxt.w[st][x]);
            else
              read_frag(s + st * 1536 + kAOff + (x - kTI) * kF6Block, nxt.a[st][x - kTI]);
            constexpr int k = f6_part_after(F, kFrags, kParts);
            if constexpr (k > 0)
              issue_part(wt, at, rbw, rba, kbi, buf, std::integral_constant<int, k * NL / kParts>{},
                         std::integral_constant<int, (k + 1) * NL / kParts>{});
          }(),
          ...);
    }(std::make_integer_sequence<int, kFrags>{});
#pragma unroll
    for (int st = 0; st < 2; ++st)
#pragma unroll
      for (int i = 0; i < kTI; ++i)
#pragma unroll
        for (int j = 0; j < kTJ; ++j) acc[i][j] = mfma_f6(cur.w[st][i], cur.a[st][j], acc[i][j]);
    f6_sched_mixed<0, 2 * kTI * kTJ, NL>();
    __builtin_amdgcn_sched_barrier(0);
  };

  // Epilogue of tile r.  Lane l holds column m = l & 31 of each 32 x 32
  // accumulator and, in registers 4b .. 4b+3, rows n = 8 b + 4 g + 0..3
  // (g = l >> 5).  For b = 2p, 2p + 1 a swap of the upper half-wavefront's
  // first value with the lower half's second gives lane l < 32 the halves
  // n = 16 p + 0..7 and lane l + 32 the halves 16 p + 8..15 of row m.
  auto epilogue = [&](int r) __attribute__((always_inline)) {
    int m0, n0;
    origin(r, m0, n0);
    const int fr = lane & 31, fg = lane >> 5;
    const int mbase = WM * kTJ * 32 + fr, nbase = WN * kTI * 32;
    const bool inside = m0 + C::kBM <= M && n0 + C::kBN <= N;
    if constexpr (ACC_OUT) {
#pragma unroll
      for (int j = 0; j < kTJ; ++j) {
        const int m = m0 + mbase + j * 32;
#pragma unroll
        for (int i = 0; i < kTI; ++i)
#pragma unroll
          for (int b = 0; b < 4; ++b) {
            const int n = n0 + nbase + i * 32 + 8 * b + 4 * fg;
            if (m < M && n < N)
              *reinterpret_cast<int4*>(acc_out + (size_t)m * N + n) =
                  make_int4((int)acc[i][j][4 * b], (int)acc[i][j][4 * b + 1],
                            (int)acc[i][j][4 * b + 2], (int)acc[i][j][4 * b + 3]);
          }
      }
    } else {
      const float* sc = reinterpret_cast<const float*>(smem + C::kRing + (r & 1) * C::kScaleSlot);
#pragma unroll
      for (int j = 0; j < kTJ; ++j) {
        const float as = sc[mbase + j * 32];
        const int m = m0 + mbase + j * 32;
#pragma unroll
        for (int i = 0; i < kTI; ++i) {
#pragma unroll
          for (int p = 0; p < 2; ++p) {
            const int nl = nbase + i * 32 + 16 * p + 4 * fg;
            const float4 ws0 = *reinterpret_cast<const float4*>(sc + 256 + nl);
            const float4 ws1 = *reinterpret_cast<const float4*>(sc + 256 + nl + 8);
            const uint2 x0 = f6_dequant4(acc[i][j][8 * p], acc[i][j][8 * p + 1], acc[i][j][8 * p + 2],
                                         acc[i][j][8 * p + 3], as, ws0);
            const uint2 x1 = f6_dequant4(acc[i][j][8 * p + 4], acc[i][j][8 * p + 5],
                                         acc[i][j][8 * p + 6], acc[i][j][8 * p + 7], as, ws1);
            const auto s0 = __builtin_amdgcn_permlane32_swap(x0.x, x1.x, false, false);
            const auto s1 = __builtin_amdgcn_permlane32_swap(x0.y, x1.y, false, false);
            const int n = n0 + nbase + i * 32 + 16 * p + 8 * fg;
            if (inside || (m < M && n < N))
              *reinterpret_cast<uint4*>(y + (size_t)m * N + n) = make_uint4(s0[0], s1[0], s0[1], s1[1]);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
  };

  // Issue targets.  In the fast shapes a stage issued three ahead is in the
  // current tile or the next (a tile has at least three stages); past the
  // workgroup's last stage the last stage is issued again into a buffer
  // nobody reads any more, so every stage issues the same loads.  The CLAMP
  // variant looks up any tile up to three ahead.
  struct Tgt {
    const uint8_t* wt;
    const uint8_t* at;
    int rbw, rba, kb;
  };
  auto tile_base = [&](int r, Tgt& tg) __attribute__((always_inline)) {
    int m0, n0;
    origin(r, m0, n0);
    tg.rbw = n0 / 32;
    tg.rba = m0 / 32;
    tg.wt = w6 + (size_t)tg.rbw * kF6Block;
    tg.at = a6 + (size_t)tg.rba * kF6Block;
  };
  auto target = [&](int r, int kb, const Tgt& cur_t, const Tgt& next_t) __attribute__((always_inline)) {
    Tgt tg;
    const int k3 = kb + 3;
    if constexpr (!CLAMP) {
      const bool in_next = k3 >= nkb;
      const bool has_next = r + 1 < ntile;
      tg = (in_next && has_next) ? next_t : cur_t;
      tg.kb = in_next ? (has_next ? k3 - nkb : nkb - 1) : k3;
    } else {
      const int w = (k3 >= nkb) + (k3 >= 2 * nkb) + (k3 >= 3 * nkb);
      const bool past = r + w >= ntile;
      tile_base(past ? ntile - 1 : r + w, tg);
      tg.kb = past ? nkb - 1 : k3 - w * nkb;
    }
    return tg;
  };

  Tgt t_cur, t_next;
  tile_base(0, t_cur);
  tile_base(1, t_next);
  issue_scales(0);
  issue_scales(1);
#pragma unroll
  for (int i = 0; i < 3; ++i) {
    const Tgt tg = target(0, i - 3, t_cur, t_next);
    issue(tg.wt, tg.at, tg.rbw, tg.rba, tg.kb, i);
  }
  // Stage 0 has landed once only stages 1 and 2 are outstanding.
  f6_wait_vmcnt<2 * NL>();
  f6_barrier();
  Frag fa, fb;
  {
    const uint8_t* s = smem;
#pragma unroll
    for (int st = 0; st < 2; ++st) {
#pragma unroll
      for (int i = 0; i < kTI; ++i) read_frag(s + st * 1536 + kWOff + i * kF6Block, fa.w[st][i]);
#pragma unroll
      for (int j = 0; j < kTJ; ++j) read_frag(s + st * 1536 + kAOff + j * kF6Block, fa.a[st][j]);
    }
  }
  int buf = 0;
  for (int r = 0; r < ntile; ++r) {
#pragma unroll
    for (int i = 0; i < kTI; ++i)
#pragma unroll
      for (int j = 0; j < kTJ; ++j) acc[i][j] = v16f_t{};
    int kb = 0;
    for (; kb + 1 < nkb; kb += 2) {
      Tgt tg = target(r, kb, t_cur, t_next);
      stage(fa, fb, buf, tg.wt, tg.at, tg.rbw, tg.rba, tg.kb);
      buf = buf == 2 ? 0 : buf + 1;
      tg = target(r, kb + 1, t_cur, t_next);
      stage(fb, fa, buf, tg.wt, tg.at, tg.rbw, tg.rba, tg.kb);
      buf = buf == 2 ? 0 : buf + 1;
    }
    if (kb < nkb) {
      const Tgt tg = target(r, kb, t_cur, t_next);
      stage(fa, fb, buf, tg.wt, tg.at, tg.rbw, tg.rba, tg.kb);
      buf = buf == 2 ? 0 : buf + 1;
      fa = fb;
    }
    epilogue(r);
    t_cur = t_next;
    tile_base(r + 2, t_next);
    if constexpr (!ACC_OUT) {
      // The scales slot of tile r is free once every wavefront is past its epilogue.
      f6_barrier();
      issue_scales(r + 2);
    }
  }
  f6_wait_vmcnt<0>();   // the re-issued tail loads land before the LDS is released
}

template <bool ACC_OUT, bool CLAMP>
__global__ void __launch_bounds__(256)
qgemm_fp6(const uint8_t* __restrict__ a6, const float* __restrict__ a_scales,
          const uint8_t* __restrict__ w6, const float* __restrict__ w_scales, int M, int N,
          int K, __half* __restrict__ y, int32_t* __restrict__ acc_out) {
  __shared__ __attribute__((aligned(1024))) uint8_t smem[F6::kLds];
  switch (__builtin_amdgcn_readfirstlane(threadIdx.x >> 6)) {
    case 0: qgemm_fp6_body<0, ACC_OUT, CLAMP>(a6, a_scales, w6, w_scales, M, N, K, y, acc_out, smem); break;
    case 1: qgemm_fp6_body<1, ACC_OUT, CLAMP>(a6, a_scales, w6, w_scales, M, N, K, y, acc_out, smem); break;
    case 2: qgemm_fp6_body<2, ACC_OUT, CLAMP>(a6, a_scales, w6, w_scales, M, N, K, y, acc_out, smem); break;
    default: qgemm_fp6_body<3, ACC_OUT, CLAMP>(a6, a_scales, w6, w_scales, M, N, K, y, acc_out, smem); break;
  }
}

}  // namespace

int64_t fp6_bytes(int64_t rows, int64_t K) { return ((rows + 31) / 32) * 32 * K * 3 / 4; }

hipError_t launch_pack_fp6(const uint8_t* codes, int64_t R, int K, uint8_t* out,
                           hipStream_t stream) {
  const int64_t nslots = ((R + 31) / 32) * (K / 128) * 64;
  if (nslots == 0) return hipSuccess;
  hipLaunchKernelGGL(pack_fp6_kernel, dim3((unsigned)((nslots + 255) / 256)), dim3(256), 0, stream,
                     codes, (int)R, K, out, nslots);
  return hipGetLastError();
}

hipError_t launch_qlinear_fp6(const uint8_t* a6, const float* a_scales, int64_t M, int K,
                              const uint8_t* w6, const float* w_scales, int64_t N, void* y,
                              int32_t* out_acc, hipStream_t stream) {
  if (M == 0) return hipSuccess;
  const int64_t tiles = ((M + F6::kBM - 1) / F6::kBM) * ((N + F6::kBN - 1) / F6::kBN);
  const int cus = device_cus();
  const int64_t grid = tiles < cus ? tiles : cus;
  // Fast shapes: at least one full tile of padded rows each way and three
  // stages per tile.
  const bool clamp = (M + 31) / 32 < F6::kABlk || (N + 31) / 32 < F6::kWBlk || K < 3 * 128;
  __half* yh = static_cast<__half*>(y);
  if (out_acc) {
    if (clamp)
      hipLaunchKernelGGL((qgemm_fp6<true, true>), dim3((unsigned)grid), dim3(256), 0, stream, a6,
                         a_scales, w6, w_scales, (int)M, (int)N, K, yh, out_acc);
    else
      hipLaunchKernelGGL((qgemm_fp6<true, false>), dim3((unsigned)grid), dim3(256), 0, stream, a6,
                         a_scales, w6, w_scales, (int)M, (int)N, K, yh, out_acc);
  } else {
    if (clamp)
      hipLaunchKernelGGL((qgemm_fp6<false, true>), dim3((unsigned)grid), dim3(256), 0, stream, a6,
                         a_scales, w6, w_scales, (int)M, (int)N, K, yh, out_acc);
    else
      hipLaunchKernelGGL((qgemm_fp6<false, false>), dim3((unsigned)grid), dim3(256), 0, stream, a6,
                         a_scales, w6, w_scales, (int)M, (int)N, K, yh, out_acc);
  }
  return hipGetLastError();
}

}  // namespace dptq
