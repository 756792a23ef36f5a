// 256 x 256 bf16 MFMA tile engine shared by the large prefill kernels.
//
// 512 threads = 8 waves laid out 2 (M) x 4 (N); each wave owns 128 x 64 of
// the tile as 4 x 2 fragments of v_mfma_f32_32x32x16_bf16 (128 fp32
// accumulators per lane).  Operands stream from global memory straight into
// LDS with global_load_lds_dwordx4 (no VGPR staging): one wave instruction
// moves 1 KB, lane i landing at byte 16*i of the destination.  A stage holds
// A [256 rows][BK] and B [256 rows][BK] in bf16; NS stages of 128 KB in total
// form a ring, so the loads of step k+NS-1 are in flight while step k is
// multiplied.  Two shapes of the ring are compiled: BK = 64 x 2 stages and
// BK = 32 x 4 stages (deeper prefetch, twice the barriers).
//
// LDS layout: a row of BK bf16 is BK/8 chunks of 16 bytes.  Logical chunk c
// of row r sits at physical chunk c ^ f(r).  A 128-bit LDS read is served 16
// lanes at a time across 64 banks (256 bytes); the 16 lanes of an MFMA
// fragment read cover 16 consecutive rows at one logical chunk, so f must
// send them to 16 distinct 16-byte bank groups:
//   128-byte rows (BK = 64): group = 8*(r & 1) + chunk  ->  f(r) = (r & 7) ^ ((r >> 3) & 1)
//   64-byte rows  (BK = 32): group = 4*(r & 3) + chunk  ->  f(r) = (r >> 2) & 3
// (the plain f(r) = r & 7 collides rows r and r + 8: two-way conflicts,
// measured as about 4 extra LDS cycles per read).  The hardware fixes where
// each lane's 16 bytes land, so the swizzle is applied on the source side:
// each lane fetches the logical chunk that belongs at its landing slot.
//
// Rows that must read as zero (inactive or out of range) point their lanes at
// a 16-byte zero block in global memory, so their LDS slots are always
// overwritten.
#pragma once

#include "common.h"

namespace wide {
namespace t256 {

constexpr int BM = 256, BN = 256, NT = 512;
constexpr int LDS_BYTES = 131072;

typedef const void __attribute__((address_space(1)))* gptr_t;
typedef void __attribute__((address_space(3)))* lptr_t;

template <int BK>
struct Ring {
  static constexpr int CPR = BK / 8;              // 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;            // rows per wave load instruction
  static constexpr int SLOTS = BM / (8 * RPI);    // load slots per lane per operand
  static constexpr int A_ELEMS = BM * BK;
  static constexpr int STAGE = (BM + BN) * BK;    // bf16 elements per stage
  static constexpr int NS = LDS_BYTES / (STAGE * 2);
  static_assert(NS >= 2 && NS <= 4, "ring of two to four stages");

  __device__ static __forceinline__ int f(int row) {
    return CPR == 8 ? ((row & 7) ^ ((row >> 3) & 1)) : ((row >> 2) & 3);
  }
  __device__ static __forceinline__ int swz(int row, int chunk) {
    return row * BK + ((chunk ^ f(row)) << 3);
  }
  // Tile row served by load slot j of this lane, and the logical chunk it
  // fetches so that it lands at physical chunk lane % CPR.
  __device__ static __forceinline__ int slot_row(int j) {
    return (wave_id() * SLOTS + j) * RPI + lane_id() / CPR;
  }
  __device__ static __forceinline__ int slot_chunk(int j) {
    return (lane_id() % CPR) ^ f(slot_row(j));
  }
  // Issue load slots [j0, j1) of one k step: a[j] / b[j] already point at
  // the lane's 16 bytes.
  __device__ static __forceinline__ void issue(uint16_t* stage, const uint16_t* const (&a)[SLOTS],
                                               const uint16_t* const (&b)[SLOTS], int j0 = 0,
                                               int j1 = SLOTS) {
    const int w = wave_id();
#pragma unroll
    for (int j = 0; j < SLOTS; ++j) {
      if (j < j0 || j >= j1) continue;
      const int r0 = (w * SLOTS + j) * RPI;
      __builtin_amdgcn_global_load_lds((gptr_t)a[j], (lptr_t)(stage + r0 * BK), 16, 0, 0);
      __builtin_amdgcn_global_load_lds((gptr_t)b[j], (lptr_t)(stage + A_ELEMS + r0 * BK), 16, 0, 0);
    }
  }
  static constexpr int LOADS_PER_STEP = 2 * SLOTS;  // per wave
};

// Wait until at most n of this wave's vector-memory operations are in
// flight (expcnt and lgkmcnt untouched).  n <= 63.
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// MFMAs of one stage.  B fragment rows brow0/brow1; A fragment fm covers rows
// wm*128 + fm*32 + lane%32 and is skipped unless bit fm of `live` is set
// (FULL: all four live, no test).  mid() runs after the first half of the
// sub-steps (the loop uses it to issue the second half of the next step's
// loads).
template <int BK, bool FULL, class Mid>
__device__ __forceinline__ void mma_stage(const uint16_t* stage, int brow0, int brow1, int live,
                                          f32x16 (&acc)[4][2], Mid mid) {
  using Rg = Ring<BK>;
  constexpr int KK = BK / 16;
  const int lane = lane_id();
  const int wm = wave_id() >> 2;
  const int l32 = lane & 31, lhi = lane >> 5;
  const uint16_t* As = stage;
  const uint16_t* Bs = stage + Rg::A_ELEMS;
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    const int ch = kk * 2 + lhi;
    const u32x4 b0 = *reinterpret_cast<const u32x4*>(&Bs[Rg::swz(brow0, ch)]);
    const u32x4 b1 = *reinterpret_cast<const u32x4*>(&Bs[Rg::swz(brow1, ch)]);
    u32x4 a[4];
#pragma unroll
    for (int fm = 0; fm < 4; ++fm)
      a[fm] = *reinterpret_cast<const u32x4*>(&As[Rg::swz(wm * 128 + fm * 32 + l32, ch)]);
#pragma unroll
    for (int fm = 0; fm < 4; ++fm) {
      if (FULL || (live & (1 << fm))) {
        acc[fm][0] = mfma32(a[fm], b0, acc[fm][0]);
        acc[fm][1] = mfma32(a[fm], b1, acc[fm][1]);
      }
    }
    if (kk == KK / 2 - 1) mid();
  }
}

// The pipelined k loop over `nsteps` steps.  src(s, a, b) fills the lane's
// source pointers of step s.  Every wave issues LOADS_PER_STEP loads per
// step, so "step s has landed" is a vmcnt bound on the younger steps.
template <int BK, bool FULL, class Src>
__device__ __forceinline__ void mainloop(uint16_t* smem, int nsteps, Src src, int brow0, int brow1,
                                         int live, f32x16 (&acc)[4][2]) {
  using Rg = Ring<BK>;
  constexpr int NS = Rg::NS, L = Rg::LOADS_PER_STEP;
  auto issue = [&](int s) {
    const uint16_t* ap[Rg::SLOTS];
    const uint16_t* bp[Rg::SLOTS];
    src(s, ap, bp);
    Rg::issue(smem + (s % NS) * Rg::STAGE, ap, bp);
  };
  // wait until step s has landed, given that steps up to `last` were issued
  auto wait_step = [&](int s, int last) {
    const int younger = last - s;  // 0 .. NS-2 steps issued after step s
    if (NS == 2 || younger <= 0) wait_vm<0>();
    else if (younger == 1) wait_vm<L>();
    else wait_vm<2 * L>();
  };
  if (nsteps <= 0) return;
  const int pro = min(NS - 1, nsteps);
  for (int s = 0; s < pro; ++s) issue(s);
  wait_step(0, pro - 1);
  __syncthreads();
  // The next step's loads go out in two halves, one before the MFMAs and one
  // half-way through them: this spreads the memory requests over the step
  // and measured about 10% faster than issuing them in one burst.
  constexpr int S = Rg::SLOTS;
  for (int kt = 0; kt < nsteps; ++kt) {
    const int nxt = kt + NS - 1;
    const bool more = nxt < nsteps;
    const uint16_t* ap[S];
    const uint16_t* bp[S];
    uint16_t* nstage = smem + (nxt % NS) * Rg::STAGE;
    if (more) {
      src(nxt, ap, bp);
      Rg::issue(nstage, ap, bp, 0, S / 2);
    }
    mma_stage<BK, FULL>(smem + (kt % NS) * Rg::STAGE, brow0, brow1, live, acc, [&]() {
      if (more) Rg::issue(nstage, ap, bp, S / 2, S);
    });
    if (kt + 1 < nsteps) wait_step(kt + 1, min(nxt, nsteps - 1));
    __syncthreads();
  }
}

__device__ __forceinline__ void zero_acc(f32x16 (&acc)[4][2]) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};
}

// Accumulator element i of fragment fm: tile row; column inside the
// 32-wide fragment is lane % 32.
__device__ __forceinline__ int acc_row(int fm, int i) {
  return (wave_id() >> 2) * 128 + fm * 32 + (i >> 2) * 8 + (lane_id() >> 5) * 4 + (i & 3);
}
__device__ __forceinline__ int acc_col() { return lane_id() & 31; }

// Workgroup id -> tile id: each XCD (workgroups are dealt round-robin to the
// 8 XCDs) walks a contiguous range of tile ids.
__device__ __forceinline__ int xcd_remap(int id, int n) {
  const int q = n / 8, r = n % 8;
  const int xcd = id % 8, local = id / 8;
  return (xcd < r) ? xcd * (q + 1) + local : r * (q + 1) + (xcd - r) * q + local;
}

}  // namespace t256
}  // namespace wide
