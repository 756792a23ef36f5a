// 256 x 256 bf16 MFMA tile engine shared by the large prefill kernels.
//
// 512 threads = 8 waves laid out 2 (M) x 4 (N); each wave owns 128 x 64 of
// the tile as 4 x 2 fragments of v_mfma_f32_32x32x16_bf16 (128 fp32
// accumulators per lane).  Operands stream from global memory straight into
// LDS with global_load_lds_dwordx4 (no VGPR staging): one wave instruction
// moves 1 KB, lane i landing at byte 16*i of the destination.  A stage holds
// A [256 rows][BK] and B [256 rows][BK] in bf16; NS stages form a ring, so
// the loads of step k+NS-1 are in flight while step k is multiplied.  The
// library launches BK = 64 x 2 stages (128 KB); the ring also takes BK = 32
// with 4 or 5 stages (a prefetch distance of 96 or 128 k at twice the
// barriers), which measured slower on MI355X.
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
constexpr int LDS_MAX = 163840;  // bytes of LDS one workgroup may use on gfx950

typedef const void __attribute__((address_space(1)))* gptr_t;
typedef void __attribute__((address_space(3)))* lptr_t;

template <int BK_, int NS_>
struct Ring {
  static constexpr int BK = BK_;
  static constexpr int NS = NS_;                  // stages in the ring
  static constexpr int CPR = BK / 8;              // 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;            // rows per wave load instruction
  static constexpr int SLOTS = BM / (8 * RPI);    // load slots per lane per operand
  static constexpr int A_ELEMS = BM * BK;
  static constexpr int STAGE = (BM + BN) * BK;    // bf16 elements per stage
  static constexpr int LDS = NS * STAGE * 2;      // bytes
  static_assert(NS >= 2 && NS <= 5 && LDS <= LDS_MAX, "ring of two to five stages");

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
  __device__ static __forceinline__ void issue_a(uint16_t* stage, const uint16_t* const (&a)[SLOTS]) {
    const int w = wave_id();
#pragma unroll
    for (int j = 0; j < SLOTS; ++j)
      __builtin_amdgcn_global_load_lds((gptr_t)a[j], (lptr_t)(stage + (w * SLOTS + j) * RPI * BK), 16, 0, 0);
  }
  __device__ static __forceinline__ void issue_b(uint16_t* stage, const uint16_t* const (&b)[SLOTS]) {
    const int w = wave_id();
#pragma unroll
    for (int j = 0; j < SLOTS; ++j)
      __builtin_amdgcn_global_load_lds((gptr_t)b[j], (lptr_t)(stage + A_ELEMS + (w * SLOTS + j) * RPI * BK), 16, 0, 0);
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

// Workgroup barrier after this wave's LDS reads have returned.  Unlike
// __syncthreads() it does not wait for the wave's outstanding global loads,
// so the deeper stages of the ring stay in flight across it; the memory
// clobber keeps the compiler from moving LDS accesses or loads across it.
__device__ __forceinline__ void stage_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// One 16-wide k sub-step of this wave's operands: B fragment rows brow0 and
// brow1, A fragment fm covering tile rows wm*128 + fm*32 + lane%32.
struct Frags {
  u32x4 a[4];
  u32x4 b0, b1;
};

// Fragments of a partial tile: the tile rows this wave multiplies that are
// active form a prefix, so NLIVE (0..4) of its A fragments are live and the
// rest are skipped at compile time (no reads, no MFMAs).
template <class Rg, int NLIVE = 4>
__device__ __forceinline__ void read_frags(const uint16_t* stage, int kk, int brow0, int brow1,
                                           Frags& f) {
  if (NLIVE == 0) return;
  const int lane = lane_id();
  const int wm = wave_id() >> 2;
  const int l32 = lane & 31, lhi = lane >> 5;
  const int ch = kk * 2 + lhi;
  const uint16_t* As = stage;
  const uint16_t* Bs = stage + Rg::A_ELEMS;
  f.b0 = *reinterpret_cast<const u32x4*>(&Bs[Rg::swz(brow0, ch)]);
  f.b1 = *reinterpret_cast<const u32x4*>(&Bs[Rg::swz(brow1, ch)]);
#pragma unroll
  for (int fm = 0; fm < NLIVE; ++fm)
    f.a[fm] = *reinterpret_cast<const u32x4*>(&As[Rg::swz(wm * 128 + fm * 32 + l32, ch)]);
}

template <int NLIVE, int F0 = 0, int F1 = 4>
__device__ __forceinline__ void mma_frags(const Frags& f, f32x16 (&acc)[4][2]) {
#pragma unroll
  for (int fm = F0; fm < (F1 < NLIVE ? F1 : NLIVE); ++fm) {
    acc[fm][0] = mfma32(f.a[fm], f.b0, acc[fm][0]);
    acc[fm][1] = mfma32(f.a[fm], f.b1, acc[fm][1]);
  }
}

// Interleave hints for a partial tile's sub-step: each MFMA followed by one
// fragment read and up to VM_PER loads while they last.
template <int MF, int RD, int VM, int VM_PER>
__device__ __forceinline__ void sched_partial() {
#pragma unroll
  for (int i = 0; i < (MF > 0 ? MF : 1); ++i) {
    if (i < MF) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if (i < RD) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    if (VM_PER > 0 && i * VM_PER < VM) __builtin_amdgcn_sched_group_barrier(0x020, VM_PER, 0);
  }
}

// The pipelined k loop over `nsteps` steps.  src(s, a, b) fills the lane's
// source pointers of step s.  Every wave issues LOADS_PER_STEP loads per
// step, so "step s has landed" is a vmcnt bound on the younger steps.
//
// Schedule of step kt (KK = BK/16 sub-steps):
//   - the loads of step kt+NS-1 go out into the stage that step kt-1 used
//     (with two stages, in sub-step 0, two after each of its first four
//     MFMAs, and they must land within the step; with more stages, spread
//     over the sub-steps);
//   - sub-step kk interleaves the LDS reads of sub-step kk+1 with its own
//     MFMAs (one read per MFMA), so LDS latency hides behind the matrix core;
//   (measured in same-process A/B runs on gate/up, down and Q/K/V: issuing
//   the stage's loads in a burst at the start of the step, or reads in a
//   burst after two MFMAs, was 2-6% slower in total)
//   - at the last sub-step the wave waits for step kt+1, meets the others at
//     the barrier (which also retires every read of step kt's stage) and
//     reads step kt+1's first fragments between its first two and its last
//     six MFMAs: the barrier wait overlaps the MFMAs already in the pipe.
//
// NLIVE < 4 (a partial tile) skips the dead fragments' reads and MFMAs at
// compile time (a branch around each fragment's MFMAs made the compiler wait
// for every LDS read before them).  A wave's A load slots cover the 32 tile
// rows of fragment (w >> 2, w & 3); AON = false (that fragment is dead; the
// two-stage ring only, where every wait is for all of the wave's loads) also
// skips those loads.
template <class Rg, int NLIVE, bool AON, class Src>
__device__ __forceinline__ void mainloop(uint16_t* smem, int nsteps, Src src, int brow0, int brow1,
                                         f32x16 (&acc)[4][2]) {
  constexpr bool FULL = NLIVE == 4;
  static_assert(AON || Rg::NS == 2, "skipped loads would upset the vmcnt bounds of deeper rings");
  constexpr int NS = Rg::NS, L = Rg::LOADS_PER_STEP, S = Rg::SLOTS, KK = Rg::BK / 16;
  constexpr int MF = 2 * NLIVE, RD = NLIVE > 0 ? NLIVE + 2 : 0;  // MFMAs and reads per sub-step
  constexpr int VM = (AON ? 2 : 1) * S, VM_PER = MF > 0 ? (VM + MF - 1) / MF : 0;  // loads per step
  auto issue_all = [&](int s) {
    const uint16_t* ap[S];
    const uint16_t* bp[S];
    src(s, ap, bp);
    Rg::issue(smem + (s % NS) * Rg::STAGE, ap, bp);
  };
  // wait until step s has landed, given that steps up to `last` were issued
  auto wait_step = [&](int s, int last) {
    const int younger = last - s;  // 0 .. NS-2 steps issued after step s
    if (NS == 2 || younger <= 0) wait_vm<0>();
    else if (younger == 1) wait_vm<L>();
    else if (NS == 3 || younger == 2) wait_vm<2 * L>();
    else wait_vm<3 * L>();
  };
  if (nsteps <= 0) return;
  const int pro = min(NS - 1, nsteps);
  if (NS == 2) {  // B's addresses need no gathered row index: send them first
    const uint16_t* ap[S];
    const uint16_t* bp[S];
    src(0, ap, bp);
    Rg::issue_b(smem, bp);
    if (AON) Rg::issue_a(smem, ap);
  } else {
    for (int s = 0; s < pro; ++s) issue_all(s);
  }
  wait_step(0, pro - 1);
  stage_barrier();
  // Sub-step kk works on fr[kk & 1] and fills fr[(kk + 1) & 1]; KK is even,
  // so the parity carries over from one step to the next without copies.
  static_assert(KK % 2 == 0, "even number of sub-steps");
  Frags fr[2];
  read_frags<Rg, NLIVE>(smem, 0, brow0, brow1, fr[0]);
  for (int kt = 0; kt < nsteps; ++kt) {
    const int nxt = kt + NS - 1;
    const bool more = nxt < nsteps;
    const uint16_t* ap[S];
    const uint16_t* bp[S];
    uint16_t* nstage = smem + (nxt % NS) * Rg::STAGE;
    const uint16_t* cstage = smem + (kt % NS) * Rg::STAGE;
    constexpr bool TWO = NS == 2;
    if (TWO) {
      // Branch-free, so the loads can sit among the MFMAs: in the last step
      // they fetch that step again into the stage nobody reads any more
      // (waited for after the loop).
      src(min(nxt, nsteps - 1), ap, bp);
    } else if (more) {
      src(nxt, ap, bp);
    }
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      if (!TWO && more) Rg::issue(nstage, ap, bp, kk * S / KK, (kk + 1) * S / KK);
      if (TWO && kk == 0) {
        // Sub-step 0 of a two-stage ring: the next step's loads (two per
        // MFMA) and the six fragment reads of sub-step 1 interleave with the
        // MFMAs.
        __builtin_amdgcn_sched_barrier(0);
        mma_frags<NLIVE, 0, 4>(fr[0], acc);
        if (AON) Rg::issue_a(nstage, ap);
        Rg::issue_b(nstage, bp);
        read_frags<Rg, NLIVE>(cstage, 1, brow0, brow1, fr[1]);
        if (FULL) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x020, 2, 0);
          }
#pragma unroll
          for (int i = 0; i < 2; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          }
          __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
        } else {
          sched_partial<MF, RD, VM, VM_PER>();
        }
        __builtin_amdgcn_sched_barrier(0);
        continue;
      }
      if (kk + 1 < KK) {
        // Inside a step: the six fragment reads of sub-step kk+1 interleave
        // with the first six MFMAs of sub-step kk (one each), so the LDS
        // sees one read per MFMA instead of a burst (measured 1-2% faster
        // than two MFMAs, six reads, six MFMAs).
        __builtin_amdgcn_sched_barrier(0);
        mma_frags<NLIVE, 0, 4>(fr[kk & 1], acc);
        read_frags<Rg, NLIVE>(cstage, kk + 1, brow0, brow1, fr[(kk + 1) & 1]);
        if (FULL) {
#pragma unroll
          for (int i = 0; i < 6; ++i) {
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
          }
          __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
        } else {
          sched_partial<MF, RD, 0, 0>();
        }
        __builtin_amdgcn_sched_barrier(0);
        continue;
      }
      // Last sub-step: the first two MFMAs go out before the barrier and the
      // next stage's first fragment reads, so the matrix core is busy while
      // they wait.
      mma_frags<NLIVE, 0, 1>(fr[kk & 1], acc);
      __builtin_amdgcn_sched_barrier(0);
      if (kt + 1 < nsteps) {
        wait_step(kt + 1, min(nxt, nsteps - 1));
        stage_barrier();
        read_frags<Rg, NLIVE>(smem + ((kt + 1) % NS) * Rg::STAGE, 0, brow0, brow1, fr[0]);
      }
      __builtin_amdgcn_sched_barrier(0);
      mma_frags<NLIVE, 1, 4>(fr[kk & 1], acc);
    }
  }
  if (NS == 2) wait_vm<0>();  // the last step's repeated loads
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
