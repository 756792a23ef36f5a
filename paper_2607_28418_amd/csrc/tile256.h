// 256 x 256 bf16 MFMA tile engine shared by the large prefill kernels.
//
// 256 threads = 4 waves laid out 2 (M) x 2 (N), one wave per SIMD; each wave
// owns 128 x 128 of the tile as 4 x 4 fragments of v_mfma_f32_32x32x16_bf16,
// 256 fp32 accumulators per lane held in the accumulation registers (AGPRs).
// Per 64-deep k step a wave reads 32 KB of fragments from LDS for 64 MFMAs
// (a 128 x 64 wave tile reads 24 KB for 32).  The MFMAs are issued through
// inline assembly with AGPR operands: with the builtin, the compiler split the
// 256 accumulators between the two register files and copied them back and
// forth inside the k loop.
//
// Operands stream from global memory straight into LDS with
// global_load_lds_dwordx4 (no VGPR staging): one wave instruction moves 1 KB,
// lane i landing at byte 16*i of the destination.  An operand stage holds
// [256 rows][64] bf16 (32 KB).  A (the token rows, gathered in the masked
// kernels) has DA stages and B (the weights) two; with DA = 3 (160 KB, all of
// LDS) A's loads run two steps ahead and B's one, so the CU's load pipe has
// work queued when a step's barrier comes, instead of draining at every step
// (measured on the dense 8192x4096x14336 shape: 1300 -> 1375 TFLOP/s with
// random operands; B deep instead of A: 1310).
//
// LDS layout: a row of 64 bf16 is 8 chunks of 16 bytes.  Logical chunk c of
// row r sits at physical chunk c ^ f(r), f(r) = (r & 7) ^ ((r >> 3) & 1).  A
// 128-bit LDS read is served 16 lanes at a time across 64 banks (256 bytes);
// the 16 lanes of a fragment read cover 16 consecutive rows at one logical
// chunk, and f sends them to 16 distinct 16-byte bank groups (the plain
// f(r) = r & 7 collides rows r and r + 8: two-way conflicts).  The hardware
// fixes where each lane's 16 bytes land, so the swizzle is applied on the
// source side: each lane fetches the logical chunk that belongs at its
// landing slot.
//
// Rows that must read as zero (inactive or out of range) point their lanes at
// a 16-byte zero block in global memory, so their LDS slots are always
// overwritten.
#pragma once

#include <type_traits>

#include "common.h"

namespace wide {
namespace t256 {

constexpr int BM = 256, BN = 256, NT = 256, BK = 64;
constexpr int LDS_MAX = 163840;  // bytes of LDS one workgroup may use on gfx950

typedef const void __attribute__((address_space(1)))* gptr_t;
typedef void __attribute__((address_space(3)))* lptr_t;

template <int DA_>
struct Ring {
  static constexpr int DA = DA_;                // A stages
  static constexpr int LEAD = DA - 1;           // steps A's loads run ahead
  static constexpr int CPR = BK / 8;            // 16-byte chunks per row
  static constexpr int RPI = 64 / CPR;          // rows per wave load instruction
  static constexpr int SLOTS = BM / (4 * RPI);  // load slots per lane per operand
  static constexpr int OP = BM * BK;            // bf16 elements of one operand stage
  static constexpr int LDS = (DA + 2) * OP * 2; // bytes
  static_assert((DA == 2 || DA == 3) && LDS <= LDS_MAX, "two or three A stages");

  __device__ static __forceinline__ uint16_t* a_stage(uint16_t* smem, int s) { return smem + (s % DA) * OP; }
  __device__ static __forceinline__ uint16_t* b_stage(uint16_t* smem, int s) { return smem + (DA + (s & 1)) * OP; }
  __device__ static __forceinline__ int f(int row) { return (row & 7) ^ ((row >> 3) & 1); }
  __device__ static __forceinline__ int swz(int row, int chunk) { return row * BK + ((chunk ^ f(row)) << 3); }
  // Tile row served by load slot j of this lane (a wave's slots cover rows
  // [64 w, 64 w + 64)), and the logical chunk it fetches so that it lands at
  // physical chunk lane % CPR.
  __device__ static __forceinline__ int slot_row(int j) {
    return (wave_id() * SLOTS + j) * RPI + lane_id() / CPR;
  }
  __device__ static __forceinline__ int slot_chunk(int j) {
    return (lane_id() % CPR) ^ f(slot_row(j));
  }
  // Load slot j of one operand stage; p points at the lane's 16 bytes.
  __device__ static __forceinline__ void issue_ptr(uint16_t* stage, const uint16_t* p, int j) {
    __builtin_amdgcn_global_load_lds((gptr_t)p, (lptr_t)(stage + (wave_id() * SLOTS + j) * RPI * BK), 16, 0, 0);
  }
  // The same through a buffer view: the lane's 16 bytes at byte voff + soff
  // (soff wave-uniform).  Lanes past the view's end land zeros.
  __device__ static __forceinline__ void issue_buf(uint16_t* stage, bufview_t v, uint32_t voff, uint32_t soff, int j) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(v, (lptr_t)(stage + (wave_id() * SLOTS + j) * RPI * BK), 16, (int)voff,
                                             (int)soff, 0, 0);
  }
};

// Operand sources.  With a buffer view (views under 2^31 bytes) each lane
// keeps one 32-bit byte offset per load slot for the whole tile and a step
// adds its k offset as a scalar; a 128-bit global address per slot and step
// cost the same loads 3-4% (measured on dense 256x256 tiles) besides the
// VALU work.  The range check covers the scalar part too, so a dead row
// (zeros) takes kOffDead: past every view, and still past it (no 32-bit
// wrap) with any scalar offset below 2^31.
constexpr uint32_t kOffDead = 0x80000000u;
constexpr int64_t kBufViewMax = (int64_t(1) << 31) - 256;  // bytes of a view the tile kernels use

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

// Nothing is scheduled across it.
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

// acc += A-fragment x B-fragment, the accumulator in AGPRs.
__device__ __forceinline__ void mfma_acc(const u32x4& a, const u32x4& b, f32x16& c) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(c) : "v"(a), "v"(b));
}

// The compiler does not see the MFMAs inside the asm, so it inserts none of
// the wait states between an accumulator's write by a VALU op and its use as
// an MFMA source, or between the last MFMA and the reads of its result.
// This fence, holding every accumulator, provides them at both ends of the
// k loop (64 wait states, more than the 8-pass MFMA's latency).
__device__ __forceinline__ void acc_fence(f32x16 (&c)[4][4]) {
  asm volatile("s_nop 15\n\ts_nop 15\n\ts_nop 15\n\ts_nop 15"
               : "+a"(c[0][0]), "+a"(c[0][1]), "+a"(c[0][2]), "+a"(c[0][3]),
                 "+a"(c[1][0]), "+a"(c[1][1]), "+a"(c[1][2]), "+a"(c[1][3]),
                 "+a"(c[2][0]), "+a"(c[2][1]), "+a"(c[2][2]), "+a"(c[2][3]),
                 "+a"(c[3][0]), "+a"(c[3][1]), "+a"(c[3][2]), "+a"(c[3][3]));
}

__device__ __forceinline__ void zero_acc(f32x16 (&acc)[4][4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};
}

// One 16-deep k sub-step of the wave's operands: A fragment fm covers tile
// rows wm*128 + fm*32 + lane%32, B fragment fn tile columns bb[fn] + lane%32.
struct Frags {
  u32x4 a[4], b[4];
};

// Fragment read r of a sub-step, in the order the MFMAs first use them:
// A0, B0, B1, B2, B3, A1, A2, A3.
// B fragment fn of a wave starts bfrag_off<BL>(fn) tile rows after its
// first, bb[0] (a multiple of 32): BL 0, four consecutive 32-row fragments;
// BL 1 (gate/up pairs), two consecutive fragments of gate rows and the same
// two of up rows, 128 rows on.  Kernels build bb[fn] = bb[0] + bfrag_off.
template <int BL>
__host__ __device__ constexpr int bfrag_off(int fn) {
  return BL == 0 ? fn * 32 : (fn >> 1) * 128 + (fn & 1) * 32;
}

// Every fragment starts at a tile row that is a multiple of 32, so its
// swizzle depends on the lane alone: the address is the fragment's row base
// times BK plus one per-lane offset per sub-step, the same for A and B.  The
// row bases are a wave-uniform value plus constants, so a sub-step's four A
// and four B reads share two address registers and differ by immediate
// offsets (an XOR over the whole row, or a base per fragment, needed one add
// per read).
template <class Rg, int BL>
__device__ __forceinline__ void read_frag(const uint16_t* as, const uint16_t* bs, int kk, const int (&bb)[4],
                                          Frags& f, int r) {
  const int lane = lane_id(), l32 = lane & 31;
  const int ch = kk * 2 + (lane >> 5);
  const int wm = wave_id() >> 1;
  const int lo = l32 * BK + ((ch ^ Rg::f(l32)) << 3);  // = swz(base + l32, ch) - base * BK
  if (r == 0 || r >= 5) {
    const int fm = r == 0 ? 0 : r - 4;
    f.a[fm] = *reinterpret_cast<const u32x4*>(as + wm * 128 * BK + lo + fm * 32 * BK);
  } else {
    f.b[r - 1] = *reinterpret_cast<const u32x4*>(bs + bb[0] * BK + lo + bfrag_off<BL>(r - 1) * BK);
  }
}

// MFMAs [Q0, Q1) of a sub-step on fragment set f (MFMA q: A fragment q / 4,
// B fragment q % 4; only the first NL A fragments are live) with RDN
// fragment reads rd(r) and LDN loads ld(l) spread among them: when they fit,
// a load after each even and a read after each odd MFMA, so no MFMA waits on
// more than one instruction's address work; else as evenly as they go.
template <int NL, int Q0, int Q1, int RDN, int LDN, class Rd, class Ld>
__device__ __forceinline__ void substep(const Frags& f, f32x16 (&acc)[4][4], Rd rd, Ld ld) {
  constexpr int QE = Q1 < 4 * NL ? Q1 : 4 * NL;
  constexpr int MF = QE > Q0 ? QE - Q0 : 0;
  if constexpr (MF == 0) {
#pragma unroll
    for (int r = 0; r < RDN; ++r) rd(r);
#pragma unroll
    for (int l = 0; l < LDN; ++l) ld(l);
    sched_fence();
  } else {
    constexpr bool HALF = 2 * RDN <= MF;
    constexpr int RPM = (RDN + MF - 1) / MF, LPM = (LDN + MF - 1) / MF;
#pragma unroll
    for (int i = 0; i < MF; ++i) {
      const int q = Q0 + i;
      mfma_acc(f.a[q >> 2], f.b[q & 3], acc[q >> 2][q & 3]);
      if (HALF) {
        if ((i & 1) && (i >> 1) < RDN) rd(i >> 1);
      } else {
#pragma unroll
        for (int t = 0; t < RPM; ++t)
          if (i * RPM + t < RDN) rd(i * RPM + t);
      }
      if (HALF && 2 * LDN <= MF) {
        if (!(i & 1) && (i >> 1) < LDN) ld(i >> 1);
      } else {
#pragma unroll
        for (int t = 0; t < LPM; ++t)
          if (i * LPM + t < LDN) ld(i * LPM + t);
      }
      sched_fence();
    }
  }
}

// The pipelined k loop over `nsteps` 64-deep steps.  koff(s) gives step s's
// k offset into the operand rows (scalar work, once per step and operand);
// lda(stage, k, j) / ldb(stage, k, j) issue load slot j of A / B at k offset
// k into the stage.  They are called beside each load, so their arithmetic
// sits between MFMAs (with one wave per SIMD, a step's address work done in
// one burst stalls the matrix core).  acc must be zeroed by the caller.
//
// Schedule of step kt (four 16-deep sub-steps, fragment sets alternating):
//   - sub-step kk interleaves the LDS reads of sub-step kk+1 with its own
//     MFMAs (one read after every other MFMA);
//   - sub-step 0 issues B of step kt+1, one load after every other MFMA;
//     sub-step 2 issues A of step kt+LEAD the same way.  B goes first: it is
//     the one needed by the end of this step when LEAD = 2.  (Same-process
//     runs on the Llama-3-8B layer prefill: A in sub-step 2 rather than 1 took
//     4% off gate/up and down; split over sub-steps 1 and 2, or B over 0 and
//     1, was as good; A before the barrier of sub-step 3 was 2-3% slower.)
//   - at the last sub-step the wave runs half its MFMAs, waits for step
//     kt+1 (A of kt+2 may stay in flight), meets the others at the barrier
//     (which also retires every read of step kt's stages) and reads step
//     kt+1's first fragments among its remaining MFMAs.
// Every wave issues the same loads in the same order each step, so "step s
// has landed" is a vmcnt bound.
//
// NL < 4 (a partial tile) skips the dead A fragments' reads and MFMAs at
// compile time.  A wave's A load slots cover tile rows [64 w, 64 w + 64);
// AON = false (all of them past the active rows) skips its A loads.
template <class Rg, int NL, bool AON, int BL, class Koff, class LdA, class LdB>
__device__ __forceinline__ void mainloop(uint16_t* smem, int nsteps, Koff koff, LdA lda, LdB ldb, const int (&bb)[4],
                                         f32x16 (&acc)[4][4]) {
  constexpr int S = Rg::SLOTS, LEAD = Rg::LEAD;
  constexpr int RDN = NL > 0 ? NL + 4 : 0;  // fragment reads per sub-step
  constexpr int PRE = 2 * NL;               // MFMAs of the last sub-step before the barrier
  acc_fence(acc);
  if (nsteps > 0) {
    const int k0 = koff(0);
#pragma unroll
    for (int j = 0; j < S; ++j) ldb(Rg::b_stage(smem, 0), k0, j);
    if (AON) {
#pragma unroll
      for (int j = 0; j < S; ++j) lda(Rg::a_stage(smem, 0), k0, j);
    }
    if (AON && LEAD == 2 && nsteps > 1) {
      const int k1 = koff(1);
#pragma unroll
      for (int j = 0; j < S; ++j) lda(Rg::a_stage(smem, 1), k1, j);
      wait_vm<S>();
    } else {
      wait_vm<0>();
    }
    stage_barrier();
    Frags f0, f1;
    if (NL > 0) {
#pragma unroll
      for (int r = 0; r < RDN; ++r) read_frag<Rg, BL>(Rg::a_stage(smem, 0), Rg::b_stage(smem, 0), 0, bb, f0, r);
    }
    // LS: issue B of kt+1; LA: A of kt+LEAD; NEXT: step kt+1 exists; WN: loads
    // allowed in flight when waiting for step kt+1
    auto step = [&](int kt, auto ls_t, auto la_t, auto next_t, auto wn_t) {
      constexpr bool LS = decltype(ls_t)::value, LA = decltype(la_t)::value && AON;
      constexpr bool NEXT = decltype(next_t)::value;
      constexpr int WN = decltype(wn_t)::value;
      const uint16_t* as = Rg::a_stage(smem, kt);
      const uint16_t* bs = Rg::b_stage(smem, kt);
      uint16_t* lb = Rg::b_stage(smem, kt + 1);
      uint16_t* la = Rg::a_stage(smem, kt + LEAD);
      const int kb = LS ? koff(kt + 1) : 0;
      const int ka = LA ? koff(kt + LEAD) : 0;
      auto rd = [&](int kk, Frags& f) { return [&, kk](int r) { read_frag<Rg, BL>(as, bs, kk, bb, f, r); }; };
      auto none = [](int) {};
      sched_fence();
      substep<NL, 0, 16, RDN, LS ? S : 0>(f0, acc, rd(1, f1), [&](int j) { ldb(lb, kb, j); });
      substep<NL, 0, 16, RDN, 0>(f1, acc, rd(2, f0), none);
      substep<NL, 0, 16, RDN, LA ? S : 0>(f0, acc, rd(3, f1), [&](int j) { lda(la, ka, j); });
      substep<NL, 0, PRE, 0, 0>(f1, acc, none, none);
      if (NEXT) {
        wait_vm<WN>();
        stage_barrier();
      }
      sched_fence();
      const uint16_t* an = Rg::a_stage(smem, kt + 1);
      const uint16_t* bn = Rg::b_stage(smem, kt + 1);
      substep<NL, PRE, 16, NEXT ? RDN : 0, 0>(f1, acc, [&](int r) { read_frag<Rg, BL>(an, bn, 0, bb, f0, r); }, none);
    };
    using T = std::true_type;
    using F = std::false_type;
    using I0 = std::integral_constant<int, 0>;
    using IS = std::integral_constant<int, AON && LEAD == 2 ? S : 0>;
    int kt = 0;
    for (; kt + LEAD < nsteps; ++kt) step(kt, T{}, T{}, T{}, IS{});
    if (LEAD == 2 && kt + 1 < nsteps) step(kt++, T{}, F{}, T{}, I0{});
    step(kt, F{}, F{}, F{}, I0{});
  }
  acc_fence(acc);
}

// Accumulator element i of A fragment fm: tile row; the column inside the
// 32-wide B fragment is lane % 32.
__device__ __forceinline__ int acc_row(int fm, int i) {
  return (wave_id() >> 1) * 128 + fm * 32 + (i >> 2) * 8 + (lane_id() >> 5) * 4 + (i & 3);
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
