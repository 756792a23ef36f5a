// Large-tile prefill kernels (256 x 256 tiles, 4 waves, direct-to-LDS loads).
//
//   wide_mn256<SWIGLU,BK>  N-axis masked projection (GEMM-MN): gate/up + SwiGLU
//                          (one tile = 256 sorted tokens x one 128-column slice
//                          of a group: 128 gate rows + 128 up rows), or plain
//                          Q/K/V (one tile = 256 tokens x 256 output columns).
//   wide_kd256<NWR, BK>    K-axis masked projection, dense-masked schedule.
//   wide_ks256<BK>         K-axis masked projection, scatter schedule (GEMM-K).
//
// Semantics, skipping levels and the two K-axis schedules are those of the
// 128-tile kernels in gemm_mn.hip / gemm_k.hip (WIDE Section 3.1 equations
// (1)-(3); Section 3.3; Appendix B, Algorithms 2 and 3); only the tile engine
// differs (tile256.h).  Tiles whose 256 rows are all active take the
// all-active path (no per-fragment tests), as the paper does for full tiles
// of a sorted column.  BK is the ring's k depth, 64.
#include "common.h"
#include "kernels.h"
#include "launch.h"
#include "tile256.h"

namespace wide {

using namespace t256;

namespace {
__device__ __attribute__((aligned(16))) uint16_t g_zero_blk[64];  // stays zero: never written

// Rings: three stages of A and two of B (160 KB, all of LDS), except the
// dense-masked K-axis kernel over more than 128 groups, which keeps 17 KB for
// its tile's mask bits and so runs two A stages.
using RingMN = Ring<3>;
template <int NWR>
using RingKD = Ring<NWR == 0 ? 2 : 3>;

// Epilogue row map.  Output rows go back to token order through a per-row
// index (the reorder, or the pattern order); fetching it per output element
// put one dependent global load in front of every store.  Instead, thread
// r < 256 fetches tile row r's token (-1 past the end) before the k loop,
// and after it the map goes through the then idle ring LDS.
// `extra` (a row's mask bits, token-order regions) goes to map[BM + r].
__device__ __forceinline__ const int* stage_row_map(uint16_t* smem, int my_row, int extra = 0) {
  int* map = reinterpret_cast<int*>(smem);
  __syncthreads();  // every wave is done with the ring
  if (threadIdx.x < BM) {
    map[threadIdx.x] = my_row;
    map[BM + threadIdx.x] = extra;
  }
  __syncthreads();
  return map;
}

// Bit b of the result: byte b of the n (<= 32) mask bytes at mr is nonzero.
// Rows of ng bytes start 16-byte aligned when 16 divides ng (the mask itself
// is 16-byte aligned), 4-byte aligned when 4 does; the loads are as wide as
// that allows.
__device__ __forceinline__ uint32_t nz4(uint32_t w) {  // bit i: byte i of w != 0
  const uint32_t m = (((w & 0x7f7f7f7fu) + 0x7f7f7f7fu) | w) & 0x80808080u;
  return ((m >> 7) & 1u) | ((m >> 14) & 2u) | ((m >> 21) & 4u) | ((m >> 28) & 8u);
}
__device__ __forceinline__ uint32_t mask_bits32(const uint8_t* mr, int n, int ng) {
  uint32_t bits = 0;
  if (n == 32 && ng % 16 == 0) {
    const u32x4 a = *reinterpret_cast<const u32x4*>(mr);
    const u32x4 b = *reinterpret_cast<const u32x4*>(mr + 16);
    bits = nz4(a[0]) | nz4(a[1]) << 4 | nz4(a[2]) << 8 | nz4(a[3]) << 12 | nz4(b[0]) << 16 |
           nz4(b[1]) << 20 | nz4(b[2]) << 24 | nz4(b[3]) << 28;
  } else if (ng % 4 == 0) {  // n is a multiple of 4 too
    for (int b = 0; b < n; b += 4) bits |= nz4(*reinterpret_cast<const uint32_t*>(mr + b)) << b;
  } else {
    for (int b = 0; b < n; ++b) bits |= (uint32_t)(mr[b] != 0) << b;
  }
  return bits;
}

// Tiles of one region that each XCD runs (the region padded to a multiple of 8).
__host__ __device__ __forceinline__ int mn256_share(int tiles) { return (tiles + 7) / 8; }

// The k loop of one tile with the wave's live A fragments and A loads:
// `act` tile rows are active, always a prefix (rows past the active count, or
// past M, come last in a tile).
template <class Rg, int BL, class Koff, class LdA, class LdB>
__device__ __forceinline__ void run_tile(uint16_t* smem, int nsteps, Koff koff, LdA lda, LdB ldb, const int (&bb)[4],
                                         int64_t act, f32x16 (&acc)[4][4]) {
  const int p = (int)(act < 0 ? 0 : act > BM ? BM : act);
  const int w = wave_id(), wm = w >> 1;
  const int nl = min(4, max(0, (p - wm * 128 + 31) / 32));  // live A fragments of the wave
  const bool aon = 64 * w < p;                              // the wave's A load rows [64 w, 64 w + 64)
  // (nl, aon): (4|3, true) full or nearly; (2|1, true|false); (0, false) -- the
  // waves of the lower half of a tile with at most 128 active rows
  switch (nl) {
    case 4: mainloop<Rg, 4, true, BL>(smem, nsteps, koff, lda, ldb, bb, acc); break;
    case 3: mainloop<Rg, 3, true, BL>(smem, nsteps, koff, lda, ldb, bb, acc); break;
    case 2:
      if (aon) mainloop<Rg, 2, true, BL>(smem, nsteps, koff, lda, ldb, bb, acc);
      else mainloop<Rg, 2, false, BL>(smem, nsteps, koff, lda, ldb, bb, acc);
      break;
    case 1:
      if (aon) mainloop<Rg, 1, true, BL>(smem, nsteps, koff, lda, ldb, bb, acc);
      else mainloop<Rg, 1, false, BL>(smem, nsteps, koff, lda, ldb, bb, acc);
      break;
    default: mainloop<Rg, 0, false, BL>(smem, nsteps, koff, lda, ldb, bb, acc); break;
  }
}
}  // namespace

// Tile order inside an XCD's share of a region: group, then sorted m-tile,
// then column tile inside the group, so the tiles an XCD runs together share
// the group's weight panel in L2 (gate/up runs m-blocked instead, see
// mn256_mblocked).  A group wider than four column tiles (one group over a
// whole projection, the M-axis case) goes column tile first: each XCD then
// covers a slice of the weight once and re-reads the gathered rows, which
// fit the last-level cache, instead of streaming the whole weight once per
// m-tile.
//
// When an XCD's share is a whole number of groups ("ordered"), it runs the
// full tiles of its groups first, then their partial last m-tiles, then the
// empty ones, so its real tiles come first.
template <int BNO>
__device__ __forceinline__ bool mn256_ordered(const MN256Args& a, const MN256Region& R) {
  const int share = mn256_share(R.tiles), per_group = R.gw / BNO * a.m_tiles;
  return a.order && R.masked == kMN256Sorted && R.gw / BNO <= 4 && 8 * share == R.tiles &&
         share % per_group == 0;
}

// "m-blocked" (gate/up): when an XCD's share is a whole number of groups, it
// runs m-tile 0 of each of its groups, then m-tile 1, and so on, over one
// half of its groups and then the other.  The tiles that run together then
// gather rows from one stretch of tokens (a sorted m-tile of any group
// covers about the same token range) instead of one group's whole token
// list, so the gathered rows are mostly shared in L2 while each group's
// weight panel is re-read once per m-tile.  Measured on the Llama-3-8B
// gate/up at T = 8192 (topk, keep 0.5): traffic from beyond L2 down 37%,
// time down 2% against group by group; blocks of 4 or 8 m-tiles per group
// cut the traffic as much but ran 7-9% slower.  Halves (7 of the XCD's 14
// groups at a time, so fewer weight panels per k step, and the first
// half's partial m-tiles run beside the second half's full ones) took
// another 2.5% off; pairs of groups did the same.
template <int BNO>
__device__ __forceinline__ bool mn256_mblocked(const MN256Args& a, const MN256Region& R) {
  const int share = mn256_share(R.tiles), per_group = R.gw / BNO * a.m_tiles;
  return a.mblock && R.masked == kMN256Sorted && R.gw / BNO <= 4 && 8 * share == R.tiles &&
         share % per_group == 0;
}

template <int BNO>
__device__ __forceinline__ void mn256_coords(const MN256Args& a, const MN256Region& R, int xcd, int local,
                                             int& g, int& m_tile, int& nt_in) {
  const int share = mn256_share(R.tiles);
  const int tile = xcd * share + local;
  const int ntpg = R.gw / BNO;  // tiles per group
  const int per_group = ntpg * a.m_tiles;
  if (mn256_mblocked<BNO>(a, R)) {
    // the XCD's groups in two halves, each walked m-tile by m-tile
    const int gps = share / per_group, parts = gps % 2 == 0 && gps >= 4 ? 2 : 1, gpp = gps / parts;
    const int per_part = gpp * ntpg * a.m_tiles, part = local / per_part, l = local % per_part;
    const int r = l % (gpp * ntpg);
    m_tile = l / (gpp * ntpg);
    g = xcd * gps + part * gpp + r / ntpg;
    nt_in = r % ntpg;
    return;
  }
  if (mn256_ordered<BNO>(a, R)) {
    const int gps = share / per_group, gb = xcd * gps, gl = gb + gps - 1;
    int n_full = 0, n_part = 0;
    for (int i = gb; i <= gl; ++i) {
      const int c = a.cnt[i];
      n_full += c / BM;
      n_part += (c % BM) != 0;
    }
    int l = local;
    if (l < n_full * ntpg) {
      for (g = gb; g < gl; ++g) {
        const int f = a.cnt[g] / BM * ntpg;
        if (l < f) break;
        l -= f;
      }
      m_tile = l / ntpg;
      nt_in = l % ntpg;
    } else if ((l -= n_full * ntpg) < n_part * ntpg) {
      for (g = gb; g < gl; ++g) {
        const int f = (a.cnt[g] % BM) != 0 ? ntpg : 0;
        if (l < f) break;
        l -= f;
      }
      m_tile = a.cnt[g] / BM;
      nt_in = l;
    } else {
      l -= n_part * ntpg;
      for (g = gb; g < gl; ++g) {
        const int e = (a.m_tiles - (a.cnt[g] + BM - 1) / BM) * ntpg;
        if (l < e) break;
        l -= e;
      }
      m_tile = (a.cnt[g] + BM - 1) / BM + l / ntpg;
      nt_in = l % ntpg;
    }
  } else {
    if (ntpg > 4) {
      nt_in = (tile / a.m_tiles) % ntpg;
      m_tile = tile % a.m_tiles;
    } else {
      nt_in = tile % ntpg;
      m_tile = (tile / ntpg) % a.m_tiles;
    }
    g = tile / per_group;
  }
}

__device__ __forceinline__ int mn256_shares(const MN256Args& a) {
  int n = mn256_share(a.reg[0].tiles);
  if (a.n_regions > 1) n += mn256_share(a.reg[1].tiles);
  if (a.n_regions > 2) n += mn256_share(a.reg[2].tiles);
  return n;
}

// The XCD's last partial round.  An XCD's 32 CUs run its real tiles in
// rounds of 32; with T real tiles the last T % 32 would leave most CUs idle
// for a whole tile's time (measured: 15-20% of Q/K/V, 7% of gate/up).  With
// a.tail those n = T % 32 tiles are cut along k into split = 32 / n chunks,
// run by 32 extra workgroups per XCD that write fp32 partial tiles; a second
// kernel adds each tile's chunks in order and applies the epilogue.  Only
// for launches whose regions are dense or ordered (real tiles first in every
// share, so a tile's rank among the XCD's real tiles is known).
struct MN256Tail {
  int real[3], before[3];  // real tiles per region share; real tiles of earlier regions
  int base, n, split;      // first tail rank, tail tiles, chunks per tail tile
};

template <int BNO>
__device__ __forceinline__ int mn256_real(const MN256Args& a, const MN256Region& R, int xcd) {
  const int share = mn256_share(R.tiles);
  if (R.masked != kMN256Sorted) return max(0, min(share, R.tiles - xcd * share));
  const int ntpg = R.gw / BNO, gps = share / (ntpg * a.m_tiles), gb = xcd * gps;
  int n = 0;
  for (int i = 0; i < gps; ++i) n += (a.cnt[gb + i] + BM - 1) / BM;
  return n * ntpg;
}

template <int BNO>
__device__ __forceinline__ MN256Tail mn256_tail(const MN256Args& a, int xcd) {
  MN256Tail t;
  t.real[0] = mn256_real<BNO>(a, a.reg[0], xcd);
  t.real[1] = a.n_regions > 1 ? mn256_real<BNO>(a, a.reg[1], xcd) : 0;
  t.real[2] = a.n_regions > 2 ? mn256_real<BNO>(a, a.reg[2], xcd) : 0;
  t.before[0] = 0;
  t.before[1] = t.real[0];
  t.before[2] = t.real[0] + t.real[1];
  const int total = t.before[2] + t.real[2];
  t.base = total / kMN256TailJobs * kMN256TailJobs;
  t.n = total - t.base;
  // at most 8 chunks: each adds a 256 KB partial tile to write and read back
  t.split = t.n ? min(kMN256TailJobs / t.n, kMN256TailMaxSplit) : 0;
  if (!a.tail || t.split < 2) {  // nothing to gain: the tiles stay whole
    t.base = total;
    t.n = t.split = 0;
  }
  return t;
}

// Region and share-local index of tail tile k (rank base + k).
__device__ __forceinline__ void mn256_tail_tile(const MN256Tail& t, int k, int& ri, int& local) {
  const int rank = t.base + k;
  ri = rank < t.before[1] ? 0 : rank < t.before[2] ? 1 : 2;
  local = rank - (ri == 0 ? 0 : ri == 1 ? t.before[1] : t.before[2]);
}

// The k range of chunk c of n over K (in whole 64-wide units, so both ring
// depths cut at the same k): steps [s0, s0 + ns) of a BK-deep ring.
template <int BK>
__device__ __forceinline__ void mn256_chunk_steps(int K, int c, int n, int& s0, int& ns) {
  const int u = K / 64;
  const int u0 = (int)((int64_t)u * c / n), u1 = (int)((int64_t)u * (c + 1) / n);
  s0 = u0 * (64 / BK);
  ns = (u1 - u0) * (64 / BK);
}

// --------------------------------------------------------------------- GEMM-MN
template <bool SWIGLU, int BK, bool BUF>
__global__ __launch_bounds__(NT, 1) void wide_mn256(MN256Args a) {
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
  static_assert(BK == t256::BK, "64-deep ring");
  using Rg = RingMN;
  constexpr int S = Rg::SLOTS;
  constexpr int BNO = SWIGLU ? 128 : 256;  // output columns per tile
  const uint16_t* zero = g_zero_blk;

  // Workgroups are dealt round-robin to the 8 XCDs.  Each region's tiles
  // (padded to a multiple of 8) are cut into 8 contiguous shares and XCD x
  // runs share x of every region in turn: a masked region whose tail tiles
  // are mostly empty then loads the XCDs as evenly as the dense regions
  // beside it (one contiguous range per XCD over all regions left the XCDs
  // holding K and V with half again the work of the others).
  const int xcd = blockIdx.x % 8;
  int local = blockIdx.x / 8;
  const int shares = mn256_shares(a);
  int ri = 0, job = -1;   // region; tail job of a tail block
  int chunk = 0, nchunks = 1;
  if (local >= shares) {  // one of the 32 tail blocks per XCD
    job = local - shares;
    const MN256Tail t = mn256_tail<BNO>(a, xcd);
    if (job >= t.n * t.split) return;
    chunk = job % t.split;
    nchunks = t.split;
    mn256_tail_tile(t, job / t.split, ri, local);
  } else {
    ri = 0;
    if (a.n_regions > 1 && local >= mn256_share(a.reg[0].tiles)) {
      local -= mn256_share(a.reg[0].tiles);
      ri = 1;
      if (a.n_regions > 2 && local >= mn256_share(a.reg[1].tiles)) {
        local -= mn256_share(a.reg[1].tiles);
        ri = 2;
      }
    }
    if (a.tail) {  // a tile of the XCD's last partial round is left to the tail blocks
      const MN256Tail t = mn256_tail<BNO>(a, xcd);
      const int real = ri == 0 ? t.real[0] : ri == 1 ? t.real[1] : t.real[2];  // no dynamic
      const int before = ri == 0 ? 0 : ri == 1 ? t.before[1] : t.before[2];   // indexing
      if (local < real && before + local >= t.base) return;
    }
  }
  const MN256Region R = ri == 0 ? a.reg[0] : ri == 1 ? a.reg[1] : a.reg[2];
  const int share = mn256_share(R.tiles);
  const int tile = xcd * share + local;
  if (tile >= R.tiles) return;  // padding
  int g, nt_in, m_tile;
  mn256_coords<BNO>(a, R, xcd, local, g, m_tile, nt_in);
  const int n0 = g * R.gw + nt_in * BNO;
  const int64_t M = a.M;
  const int K = a.K;
  const bool sorted = R.masked == kMN256Sorted;
  const int32_t* rows = sorted ? a.idx + (int64_t)g * M : nullptr;
  const int64_t cnt = sorted ? (int64_t)a.cnt[g] : M;
  const int64_t m0 = (int64_t)m_tile * BM;
  const int tid = threadIdx.x;

  // Token-order region: thread r < 256 holds row r's mask bits over the
  // tile's groups (bit i: group n0 / mask_G + i), for the epilogue.
  const bool tok_order = R.masked == kMN256TokenOrder;
  uint32_t rbits = 0;
  bool empty = m0 >= cnt;  // l = 0: the whole tile is inactive for group g
  if (tok_order) {
    const int gpt = BNO / a.mask_G;
    if (tid < BM && m0 + tid < M) {
      const uint8_t* mr = a.mask + (m0 + tid) * a.mask_ng + n0 / a.mask_G;
      for (int i = 0; i < gpt; ++i) rbits |= (uint32_t)(mr[i] != 0) << i;
    }
    // l = 0: no (row, group) of the tile is active.  (The flag lives in the
    // ring's LDS, not yet in use: a block-wide vote would take static LDS,
    // which the five-stage ring leaves none of.)
    int* flag = reinterpret_cast<int*>(smem);
    if (tid == 0) *flag = 0;
    __syncthreads();
    if (rbits) *flag = 1;
    __syncthreads();
    empty = *flag == 0;
    __syncthreads();  // before the ring's loads overwrite the flag
  }

  if (empty) {
    if (R.skip_zero) return;
    constexpr int CH = BNO / 8;
    int my_row = -1;
    if (tid < BM && m0 + tid < M) my_row = rows ? rows[m0 + tid] : (int)(m0 + tid);
    const int* map = stage_row_map(smem, my_row);
#pragma unroll 4
    for (int i = tid; i < BM * CH; i += NT) {
      const int t = map[i / CH];
      if (t >= 0) stg16(R.out + (int64_t)t * R.ldo + n0 + (i % CH) * 8, u32x4{0, 0, 0, 0});
    }
    return;
  }

  // Sources of the lane's load slots.  l = 1: rows past the active prefix
  // read zeros.  Under SwiGLU waves 0 and 1 load gate rows, 2 and 3 up rows.
  const uint16_t* wpanel = uniform_ptr((SWIGLU && wave_id() >= 2 ? R.w1 : R.w0) + (int64_t)n0 * K);
  const bufview_t va = buf_view(uniform_ptr(a.x), BUF ? (uint32_t)(M * K * 2) : 0u);
  const bufview_t vb = buf_view(wpanel, BUF ? (uint32_t)((SWIGLU ? 128 : 256) * K * 2) : 0u);
  uint32_t aoff[S], boff[S];
  const uint16_t* abase[S];
  const uint16_t* bbase[S];
#pragma unroll
  for (int j = 0; j < S; ++j) {
    const int rr = Rg::slot_row(j);
    const int c8 = Rg::slot_chunk(j) * 8;
    const int64_t p = m0 + rr;
    const int64_t arow = p < cnt ? (rows ? (int64_t)rows[p] : p) : -1;
    const int64_t brow = SWIGLU ? (rr & 127) : rr;
    if (BUF) {
      aoff[j] = arow >= 0 ? (uint32_t)((arow * K + c8) * 2) : kOffDead;
      boff[j] = (uint32_t)((brow * K + c8) * 2);
    } else {
      abase[j] = arow >= 0 ? a.x + arow * K + c8 : nullptr;
      bbase[j] = wpanel + brow * K + c8;
    }
  }
  // B fragments of the wave: SwiGLU pairs gate column c (B rows 0..127) with
  // up column c (B rows 128..255), so a wave takes 64 gate rows (fragments 0
  // and 1) and the same 64 up rows (fragments 2 and 3)
  const int wn = wave_id() & 1;
  constexpr int BL = SWIGLU ? 1 : 0;
  int bb[4];
#pragma unroll
  for (int fn = 0; fn < 4; ++fn) bb[fn] = (SWIGLU ? wn * 64 : wn * 128) + bfrag_off<BL>(fn);

  f32x16 acc[4][4];
  zero_acc(acc);
  int s0 = 0, ns = K / BK;  // a tail chunk runs its share of the k steps
  if (job >= 0) mn256_chunk_steps<BK>(K, chunk, nchunks, s0, ns);
  auto koff = [&](int s) { return (s0 + s) * BK; };
  auto lda = [&](uint16_t* st, int k0, int j) {
    if (BUF) Rg::issue_buf(st, va, aoff[j], 2u * k0, j);
    else Rg::issue_ptr(st, abase[j] ? abase[j] + k0 : zero, j);
  };
  auto ldb = [&](uint16_t* st, int k0, int j) {
    if (BUF) Rg::issue_buf(st, vb, boff[j], 2u * k0, j);
    else Rg::issue_ptr(st, bbase[j] + k0, j);
  };
  int my_row = -1;
  if (job < 0 && tid < BM && m0 + tid < M) my_row = rows ? rows[m0 + tid] : (int)(m0 + tid);
  // l = 2: fragments wholly past the active prefix issue no MFMA
  run_tile<Rg, BL>(smem, ns, koff, lda, ldb, bb, cnt - m0, acc);
  const int col = acc_col();

  if (job >= 0) {  // tail chunk: fp32 partial tile [256 rows][256 B-tile rows]
    float* P = a.tail_ws + ((int64_t)xcd * kMN256TailJobs + job) * (BM * BN);
#pragma unroll
    for (int fm = 0; fm < 4; ++fm)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int r = acc_row(fm, i);
#pragma unroll
        for (int fn = 0; fn < 4; ++fn) P[r * BN + bb[fn] + col] = acc[fm][fn][i];
      }
    return;
  }

  // Epilogue: rows back to token order; rows past cnt hold +0 accumulators.
  // A token-order region stores +0 where the row's group is inactive.  The
  // bf16 tile goes through the idle ring LDS (after the row map), rows
  // padded by 16 bytes, so that each lane then stores whole 16-byte pieces of
  // an output row: 8 times fewer store instructions than a 2-byte store per
  // accumulator, which is how the MFMA layout holds them (those stores cost
  // gate/up 3%; staged, gate/up is 1.5% faster).
  const int* map = stage_row_map(smem, my_row, (int)rbits);
  const int gsh = tok_order ? __builtin_ctz(a.mask_G) : 0;
  constexpr int NO = SWIGLU ? 2 : 4;  // output fragments of the wave
  constexpr int PITCH = BNO + 8;      // bf16 per staged row
  static_assert(2 * BM * (int)sizeof(int) + BM * PITCH * 2 <= Rg::LDS, "row map and staged tile fit the ring");
  uint16_t* ot = smem + 2 * BM * (int)(sizeof(int) / sizeof(uint16_t));
#pragma unroll
  for (int fm = 0; fm < 4; ++fm) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int r = acc_row(fm, i);
      const int rb = tok_order ? map[BM + r] : 0;
#pragma unroll
      for (int fn = 0; fn < NO; ++fn) {
        const int c = bb[fn] + col;  // output column in the tile
        const bool on = !tok_order || ((rb >> (c >> gsh)) & 1);
        const float v = SWIGLU ? silu(acc[fm][fn][i]) * acc[fm][fn + 2][i] : acc[fm][fn][i];
        ot[r * PITCH + c] = f32_to_bf16_hw(on ? v : 0.f);
      }
    }
  }
  __syncthreads();
  constexpr int CPR = BNO / 8;  // 16-byte pieces per output row
#pragma unroll 4
  for (int q = tid; q < BM * CPR; q += NT) {
    const int r = q / CPR, c8 = q % CPR;
    const int t = map[r];
    if (t >= 0)
      stg16(R.out + (int64_t)t * R.ldo + n0 + c8 * 8, *reinterpret_cast<const u32x4*>(ot + r * PITCH + c8 * 8));
  }
}

// Finish the XCDs' tail tiles: add each tile's chunks in order, then the
// mn256 epilogue (SwiGLU or plain, rows back to token order).  Workgroup
// (xcd, k, rb) takes rows [16 rb, 16 rb + 16) of tail tile k; each thread
// loads the chunks of its elements together (independent loads) and adds
// them in chunk order.
constexpr int kTailRows = 16;
template <bool SWIGLU>
__global__ __launch_bounds__(NT) void wide_mn256_tail(MN256Args a) {
  constexpr int BNO = SWIGLU ? 128 : 256;
  constexpr int PER = kTailRows * BNO / NT;  // elements per thread
  __shared__ int map[kTailRows];
  static_assert(kTailRows <= NT, "one thread per row for the row map");
  const int rb = blockIdx.x % (BM / kTailRows);
  const int k = (blockIdx.x / (BM / kTailRows)) % kMN256TailJobs;
  const int xcd = blockIdx.x / (BM / kTailRows * kMN256TailJobs);
  const MN256Tail t = mn256_tail<BNO>(a, xcd);
  if (k >= t.n) return;
  int ri, local, g, m_tile, nt_in;
  mn256_tail_tile(t, k, ri, local);
  const MN256Region R = ri == 0 ? a.reg[0] : ri == 1 ? a.reg[1] : a.reg[2];
  mn256_coords<BNO>(a, R, xcd, local, g, m_tile, nt_in);
  const int n0 = g * R.gw + nt_in * BNO;
  const int32_t* rows = R.masked ? a.idx + (int64_t)g * a.M : nullptr;
  const int64_t p0 = (int64_t)m_tile * BM + rb * kTailRows;
  const int tid = threadIdx.x;
  if (tid < kTailRows) map[tid] = p0 + tid < a.M ? (rows ? rows[p0 + tid] : (int)(p0 + tid)) : -1;
  __syncthreads();
  const float* P = a.tail_ws + ((int64_t)xcd * kMN256TailJobs + k * t.split) * (BM * BN);
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int i = e * NT + tid;
    const int r = i / BNO, c = i % BNO;
    const int tok = map[r];
    const float* Pe = P + (rb * kTailRows + r) * BN + c;
    float v0[kMN256TailMaxSplit], v1[kMN256TailMaxSplit];
#pragma unroll
    for (int q = 0; q < kMN256TailMaxSplit; ++q) {
      const bool on = q < t.split;
      const float* Pq = Pe + (int64_t)(on ? q : 0) * (BM * BN);  // in range whether or not used
      v0[q] = on ? Pq[0] : 0.f;
      v1[q] = SWIGLU && on ? Pq[128] : 0.f;
    }
    float s0 = 0.f, s1 = 0.f;
#pragma unroll
    for (int q = 0; q < kMN256TailMaxSplit; ++q) {  // chunk order
      s0 += v0[q];
      s1 += v1[q];
    }
    if (tok < 0) continue;
    const bool on = R.masked != kMN256TokenOrder || a.mask[(int64_t)tok * a.mask_ng + (n0 + c) / a.mask_G] != 0;
    R.out[(int64_t)tok * R.ldo + n0 + c] = f32_to_bf16_hw(on ? (SWIGLU ? silu(s0) * s1 : s0) : 0.f);
  }
}

// ----------------------------------------------------------- K-axis, dense-masked
// NWR: mask words (32 groups each) of the lane's slot rows held in registers
// for the whole k loop (1: up to 32 groups, 4: up to 128); 0 reads them from
// LDS at every step.
// Tile order of the dense-masked K axis.  One workgroup fits a CU, so the
// chip runs the tiles in rounds of 256.  When the column tiles divide a
// round (n_tiles even, 256 / n_tiles a multiple of 4), round r covers the
// m-tiles [r*mr, (r+1)*mr) (mr = 256 / n_tiles) times every column tile, and
// XCD x takes a block of mr/4 m-tiles x n_tiles/2 column tiles of it: a
// round's operands (mr row panels and all of W) then fit the last-level
// cache, and the tiles of one XCD share 12 k slices per step in its L2
// (Llama-3-8B down, 8192 x 4096 x 14336: 4-6% faster than walking the m-tiles
// of each XCD's contiguous range in turn, which needs 18 and, chip-wide,
// every row panel in each round).  Tiles past the last full round, and
// shapes the blocks do not fit, keep that m-major walk.
__device__ __forceinline__ void kd256_coords(int n_tiles, int m_tiles, int& m_tile, int& n_tile) {
  const int total = m_tiles * n_tiles;
  const bool blocks = n_tiles % 2 == 0 && n_tiles <= 256 && 256 % n_tiles == 0 && (256 / n_tiles) % 4 == 0;
  const int rounds = blocks ? total / 256 : 0;
  const int id = blockIdx.x;
  if (id < rounds * 256) {
    const int xcd = id % 8, local = id / 8;  // workgroups are dealt round-robin to the 8 XCDs
    const int r = local / 32, q = local % 32;
    const int mr = 256 / n_tiles, bm = mr / 4, bn = n_tiles / 2;
    m_tile = r * mr + (xcd % 4) * bm + q % bm;
    n_tile = (xcd / 4) * bn + q / bm;
    return;
  }
  const int base = rounds * 256;
  const int tile = base + xcd_remap(id - base, total - base);  // m-major: n-tiles share the A panel
  m_tile = tile / n_tiles;
  n_tile = tile % n_tiles;
}

// Mask tables of a dense-masked tile: the rows' mask bits, the groups some
// row uses (ascending), their union and count.  With NWR > 0 they live in the
// ring's LDS before its first load and move to registers (the ring then takes
// all of LDS); with NWR = 0 they sit past a ring of two A stages.
struct KdTables {
  uint32_t mbits[BM][kKd256MaxGroups / 32];
  uint16_t groups[kKd256MaxGroups];
  uint32_t uni[kKd256MaxGroups / 32];
  int n_live;
};
template <int NWR>
constexpr int kd256_lds() {
  return NWR == 0 ? RingKD<0>::LDS + (int)sizeof(KdTables) : RingKD<NWR>::LDS;
}
static_assert(kd256_lds<0>() <= LDS_MAX && (int)sizeof(KdTables) <= RingKD<4>::LDS, "tables fit");

template <int NWR, int BK, bool BUF>
__global__ __launch_bounds__(NT, 1) void wide_kd256(KArgs a) {
  static_assert(BK == t256::BK, "64-deep ring");
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
  using Rg = RingKD<NWR>;
  constexpr int S = Rg::SLOTS;
  KdTables& tb = *reinterpret_cast<KdTables*>(reinterpret_cast<char*>(smem) + (NWR == 0 ? Rg::LDS : 0));
  const uint16_t* zero = g_zero_blk;
  const int n_tiles = a.N / BN;
  int m_tile, n_tile;
  kd256_coords(n_tiles, (int)((a.M + BM - 1) / BM), m_tile, n_tile);
  const int64_t m0 = (int64_t)m_tile * BM;
  const int n0 = n_tile * BN;
  const int ng = a.K / a.G;
  const int nw = (ng + 31) / 32;
  const int tid = threadIdx.x;

  if (tid < nw) tb.uni[tid] = 0u;
  __syncthreads();
  // Tile row r is token m0 + r, or perm[m0 + r] when the rows are ordered by
  // mask pattern (rows that share groups then share the tile).
  auto token = [&](int64_t p) -> int64_t { return a.perm ? (int64_t)a.perm[p] : p; };
  for (int i = tid; i < BM * nw; i += NT) {
    const int r = i / nw, wd = i % nw;
    const int64_t p = m0 + r;
    const int64_t t = p < a.M ? token(p) : a.M;
    uint32_t bits = 0;
    if (t < a.M) bits = mask_bits32(a.mask + t * ng + wd * 32, min(32, ng - wd * 32), ng);
    tb.mbits[r][wd] = bits;
    if (bits) atomicOr(&tb.uni[wd], bits);
  }
  __syncthreads();
  // groups some row of the tile uses, ascending: thread g places group g at
  // the count of union bits below it (no serial pass over the union)
  for (int gi = tid; gi < nw * 32; gi += NT) {
    const int wd = gi >> 5, b = gi & 31;
    int pos = __builtin_popcount(tb.uni[wd] & ((1u << b) - 1u));
    for (int i = 0; i < wd; ++i) pos += __builtin_popcount(tb.uni[i]);
    if ((tb.uni[wd] >> b) & 1u) tb.groups[pos] = (uint16_t)gi;
    if (gi == 0) {
      int n = 0;
      for (int i = 0; i < nw; ++i) n += __builtin_popcount(tb.uni[i]);
      tb.n_live = n;
    }
  }
  __syncthreads();
  const int spg = a.G / BK;  // k steps per group
  const int nsteps = __builtin_amdgcn_readfirstlane(tb.n_live) * spg;

  int srow[S];
  const uint16_t* wpanel = uniform_ptr(a.w + (int64_t)n0 * a.K);
  const bufview_t va = buf_view(uniform_ptr(a.a), BUF ? (uint32_t)(a.M * a.K * 2) : 0u);
  const bufview_t vb = buf_view(wpanel, BUF ? (uint32_t)(BN * a.K * 2) : 0u);
  uint32_t aoff[S], boff[S];
  const uint16_t* abase[S];
  const uint16_t* bbase[S];
#pragma unroll
  for (int j = 0; j < S; ++j) {
    const int rr = Rg::slot_row(j);
    const int c8 = Rg::slot_chunk(j) * 8;
    const int64_t p = m0 + rr;
    const int64_t arow = p < a.M ? token(p) : -1;
    srow[j] = rr;
    if (BUF) {
      aoff[j] = arow >= 0 ? (uint32_t)((arow * a.K + c8) * 2) : kOffDead;
      boff[j] = (uint32_t)(((int64_t)rr * a.K + c8) * 2);
    } else {
      abase[j] = arow >= 0 ? a.a + arow * a.K + c8 : nullptr;
      bbase[j] = wpanel + (int64_t)rr * a.K + c8;
    }
  }
  const int lane = lane_id(), wn = wave_id() & 1;
  int bb[4];
#pragma unroll
  for (int fn = 0; fn < 4; ++fn) bb[fn] = wn * 128 + bfrag_off<0>(fn);

  f32x16 acc[4][4];
  zero_acc(acc);
  // Every step needs, per slot row, one bit of its mask row.  Reading them
  // from LDS at each step put several dependent LDS round trips in front of
  // the step's loads; with NWR > 0 the rows' mask words sit in registers,
  // inverted (rows past M hold zero words, all ones inverted, so their
  // blocks read as zeros), and so does the union's group list: lane l holds
  // groups l and 64 + l, and a step takes its group with a readlane.
  // (words past the row's last group are never selected: any value will do)
  uint64_t nlo[S], nhi[S];
#pragma unroll
  for (int j = 0; j < S; ++j) {
    nlo[j] = nhi[j] = ~0ull;
    if (NWR >= 1) nlo[j] = ~(uint64_t)tb.mbits[srow[j]][0];
    if (NWR >= 4) {
      nlo[j] = ~((uint64_t)tb.mbits[srow[j]][0] | (uint64_t)tb.mbits[srow[j]][1] << 32);
      nhi[j] = ~((uint64_t)tb.mbits[srow[j]][2] | (uint64_t)tb.mbits[srow[j]][3] << 32);
    }
  }
  const int glo = NWR >= 1 ? tb.groups[lane] : 0;
  const int ghi = NWR >= 4 ? tb.groups[64 + lane] : 0;
  if (NWR > 0) __syncthreads();  // the ring's first loads overwrite the tables
  auto group = [&](int gi) -> int {  // gi-th group of the tile's union
    if (NWR == 1) return __builtin_amdgcn_readlane(glo, gi);
    if (NWR == 4) {  // both reads and a scalar select: no branch in the k loop
      const int lo = __builtin_amdgcn_readlane(glo, gi & 63), hi = __builtin_amdgcn_readlane(ghi, gi & 63);
      return gi < 64 ? lo : hi;
    }
    return __builtin_amdgcn_readfirstlane(tb.groups[gi]);  // one LDS word, the same for every lane
  };
  const int lg = __builtin_ctz(a.G), lsp = lg - 6;  // G is a power of two, at least BK
  auto koff = [&](int s) {
    const int gi = s >> lsp;
    return group(gi) * a.G + (s & (spg - 1)) * BK;
  };
  // Inactive (t, g) blocks are never read.  Bit 31 of `dead` is set for
  // them: the inverted mask bit shifted up to bit 31 (one 64-bit shift by a
  // uniform amount) and merged into the row's view offset.  A row's offset
  // plus any step's k offset is a byte inside the view, below 2^31, so with
  // bit 31 added the sum is past the view and below 2^32 (no wrap).  Four
  // vector instructions per load where a compare and a select took six.
  auto lda = [&](uint16_t* st, int k0, int j) {
    const int gg = k0 >> lg;
    uint32_t dead;
    if (NWR == 0)
      dead = (tb.mbits[srow[j]][gg >> 5] >> (gg & 31)) & 1u ? 0u : kOffDead;
    else if (NWR == 1)
      dead = (uint32_t)nlo[j] << (31 - gg);
    else
      dead = (uint32_t)(((gg < 64 ? nlo[j] : nhi[j]) << (63 - (gg & 63))) >> 32);
    dead &= kOffDead;
    if (BUF) Rg::issue_buf(st, va, dead | aoff[j], 2u * k0, j);
    else Rg::issue_ptr(st, dead ? zero : abase[j] + k0, j);
  };
  auto ldb = [&](uint16_t* st, int k0, int j) {
    if (BUF) Rg::issue_buf(st, vb, boff[j], 2u * k0, j);
    else Rg::issue_ptr(st, bbase[j] + k0, j);
  };
  int my_row = -1;
  if (tid < BM && m0 + tid < a.M) my_row = (int)token(m0 + tid);
  run_tile<Rg, 0>(smem, nsteps, koff, lda, ldb, bb, a.M - m0, acc);

  const int* map = stage_row_map(smem, my_row);
  const int col = acc_col();
#pragma unroll
  for (int fm = 0; fm < 4; ++fm)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int t = map[acc_row(fm, i)];
      if (t < 0) continue;
      uint16_t* o = a.y + (int64_t)t * a.N + n0 + col;
#pragma unroll
      for (int fn = 0; fn < 4; ++fn) o[bb[fn]] = f32_to_bf16_hw(acc[fm][fn][i]);
    }
}

// -------------------------------------------------------------- K-axis, scatter
// One workgroup owns (sorted-position tile, 256 output columns, a run of
// a.pack K-groups) and runs the groups in turn, each with its own pipeline
// prologue and accumulator (Appendix B, Algorithm 3 and its outer loop that
// packs K-groups into one CTA).  When the column tiles divide among the 8
// XCDs, workgroup ids are dealt so that every workgroup adding into a column
// slab runs on the same XCD.
template <int BK, bool BUF>
__global__ __launch_bounds__(NT, 1) void wide_ks256(KArgs a) {
  static_assert(BK == t256::BK, "64-deep ring");
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];
  using Rg = RingMN;
  constexpr int S = Rg::SLOTS;
  const uint16_t* zero = g_zero_blk;
  const int n_tiles = a.N / BN;
  const int m_tiles = (int)((a.M + BM - 1) / BM);
  const int ng = a.K / a.G;
  const int n_splits = (ng + a.pack - 1) / a.pack;
  int n_tile, m_tile, split;
  if (n_tiles % 8 == 0) {  // column slab of the workgroup's XCD (dispatch is round-robin over XCDs)
    const int xcd = blockIdx.x % 8, local = blockIdx.x / 8, per = n_tiles / 8;
    n_tile = xcd * per + local % per;
    m_tile = (local / per) % m_tiles;
    split = local / per / m_tiles;
  } else {
    const int tile = xcd_remap(blockIdx.x, gridDim.x);
    n_tile = tile % n_tiles;
    m_tile = (tile / n_tiles) % m_tiles;
    split = tile / (n_tiles * m_tiles);
  }
  if (split >= n_splits) return;
  const int g_end = min(ng, (split + 1) * a.pack);
  const int64_t m0 = (int64_t)m_tile * BM;
  const int n0 = n_tile * BN;
  const int wn = wave_id() & 1;
  int bb[4];
#pragma unroll
  for (int fn = 0; fn < 4; ++fn) bb[fn] = wn * 128 + bfrag_off<0>(fn);
  const int col = acc_col();
  const int* map = reinterpret_cast<const int*>(smem);
  const uint16_t* wpanel = uniform_ptr(a.w + (int64_t)n0 * a.K);
  const bufview_t va = buf_view(uniform_ptr(a.a), BUF ? (uint32_t)(a.M * a.K * 2) : 0u);
  const bufview_t vb = buf_view(wpanel, BUF ? (uint32_t)(BN * a.K * 2) : 0u);
  for (int g = split * a.pack; g < g_end; ++g) {
    const int64_t cnt = a.cnt[g];
    if (m0 >= cnt) continue;  // l = 0 for this group
    const int32_t* rows = a.idx + (int64_t)g * a.M;
    uint32_t aoff[S], boff[S];
    const uint16_t* abase[S];
    const uint16_t* bbase[S];
#pragma unroll
    for (int j = 0; j < S; ++j) {
      const int rr = Rg::slot_row(j);
      const int c8 = Rg::slot_chunk(j) * 8;
      const int64_t p = m0 + rr;
      const int64_t arow = p < cnt ? (int64_t)rows[p] : -1;  // l = 1
      if (BUF) {
        aoff[j] = arow >= 0 ? (uint32_t)((arow * a.K + c8) * 2) : kOffDead;
        boff[j] = (uint32_t)(((int64_t)rr * a.K + c8) * 2);
      } else {
        abase[j] = arow >= 0 ? a.a + arow * a.K + c8 : nullptr;
        bbase[j] = wpanel + (int64_t)rr * a.K + c8;
      }
    }
    f32x16 acc[4][4];
    zero_acc(acc);
    const int kbeg = g * a.G;
    auto koff = [&](int s) { return kbeg + s * BK; };
    auto lda = [&](uint16_t* st, int k0, int j) {
      if (BUF) Rg::issue_buf(st, va, aoff[j], 2u * k0, j);
      else Rg::issue_ptr(st, abase[j] ? abase[j] + k0 : zero, j);
    };
    auto ldb = [&](uint16_t* st, int k0, int j) {
      if (BUF) Rg::issue_buf(st, vb, boff[j], 2u * k0, j);
      else Rg::issue_ptr(st, bbase[j] + k0, j);
    };
    int my_row = -1;
    if ((int)threadIdx.x < BM && m0 + (int)threadIdx.x < cnt) my_row = rows[m0 + threadIdx.x];
    __syncthreads();  // the previous group's epilogue is done with the row map in the ring
    run_tile<Rg, 0>(smem, a.G / BK, koff, lda, ldb, bb, cnt - m0, acc);  // l = 2: dead fragments skipped
    stage_row_map(smem, my_row);
#pragma unroll
    for (int fm = 0; fm < 4; ++fm) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int t = map[acc_row(fm, i)];
        if (t < 0) continue;
        float* o = a.acc32 + (int64_t)t * a.N + n0 + col;
#pragma unroll
        for (int fn = 0; fn < 4; ++fn) unsafeAtomicAdd(o + bb[fn], acc[fm][fn][i]);
      }
    }
  }
}

// ------------------------------------------------------------------ launchers
namespace {
template <class F>
hipError_t allow_big_lds(F* f, int bytes) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(f),
                             hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
}

// Raise the dynamic-LDS limit of one kernel instance once per process.
template <auto Kern, int Bytes>
hipError_t prepare() {
  static const hipError_t e = allow_big_lds(Kern, Bytes);
  return e;
}
}  // namespace

#define WIDE_RING_LAUNCH(NAME, KERN, LDSB, GRID, STREAM, ARGS)                                    \
  do {                                                                                            \
    hipError_t e_ = prepare<KERN, LDSB>();                                                        \
    if (e_ != hipSuccess) return e_;                                                              \
    WIDE_LAUNCH_NAMED(NAME "/bk64", (KERN), dim3(GRID), dim3(NT), LDSB, STREAM, ARGS);            \
  } while (0)

// Buffer-view sources when the token-row operand fits a view (2 GB); the
// same kernels on 64-bit addresses beyond.
bool views_fit(int64_t rows, int K) { return rows * (int64_t)K * 2 <= kBufViewMax; }

hipError_t launch_mn256(const MN256Args& a, bool swiglu, hipStream_t s) {
  int64_t total = 0;
  for (int i = 0; i < a.n_regions; ++i) total += 8 * (int64_t)mn256_share(a.reg[i].tiles);
  if (total == 0) return hipSuccess;
  if (a.tail) total += 8 * kMN256TailJobs;  // the tail blocks of every XCD, dispatched last
  const bool buf = views_fit(a.M, a.K);
  if (swiglu && buf)
    WIDE_RING_LAUNCH("wide_mn256<true>", (wide_mn256<true, 64, true>), RingMN::LDS, (unsigned)total, s, a);
  else if (swiglu)
    WIDE_RING_LAUNCH("wide_mn256<true>", (wide_mn256<true, 64, false>), RingMN::LDS, (unsigned)total, s, a);
  else if (buf)
    WIDE_RING_LAUNCH("wide_mn256<false>", (wide_mn256<false, 64, true>), RingMN::LDS, (unsigned)total, s, a);
  else
    WIDE_RING_LAUNCH("wide_mn256<false>", (wide_mn256<false, 64, false>), RingMN::LDS, (unsigned)total, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !a.tail) return e;
  const dim3 tg(8 * kMN256TailJobs * (BM / kTailRows));
  if (swiglu)
    WIDE_LAUNCH(wide_mn256_tail<true>, tg, dim3(NT), 0, s, a);
  else
    WIDE_LAUNCH(wide_mn256_tail<false>, tg, dim3(NT), 0, s, a);
  return hipGetLastError();
}

bool mn256_tail_ok(const MN256Args& a, int bno) {
  for (int i = 0; i < a.n_regions; ++i) {
    const MN256Region& R = a.reg[i];
    if (R.masked != kMN256Sorted) continue;  // dense and token-order regions: every tile is real
    const int share = mn256_share(R.tiles), per_group = R.gw / bno * a.m_tiles;
    if (!(a.order && !a.mblock && R.gw / bno <= 4 && 8 * share == R.tiles && share % per_group == 0))
      return false;
  }
  return true;
}

hipError_t launch_kd256(const KArgs& a, hipStream_t s) {
  const int64_t m_tiles = (a.M + BM - 1) / BM;
  const int64_t total = m_tiles * (a.N / BN);
  if (total == 0) return hipSuccess;
  if (a.K / a.G > kKd256MaxGroups) return hipErrorInvalidValue;
  const int ng = a.K / a.G;
  const bool buf = views_fit(a.M, a.K);
  if (ng <= 32 && buf)
    WIDE_RING_LAUNCH("wide_kd256<1>", (wide_kd256<1, 64, true>), kd256_lds<1>(), (unsigned)total, s, a);
  else if (ng <= 32)
    WIDE_RING_LAUNCH("wide_kd256<1>", (wide_kd256<1, 64, false>), kd256_lds<1>(), (unsigned)total, s, a);
  else if (ng <= 128 && buf)
    WIDE_RING_LAUNCH("wide_kd256<4>", (wide_kd256<4, 64, true>), kd256_lds<4>(), (unsigned)total, s, a);
  else if (ng <= 128)
    WIDE_RING_LAUNCH("wide_kd256<4>", (wide_kd256<4, 64, false>), kd256_lds<4>(), (unsigned)total, s, a);
  else if (buf)
    WIDE_RING_LAUNCH("wide_kd256<0>", (wide_kd256<0, 64, true>), kd256_lds<0>(), (unsigned)total, s, a);
  else
    WIDE_RING_LAUNCH("wide_kd256<0>", (wide_kd256<0, 64, false>), kd256_lds<0>(), (unsigned)total, s, a);
  return hipGetLastError();
}

hipError_t launch_ks256(const KArgs& a, hipStream_t s) {
  const int64_t m_tiles = (a.M + BM - 1) / BM;
  const int pack = a.pack > 0 ? a.pack : 1;
  const int64_t splits = (a.K / a.G + pack - 1) / pack;
  const int64_t total = splits * m_tiles * (a.N / BN);
  if (total == 0) return hipSuccess;
  if (views_fit(a.M, a.K))
    WIDE_RING_LAUNCH("wide_ks256", (wide_ks256<64, true>), RingMN::LDS, (unsigned)total, s, a);
  else
    WIDE_RING_LAUNCH("wide_ks256", (wide_ks256<64, false>), RingMN::LDS, (unsigned)total, s, a);
  return hipGetLastError();
}

}  // namespace wide
