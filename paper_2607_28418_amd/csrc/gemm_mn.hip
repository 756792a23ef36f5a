// Prefill N-axis masked GEMM ("GEMM-MN"), bf16 MFMA on gfx950.
//
// Computes out[t, n] = x_t . w[n] for the output columns n of a routing group
// g and only for tokens active in g (WIDE Section 3.1, equations (1) and (3):
// W_q, W_gate and W_up pruned over their out-features), writing +0 for the
// inactive tokens.  The rows of each group are taken in the order of the mask
// reorder, so the active tokens of g are the prefix idx[g][0:cnt[g]]
// (Section 3.3); a tile of BM consecutive sorted positions is then entirely
// active, entirely inactive, or the single boundary tile of the group
// (Appendix B, the GEMM-MN description and Algorithm 2).
//
// Skipping, in the paper's three levels:
//   l = 0  a tile whose first sorted position is >= cnt[g] does no loads and
//          no MFMA; it only writes the +0 rows its positions stand for;
//   l = 1  in the boundary tile, A rows at positions >= cnt[g] are not loaded
//          (their LDS rows are zero-filled);
//   l = 2  a wave whose 32-row MFMA fragment lies wholly at positions >=
//          cnt[g] issues no MFMA for it (wave-uniform branch).
//
// Tile: BM = 128 sorted tokens x 128 weight rows x BK = 64, 256 threads as a
// 2x2 grid of waves, each wave 64 x 64 with 32x32x16 MFMAs.  In SwiGLU mode
// the 128 weight rows are 64 gate rows and the 64 up rows of the same
// output columns; each wave holds the matching gate and up fragments, so
// silu(gate) * up is formed in registers and only H is stored.  Operands pass
// through a double-buffered LDS ring (2 x 32 KB) whose 16-byte chunks are
// XOR-swizzled by row, which keeps both the stores and the MFMA-fragment
// reads free of bank conflicts without padding.
#include "common.h"
#include "launch.h"
#include "kernels.h"

namespace wide {

namespace {

constexpr int BM = 128;
constexpr int BK = 64;
constexpr int NT = 256;        // threads

// Workgroup id -> tile id such that each of the 8 XCDs (which receive
// workgroups round-robin) walks a contiguous range of tiles; tiles that
// share a weight tile then share that XCD's L2.
__device__ __forceinline__ int xcd_remap(int id, int n) {
  const int q = n / 8, r = n % 8;
  const int xcd = id % 8, local = id / 8;
  return (xcd < r) ? xcd * (q + 1) + local : r * (q + 1) + (xcd - r) * q + local;
}

__device__ __forceinline__ int swz(int row, int chunk) {  // element offset in a [rows][64] tile
  // 16 lanes of a 128-bit LDS read hit 64 banks together: keep rows r and
  // r + 8 on different chunks (see tile256.h)
  return row * BK + ((chunk ^ ((row & 7) ^ ((row >> 3) & 1))) << 3);
}

}  // namespace

template <bool SWIGLU>
__global__ __launch_bounds__(NT, 2) void wide_gemm_mn(MNArgs a) {
  constexpr int BNO = SWIGLU ? 64 : 128;   // output columns per tile
  __shared__ __attribute__((aligned(16))) uint16_t lds[2][2][BM * BK];

  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int n_tile = tile / a.m_tiles;
  const int m_tile = tile % a.m_tiles;

  int nt = n_tile;
  MNRegion R = a.reg[0];
  if (a.n_regions > 1 && nt >= a.reg[0].n_tiles) {
    nt -= a.reg[0].n_tiles;
    R = a.reg[1];
    if (a.n_regions > 2 && nt >= a.reg[1].n_tiles) {
      nt -= a.reg[1].n_tiles;
      R = a.reg[2];
    }
  }
  const int n0 = nt * BNO;
  const int64_t M = a.M;
  const int K = a.K;
  const int64_t m0 = (int64_t)m_tile * BM;
  const int32_t* rows = nullptr;
  int64_t cnt = M;
  if (R.masked) {
    const int g = n0 / a.G;
    rows = a.idx + (int64_t)g * M;
    cnt = a.cnt[g];
  }
  const int tid = threadIdx.x;

  if (m0 >= cnt) {
    // l = 0: every token at these sorted positions is inactive for g.
    const int64_t pend = min(m0 + BM, M);
    constexpr int CH = BNO / 8;  // 16-byte chunks per output row
    for (int i = tid; i < BM * CH; i += NT) {
      const int64_t p = m0 + i / CH;
      if (p < pend) {
        const int64_t t = rows ? rows[p] : p;
        stg16(R.out + t * R.ldo + n0 + (i % CH) * 8, u32x4{0, 0, 0, 0});
      }
    }
    return;
  }

  // Per-thread global-load assignments: 4 A rows and 4 weight rows.
  const int lrow = tid / 8, lch = tid % 8;
  const uint16_t* ap[4];
  const uint16_t* bp[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = lrow + 32 * i;
    const int64_t p = m0 + r;
    ap[i] = nullptr;
    if (p < cnt) {
      const int64_t t = rows ? rows[p] : p;
      ap[i] = a.x + t * K + lch * 8;
    }
    if (SWIGLU) {
      bp[i] = (r < 64) ? R.w0 + (int64_t)(n0 + r) * K + lch * 8
                       : R.w1 + (int64_t)(n0 + r - 64) * K + lch * 8;
    } else {
      bp[i] = R.w0 + (int64_t)(n0 + r) * K + lch * 8;
    }
  }

  const int w = wave_id(), lane = lane_id();
  const int wm = w >> 1, wn = w & 1;
  const int l32 = lane & 31, lhi = lane >> 5;
  // l = 2: fragment fm of this wave is live iff its first sorted row < cnt.
  const bool frag_live0 = m0 + wm * 64 < cnt;
  const bool frag_live1 = m0 + wm * 64 + 32 < cnt;

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};

  u32x4 ra[4], rb[4];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ra[i] = ap[i] ? ldg16(ap[i] + k0) : u32x4{0, 0, 0, 0};
      rb[i] = ldg16(bp[i] + k0);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = lrow + 32 * i;
      *reinterpret_cast<u32x4*>(&lds[buf][0][swz(r, lch)]) = ra[i];
      *reinterpret_cast<u32x4*>(&lds[buf][1][swz(r, lch)]) = rb[i];
    }
  };

  const int nk = K / BK;
  gload(0);
  lstore(0);
  __syncthreads();

  // Fragment rows inside the tile.
  const int arow0 = wm * 64 + l32, arow1 = arow0 + 32;
  int brow0, brow1;
  if (SWIGLU) {
    brow0 = wn * 32 + l32;        // gate rows
    brow1 = 64 + wn * 32 + l32;   // up rows, same output columns
  } else {
    brow0 = wn * 64 + l32;
    brow1 = brow0 + 32;
  }

  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * BK);
    const uint16_t* As = lds[buf][0];
    const uint16_t* Bs = lds[buf][1];
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int ch = kk * 2 + lhi;
      const u32x4 b0 = *reinterpret_cast<const u32x4*>(&Bs[swz(brow0, ch)]);
      const u32x4 b1 = *reinterpret_cast<const u32x4*>(&Bs[swz(brow1, ch)]);
      if (frag_live0) {
        const u32x4 a0 = *reinterpret_cast<const u32x4*>(&As[swz(arow0, ch)]);
        acc[0][0] = mfma32(a0, b0, acc[0][0]);
        acc[0][1] = mfma32(a0, b1, acc[0][1]);
      }
      if (frag_live1) {
        const u32x4 a1 = *reinterpret_cast<const u32x4*>(&As[swz(arow1, ch)]);
        acc[1][0] = mfma32(a1, b0, acc[1][0]);
        acc[1][1] = mfma32(a1, b1, acc[1][1]);
      }
    }
    if (kt + 1 < nk) lstore(buf ^ 1);
    __syncthreads();
  }

  // Epilogue: scatter rows back to token order.  Positions in [cnt, M) hold
  // inactive tokens whose accumulators are exactly +0, so they store +0.
#pragma unroll
  for (int fm = 0; fm < 2; ++fm) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int r = wm * 64 + fm * 32 + (i >> 2) * 8 + lhi * 4 + (i & 3);
      const int64_t p = m0 + r;
      if (p >= M) continue;
      const int64_t t = rows ? rows[p] : p;
      uint16_t* o = R.out + t * R.ldo + n0;
      if (SWIGLU) {
        const float h = silu(acc[fm][0][i]) * acc[fm][1][i];
        o[wn * 32 + l32] = f32_to_bf16(h);
      } else {
        o[wn * 64 + l32] = f32_to_bf16(acc[fm][0][i]);
        o[wn * 64 + 32 + l32] = f32_to_bf16(acc[fm][1][i]);
      }
    }
  }
}

hipError_t launch_gemm_mn(const MNArgs& a, bool swiglu, hipStream_t s) {
  int n_tiles = 0;
  for (int i = 0; i < a.n_regions; ++i) n_tiles += a.reg[i].n_tiles;
  const int64_t total = (int64_t)n_tiles * a.m_tiles;
  if (total == 0) return hipSuccess;
  if (swiglu)
    WIDE_LAUNCH((wide_gemm_mn<true>), dim3((unsigned)total), dim3(NT), 0, s, a);
  else
    WIDE_LAUNCH((wide_gemm_mn<false>), dim3((unsigned)total), dim3(NT), 0, s, a);
  return hipGetLastError();
}

}  // namespace wide
