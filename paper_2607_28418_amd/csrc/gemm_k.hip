// Prefill K-axis masked GEMM ("GEMM-K"), bf16 MFMA on gfx950.
//
//   y[t, n] = sum over groups g active for t of sum_{k in group g} a[t, k] w[n, k]
//
// (WIDE Section 3.1, equations (2)-(3): W_o and W_down pruned over their
// in-features; Appendix B gives this sum as the definition of GEMM-K.)  The
// activations of inactive (t, g) blocks are never read.
//
// Two schedules compute it:
//
//  * scatter (the paper's GEMM-K, Appendix B, Algorithm 3): one tile per
//    (group g, 128 sorted positions of g, 128 output columns).  Rows come from
//    the mask reorder, so a tile is fully active, fully inactive (early exit,
//    l = 0) or the group's boundary tile (inactive rows not loaded, l = 1; dead
//    MFMA fragments skipped, l = 2).  Each tile reduces only over its group's
//    G in-features and adds its partial sums into an fp32 buffer with
//    hardware float atomics; a final pass rounds that buffer to bf16.  FLOPs
//    scale with the active fraction, but every active (token, group) pair
//    costs N atomic adds.
//
//  * dense-masked: one tile per (128 tokens in their own order, 128 output
//    columns), reducing over all K.  Inactive (t, g) blocks are replaced by
//    zeros while A is staged into LDS (never loaded), so the result is the
//    same sum; FLOPs are those of the dense product, but there are no atomics
//    and each output is written once, already in bf16.
//
// The host picks the schedule per call (see the dispatch in api.cpp).  Tile
// geometry, LDS swizzle and MFMA layout follow the GEMM-MN kernel: 256
// threads as 2x2 waves, each 64x64 with 32x32x16 bf16 MFMAs, BK = 64,
// double-buffered XOR-swizzled LDS.
#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace wide {

namespace {

constexpr int BM = kKTileM, BN = kKTileN, BK = kKTileK, NT = 256;

__device__ __forceinline__ int swz(int row, int chunk) {
  // 16 lanes of a 128-bit LDS read hit 64 banks together: keep rows r and
  // r + 8 on different chunks (see tile256.h)
  return row * BK + ((chunk ^ ((row & 7) ^ ((row >> 3) & 1))) << 3);
}

__device__ __forceinline__ int xcd_remap(int id, int n) {
  const int q = n / 8, r = n % 8;
  const int xcd = id % 8, local = id / 8;
  return (xcd < r) ? xcd * (q + 1) + local : r * (q + 1) + (xcd - r) * q + local;
}

// One BM x BN tile over the k range [kbeg, kend).  ap[i] are the four A-row
// base pointers of this thread (nullptr: the row is not loaded) and am[i] the
// matching mask rows (nullptr: no per-group masking).
struct TileIO {
  const uint16_t* ap[4];
  const uint8_t* am[4];
  const uint16_t* bp[4];
};

// `tu` (nullable) marks the groups with at least one active token in this
// tile; k steps of the other groups are skipped entirely (no loads, no MFMA).
__device__ __forceinline__ int next_step(int k, int kend, int G, const uint8_t* tu) {
  if (tu) {
    while (k < kend && tu[k / G] == 0) k = (k / G + 1) * G;
  }
  return k < kend ? k : kend;
}

__device__ __forceinline__ void tile_mainloop(uint16_t (*lds)[2][BM * BK], const TileIO& io,
                                              int kbeg, int kend, int G, const uint8_t* tu,
                                              bool live0, bool live1, f32x16 (&acc)[2][2]) {
  const int tid = threadIdx.x;
  const int lrow = tid / 8, lch = tid % 8;
  const int w = wave_id(), lane = lane_id();
  const int wm = w >> 1, wn = w & 1;
  const int l32 = lane & 31, lhi = lane >> 5;
  u32x4 ra[4], rb[4];
  auto gload = [&](int k0) {
    const int g = k0 / G;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const bool on = io.ap[i] && (!io.am[i] || io.am[i][g] != 0);
      ra[i] = on ? ldg16(io.ap[i] + k0) : u32x4{0, 0, 0, 0};
      rb[i] = ldg16(io.bp[i] + k0);
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
  int kc = next_step(kbeg, kend, G, tu);
  if (kc >= kend) return;
  gload(kc);
  lstore(0);
  __syncthreads();
  const int arow0 = wm * 64 + l32, arow1 = arow0 + 32;
  const int brow0 = wn * 64 + l32, brow1 = brow0 + 32;
  for (int buf = 0; kc < kend; buf ^= 1) {
    const int kn = next_step(kc + BK, kend, G, tu);
    if (kn < kend) gload(kn);
    const uint16_t* As = lds[buf][0];
    const uint16_t* Bs = lds[buf][1];
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int ch = kk * 2 + lhi;
      const u32x4 b0 = *reinterpret_cast<const u32x4*>(&Bs[swz(brow0, ch)]);
      const u32x4 b1 = *reinterpret_cast<const u32x4*>(&Bs[swz(brow1, ch)]);
      if (live0) {
        const u32x4 a0 = *reinterpret_cast<const u32x4*>(&As[swz(arow0, ch)]);
        acc[0][0] = mfma32(a0, b0, acc[0][0]);
        acc[0][1] = mfma32(a0, b1, acc[0][1]);
      }
      if (live1) {
        const u32x4 a1 = *reinterpret_cast<const u32x4*>(&As[swz(arow1, ch)]);
        acc[1][0] = mfma32(a1, b0, acc[1][0]);
        acc[1][1] = mfma32(a1, b1, acc[1][1]);
      }
    }
    if (kn < kend) lstore(buf ^ 1);
    __syncthreads();
    kc = kn;
  }
}

}  // namespace

__global__ __launch_bounds__(NT, 2) void wide_gemm_k_dense_masked(KArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[2][2][BM * BK];
  const int n_tiles = a.N / BN;
  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int m_tile = tile / n_tiles, n_tile = tile % n_tiles;
  const int64_t m0 = (int64_t)m_tile * BM;
  const int n0 = n_tile * BN;
  const int n_groups = a.K / a.G;
  const int tid = threadIdx.x, lrow = tid / 8, lch = tid % 8;
  TileIO io;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = lrow + 32 * i;
    const int64_t t = m0 + r;
    io.ap[i] = (t < a.M) ? a.a + t * a.K + lch * 8 : nullptr;
    io.am[i] = (t < a.M) ? a.mask + t * n_groups : nullptr;
    io.bp[i] = a.w + (int64_t)(n0 + r) * a.K + lch * 8;
  }
  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};
  const int wm = wave_id() >> 1;
  const bool live0 = m0 + wm * 64 < a.M, live1 = m0 + wm * 64 + 32 < a.M;
  tile_mainloop(lds, io, 0, a.K, a.G, a.tile_union + m_tile * (int64_t)n_groups, live0, live1, acc);

  const int lane = lane_id(), wn = wave_id() & 1;
  const int l32 = lane & 31, lhi = lane >> 5;
#pragma unroll
  for (int fm = 0; fm < 2; ++fm)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int64_t t = m0 + wm * 64 + fm * 32 + (i >> 2) * 8 + lhi * 4 + (i & 3);
      if (t >= a.M) continue;
      uint16_t* o = a.y + t * a.N + n0 + wn * 64;
      o[l32] = f32_to_bf16(acc[fm][0][i]);
      o[32 + l32] = f32_to_bf16(acc[fm][1][i]);
    }
}

__global__ __launch_bounds__(NT, 2) void wide_gemm_k_scatter(KArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t lds[2][2][BM * BK];
  const int n_tiles = a.N / BN;
  const int m_tiles = (int)((a.M + BM - 1) / BM);
  // tile order: n fastest, then sorted m-tile, then group
  const int tile = xcd_remap(blockIdx.x, gridDim.x);
  const int n_tile = tile % n_tiles;
  const int m_tile = (tile / n_tiles) % m_tiles;
  const int g = tile / (n_tiles * m_tiles);
  const int64_t cnt = a.cnt[g];
  const int64_t m0 = (int64_t)m_tile * BM;
  if (m0 >= cnt) return;  // l = 0: no active token at these positions
  const int n0 = n_tile * BN;
  const int32_t* rows = a.idx + (int64_t)g * a.M;
  const int tid = threadIdx.x, lrow = tid / 8, lch = tid % 8;
  TileIO io;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = lrow + 32 * i;
    const int64_t p = m0 + r;
    io.ap[i] = (p < cnt) ? a.a + (int64_t)rows[p] * a.K + lch * 8 : nullptr;  // l = 1
    io.am[i] = nullptr;  // rows < cnt are active for g by construction
    io.bp[i] = a.w + (int64_t)(n0 + r) * a.K + lch * 8;
  }
  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};
  const int wm = wave_id() >> 1;
  const bool live0 = m0 + wm * 64 < cnt, live1 = m0 + wm * 64 + 32 < cnt;  // l = 2
  tile_mainloop(lds, io, g * a.G, (g + 1) * a.G, a.G, nullptr, live0, live1, acc);

  const int lane = lane_id(), wn = wave_id() & 1;
  const int l32 = lane & 31, lhi = lane >> 5;
#pragma unroll
  for (int fm = 0; fm < 2; ++fm) {
    if (!(fm == 0 ? live0 : live1)) continue;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int64_t p = m0 + wm * 64 + fm * 32 + (i >> 2) * 8 + lhi * 4 + (i & 3);
      if (p >= cnt) continue;
      float* o = a.acc32 + (int64_t)rows[p] * a.N + n0 + wn * 64;
      unsafeAtomicAdd(o + l32, acc[fm][0][i]);
      unsafeAtomicAdd(o + 32 + l32, acc[fm][1][i]);
    }
  }
}

// tu[mt][g] = 1 iff some token of the tile_m-token tile mt is active in group g.
__global__ __launch_bounds__(256) void wide_tile_union(const uint8_t* __restrict__ mask,
                                                       int64_t M, int n_groups, int tile_m,
                                                       uint8_t* __restrict__ tu) {
  const int64_t t0 = (int64_t)blockIdx.x * tile_m;
  const int64_t tn = min((int64_t)tile_m, M - t0);
  for (int g = threadIdx.x; g < n_groups; g += blockDim.x) {
    uint8_t any = 0;
    for (int64_t r = 0; r < tn && !any; ++r) any = mask[(t0 + r) * n_groups + g] != 0;
    tu[blockIdx.x * (int64_t)n_groups + g] = any;
  }
}

hipError_t launch_tile_union(const uint8_t* mask, int64_t M, int n_groups, int tile_m, uint8_t* tu,
                             hipStream_t s) {
  const int64_t m_tiles = (M + tile_m - 1) / tile_m;
  if (m_tiles == 0) return hipSuccess;
  WIDE_LAUNCH(wide_tile_union, dim3((unsigned)m_tiles), dim3(256), 0, s, mask, M, n_groups, tile_m, tu);
  return hipGetLastError();
}

__global__ void wide_zero_f32(float* __restrict__ p, int64_t n) {
  const int64_t n4 = n / 4;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride)
    reinterpret_cast<f32x4*>(p)[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int64_t i = n4 * 4 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
    p[i] = 0.f;
}

__global__ void wide_f32_to_bf16(const float* __restrict__ src, uint16_t* __restrict__ dst,
                                 int64_t n) {
  const int64_t n8 = n / 8;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n8; i += stride) {
    const f32x4 v0 = reinterpret_cast<const f32x4*>(src)[2 * i];
    const f32x4 v1 = reinterpret_cast<const f32x4*>(src)[2 * i + 1];
    u32x4 o;
    o[0] = pack_bf16x2(v0[0], v0[1]);
    o[1] = pack_bf16x2(v0[2], v0[3]);
    o[2] = pack_bf16x2(v1[0], v1[1]);
    o[3] = pack_bf16x2(v1[2], v1[3]);
    reinterpret_cast<u32x4*>(dst)[i] = o;
  }
  for (int64_t i = n8 * 8 + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
    dst[i] = f32_to_bf16(src[i]);
}

static unsigned elementwise_blocks(int64_t n, int per_thread) {
  const int64_t work = (n + per_thread - 1) / per_thread;
  int64_t b = (work + 255) / 256;
  if (b > 256 * 16) b = 256 * 16;
  if (b < 1) b = 1;
  return (unsigned)b;
}

hipError_t launch_gemm_k_dense_masked(const KArgs& a, hipStream_t s) {
  const int64_t m_tiles = (a.M + BM - 1) / BM;
  const int64_t total = m_tiles * (a.N / BN);
  if (total == 0) return hipSuccess;
  hipError_t e = launch_tile_union(a.mask, a.M, a.K / a.G, BM, a.tile_union, s);
  if (e != hipSuccess) return e;
  WIDE_LAUNCH(wide_gemm_k_dense_masked, dim3((unsigned)total), dim3(NT), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gemm_k_scatter(const KArgs& a, hipStream_t s) {
  const int64_t m_tiles = (a.M + BM - 1) / BM;
  const int64_t total = (int64_t)(a.K / a.G) * m_tiles * (a.N / BN);
  if (total == 0) return hipSuccess;
  WIDE_LAUNCH(wide_gemm_k_scatter, dim3((unsigned)total), dim3(NT), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_zero_f32(float* p, int64_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  WIDE_LAUNCH(wide_zero_f32, dim3(elementwise_blocks(n, 4)), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

hipError_t launch_f32_to_bf16(const float* src, uint16_t* dst, int64_t n, hipStream_t s) {
  if (n == 0) return hipSuccess;
  WIDE_LAUNCH(wide_f32_to_bf16, dim3(elementwise_blocks(n, 8)), dim3(256), 0, s, src, dst, n);
  return hipGetLastError();
}

}  // namespace wide
