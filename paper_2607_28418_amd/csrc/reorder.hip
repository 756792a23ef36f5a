// Mask reordering: per-group stable partition of the routing mask.
//
// WIDE Section 3.3 sorts every routing column of the mask in descending order
// so that a group's active tokens form a contiguous prefix (Appendix B,
// Algorithm 1).  With ties kept in token order this is a stable partition:
// idx[g][0:cnt[g]] = active tokens ascending, idx[g][cnt[g]:M] = the rest.
//
// Up to 32768 tokens a single kernel does it (wide_reorder_fused, below).
// Beyond, three short kernels, no host synchronisation.  The mask is cut into chunks
// of 64 tokens, one wave each (one token per lane):
//   count    the chunk's mask rows (64 x n_groups bytes, contiguous in
//            memory) are staged in LDS with coalesced loads, in slabs of 512
//            groups; for every group a wave ballot over the 64 tokens gives
//            the chunk's active count, stored transposed as ccnt[g][chunk];
//   scan     one workgroup per group: block-wide exclusive prefix of
//            ccnt[g][:] over chunks (coff[g][chunk]) and the total counts[g];
//   scatter  the chunk's rows are staged again; per group the ballot and
//            mbcnt give each token its rank among the chunk's active (or
//            inactive) tokens, and coff[g][chunk] / counts[g] place it.
#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace wide {

namespace {
constexpr int kChunk = 64;     // tokens per chunk = one wave
constexpr int kSlab = 512;     // groups staged in LDS at a time (32 KB)
constexpr int kScanThreads = 256;

// Stage mask[t0 .. t0+rows)[g0 .. g0+gn) into s[r * gn + j] (bytes).  Whole
// rows are one contiguous run: copied 16 bytes per lane when the run is
// 16-byte aligned, so that many loads are in flight at once.
__device__ __forceinline__ void stage_mask(const uint8_t* __restrict__ mask, int64_t t0, int rows,
                                           int n_groups, int g0, int gn, uint8_t* s) {
  const int n = rows * gn;
  if (gn == n_groups) {
    const uint8_t* src = mask + t0 * n_groups;
    int done = 0;
    if ((reinterpret_cast<uintptr_t>(src) & 15) == 0) {
      const int nv = n / 16;
#pragma unroll 4
      for (int i = threadIdx.x; i < nv; i += kChunk)
        *reinterpret_cast<u32x4*>(s + 16 * i) = ldg16(src + 16 * i);
      done = nv * 16;
    }
    for (int i = done + threadIdx.x; i < n; i += kChunk) s[i] = src[i];
  } else {
#pragma unroll 4
    for (int i = threadIdx.x; i < n; i += kChunk) {
      const int r = i / gn, j = i % gn;
      s[i] = mask[(t0 + r) * n_groups + g0 + j];
    }
  }
}
}  // namespace

__global__ __launch_bounds__(kChunk) void wide_reorder_count(const uint8_t* __restrict__ mask,
                                                             int64_t M, int n_groups, int n_chunks,
                                                             int32_t* __restrict__ ccnt) {
  __shared__ uint8_t s[kChunk * kSlab];
  const int c = blockIdx.x;
  const int64_t t0 = (int64_t)c * kChunk;
  const int rows = (int)min((int64_t)kChunk, M - t0);
  const int lane = threadIdx.x;
  for (int g0 = 0; g0 < n_groups; g0 += kSlab) {
    const int gn = min(kSlab, n_groups - g0);
    stage_mask(mask, t0, rows, n_groups, g0, gn, s);
    __syncthreads();
    for (int j = 0; j < gn; ++j) {
      const bool a = lane < rows && s[lane * gn + j] != 0;
      const uint64_t b = __ballot(a);
      if (lane == 0) ccnt[(int64_t)(g0 + j) * n_chunks + c] = __popcll(b);
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(kScanThreads) void wide_reorder_scan(const int32_t* __restrict__ ccnt,
                                                                  int n_chunks,
                                                                  int32_t* __restrict__ coff,
                                                                  int32_t* __restrict__ counts) {
  __shared__ int32_t wsum[kScanThreads / kWave];
  const int g = blockIdx.x;
  const int32_t* in = ccnt + (int64_t)g * n_chunks;
  int32_t* out = coff + (int64_t)g * n_chunks;
  const int lane = lane_id(), w = wave_id();
  int32_t run = 0;
  for (int base = 0; base < n_chunks; base += kScanThreads) {
    const int c = base + threadIdx.x;
    const int32_t v = c < n_chunks ? in[c] : 0;
    // inclusive scan inside the wave
    int32_t x = v;
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
      const int32_t y = __shfl_up(x, d, kWave);
      if (lane >= d) x += y;
    }
    if (lane == kWave - 1) wsum[w] = x;
    __syncthreads();
    int32_t before = run;
    for (int i = 0; i < w; ++i) before += wsum[i];
    int32_t tile_total = 0;
    for (int i = 0; i < kScanThreads / kWave; ++i) tile_total += wsum[i];
    if (c < n_chunks) out[c] = before + x - v;
    run += tile_total;
    __syncthreads();
  }
  if (threadIdx.x == 0) counts[g] = run;
}

__global__ __launch_bounds__(kChunk) void wide_reorder_scatter(const uint8_t* __restrict__ mask,
                                                               int64_t M, int n_groups,
                                                               int n_chunks,
                                                               const int32_t* __restrict__ coff,
                                                               const int32_t* __restrict__ counts,
                                                               int32_t* __restrict__ idx) {
  __shared__ uint8_t s[kChunk * kSlab];
  __shared__ int32_t s_off[kSlab], s_cnt[kSlab];
  const int c = blockIdx.x;
  const int64_t t0 = (int64_t)c * kChunk;
  const int rows = (int)min((int64_t)kChunk, M - t0);
  const int lane = threadIdx.x;
  const int64_t t = t0 + lane;
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const uint64_t valid = __ballot(lane < rows);
  for (int g0 = 0; g0 < n_groups; g0 += kSlab) {
    const int gn = min(kSlab, n_groups - g0);
    stage_mask(mask, t0, rows, n_groups, g0, gn, s);
    for (int j = lane; j < gn; j += kChunk) {  // independent loads, all in flight
      s_off[j] = coff[(int64_t)(g0 + j) * n_chunks + c];
      s_cnt[j] = counts[g0 + j];
    }
    __syncthreads();
    for (int j = 0; j < gn; ++j) {
      const int g = g0 + j;
      const bool a = lane < rows && s[lane * gn + j] != 0;
      const uint64_t b = __ballot(a);
      if (lane < rows) {
        const int32_t off = s_off[j];  // active tokens in earlier chunks
        int32_t* out = idx + (int64_t)g * M;
        if (a) {
          out[off + __popcll(b & below)] = (int32_t)t;
        } else {
          const int64_t inact_before = t0 - off;  // inactive tokens in earlier chunks
          out[s_cnt[j] + inact_before + __popcll(valid & ~b & below)] = (int32_t)t;
        }
      }
    }
    __syncthreads();
  }
}

// Single-kernel variant for M <= 32768: one workgroup of 1024 threads per
// group.  Thread tid owns tokens i*1024 + tid (i < 32); their mask bytes are
// loaded up front into a bit set, so the only memory latency is one round of
// independent loads.  Ballots give per-(chunk, wave) active counts; one
// block-wide exclusive scan over those (token order = (chunk, wave, lane))
// gives every token its rank among the active tokens, and the inactive
// tokens follow at cnt + (t - active tokens before t).
namespace {
constexpr int kFusedThreads = 1024;
constexpr int kFusedChunks = 32;
constexpr int kFusedWaves = kFusedThreads / kWave;
}  // namespace

__global__ __launch_bounds__(kFusedThreads) void wide_reorder_fused(const uint8_t* __restrict__ mask,
                                                                     int M, int n_groups,
                                                                     int32_t* __restrict__ idx,
                                                                     int32_t* __restrict__ counts) {
  __shared__ int32_t s_cnt[kFusedChunks * kFusedWaves];
  __shared__ int32_t s_wsum[kFusedWaves];
  const int g = blockIdx.x, tid = threadIdx.x;
  const int w = wave_id(), lane = lane_id();
  const int nch = (M + kFusedThreads - 1) / kFusedThreads;
  uint32_t bits = 0;
  for (int i0 = 0; i0 < nch; i0 += 8) {  // eight independent loads per round, no branches
    uint8_t v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int t = (i0 + j) * kFusedThreads + tid;
      v[j] = mask[(t < M ? (int64_t)t * n_groups : 0) + g];
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int t = (i0 + j) * kFusedThreads + tid;
      bits |= (uint32_t)(t < M && v[j] != 0) << (i0 + j);
    }
  }
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int i = 0; i < nch; ++i) {
    const uint64_t b = __ballot((bits >> i) & 1u);
    if (lane == 0) s_cnt[i * kFusedWaves + w] = __popcll(b);
  }
  __syncthreads();
  // exclusive scan of the nch*16 (chunk, wave) counts, in token order
  const int n = nch * kFusedWaves;
  const int32_t v = tid < n ? s_cnt[tid] : 0;
  int32_t x = v;
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    const int32_t y = __shfl_up(x, d, kWave);
    if (lane >= d) x += y;
  }
  if (lane == kWave - 1) s_wsum[w] = x;
  __syncthreads();
  int32_t before = 0, cnt = 0;
  for (int i = 0; i < kFusedWaves; ++i) {
    before += i < w ? s_wsum[i] : 0;
    cnt += s_wsum[i];
  }
  if (tid < n) s_cnt[tid] = before + x - v;
  __syncthreads();
  if (tid == 0) counts[g] = cnt;
  int32_t* out = idx + (int64_t)g * M;
  for (int i = 0; i < nch; ++i) {
    const int t = i * kFusedThreads + tid;
    const bool a = (bits >> i) & 1u;
    const uint64_t b = __ballot(a);
    if (t < M) {
      const int32_t act_before = s_cnt[i * kFusedWaves + w] + __popcll(b & below);
      out[a ? act_before : cnt + (t - act_before)] = t;
    }
  }
}

// Host-side launcher (called from api.cpp after validation).  ccnt and coff
// each hold n_groups * ceil(M / 64) ints (unused by the single-kernel path).
hipError_t launch_reorder(const uint8_t* mask, int64_t M, int n_groups, int32_t* idx,
                          int32_t* counts, int32_t* ccnt, int32_t* coff, hipStream_t s) {
  const int64_t n_chunks64 = (M + kChunk - 1) / kChunk;
  if (n_chunks64 > 0x7fffffff) return hipErrorInvalidValue;
  const int n_chunks = (int)n_chunks64;
  if (M > 0 && M <= (int64_t)kFusedThreads * kFusedChunks) {
    WIDE_LAUNCH(wide_reorder_fused, dim3(n_groups), dim3(kFusedThreads), 0, s, mask, (int)M, n_groups,
                idx, counts);
    return hipGetLastError();
  }
  if (n_chunks > 0)
    WIDE_LAUNCH(wide_reorder_count, dim3(n_chunks), dim3(kChunk), 0, s, mask, M, n_groups,
                n_chunks, ccnt);
  WIDE_LAUNCH(wide_reorder_scan, dim3(n_groups), dim3(kScanThreads), 0, s, ccnt, n_chunks, coff,
              counts);
  if (n_chunks > 0)
    WIDE_LAUNCH(wide_reorder_scatter, dim3(n_chunks), dim3(kChunk), 0, s, mask, M, n_groups,
                n_chunks, coff, counts, idx);
  return hipGetLastError();
}

// ---- token order by mask pattern ---------------------------------------------
//
// For a K-axis projection with few groups (attention's head groups), tokens
// that share a mask row share their set of active groups.  Ordering the
// tokens by that row makes the rows of one 256-row tile share most of their
// groups, so the dense-masked K-axis kernel can skip the k steps of every
// group none of the tile's rows uses.  The sort key is the row's rank in the
// reflected binary Gray code (the row's bits, read as a Gray codeword, decoded
// to binary): neighbouring patterns then differ in one group, and a tile that
// straddles several of them spans fewer groups than in plain binary order
// (for 4 of 8 groups per token, 5.75 instead of 6.2 of 8 on average).
// Any order within a pattern is fine (each output row's sum is the same: a
// skipped group only ever adds exact zeros), so the scatter takes positions
// inside a chunk with LDS atomics.  Three short kernels: per-chunk pattern
// histograms, one exclusive scan over (pattern, chunk), the scatter.
namespace {
constexpr int kPatChunk = 1024;  // tokens per workgroup
constexpr int kPatMaxGroups = 8;
constexpr int kPatKeys = 1 << kPatMaxGroups;

__device__ __forceinline__ int pattern_of(const uint8_t* mask, int64_t t, int ng) {
  int key = 0;
  for (int g = 0; g < ng; ++g) key |= (mask[t * ng + g] != 0) << g;
  key ^= key >> 1;  // Gray decode of an 8-bit word: prefix XOR from the top bit down
  key ^= key >> 2;
  key ^= key >> 4;
  return key;
}

__global__ __launch_bounds__(kPatChunk) void wide_pattern_count(const uint8_t* mask, int64_t M, int ng,
                                                                int n_chunks, int32_t* hist) {
  __shared__ int h[kPatKeys];
  const int tid = threadIdx.x;
  for (int i = tid; i < kPatKeys; i += kPatChunk) h[i] = 0;
  __syncthreads();
  const int64_t t = (int64_t)blockIdx.x * kPatChunk + tid;
  if (t < M) atomicAdd(&h[pattern_of(mask, t, ng)], 1);
  __syncthreads();
  for (int i = tid; i < kPatKeys; i += kPatChunk) hist[(int64_t)i * n_chunks + blockIdx.x] = h[i];
}

// hist [key][chunk] -> exclusive prefix in (key, chunk) order, in place.
__global__ __launch_bounds__(1024) void wide_pattern_scan(int32_t* hist, int n) {
  __shared__ int64_t part[1024];
  const int tid = threadIdx.x;
  const int per = (n + 1023) / 1024;
  const int b = tid * per, e = min(n, b + per);
  int64_t s = 0;
  for (int i = b; i < e; ++i) s += hist[i];
  part[tid] = s;
  __syncthreads();
  for (int o = 1; o < 1024; o <<= 1) {  // inclusive scan of the thread sums
    const int64_t v = tid >= o ? part[tid - o] : 0;
    __syncthreads();
    part[tid] += v;
    __syncthreads();
  }
  int64_t run = tid ? part[tid - 1] : 0;
  for (int i = b; i < e; ++i) {
    const int c = hist[i];
    hist[i] = (int32_t)run;
    run += c;
  }
}

__global__ __launch_bounds__(kPatChunk) void wide_pattern_scatter(const uint8_t* mask, int64_t M, int ng,
                                                                  int n_chunks, const int32_t* off,
                                                                  int32_t* perm) {
  __shared__ int cur[kPatKeys];
  const int tid = threadIdx.x;
  for (int i = tid; i < kPatKeys; i += kPatChunk) cur[i] = off[(int64_t)i * n_chunks + blockIdx.x];
  __syncthreads();
  const int64_t t = (int64_t)blockIdx.x * kPatChunk + tid;
  if (t < M) perm[atomicAdd(&cur[pattern_of(mask, t, ng)], 1)] = (int32_t)t;
}
// Up to kPatFusedMax tokens: one workgroup does all three passes (histogram,
// scan and scatter through LDS), saving two launches.  Each token's key is
// computed once (from one 8-byte load when the mask has 8 groups) and kept
// in LDS for the scatter; the loads of a thread's tokens go out together.
constexpr int kPatFusedMax = 32768;
static_assert(kPatKeys == 256, "the fused scan gives each of 64 lanes four keys");
__device__ __forceinline__ int pattern_key8(const uint8_t* mask, int64_t t) {
  const uint2 w = *reinterpret_cast<const uint2*>(mask + t * 8);
  int key = 0;
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    key |= (((w.x >> (8 * b)) & 0xffu) != 0) << b;
    key |= (((w.y >> (8 * b)) & 0xffu) != 0) << (4 + b);
  }
  key ^= key >> 1;  // Gray decode, as in pattern_of
  key ^= key >> 2;
  key ^= key >> 4;
  return key;
}
__global__ __launch_bounds__(1024) void wide_pattern_fused(const uint8_t* mask, int M, int ng, int32_t* perm) {
  __shared__ int cnt[kPatKeys];
  __shared__ uint8_t keys[kPatFusedMax];
  const int tid = threadIdx.x;
  for (int i = tid; i < kPatKeys; i += 1024) cnt[i] = 0;
  __syncthreads();
#pragma unroll 8
  for (int k = 0; k < kPatFusedMax / 1024; ++k) {
    const int t = tid + k * 1024;
    if (t < M) {
      const int key = ng == 8 ? pattern_key8(mask, t) : pattern_of(mask, t, ng);
      keys[t] = (uint8_t)key;
      atomicAdd(&cnt[key], 1);
    }
  }
  __syncthreads();
  if (tid < 64) {  // exclusive scan of the 256 counts by one wave, four per lane
    int v[4], sum = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[i] = cnt[tid * 4 + i];
      sum += v[i];
    }
    int incl = sum;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int y = __shfl_up(incl, o, 64);
      if (tid >= o) incl += y;
    }
    int run = incl - sum;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      cnt[tid * 4 + i] = run;
      run += v[i];
    }
  }
  __syncthreads();
#pragma unroll 8
  for (int k = 0; k < kPatFusedMax / 1024; ++k) {
    const int t = tid + k * 1024;
    if (t < M) perm[atomicAdd(&cnt[keys[t]], 1)] = t;
  }
}
}  // namespace

size_t pattern_scratch_ints(int64_t M) { return (size_t)kPatKeys * (size_t)((M + kPatChunk - 1) / kPatChunk); }

hipError_t launch_pattern_order(const uint8_t* mask, int64_t M, int n_groups, int32_t* perm, int32_t* scratch,
                                hipStream_t s) {
  if (M == 0) return hipSuccess;
  if (n_groups > kPatMaxGroups) return hipErrorInvalidValue;
  const int64_t nc64 = (M + kPatChunk - 1) / kPatChunk;
  if (nc64 * kPatKeys > 0x7fffffff) return hipErrorInvalidValue;
  const int nc = (int)nc64;
  if (M <= kPatFusedMax) {
    WIDE_LAUNCH(wide_pattern_fused, dim3(1), dim3(1024), 0, s, mask, (int)M, n_groups, perm);
    return hipGetLastError();
  }
  WIDE_LAUNCH(wide_pattern_count, dim3(nc), dim3(kPatChunk), 0, s, mask, M, n_groups, nc, scratch);
  WIDE_LAUNCH(wide_pattern_scan, dim3(1), dim3(1024), 0, s, scratch, nc * kPatKeys);
  WIDE_LAUNCH(wide_pattern_scatter, dim3(nc), dim3(kPatChunk), 0, s, mask, M, n_groups, nc, scratch, perm);
  return hipGetLastError();
}

size_t reorder_scratch_ints(int64_t M, int n_groups) {
  const int64_t n_chunks = (M + kChunk - 1) / kChunk;
  return (size_t)(n_chunks * n_groups);
}

// Routing columns merged r at a time: out[t][b] = 1 when any of groups
// [b r, (b+1) r) is active for token t, else 0.  The K axis of groups
// narrower than its 64-wide k step works on these blocks (the inactive
// groups inside an active block hold exact zeros in H).
__global__ __launch_bounds__(256) void wide_mask_merge(const uint8_t* __restrict__ mask, int64_t M, int ng, int r,
                                                       uint8_t* __restrict__ out) {
  const int nb = ng / r;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= M * nb) return;
  const int64_t t = i / nb;
  const int b = (int)(i % nb);
  const uint8_t* p = mask + t * ng + (int64_t)b * r;
  int on = 0;
  for (int j = 0; j < r; ++j) on |= p[j];
  out[i] = on != 0;
}

hipError_t launch_mask_merge(const uint8_t* mask, int64_t M, int n_groups, int r, uint8_t* out, hipStream_t s) {
  const int64_t n = M * (n_groups / r);
  if (n == 0) return hipSuccess;
  WIDE_LAUNCH(wide_mask_merge, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, mask, M, n_groups, r, out);
  return hipGetLastError();
}

}  // namespace wide
