// Mask reordering: per-group stable partition of the routing mask.
//
// WIDE Section 3.3 sorts every routing column of the mask in descending order
// so that a group's active tokens form a contiguous prefix (Appendix B,
// Algorithm 1).  With ties kept in token order this is a stable partition:
// idx[g][0:cnt[g]] = active tokens ascending, idx[g][cnt[g]:M] = the rest.
//
// Three short kernels, all wave64, no host synchronisation:
//   count   one workgroup per chunk of 256 tokens; each wave ballots the
//           active bits of its 64 tokens per group and the chunk's count per
//           group lands in chunk_cnt[chunk][g];
//   scan    one thread per group: exclusive prefix of the chunk counts over
//           chunks (chunk_off[chunk][g]) and the group total (counts[g]);
//   scatter one workgroup per chunk again; ballot + mbcnt give each token its
//           rank among the active (or inactive) tokens of its wave, an LDS
//           exchange of the four wave totals gives the rank inside the chunk,
//           and chunk_off places it in the group's list.
#include "common.h"
#include "launch.h"

namespace wide {

constexpr int kChunk = 256;          // tokens per workgroup (4 waves)
constexpr int kChunkWaves = kChunk / kWave;

__global__ __launch_bounds__(kChunk) void wide_reorder_count(
    const uint8_t* __restrict__ mask, int64_t M, int n_groups,
    int32_t* __restrict__ chunk_cnt) {
  __shared__ int32_t wcnt[kChunkWaves][64];
  const int64_t t = (int64_t)blockIdx.x * kChunk + threadIdx.x;
  const bool in_range = t < M;
  const uint8_t* row = mask + t * n_groups;
  const int w = wave_id();
  for (int g0 = 0; g0 < n_groups; g0 += 64) {
    const int gn = min(64, n_groups - g0);
    for (int j = 0; j < gn; ++j) {
      const bool a = in_range && row[g0 + j] != 0;
      const uint64_t b = __ballot(a);
      if (lane_id() == 0) wcnt[w][j] = __popcll(b);
    }
    __syncthreads();
    if (threadIdx.x < gn) {
      int s = 0;
      for (int i = 0; i < kChunkWaves; ++i) s += wcnt[i][threadIdx.x];
      chunk_cnt[(int64_t)blockIdx.x * n_groups + g0 + threadIdx.x] = s;
    }
    __syncthreads();
  }
}

__global__ __launch_bounds__(256) void wide_reorder_scan(
    const int32_t* __restrict__ chunk_cnt, int n_chunks, int n_groups,
    int32_t* __restrict__ chunk_off, int32_t* __restrict__ counts) {
  const int g = blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= n_groups) return;
  int32_t run = 0;
  for (int c = 0; c < n_chunks; ++c) {
    const int64_t o = (int64_t)c * n_groups + g;
    const int32_t v = chunk_cnt[o];
    chunk_off[o] = run;
    run += v;
  }
  counts[g] = run;
}

__global__ __launch_bounds__(kChunk) void wide_reorder_scatter(
    const uint8_t* __restrict__ mask, int64_t M, int n_groups,
    const int32_t* __restrict__ chunk_off, const int32_t* __restrict__ counts,
    int32_t* __restrict__ idx) {
  __shared__ int32_t wact[2][kChunkWaves];
  const int64_t c0 = (int64_t)blockIdx.x * kChunk;
  const int64_t t = c0 + threadIdx.x;
  const bool in_range = t < M;
  const uint8_t* row = mask + t * n_groups;
  const int w = wave_id();
  const int lane = lane_id();
  const uint64_t below = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  const uint64_t valid_wave = __ballot(in_range);
  for (int g = 0; g < n_groups; ++g) {
    const bool a = in_range && row[g] != 0;
    const uint64_t b = __ballot(a);
    const int buf = g & 1;
    if (lane == 0) wact[buf][w] = __popcll(b);
    __syncthreads();
    int act_before = 0, tok_before = 0;
    for (int i = 0; i < w; ++i) {
      act_before += wact[buf][i];
      tok_before += kWave;
    }
    if (in_range) {
      const int32_t off = chunk_off[blockIdx.x * (int64_t)n_groups + g];
      int32_t* out = idx + (int64_t)g * M;
      const int r_act = __popcll(b & below);
      if (a) {
        out[off + act_before + r_act] = (int32_t)t;
      } else {
        const int r_inact = __popcll(valid_wave & ~b & below);
        const int64_t inact_before_chunk = c0 - off;  // inactive tokens in earlier chunks
        out[counts[g] + inact_before_chunk + (tok_before - act_before) + r_inact] = (int32_t)t;
      }
    }
    // wact[buf] is rewritten two groups later, after the next barrier.
  }
}

// Host-side launcher (called from api.cpp after validation).
hipError_t launch_reorder(const uint8_t* mask, int64_t M, int n_groups,
                          int32_t* idx, int32_t* counts, int32_t* chunk_cnt,
                          int32_t* chunk_off, hipStream_t s) {
  if (M == 0) {
    const int blocks = (n_groups + 255) / 256;
    // counts of an empty column are zero: one scan over zero chunks.
    WIDE_LAUNCH(wide_reorder_scan, dim3(blocks), dim3(256), 0, s,
                chunk_cnt, 0, n_groups, chunk_off, counts);
    return hipGetLastError();
  }
  const int n_chunks = (int)((M + kChunk - 1) / kChunk);
  WIDE_LAUNCH(wide_reorder_count, dim3(n_chunks), dim3(kChunk), 0, s,
              mask, M, n_groups, chunk_cnt);
  WIDE_LAUNCH(wide_reorder_scan, dim3((n_groups + 255) / 256), dim3(256), 0, s,
              chunk_cnt, n_chunks, n_groups, chunk_off, counts);
  WIDE_LAUNCH(wide_reorder_scatter, dim3(n_chunks), dim3(kChunk), 0, s,
              mask, M, n_groups, chunk_off, counts, idx);
  return hipGetLastError();
}

size_t reorder_scratch_ints(int64_t M, int n_groups) {
  const int64_t n_chunks = (M + kChunk - 1) / kChunk;
  return (size_t)(n_chunks * n_groups);
}

}  // namespace wide
