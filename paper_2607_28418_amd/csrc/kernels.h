// Kernel argument blocks and host launchers of libwide (internal).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <atomic>

namespace wide {

// ---- mask reorder ---------------------------------------------------------
hipError_t launch_reorder(const uint8_t* mask, int64_t M, int n_groups,
                          int32_t* idx, int32_t* counts, int32_t* chunk_cnt,
                          int32_t* chunk_off, hipStream_t s);
size_t reorder_scratch_ints(int64_t M, int n_groups);
// Token order by mask pattern (n_groups <= 8): perm[M] lists the tokens
// grouped by their mask row.  scratch: pattern_scratch_ints(M) ints.
constexpr int kPatternMaxGroups = 8;
size_t pattern_scratch_ints(int64_t M);
hipError_t launch_pattern_order(const uint8_t* mask, int64_t M, int n_groups, int32_t* perm, int32_t* scratch,
                                hipStream_t s);
// out [M][n_groups / r] uint8: 1 where any of r consecutive groups is active.
hipError_t launch_mask_merge(const uint8_t* mask, int64_t M, int n_groups, int r, uint8_t* out, hipStream_t s);
// Groups narrower than this run the K axis on merged blocks of this width.
constexpr int kKMergeWidth = 64;

// ---- prefill N-axis GEMM ---------------------------------------------------
// A region is a run of output tiles sharing one weight (or gate/up pair) and
// one output tensor; Q, K and V of one projection call are three regions.
struct MNRegion {
  const uint16_t* w0;  // weight [N][K] (gate weight in SwiGLU mode)
  const uint16_t* w1;  // up weight in SwiGLU mode, else unused
  uint16_t* out;       // [M][ldo]
  int ldo;             // output row stride in elements
  int n_tiles;         // output tiles in this region
  int masked;          // 1: rows follow idx/cnt of the tile's group; 0: dense
};

struct MNArgs {
  const uint16_t* x;   // [M][K]
  int64_t M;
  int K;
  const int32_t* idx;  // [n_groups][M]
  const int32_t* cnt;  // [n_groups]
  int G;               // group width in output columns
  int m_tiles;
  int n_regions;
  MNRegion reg[3];
};

constexpr int kMNTileM = 128;
constexpr int kMNTileNSwiglu = 64;
constexpr int kMNTileNPlain = 128;
constexpr int kMNTileK = 64;

hipError_t launch_gemm_mn(const MNArgs& a, bool swiglu, hipStream_t s);

// ---- prefill K-axis GEMM ---------------------------------------------------
struct KArgs {
  const uint16_t* a;   // [M][K] activations (H or attention output)
  const uint16_t* w;   // [N][K]
  const uint8_t* mask; // [M][K/G]
  const int32_t* idx;  // [n_groups][M]   (scatter variant)
  const int32_t* cnt;  // [n_groups]      (scatter variant)
  float* acc32;        // [M][N] fp32 accumulation (scatter variant)
  uint16_t* y;         // [M][N] bf16 output (dense-masked variant)
  uint8_t* tile_union; // [ceil(M/128)][K/G] scratch (dense-masked variant)
  const int32_t* perm; // optional [M]: tile rows are tokens perm[m0 + r] (256-tile dense-masked)
  int64_t M;
  int K, N, G;
  int pack;            // 256-tile scatter: K-groups run in turn by one workgroup (>= 1)
};

constexpr int kKTileM = 128;
constexpr int kKTileN = 128;
constexpr int kKTileK = 64;

hipError_t launch_gemm_k_dense_masked(const KArgs& a, hipStream_t s);
inline size_t tile_union_bytes(int64_t M, int n_groups) {
  return (size_t)((M + kKTileM - 1) / kKTileM) * (size_t)n_groups;
}
hipError_t launch_gemm_k_scatter(const KArgs& a, hipStream_t s);
hipError_t launch_tile_union(const uint8_t* mask, int64_t M, int n_groups, int tile_m, uint8_t* tu,
                             hipStream_t s);

// ---- large-tile (256 x 256) prefill kernels ----------------------------------------
// A region of the large-tile GEMM-MN: output columns [0, N) of one tensor cut
// into groups of `gw` columns (gw = G for a masked region, gw = N for a dense
// one); tiles = (N / gw) * m_tiles * (gw / tile_cols).
// masked: 0 dense; 1 (kMN256Sorted) rows of a tile follow the reorder of its
// group (gw = G, a multiple of the tile width); 2 (kMN256TokenOrder) groups
// narrower than a tile: rows in token order, every output (t, n) written
// as the product when group n / mask_G is active for t, else +0 (gw = N, as
// for a dense region).
constexpr int kMN256Sorted = 1, kMN256TokenOrder = 2;
struct MN256Region {
  const uint16_t* w0;
  const uint16_t* w1;
  uint16_t* out;
  int ldo;
  int gw;
  int masked;
  int tiles;
  int skip_zero;  // 1: leave the output blocks of inactive rows unwritten (no reader needs them)
};

struct MN256Args {
  const uint16_t* x;
  int64_t M;
  int K;
  const int32_t* idx;
  const int32_t* cnt;
  int m_tiles;
  int n_regions;
  int order;  // 1: each XCD runs its groups' full tiles, then the partial, then the empty ones
  int mblock; // 1: each XCD runs m-tile 0 of all its groups, then m-tile 1, ... (gate/up)
  int tail;   // 1: split each XCD's last partial round of tiles along k (regions dense or ordered)
  float* tail_ws;  // kMN256TailFloats floats when tail
  const uint8_t* mask;  // [M][mask_ng]: the routing mask (token-order regions only)
  int mask_ng, mask_G;
  MN256Region reg[3];
};
constexpr int kMN256TailJobs = 32;  // tail workgroups per XCD (its CUs)
constexpr int kMN256TailMaxSplit = 8;  // chunks per tail tile at most
constexpr size_t kMN256TailFloats = (size_t)8 * kMN256TailJobs * 256 * 256;
// Host view of the launch condition: every region dense, or masked with the
// ordered tile order (bno: output columns per tile, 128 with SwiGLU else 256).
bool mn256_tail_ok(const MN256Args& a, int bno);

constexpr int kT256 = 256;
hipError_t launch_mn256(const MN256Args& a, bool swiglu, hipStream_t s);
hipError_t launch_kd256(const KArgs& a, hipStream_t s);
hipError_t launch_ks256(const KArgs& a, hipStream_t s);
constexpr int kKd256MaxGroups = 512;
hipError_t launch_zero_f32(float* p, int64_t n, hipStream_t s);
hipError_t launch_f32_to_bf16(const float* src, uint16_t* dst, int64_t n, hipStream_t s);

// ---- decode GEMV ------------------------------------------------------------
struct GVRegion {
  const uint16_t* w0;  // [N][K] (gate in SwiGLU mode)
  const uint16_t* w1;  // up in SwiGLU mode
  uint16_t* out;       // [B][ldo]
  int ldo;
  int n_blocks;        // 16-column blocks in this region
  int masked;
  int col0;            // first column of the region in the concatenated output space
};

struct GVNArgs {
  const uint16_t* x;   // [B][K]
  const uint8_t* mask; // [B][n_groups]
  int B, K, G, n_groups;
  int n_regions;
  GVRegion reg[3];
  int k_split;         // workgroups sharing one column run's k steps
  float* part;         // [k_split][NV][B][total columns] partials when k_split > 1
  int swiglu;          // gate/up pair + SwiGLU (NV = 2) rather than plain columns
};
// Decode N-axis split: enough workgroups to fill the chip (see gemv.hip).
int gemv_n_split(const GVNArgs& a);
size_t gemv_n_part_floats(const GVNArgs& a, bool swiglu);

struct GVKArgs {
  const uint16_t* a;   // [B][K]
  const uint16_t* w;   // [N][K]
  const uint8_t* mask; // [B][K/G]
  uint16_t* y;         // [B][N]
  int B, K, N, G, n_groups;  // G >= 64; n_groups = K / G
  int k_split;         // workgroups sharing one row block's union steps
  float* part;         // [k_split][B][N] partial sums when k_split > 1
  int merge;           // mask columns per group of G (> 1: routing groups of G / merge merged)
};
// Decode K-axis: output rows per workgroup (16 * gemv_k_ncb) and the split of
// the union steps over workgroups (see gemv.hip).
int gemv_k_ncb(int N, int B, int K);
int gemv_k_split(int N, int B, int K);

// Decode tuning overrides, 0 = automatic (wide_set_option keys gemv_n_ncb,
// gemv_n_split, gemv_k_ncb, gemv_k_split).
struct DecodeTuning {
  std::atomic<int> n_ncb, n_split, k_ncb, k_split;
};
DecodeTuning& decode_tuning();

constexpr int kDecodeMaxB = 64;

// ---- bottleneck router (router.hip)
constexpr int kRouterMaxRank = 32;
struct RouterArgs {
  const uint16_t* x;   // [M][D] bf16
  const uint16_t* w1;  // [r][D] bf16 (W1 transposed)
  const uint16_t* w2;  // [2 ng][r] bf16 (W2 transposed)
  uint8_t* mask;       // [M][ng] out
  float* logits;       // optional [M][2 ng] out
  int64_t M;
  int D, r, ng;        // D % 64 == 0, 1 <= r <= 32
};
hipError_t launch_router(const RouterArgs& a, hipStream_t s);

// ---- masked attention, prefill (attention.hip)
constexpr int kAttnHeadDim = 128;
struct AttnArgs {
  const uint16_t* q;        // [n_seq*T_q][n_q*128] bf16
  const uint16_t* k;        // [n_seq*T_k][n_kv*128] bf16
  uint16_t* vt;             // workspace: V^T [n_seq][n_kv][128][T_kp] bf16
  uint16_t* o;              // [n_seq*T_q][n_q*128] bf16 out
  const int32_t* idx;       // [ng][M] reorder of the mask (M = n_seq*T_q)
  const int32_t* cnt;       // [ng]
  const int32_t* seq_off;   // set by launch_attention
  int64_t M;
  int n_seq, T_q, T_k, T_kp;  // T_kp = T_k rounded up to 64
  int n_q, n_kv, ng, hpg, qpk, causal;
  int n_slots;              // set by launch_attention
  float scale_log2;         // log2(e) / sqrt(128)
  // Key-range split (causal, one sequence): null when off.  sched holds
  // attn_sched_ints(split_tiles) ints, part attn_part_floats() floats.
  int32_t* sched;
  float* part;
  int split_tiles;
  const int32_t* leftpad;   // optional [n_seq]: keys j < leftpad[b] of sequence b are hidden (no split then)
  int split_rounds;         // set by launch_attention
};
// The split: a launch whose active query tiles number at most split_tiles
// cuts each tile's causal key range into chunks of equal length (at most
// kAttnMaxChunks per tile, at most kAttnMaxUnits in all, about
// g_attn_split_rounds units per resident workgroup slot; split_tiles is at
// most half of kAttnMaxUnits, which leaves room for the chunks).  sched = {units,
// tiles, chunk length, list[kAttnMaxUnits], (head block << 16 | slot),
// chunks, first unit [split_tiles each]}.
constexpr int kAttnMaxChunks = 8;
constexpr int kAttnMaxUnits = 2048;
constexpr int kAttnMaxSplitTiles = kAttnMaxUnits / 2;
constexpr int kAttnSlots = 512;  // workgroups resident at once: 2 per CU on 256 CUs
constexpr int kAttnMaxSplitHB = 256;
constexpr int kAttnMaxChunkTiles = 1024;
constexpr int kAttnSchedHead = 3;
constexpr int kAttnPartO = 4 * 16 * 64 * 4;  // floats of one unit's O^T partial (4 waves)
inline size_t attn_sched_ints(int split_tiles) {
  return kAttnSchedHead + kAttnMaxUnits + (size_t)split_tiles * 3;
}
inline size_t attn_part_floats() { return (size_t)kAttnMaxUnits * (kAttnPartO + 4 * 64 * 2); }
// Query tiles the split is sized for (0: no split for this shape or option).
int attn_split_tiles(int64_t n_seq, int T_q, int T_k, int n_q, int hpg, int qpk);
// seq_off: workspace of ng*(n_seq+1) ints (used when n_seq > 1).
hipError_t launch_attention(AttnArgs a, const uint16_t* v, int32_t* seq_off, hipStream_t s);
int attn_heads_per_block(int hpg, int qpk);
int attn_slots(int T_q, int hb);
extern std::atomic<int> g_attn_split_rounds;  // units per resident workgroup slot the split aims at (1..8)
extern std::atomic<int> g_attn_split;  // split the causal key ranges when at most this many query tiles exist (0: never)

// ---- masked attention, decode (attention_decode.hip)
struct AttnDecArgs {
  const uint16_t* q;        // [B][n_q*128] bf16, one query token per sequence
  const uint16_t* k;        // bf16 key cache: [B][L][n_kv*128], or [B][n_kv][L][128] if head_major
  const uint16_t* v;        // bf16 value cache, same layout
  uint16_t* o;              // [B][n_q*128] bf16 out
  const uint8_t* mask;      // [B][ng]
  const int32_t* kv_len;    // optional [B]: keys [0, kv_len[b]) are attended (NULL: L)
  float* part;              // workspace [B][n_q][n_chunks][2 + 128]
  int B, L, n_q, n_kv, ng, hpg, qpk;
  int head_major;           // cache layout (see k)
  int chunk, n_chunks;      // keys per workgroup (multiple of 64), ceil(L / chunk)
  float scale_log2;
};
int attn_decode_chunk(int B, int n_kv, int L);
hipError_t launch_attention_decode(AttnDecArgs a, hipStream_t s);

hipError_t launch_gemv_n(const GVNArgs& a, bool swiglu, hipStream_t s);
hipError_t launch_gemv_k(const GVKArgs& a, hipStream_t s);

// ---- fp32 path ---------------------------------------------------------------
struct F32NArgs {
  const float* x; const float* w0; const float* w1; float* out;
  const uint8_t* mask;  // nullptr => dense
  int64_t M; int K, N, ldo, G, n_groups;
};
struct F32KArgs {
  const float* a; const float* w; const uint8_t* mask; float* y;
  int64_t M; int K, N, G, n_groups;
};
hipError_t launch_f32_nproj(const F32NArgs& a, bool swiglu, hipStream_t s);
hipError_t launch_f32_kproj(const F32KArgs& a, hipStream_t s);

}  // namespace wide
