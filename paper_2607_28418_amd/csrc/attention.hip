// Head-group masked attention at prefill on gfx950 (WIDE Section 3.1,
// equations (1)-(2); Appendix B, Algorithm 4).
//
// An active (token, head group) gets standard scaled dot-product attention
// over the keys of its sequence (with causal masking, the keys up to its own
// position, queries being the last T_q of T_k positions); an inactive one
// outputs +0.  The mask reorder of the projections is reused: idx[g] lists
// group g's active tokens in ascending order, so one sequence's active rows
// are a contiguous run of it, and query tiles are cut from that run (rows of
// one tile are active by construction, the paper's s^(1) gather).
//
// Work split: one workgroup of four waves per (query tile, head block).  A
// head block is HB query heads of one group that read one KV head (HB = 4 for
// Llama-3-8B, where a group is exactly the four heads of a KV head); the four
// waves are HB heads x (4/HB) blocks of 32 rows, so K/V tiles loaded once
// into LDS serve all of them.  Per wave and key tile (64 keys):
//   S^T[keys][queries] = K Q^T     16 MFMA 32x32x16 (A = K from LDS, B = Q^T
//                                  held in registers for the whole loop)
//   online softmax per query lane  (a query's 64 scores sit in lanes l and
//                                  l^32, so the row max is one swap)
//   O^T[d][queries] += V^T P^T     16 MFMA (A = V^T from LDS, B = P^T from
//                                  the S^T registers, rounded to bf16)
// Keeping the transposed products puts every per-query quantity (running
// max, sum, rescale factor) in one lane.  The A operand of the first product
// loads its 32 key rows in a permuted order chosen so that each lane's S^T
// registers hold 8 consecutive keys per 16-key step, which is exactly the k
// layout the second product's B operand needs; V therefore only has to be
// transposed (by the prep kernel below, into the workspace), not permuted.
//
// Skipping, following Algorithm 4: tiles past a sequence's active count
// exit (l = 0) after clearing their share of the inactive rows; the causal
// key range of a tile stops at its last row's position (rows are sorted);
// a wave whose rows see none of a key tile issues no MFMA for it (l = 2);
// only key tiles crossing a row's causal limit evaluate the per-element
// mask.  With left padding (Algorithm 4's first key leftpad(b)) a tile's key
// range starts at the tile holding key leftpad(b), that tile masks the keys
// before it, and a query that sees no key at all stores +0.
#include "common.h"
#include "kernels.h"
#include "launch.h"
#include "tile256.h"

namespace wide {

std::atomic<int> g_attn_split_rounds{1};
std::atomic<int> g_attn_split{1024};  // key-range split when at most this many query tiles are active (0: never)

namespace {

__host__ __device__ inline int attn_hb_of(int hpg, int qpk) {
  if (hpg % 4 == 0 && qpk % 4 == 0) return 4;
  if (hpg % 2 == 0 && qpk % 2 == 0) return 2;
  return 1;
}

using t256::gptr_t;
using t256::lptr_t;

constexpr int kHd = 128;               // head dimension
constexpr int kBN = 64;                // keys per tile
constexpr int kAT = 256;               // threads per workgroup (4 waves)
constexpr int kKSub = 64 * 64;         // one K half-tile [64 keys][64 dims]
constexpr int kVt = kHd * kBN;         // V^T tile [128 dims][64 keys]

// LDS rows are 64 bf16 = 8 chunks of 16 bytes; logical chunk c of row r sits
// at physical chunk c ^ f(r), which spreads the 16 rows that one 16-lane
// phase of a 128-bit read touches over distinct bank groups.
__device__ __forceinline__ int swz_f(int r) { return (r & 7) ^ ((r >> 3) & 1); }
__device__ __forceinline__ int swz(int r, int c) { return r * 64 + ((c ^ swz_f(r)) << 3); }

__device__ __forceinline__ u32x4 lds16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// HB: query heads per workgroup (sharing one KV head); QB: 32-query blocks
// per wave.  The launcher instantiates QB = 1: with QB = 2 every K / V^T
// fragment read from LDS feeds two MFMAs (one per query block), halving the
// LDS reads per MFMA, but at one wave per SIMD it ran slower on MI355X.
template <int HB, int QB>
__global__ __launch_bounds__(kAT, QB == 1 ? 2 : 1) void wide_attn_fwd(AttnArgs a) {
  constexpr int RB = 4 / HB;         // row blocks (of 32*QB rows) per workgroup
  constexpr int WR = 32 * QB;        // query rows per wave
  constexpr int BMW = WR * RB;       // query rows per workgroup
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * (2 * kKSub + kVt)];  // 64 KB

  const int per_hb = a.n_seq * a.n_slots;
  const int n_classic = a.n_q / HB * per_hb;
  const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
  const int64_t ldq = (int64_t)a.n_q * kHd;
  const int64_t M = a.M;
  int hbk, b, slot;
  auto classic = [&](int lid) {
    hbk = lid / per_hb;
    const int rem = lid - hbk * per_hb;
    b = rem / a.n_slots;
    slot = a.n_slots - 1 - (rem - b * a.n_slots);  // long key ranges first
  };
  auto rows_of = [&](int hk, int bb, int& s0, int& s1) {  // active run of (sequence bb, group of hk)
    const int gg = hk * HB / a.hpg;
    s0 = 0;
    s1 = a.cnt[gg];
    if (a.seq_off) {
      s0 = a.seq_off[gg * (a.n_seq + 1) + bb];
      s1 = a.seq_off[gg * (a.n_seq + 1) + bb + 1];
    }
  };

  // Inactive rows of a sequence sit at idx_g[cnt_g + (b*T_q - s0) ...]; slot
  // i of the classic mapping clears rows [i*BMW, (i+1)*BMW) of that run for
  // its HB heads.
  if ((int)blockIdx.x < n_classic) {
    classic(t256::xcd_remap(blockIdx.x, n_classic));
    constexpr int CPR = HB * kHd / 8;  // 16-byte chunks per row
    int s0, s1;
    rows_of(hbk, b, s0, s1);
    const int gg = hbk * HB / a.hpg;
    const int64_t ib = (int64_t)a.cnt[gg] + ((int64_t)b * a.T_q - s0);
    const int r0 = slot * BMW, r1 = min(a.T_q - (s1 - s0), r0 + BMW);
    const int32_t* ig = a.idx + (int64_t)gg * M;
    for (int i = tid; i < (r1 - r0) * CPR; i += kAT) {
      const int64_t t = ig[ib + r0 + i / CPR];
      stg16(a.o + t * ldq + (int64_t)(hbk * HB) * kHd + (i % CPR) * 8, u32x4{0, 0, 0, 0});
    }
  }
  // The work unit: the classic (head block, sequence, slot), or, when the
  // schedule pass split the key ranges, entry blockIdx.x of its list (a
  // tile's key chunk; longest chunks first).
  int chunk = 0, n_chunk = 1, part_unit = 0, chunk_tiles = 0;
  if (QB == 1 && a.sched && a.sched[0] > 0) {
    if ((int)blockIdx.x >= a.sched[0]) return;
    const int e = a.sched[kAttnSchedHead + blockIdx.x];
    const int rank = e / kAttnMaxChunks;
    chunk = e - rank * kAttnMaxChunks;
    const int32_t* tab = a.sched + kAttnSchedHead + kAttnMaxUnits;
    hbk = tab[rank] >> 16;
    slot = tab[rank] & 0xffff;
    b = 0;
    n_chunk = tab[a.split_tiles + rank];
    part_unit = tab[2 * a.split_tiles + rank] + chunk;
    chunk_tiles = a.sched[2];
  } else {
    if ((int)blockIdx.x >= n_classic) return;
    classic(t256::xcd_remap(blockIdx.x, n_classic));
  }
  const int h0 = hbk * HB;
  const int g = h0 / a.hpg, hkv = h0 / a.qpk;
  const int32_t* idx_g = a.idx + (int64_t)g * M;
  int s0, s1;
  rows_of(hbk, b, s0, s1);
  const int c = s1 - s0;  // active rows of (sequence b, group g)
  const int64_t seq0 = (int64_t)b * a.T_q;
  const int m0 = slot * BMW;
  if (m0 >= c) return;  // l = 0: no active row in this tile

  const int delta = a.T_k - a.T_q;
  auto limit_of = [&](int64_t t) {  // last visible key of token t
    return a.causal ? (int)(t - seq0) + delta : a.T_k - 1;
  };
  const int rb = w / HB, h = h0 + (w - rb * HB);
  const int wr0 = m0 + rb * WR;
  const bool wave_live = wr0 < c;
  const int wr1 = min(c, wr0 + WR);
  const int l32 = lane & 31, hi = lane >> 5;
  bool valid[QB];
  int64_t t[QB];
  int plim[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int myr = wr0 + 32 * qb + l32;
    valid[qb] = myr < c;
    t[qb] = valid[qb] ? (int64_t)idx_g[s0 + myr] : 0;
    plim[qb] = valid[qb] ? limit_of(t[qb]) : -1;
  }
  // rows ascend by position, so the first and last rows bound the limits
  const int wmin = wave_live ? limit_of(idx_g[s0 + wr0]) : -1;
  const int wmax = wave_live ? limit_of(idx_g[s0 + wr1 - 1]) : -1;
  const int gmax = limit_of(idx_g[s0 + min(c, m0 + BMW) - 1]);
  // First visible key of the sequence (left padding; clamped into [0, T_k]).
  const int lp = a.leftpad ? min(max(a.leftpad[b], 0), a.T_k) : 0;
  // This unit's key tiles [jlo, jhi): the tile's whole causal range (from
  // the tile of the first visible key), or one chunk of it.
  const int jlo = n_chunk > 1 ? chunk * chunk_tiles : lp / kBN;
  const int n_tiles = n_chunk > 1 ? min((gmax + kBN) / kBN, jlo + chunk_tiles) : (gmax + kBN) / kBN;

  // Q^T fragments (B operand): d-step s holds dims 16s + 8*hi .. +8 of the row.
  u32x4 qf[QB][8];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const uint16_t* qrow = a.q + t[qb] * ldq + (int64_t)h * kHd + hi * 8;
#pragma unroll
    for (int s = 0; s < 8; ++s) qf[qb][s] = valid[qb] ? ldg16(qrow + 16 * s) : u32x4{0, 0, 0, 0};
  }

  // Loads: a K tile and a V^T tile are 16 instructions of 1 KB (8 LDS rows
  // each).  Waves 0-1 load K (dims 0-63 / 64-127), waves 2-3 the 128 rows of
  // V^T; each ring has two stages.  A lane keeps a 32-bit byte offset per
  // instruction from a per-tile uniform base.
  const int64_t ldk = (int64_t)a.n_kv * kHd;
  const bool kwave = w < 2;
  const char* kb0 = reinterpret_cast<const char*>(a.k + (int64_t)b * a.T_k * ldk + hkv * kHd + (w & 1) * 64);
  const char* vb0 = reinterpret_cast<const char*>(a.vt + ((int64_t)b * a.n_kv + hkv) * kHd * (int64_t)a.T_kp);
  uint32_t off[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    const int r = kwave ? q * 8 + lane / 8 : (w - 2) * 64 + q * 8 + lane / 8;
    const int lc = (lane & 7) ^ swz_f(r);
    off[q] = kwave ? (uint32_t)((r * ldk + lc * 8) * 2) : (uint32_t)(((int64_t)r * a.T_kp + lc * 8) * 2);
  }
  uint16_t* const kst = smem;                 // K ring: 2 x [2 halves][64 keys][64 dims]
  uint16_t* const vst = smem + 2 * 2 * kKSub;  // V^T ring: 2 x [128 dims][64 keys]
  auto issue_k = [&](int jt) {  // waves 0-1
    const int j0 = jt * kBN;
    uint16_t* dst = kst + (jt & 1) * 2 * kKSub + w * kKSub;
    const char* base = kb0 + (int64_t)j0 * ldk * 2;
    if (j0 + kBN <= a.T_k) {
#pragma unroll
      for (int q = 0; q < 8; ++q)
        __builtin_amdgcn_global_load_lds((gptr_t)(base + off[q]), (lptr_t)(dst + q * 8 * 64), 16, 0, 0);
    } else {  // last, partial tile: rows past the end re-read the last key (finite, masked)
      const int kmax = a.T_k - 1 - j0;
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        const int r = q * 8 + lane / 8;
        const int lc = (lane & 7) ^ swz_f(r);
        const uint32_t o = (uint32_t)((min(r, kmax) * ldk + lc * 8) * 2);
        __builtin_amdgcn_global_load_lds((gptr_t)(base + o), (lptr_t)(dst + q * 8 * 64), 16, 0, 0);
      }
    }
  };
  auto issue_v = [&](int jt) {  // waves 2-3
    uint16_t* dst = vst + (jt & 1) * kVt + (w - 2) * 64 * 64;
    const char* base = vb0 + (int64_t)jt * kBN * 2;
#pragma unroll
    for (int q = 0; q < 8; ++q)
      __builtin_amdgcn_global_load_lds((gptr_t)(base + off[q]), (lptr_t)(dst + q * 8 * 64), 16, 0, 0);
  };

  // K rows in the A operand: lane row x = 8j + 4h' + i loads key
  // 16(j/2) + 8h' + 4(j%2) + i, so S^T register r of lane half hi holds key
  // 16(r/8) + 8*hi + r%8 of its 32-key block.
  const int pi = 16 * (l32 >> 4) + 8 * ((l32 >> 2) & 1) + 4 * ((l32 >> 3) & 1) + (l32 & 3);

  f32x16 O[QB][4];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int i = 0; i < 4; ++i) O[qb][i] = f32x16{};
  float m[QB], z[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m[qb] = -INFINITY;
    z[qb] = 0.0f;
  }
  const float sc = a.scale_log2;

  // S^T of key tile jt for this wave's queries (two 32-key blocks each).
  auto qk = [&](int jt, f32x16 (&S)[QB][2]) {
    const uint16_t* st = kst + (jt & 1) * 2 * kKSub;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      S[qb][0] = f32x16{};
      S[qb][1] = f32x16{};
    }
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const uint16_t* ks = st + (s >> 2) * kKSub;
      const int ch = 2 * (s & 3) + hi;
      const u32x4 k0 = lds16(ks + swz(pi, ch));
      const u32x4 k1 = lds16(ks + swz(32 + pi, ch));
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        S[qb][0] = mfma32(k0, qf[qb][s], S[qb][0]);
        S[qb][1] = mfma32(k1, qf[qb][s], S[qb][1]);
      }
    }
  };
  // Online softmax of tile jt's scores per query block (masking and the new
  // row maximum, then the exponentials and the rescale) and O^T += V^T P^T.
  auto softmax_pv = [&](int jt, f32x16 (&S)[QB][2]) {
    const int j0 = jt * kBN;
    // Per-element mask only where the tile crosses some row's limit or holds
    // the first visible key; every other tile is fully visible to the wave.
    if (j0 + kBN - 1 > wmin || j0 < lp) {
      const int lo = lp - j0 - 8 * hi;  // key offsets below this are padding
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const int lim = plim[qb] - j0 - 8 * hi;  // key offset past which this row sees nothing
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int ko = 32 * kb + 16 * (r >> 3) + (r & 7);
            S[qb][kb][r] = ko > lim || ko < lo ? -INFINITY : S[qb][kb][r];
          }
      }
    }
    float alpha[QB];
    bool moved = false;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, S[qb][kb][r]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float mnew = fmaxf(m[qb], mx * sc);
      const float muse = mnew == -INFINITY ? 0.0f : mnew;  // a row with nothing visible yet
      alpha[qb] = fast_exp2(m[qb] - muse);
      m[qb] = mnew;
      moved = moved || alpha[qb] != 1.0f;
      float zs = 0.0f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = fast_exp2(fmaf(S[qb][kb][r], sc, -muse));
          S[qb][kb][r] = p;
          zs += p;
        }
      }
      z[qb] = z[qb] * alpha[qb] + zs;
    }
    if (__any(moved)) {  // lazy rescale: skipped once the maxima settle
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int db = 0; db < 4; ++db) O[qb][db] *= alpha[qb];
    }
    const uint16_t* vts = vst + (jt & 1) * kVt;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int p = 0; p < 2; ++p) {
        u32x4 pf[QB];
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
          for (int e = 0; e < 4; ++e)
            pf[qb][e] = pack_bf16x2_hw(S[qb][kb][8 * p + 2 * e], S[qb][kb][8 * p + 2 * e + 1]);
        const int ch = 4 * kb + 2 * p + hi;
#pragma unroll
        for (int db = 0; db < 4; ++db) {
          const u32x4 vf = lds16(vts + swz(32 * db + l32, ch));
#pragma unroll
          for (int qb = 0; qb < QB; ++qb) O[qb][db] = mfma32(vf, pf[qb], O[qb][db]);
        }
      }
    }
  };

  // Key tiles this wave sees at all (a prefix of the workgroup's range).
  const int wtiles = wave_live ? min(n_tiles, (wmax + kBN) / kBN) : 0;
  // Pipeline: iteration jt loads K of tile jt+2 and V of tile jt+1, computes
  // the scores of tile jt+1 and then the softmax and P.V of tile jt, so the
  // matrix core has independent work while the softmax runs.  Everything
  // issued in one iteration lands before the next one starts.
  if (jlo >= n_tiles) {
    // left padding hides every key of this tile's rows: nothing to stream
  } else if constexpr (QB == 1) {
    if (kwave) {
      issue_k(jlo);
      if (jlo + 1 < n_tiles) issue_k(jlo + 1);
    } else {
      issue_v(jlo);
    }
    t256::wait_vm<0>();
    t256::stage_barrier();
    f32x16 Sa[QB][2], Sb[QB][2];
    if (jlo < wtiles) qk(jlo, Sa);
    auto step = [&](int jt, f32x16 (&Sc)[QB][2], f32x16 (&Sn)[QB][2]) {
      t256::wait_vm<0>();
      t256::stage_barrier();
      if (kwave) {
        if (jt + 2 < n_tiles) issue_k(jt + 2);
      } else {
        if (jt + 1 < n_tiles) issue_v(jt + 1);
      }
      if (jt + 1 < wtiles) qk(jt + 1, Sn);
      if (jt < wtiles) softmax_pv(jt, Sc);  // l = 2: tiles past the wave's rows issue no MFMA
    };
    for (int jt = jlo; jt < n_tiles; jt += 2) {
      step(jt, Sa, Sb);
      if (jt + 1 < n_tiles) step(jt + 1, Sb, Sa);
    }
  } else {
    // Two query blocks already give the matrix core independent work, and
    // the registers for a second score tile are not there: scores of tile jt
    // are computed in its own step.
    // Both rings run one tile ahead: iteration jt loads K and V of tile jt+1
    // into the stages tile jt-1 used.
    f32x16 S[QB][2];
    if (kwave) issue_k(jlo);
    else issue_v(jlo);
    for (int jt = jlo; jt < n_tiles; ++jt) {
      t256::wait_vm<0>();
      t256::stage_barrier();
      if (jt + 1 < n_tiles) {
        if (kwave) issue_k(jt + 1);
        else issue_v(jt + 1);
      }
      if (jt < wtiles) {  // l = 2: tiles past the wave's rows issue no MFMA
        qk(jt, S);
        softmax_pv(jt, S);
      }
    }
  }

  if (QB == 1 && n_chunk > 1) {
    // One chunk of a split key range: the unnormalised O^T registers, the
    // running maximum and this lane half's sum go to the unit's partial
    // slot, lane-major so that every store of the wave is 1 KB contiguous;
    // wide_attn_merge combines the chunks.
    float4* po = reinterpret_cast<float4*>(a.part) + ((int64_t)part_unit * 4 + w) * (QB * 16 * kWave);
    float2* pm = reinterpret_cast<float2*>(a.part + (int64_t)kAttnMaxUnits * kAttnPartO) +
                 ((int64_t)part_unit * 4 + w) * (QB * kWave);
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      pm[qb * kWave + lane] = make_float2(m[qb], z[qb]);
#pragma unroll
      for (int db = 0; db < 4; ++db)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          po[((qb * 4 + db) * 4 + j) * kWave + lane] =
              make_float4(O[qb][db][4 * j], O[qb][db][4 * j + 1], O[qb][db][4 * j + 2], O[qb][db][4 * j + 3]);
    }
    return;
  }
  // Epilogue: the two halves of a query's sum, normalise, scatter the row.
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const float zt = z[qb] + __shfl_xor(z[qb], 32);
    if (!valid[qb]) continue;
    const float inv = zt > 0.0f ? 1.0f / zt : 0.0f;  // no visible key (left padding): +0
    uint16_t* orow = a.o + t[qb] * ldq + (int64_t)h * kHd + 4 * hi;
#pragma unroll
    for (int db = 0; db < 4; ++db) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        uint2 v;
        v.x = pack_bf16x2_hw(O[qb][db][4 * j] * inv, O[qb][db][4 * j + 1] * inv);
        v.y = pack_bf16x2_hw(O[qb][db][4 * j + 2] * inv, O[qb][db][4 * j + 3] * inv);
        *reinterpret_cast<uint2*>(orow + 32 * db + 8 * j) = v;
      }
    }
  }
}

// Exclusive prefix sum, in place, of n <= 16 * 64 LDS values taken in the
// order v[0], v[1], ... (or v[top], v[top - 1], ... when rev), by one wave;
// returns the total.
__device__ int wave_exscan(int* v, int n, bool rev, int top) {
  const int lane = lane_id();
  int x[16], s = 0;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const int i = lane * 16 + k;
    x[k] = i < n ? v[rev ? top - i : i] : 0;
    s += x[k];
  }
  int inc = s;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int y = __shfl_up(inc, o, kWave);
    if (lane >= o) inc += y;
  }
  int ex = inc - s;
#pragma unroll
  for (int k = 0; k < 16; ++k) {
    const int i = lane * 16 + k;
    if (i < n) v[rev ? top - i : i] = ex;
    ex += x[k];
  }
  return __shfl(inc, kWave - 1, kWave);
}

// Schedule of the key-range split (one workgroup; causal, one sequence).
// The active query tiles are numbered head block by head block.  With W key
// tiles of work over all of them, the chunk length is the smallest that
// keeps a tile to kAttnMaxChunks chunks and the launch to kAttnMaxUnits
// units, and at least W / (split_rounds * kAttnSlots), so that each resident
// workgroup slot runs about split_rounds units; at most the key tiles of the
// whole range (no tile spans more).  A tile whose causal range
// spans nt key tiles becomes ceil(nt / chunk) units (one, written straight
// to the output, when nt <= chunk), listed by their number of key tiles,
// largest first, so that the dispatcher hands out the long ones while every
// CU is still busy.  More active tiles than split_tiles: no split (units = 0).
__device__ void attn_schedule(const AttnArgs& a, int hb, int bmw) {
  __shared__ int tpre[kAttnMaxSplitHB + 1];
  __shared__ int hist[kAttnMaxChunkTiles + 1];
  __shared__ int nt_of[kAttnMaxSplitTiles];
  __shared__ int tsum[kAT];
  __shared__ int work, chl, n_units;
  const int tid = threadIdx.x, n_hb = a.n_q / hb;
  int32_t* sched = a.sched;
  int32_t* list = sched + kAttnSchedHead;
  int32_t* tab = list + kAttnMaxUnits;
  int32_t* nch = tab + a.split_tiles;
  int32_t* ubase = nch + a.split_tiles;
  if (tid < n_hb) tpre[tid] = (a.cnt[tid * hb / a.hpg] + bmw - 1) / bmw;  // n_hb <= kAT
  if (tid == 0) work = 0;
  __syncthreads();
  if (tid < kWave) {
    const int t = wave_exscan(tpre, n_hb, false, 0);
    if (tid == 0) tpre[n_hb] = t;
  }
  __syncthreads();
  const int total = tpre[n_hb];
  if (total == 0 || total > a.split_tiles) {
    if (tid == 0) {
      sched[0] = 0;
      sched[1] = 0;
      sched[2] = 0;
    }
    return;
  }
  const int delta = a.T_k - a.T_q;
  static_assert(kAttnMaxSplitTiles <= 4 * kAT, "four tiles per thread");
  int last_tok[4];  // each tile's last row: four independent loads in flight
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int i = tid + q * kAT;
    last_tok[q] = 0;
    if (i < total) {
      int h = 0;
      while (tpre[h + 1] <= i) ++h;
      const int slot = i - tpre[h], gg = h * hb / a.hpg;
      const int last = min(a.cnt[gg], (slot + 1) * bmw) - 1;
      last_tok[q] = a.idx[(int64_t)gg * a.M + last];
      tab[i] = h << 16 | slot;
    }
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int i = tid + q * kAT;
    if (i < total) {
      const int nt = (last_tok[q] + delta + kBN) / kBN;  // key tiles of the tile
      nt_of[i] = nt;
      atomicAdd(&work, nt);
    }
  }
  __syncthreads();
  if (tid == 0) {
    const int nkt = (a.T_k + kBN - 1) / kBN, per_round = a.split_rounds * kAttnSlots;
    int ch = (nkt + kAttnMaxChunks - 1) / kAttnMaxChunks;
    ch = max(ch, (work + per_round - 1) / per_round);
    // sum of ceil(nt / ch) <= work / ch + total <= kAttnMaxUnits
    ch = max(ch, (work + (kAttnMaxUnits - total) - 1) / (kAttnMaxUnits - total));
    // No tile spans more than nkt key tiles: a longer chunk splits nothing,
    // and nkt <= kAttnMaxChunkTiles bounds the size histogram.
    chl = min(ch, nkt);
  }
  for (int i = tid; i <= kAttnMaxChunkTiles; i += kAT) hist[i] = 0;
  __syncthreads();
  const int ch = chl;
  // Each thread's contiguous run of tiles: chunk counts, their sum, the sizes.
  const int per = (total + kAT - 1) / kAT, i0 = min(total, tid * per), i1 = min(total, i0 + per);
  int mine = 0;
  for (int i = i0; i < i1; ++i) {
    const int nt = nt_of[i], nc = (nt + ch - 1) / ch;
    nch[i] = nc;
    mine += nc;
    for (int c = 0; c < nc; ++c) atomicAdd(&hist[min(ch, nt - c * ch)], 1);
  }
  tsum[tid] = mine;
  __syncthreads();
  if (tid < kWave) {
    n_units = wave_exscan(tsum, kAT, false, 0);
  } else if (tid < 2 * kWave) {  // start of each size's run, largest size first
    wave_exscan(hist + 1, ch, true, ch - 1);
  }
  __syncthreads();
  if (tid == 0) {
    sched[0] = n_units;
    sched[1] = total;
    sched[2] = ch;
  }
  int u = tsum[tid];
  for (int i = i0; i < i1; ++i) {
    const int nt = nt_of[i], nc = (nt + ch - 1) / ch;
    ubase[i] = u;
    u += nc;
    for (int c = 0; c < nc; ++c) list[atomicAdd(&hist[min(ch, nt - c * ch)], 1)] = i * kAttnMaxChunks + c;
  }
}

// Merge of a split tile's chunks: with m_c the chunks' running maxima (log2
// units) and M their maximum, O = sum_c 2^(m_c - M) O_c and the sum likewise,
// added in chunk order; then the epilogue of wide_attn_fwd.  One workgroup
// per listed tile, its waves laid out as the attention kernel's.
template <int HB>
__global__ __launch_bounds__(kAT) void wide_attn_merge(AttnArgs a) {
  constexpr int WR = 32, BMW = WR * (4 / HB);
  const int rank = blockIdx.x;
  if (rank >= a.sched[1]) return;
  const int32_t* tab = a.sched + kAttnSchedHead + kAttnMaxUnits;
  const int nc = tab[a.split_tiles + rank];
  if (nc <= 1) return;
  const int hbk = tab[rank] >> 16, slot = tab[rank] & 0xffff, u0 = tab[2 * a.split_tiles + rank];
  const int lane = lane_id(), w = wave_id(), l32 = lane & 31, hi = lane >> 5;
  const int rb = w / HB, h = hbk * HB + (w - rb * HB), g = hbk * HB / a.hpg;
  const int myr = slot * BMW + rb * WR + l32;
  const bool valid = myr < a.cnt[g];
  const float4* po = reinterpret_cast<const float4*>(a.part);
  const float2* pm = reinterpret_cast<const float2*>(a.part + (int64_t)kAttnMaxUnits * kAttnPartO);
  float mc[kAttnMaxChunks], zc[kAttnMaxChunks];
  float mx = -INFINITY;
#pragma unroll
  for (int c = 0; c < kAttnMaxChunks; ++c) {
    const float2 v = c < nc ? pm[((int64_t)(u0 + c) * 4 + w) * kWave + lane]
                            : make_float2(-INFINITY, 0.0f);
    mc[c] = v.x;
    zc[c] = v.y;
    mx = fmaxf(mx, v.x);
  }
  const float muse = mx == -INFINITY ? 0.0f : mx;  // a wave with no valid row
  float4 o[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) o[i] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
  float zs = 0.0f;
#pragma unroll
  for (int c = 0; c < kAttnMaxChunks; ++c) {
    if (c >= nc) break;
    const float wc = fast_exp2(mc[c] - muse);
    zs += wc * zc[c];
    const float4* src = po + ((int64_t)(u0 + c) * 4 + w) * (16 * kWave) + lane;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float4 v = src[i * kWave];
      o[i].x += wc * v.x;
      o[i].y += wc * v.y;
      o[i].z += wc * v.z;
      o[i].w += wc * v.w;
    }
  }
  const float zt = zs + __shfl_xor(zs, 32);
  if (!valid) return;
  const float inv = 1.0f / zt;
  const int64_t t = a.idx[(int64_t)g * a.M + myr];
  uint16_t* orow = a.o + t * ((int64_t)a.n_q * kHd) + (int64_t)h * kHd + 4 * hi;
#pragma unroll
  for (int db = 0; db < 4; ++db) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float4 v = o[db * 4 + j];
      uint2 u;
      u.x = pack_bf16x2_hw(v.x * inv, v.y * inv);
      u.y = pack_bf16x2_hw(v.z * inv, v.w * inv);
      *reinterpret_cast<uint2*>(orow + 32 * db + 8 * j) = u;
    }
  }
}

// Prep: V [n_seq*T_k][n_kv*128] -> V^T [n_seq][n_kv][128][T_kp] (zero past
// T_k), one workgroup per (sequence, KV head, 64 keys); then, when there is
// more than one sequence, one wave per (group, sequence boundary) finds where
// each sequence's active run starts in idx[g] (a 64-way search of the sorted
// list).
__global__ __launch_bounds__(kAT) void wide_attn_prep(AttnArgs a, const uint16_t* v, int32_t* seq_off,
                                                      int n_vt_blocks) {
  const int tid = threadIdx.x;
  int blk = blockIdx.x;
  if (a.sched) {  // block 0: the split's schedule, dispatched first
    if (blk == 0) {
      const int hb = attn_hb_of(a.hpg, a.qpk);
      attn_schedule(a, hb, 32 * (4 / hb));
      return;
    }
    --blk;
  }
  if (blk < n_vt_blocks) {
    // Thread (kc, dc) of the first 128 moves the 8 x 8 block of keys
    // kt*64 + 8kc.. and dims 8dc..: eight 16-byte row loads, a transpose in
    // registers, eight 16-byte stores.  A wave's loads cover 8 key rows x 128
    // contiguous bytes, its stores 8 dim rows x 128 contiguous bytes.
    if (tid >= 128) return;
    const int nkt = a.T_kp / 64;
    const int kt = blk % nkt;
    const int bh = blk / nkt;  // b * n_kv + hkv
    const int b = bh / a.n_kv, hkv = bh - b * a.n_kv;
    const int64_t ldk = (int64_t)a.n_kv * kHd;
    const int kc = tid & 7, dc = tid >> 3;
    const int k0 = kt * 64 + kc * 8;
    u32x4 in[8];
#pragma unroll
    for (int i = 0; i < 8; ++i)
      in[i] = k0 + i < a.T_k ? ldg16(v + ((int64_t)b * a.T_k + k0 + i) * ldk + hkv * kHd + dc * 8)
                             : u32x4{0, 0, 0, 0};
    uint16_t* vt = a.vt + (int64_t)bh * kHd * a.T_kp + k0;
#pragma unroll
    for (int e = 0; e < 8; ++e) {  // dim 8dc + e: keys k0 .. k0 + 7, two per word
      u32x4 o;
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const uint32_t lo = in[2 * j][e >> 1], hi = in[2 * j + 1][e >> 1];
        o[j] = (e & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
      }
      stg16(vt + (int64_t)(dc * 8 + e) * a.T_kp, o);
    }
    return;
  }
  // sequence offsets
  const int wv = (blk - n_vt_blocks) * (kAT / kWave) + wave_id();
  const int nb = a.n_seq + 1;
  if (wv >= a.ng * nb) return;
  const int g = wv / nb, b = wv - g * nb;
  const int lane = lane_id();
  const int32_t* idx_g = a.idx + (int64_t)g * a.M;
  const int cnt = a.cnt[g];
  const int64_t key = (int64_t)b * a.T_q;
  int lo = 0, hi = cnt;  // first position in [lo, hi] whose token is >= key
  if (b == a.n_seq) {
    lo = cnt;
  } else {
    while (hi - lo > 64) {
      const int step = (hi - lo + 63) / 64;
      const int p = lo + lane * step;
      const bool below = p < hi && idx_g[p] < key;
      const int k = __popcll(__ballot(below));
      if (k == 0) { hi = lo; break; }
      const int nlo = lo + (k - 1) * step + 1;
      hi = min(hi, lo + k * step);
      lo = nlo;
    }
    const int p = lo + lane;
    const bool below = p < hi && idx_g[p] < key;
    lo += __popcll(__ballot(below));
  }
  if (lane == 0) seq_off[g * nb + b] = lo;
}

}  // namespace

int attn_heads_per_block(int hpg, int qpk) { return attn_hb_of(hpg, qpk); }

int attn_slots(int T_q, int hb) { return (T_q + 32 * (4 / hb) - 1) / (32 * (4 / hb)); }

int attn_split_tiles(int64_t n_seq, int T_q, int T_k, int n_q, int hpg, int qpk) {
  const int hb = attn_hb_of(hpg, qpk);
  const int nkt = (T_k + 63) / 64;
  if (!g_attn_split || n_seq != 1 || nkt < 8 || nkt > kAttnMaxChunkTiles ||
      n_q / hb > kAttnMaxSplitHB)
    return 0;
  return (int)std::min<int64_t>(g_attn_split.load(), (int64_t)(n_q / hb) * attn_slots(T_q, hb));
}

hipError_t launch_attention(AttnArgs a, const uint16_t* v, int32_t* seq_off, hipStream_t s) {
  if (a.M == 0) return hipSuccess;
  const int hb = attn_heads_per_block(a.hpg, a.qpk);
  a.n_slots = attn_slots(a.T_q, hb);
  if (!a.causal || !a.sched || !a.part || a.split_tiles <= 0 || a.leftpad) {
    a.sched = nullptr;
    a.part = nullptr;
    a.split_tiles = 0;
  }
  a.split_rounds = g_attn_split_rounds;
  const int n_vt = a.n_seq * a.n_kv * (a.T_kp / 64);
  const int n_off = a.n_seq > 1 ? (a.ng * (a.n_seq + 1) + 3) / 4 : 0;
  WIDE_LAUNCH(wide_attn_prep, dim3((unsigned)(n_vt + n_off + (a.sched ? 1 : 0))), dim3(kAT), 0, s, a, v, seq_off,
              n_vt);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  a.seq_off = a.n_seq > 1 ? seq_off : nullptr;
  const int64_t n_classic = (int64_t)(a.n_q / hb) * a.n_seq * a.n_slots;
  const int64_t max_units = std::min<int64_t>(kAttnMaxUnits, (int64_t)a.split_tiles * kAttnMaxChunks);
  const dim3 grid((unsigned)std::max<int64_t>(n_classic, a.sched ? max_units : 0));
  if (hb == 4) WIDE_LAUNCH_NAMED("wide_attn_fwd", (wide_attn_fwd<4, 1>), grid, dim3(kAT), 0, s, a);
  else if (hb == 2) WIDE_LAUNCH_NAMED("wide_attn_fwd", (wide_attn_fwd<2, 1>), grid, dim3(kAT), 0, s, a);
  else WIDE_LAUNCH_NAMED("wide_attn_fwd", (wide_attn_fwd<1, 1>), grid, dim3(kAT), 0, s, a);
  if (a.sched) {
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const dim3 mg((unsigned)a.split_tiles);
    if (hb == 4) WIDE_LAUNCH_NAMED("wide_attn_merge", wide_attn_merge<4>, mg, dim3(kAT), 0, s, a);
    else if (hb == 2) WIDE_LAUNCH_NAMED("wide_attn_merge", wide_attn_merge<2>, mg, dim3(kAT), 0, s, a);
    else WIDE_LAUNCH_NAMED("wide_attn_merge", wide_attn_merge<1>, mg, dim3(kAT), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace wide
