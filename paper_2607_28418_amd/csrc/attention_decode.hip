// Head-group masked attention at decode on gfx950 (WIDE Section 3.1,
// equations (1)-(2); Appendix B: for decoding the reorder is bypassed, the
// routing is checked per block, and the online softmax is split over the
// keys; Appendix C on GQA packing).
//
// One query token per sequence attends to the sequence's cached keys
// [0, kv_len).  Decode attention is bound by reading the KV cache, so the
// point of the mask is to read less of it.  A work item is (sequence, KV
// head, chunk of keys) and packs every query head of that KV head (GQA
// packing); an item none of whose heads' groups is active for the token
// returns before touching the cache (l = 0), so an inactive KV head of a
// token costs no HBM traffic.
//
// Each wave is one work item and runs alone (no barriers), streaming its
// chunk in 16-key units straight into registers with three units in flight
// (the bytes in flight per CU, not the arithmetic, set the rate here):
//   scores  S^T[16 keys][16 heads] = K Q^T: four v_mfma_f32_16x16x32_bf16,
//           K rows as the A operand (16 bytes of a row per lane), the packed
//           heads' q as the B operand (columns past the heads are zero);
//   softmax online per head column, in fp32;
//   P.V     on the vector ALUs in fp32: lane = (one of 4 keys of each group
//           of 4, 8 of the 128 dims); the probabilities and rescale factors
//           pass through a per-wave LDS scratch.
// Per (token, head, chunk) the wave leaves (max, sum, unnormalised o) in the
// workspace; a second kernel merges the chunks (and writes +0 for inactive
// heads).
#include "common.h"
#include "kernels.h"
#include "launch.h"
#include "tile256.h"

namespace wide {
namespace {

constexpr int kHd = 128;
constexpr int kDT = 256;    // threads per workgroup: 4 independent waves
constexpr int kU = 16;      // keys per unit
constexpr int kDepth = 3;   // units in flight per wave

// Lanes of one wave exchange values through LDS: the fences tell the
// compiler that other lanes read what this lane wrote (and the reverse), so
// it neither forwards stale values nor moves accesses across this point.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

struct Unit {
  u32x4 k[4];  // lane: key row lane%16, dims 32s + 8*(lane/16) .. +8
  u32x4 v[4];  // lane: key 4i + lane/16, dims 8*(lane%16) .. +8
};

// HMAX: the most query heads per KV head this instance serves (qpk <= HMAX).
template <int HMAX>
__global__ __launch_bounds__(kDT) void wide_attn_decode(AttnDecArgs a) {
  constexpr int HB = HMAX < 4 ? HMAX : 4;  // head columns per LDS read group
  __shared__ __attribute__((aligned(16))) float s_p[4][kU][16];  // per wave: p[key][head]
  __shared__ __attribute__((aligned(16))) float s_al[4][16];     // per wave: rescale per head
  const int w = wave_id(), lane = lane_id();
  // Work items in (sequence, KV head, chunk) order, four per workgroup; each
  // XCD (workgroups are dealt round-robin to the 8 XCDs) takes a contiguous
  // range of them, i.e. whole sequences, so masks that switch whole KV heads
  // off still leave every XCD the same share of the work.
  const int64_t item = (int64_t)t256::xcd_remap(blockIdx.x, gridDim.x) * 4 + w;
  if (item >= (int64_t)a.B * a.n_kv * a.n_chunks) return;
  const int c = (int)(item % a.n_chunks);
  const int bh = (int)(item / a.n_chunks);
  const int b = bh / a.n_kv, hkv = bh - b * a.n_kv;
  const int len = a.kv_len ? min(a.kv_len[b], a.L) : a.L;
  const int j_begin = c * a.chunk;
  const int j_end = min(len, j_begin + a.chunk);
  const uint8_t* mrow = a.mask + (int64_t)b * a.ng;
  uint32_t act = 0;  // active query heads of this KV head, bit i = head hkv*qpk + i
  for (int i = 0; i < a.qpk; ++i)
    if (mrow[(hkv * a.qpk + i) / a.hpg]) act |= 1u << i;
  if (act == 0 || j_begin >= j_end) return;  // l = 0: no cache read for this item

  const int l16 = lane & 15, g4 = lane >> 4;
  // B operand: column = head l16 (zero unless an active packed head), dims 32s + 8*g4
  u32x4 qf[4];
  {
    const bool qa = l16 < a.qpk && ((act >> l16) & 1u);
    const uint16_t* qp = a.q + (int64_t)b * a.n_q * kHd + (int64_t)(hkv * a.qpk + (qa ? l16 : 0)) * kHd + 8 * g4;
#pragma unroll
    for (int s = 0; s < 4; ++s) qf[s] = qa ? ldg16(qp + 32 * s) : u32x4{0, 0, 0, 0};
  }
  // token-major cache: row (b, key) holds all KV heads; head-major: the
  // (b, KV head) cache is one contiguous [L][128] block
  const int64_t ldk = a.head_major ? kHd : (int64_t)a.n_kv * kHd;
  const int64_t cache0 = a.head_major ? ((int64_t)b * a.n_kv + hkv) * a.L * kHd
                                      : (int64_t)b * a.L * ldk + hkv * kHd;
  auto load = [&](int j0, Unit& u) {  // rows past kv_len re-read the last key (finite, p = 0)
    const uint16_t* kp = a.k + cache0 + (int64_t)min(j0 + l16, len - 1) * ldk + 8 * g4;
#pragma unroll
    for (int s = 0; s < 4; ++s) u.k[s] = ldg16(kp + 32 * s);
#pragma unroll
    for (int i = 0; i < 4; ++i) u.v[i] = ldg16(a.v + cache0 + (int64_t)min(j0 + 4 * i + g4, len - 1) * ldk + 8 * l16);
  };

  float m = -INFINITY, zl = 0.0f;  // running max of head column l16; this lane's share of its sum
  float acc[HMAX][8];
#pragma unroll
  for (int h = 0; h < HMAX; ++h)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[h][e] = 0.0f;
  const float sc = a.scale_log2;

  auto process = [&](int j0, const Unit& U) {
    f32x4 S = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int s = 0; s < 4; ++s) S = mfma16(U.k[s], qf[s], S);  // lane: keys 4*g4 + r, head l16
    float sv[4], mx = -INFINITY;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      sv[r] = j0 + 4 * g4 + r < j_end ? S[r] * sc : -INFINITY;
      mx = fmaxf(mx, sv[r]);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16));
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float mnew = fmaxf(m, mx);  // finite: the unit has a key before j_end
    const float alpha = __builtin_amdgcn_exp2f(m - mnew);
    m = mnew;
    float ps = 0.0f, pr[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      pr[r] = __builtin_amdgcn_exp2f(sv[r] - mnew);
      ps += pr[r];
    }
    zl = zl * alpha + ps;
    wave_lds_sync();  // the previous unit's reads of the scratch are done
#pragma unroll
    for (int r = 0; r < 4; ++r) s_p[w][4 * g4 + r][l16] = pr[r];
    if (g4 == 0) s_al[w][l16] = alpha;
    wave_lds_sync();  // this unit's values are visible to every lane of the wave
    // Up to four head columns, every column up to HMAX is carried, active or
    // not (an inactive or padding column has a zero query: finite scores,
    // discarded at the end), so the unit's arithmetic is straight-line code
    // (3-5% faster at Llama-3-8B's four heads per KV head); wider instances
    // test each head (the registers would not hold more).
#pragma unroll
    for (int h4 = 0; h4 < HMAX; h4 += HB) {
      float al[HB];  // (element reads through float: the writes above are float)
#pragma unroll
      for (int t = 0; t < HB; ++t) al[t] = s_al[w][h4 + t];
#pragma unroll
      for (int h = h4; h < h4 + HB; ++h)
        if (HMAX <= 4 || ((act >> h) & 1u))
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[h][e] *= al[h - h4];
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float vf[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        vf[2 * e] = __uint_as_float(U.v[i][e] << 16);
        vf[2 * e + 1] = __uint_as_float(U.v[i][e] & 0xffff0000u);
      }
#pragma unroll
      for (int h4 = 0; h4 < HMAX; h4 += HB) {
        float p4[HB];
#pragma unroll
        for (int t = 0; t < HB; ++t) p4[t] = s_p[w][4 * i + g4][h4 + t];
#pragma unroll
        for (int h = h4; h < h4 + HB; ++h)
          if (HMAX <= 4 || ((act >> h) & 1u))
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[h][e] = fmaf(p4[h - h4], vf[e], acc[h][e]);
      }
    }
  };

  // Full groups of kDepth units run branch-free, so the compiler can wait
  // for exactly the unit about to be used (the two younger ones stay in
  // flight); prefetches past the last unit re-read it (from L2) instead of
  // branching.  The last 0-2 units are processed after the loop.
  const int nunits = (j_end - j_begin + kU - 1) / kU;
  const int last = nunits - 1;
  Unit buf[kDepth];
#pragma unroll
  for (int d = 0; d < kDepth; ++d) load(j_begin + min(d, last) * kU, buf[d]);
  const int nfull = nunits / kDepth;
  for (int g = 0; g < nfull; ++g) {
#pragma unroll
    for (int d = 0; d < kDepth; ++d) {
      process(j_begin + (g * kDepth + d) * kU, buf[d]);
      load(j_begin + min((g + 1) * kDepth + d, last) * kU, buf[d]);
    }
  }
#pragma unroll
  for (int d = 0; d < kDepth - 1; ++d)
    if (nfull * kDepth + d < nunits) process(j_begin + (nfull * kDepth + d) * kU, buf[d]);

  // partials: (max, sum, o[128]) per (token, head, chunk)
  float z = zl + __shfl_xor(zl, 16);
  z += __shfl_xor(z, 32);
#pragma unroll
  for (int h = 0; h < HMAX; ++h) {
    if (!((act >> h) & 1u)) continue;
    float o8[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {  // add the four key groups
      float v = acc[h][e];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      o8[e] = v;
    }
    float* part = a.part + (((int64_t)b * a.n_q + hkv * a.qpk + h) * a.n_chunks + c) * (kHd + 2);
    if (lane == h) {
      part[0] = m;
      part[1] = z;
    }
    if (g4 == 0) {
#pragma unroll
      for (int e = 0; e < 8; ++e) part[2 + 8 * l16 + e] = o8[e];
    }
  }
}

// Merge of the chunks: one wave per (token, query head).  Lanes take the
// chunks for the maximum and the sum (64 at a time); for the output, lane =
// two dims, and each chunk's weight comes out of its lane by readlane.
__global__ __launch_bounds__(kDT) void wide_attn_decode_merge(AttnDecArgs a) {
  const int gw = blockIdx.x * (kDT / kWave) + wave_id();
  if (gw >= a.B * a.n_q) return;
  const int b = gw / a.n_q, h = gw - b * a.n_q;
  const int lane = lane_id();
  uint16_t* orow = a.o + (int64_t)b * a.n_q * kHd + (int64_t)h * kHd + 2 * lane;
  const int len = a.kv_len ? min(a.kv_len[b], a.L) : a.L;
  if (!a.mask[(int64_t)b * a.ng + h / a.hpg] || len <= 0) {  // inactive head: +0
    *reinterpret_cast<uint32_t*>(orow) = 0u;
    return;
  }
  const int nc = (len + a.chunk - 1) / a.chunk;
  const float* part = a.part + ((int64_t)b * a.n_q + h) * a.n_chunks * (kHd + 2);
  float mx = -INFINITY;
  for (int c0 = 0; c0 < nc; c0 += kWave)
    if (c0 + lane < nc) mx = fmaxf(mx, part[(c0 + lane) * (kHd + 2)]);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
  float z = 0.0f, o0 = 0.0f, o1 = 0.0f;
  for (int c0 = 0; c0 < nc; c0 += kWave) {
    const int c = c0 + lane;
    float f = 0.0f;
    if (c < nc) {
      f = __builtin_amdgcn_exp2f(part[c * (kHd + 2)] - mx);
      z = fmaf(f, part[c * (kHd + 2) + 1], z);
    }
    const int cnt = min(kWave, nc - c0);
    for (int j = 0; j < cnt; ++j) {
      const float fj = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(f), j));
      const float* pc = part + (c0 + j) * (kHd + 2) + 2 + 2 * lane;
      o0 = fmaf(fj, pc[0], o0);
      o1 = fmaf(fj, pc[1], o1);
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) z += __shfl_xor(z, o);
  const float inv = 1.0f / z;
  *reinterpret_cast<uint32_t*>(orow) = pack_bf16x2_hw(o0 * inv, o1 * inv);
}

}  // namespace

int attn_decode_chunk(int B, int n_kv, int L) {
  int ch = 2048;  // keys per work item (wave): enough items to fill the chip
  while (ch > 64 && (int64_t)B * n_kv * ((L + ch - 1) / ch) < 4096) ch /= 2;
  return ch;
}

hipError_t launch_attention_decode(AttnDecArgs a, hipStream_t s) {
  if (a.B == 0) return hipSuccess;
  const int64_t items = (int64_t)a.B * a.n_kv * a.n_chunks;
  const dim3 grid((unsigned)((items + 3) / 4));
  if (a.qpk == 1) WIDE_LAUNCH_NAMED("wide_attn_decode", (wide_attn_decode<1>), grid, dim3(kDT), 0, s, a);
  else if (a.qpk == 2) WIDE_LAUNCH_NAMED("wide_attn_decode", (wide_attn_decode<2>), grid, dim3(kDT), 0, s, a);
  else if (a.qpk <= 4) WIDE_LAUNCH_NAMED("wide_attn_decode", (wide_attn_decode<4>), grid, dim3(kDT), 0, s, a);
  else if (a.qpk <= 8) WIDE_LAUNCH_NAMED("wide_attn_decode", (wide_attn_decode<8>), grid, dim3(kDT), 0, s, a);
  else WIDE_LAUNCH_NAMED("wide_attn_decode", (wide_attn_decode<16>), grid, dim3(kDT), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int waves = a.B * a.n_q;
  WIDE_LAUNCH(wide_attn_decode_merge, dim3((unsigned)((waves + 3) / 4)), dim3(kDT), 0, s, a);
  return hipGetLastError();
}

}  // namespace wide
