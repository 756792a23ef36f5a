// Head-group masked attention at decode on gfx950 (WIDE Section 3.1,
// equations (1)-(2); Appendix B: for decoding the reorder is bypassed, the
// routing is checked per block, and the online softmax is split over the
// keys; Appendix C on GQA packing).
//
// One query token per sequence attends to the sequence's cached keys
// [0, kv_len).  Decode attention is bound by reading the KV cache, so the
// point of the mask is to read less of it: a workgroup owns (sequence, KV
// head, chunk of keys) and packs every query head of that KV head (GQA
// packing); it exits before touching the cache when none of those heads'
// groups is active for the token (l = 0), so an inactive KV head of a token
// costs no HBM traffic.
//
// Inside a workgroup the chunk streams through LDS in 64-key steps (K and V,
// 16 KB each, two stages, direct-to-LDS loads).  The arithmetic is small
// next to the bytes (4 heads x 128 dims x 4 FLOPs per 512-byte key) and runs
// on the vector ALUs in fp32:
//   scores: lane = key; the lane's K row against the head's q (bf16 pairs
//           through v_dot2 with fp32 sums), q read from LDS by broadcast;
//   softmax: online per head over the chunk (max and sums across the wave);
//   P.V:    lane = (one of 4 key slots, 8 of the 128 dims); a key's
//           probability moves from its lane by a cross-lane permute and
//           16 bytes of its V row come from LDS; the 4 slots are added at
//           the end of the chunk.
// Per (token, head, chunk) the kernel leaves (max, sum, unnormalised o) in
// the workspace; a second kernel merges the chunks (and writes +0 for
// inactive heads).
#include "common.h"
#include "kernels.h"
#include "launch.h"
#include "tile256.h"

namespace wide {
namespace {

using t256::gptr_t;
using t256::lptr_t;

constexpr int kHd = 128;
constexpr int kDT = 256;          // threads per workgroup (4 waves)
constexpr int kKeys = 64;         // keys per LDS step
constexpr int kRowEl = kKeys * kHd;  // bf16 elements of one 64-key tile

typedef __bf16 bf16x2_v __attribute__((ext_vector_type(2)));

// LDS rows are 128 bf16 = 16 chunks of 16 bytes; logical chunk c of row r
// sits at physical chunk c ^ (r & 15), so the 64 lanes of a score step
// (one row each, same logical chunk) spread over all bank groups.
__device__ __forceinline__ int dswz(int r, int c) { return r * kHd + ((c ^ (r & 15)) << 3); }

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_v, a), __builtin_bit_cast(bf16x2_v, b), c,
                                         false);
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// HPW: query heads handled by each of the 4 waves (qpk <= 4 * HPW).
template <int HPW>
__global__ __launch_bounds__(kDT) void wide_attn_decode(AttnDecArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t sk[2][kRowEl];
  __shared__ __attribute__((aligned(16))) uint16_t sv[2][kRowEl];
  __shared__ __attribute__((aligned(16))) uint16_t sq[4 * HPW][kHd];

  const int c = blockIdx.x % a.n_chunks;
  const int bh = blockIdx.x / a.n_chunks;
  const int b = bh / a.n_kv, hkv = bh - b * a.n_kv;
  const int len = a.kv_len ? min(a.kv_len[b], a.L) : a.L;
  const int j_begin = c * a.chunk;
  const int j_end = min(len, j_begin + a.chunk);
  const uint8_t* mrow = a.mask + (int64_t)b * a.ng;
  uint32_t act = 0;  // active query heads of this KV head, bit i = head hkv*qpk + i
  for (int i = 0; i < a.qpk; ++i)
    if (mrow[(hkv * a.qpk + i) / a.hpg]) act |= 1u << i;
  if (act == 0 || j_begin >= j_end) return;  // l = 0: no cache read for this block

  const int tid = threadIdx.x, lane = lane_id(), w = wave_id();
  // q of the packed heads -> LDS (inactive heads' rows are never read)
  const int64_t ldq = (int64_t)a.n_q * kHd;
  for (int i = tid; i < a.qpk * (kHd / 8); i += kDT) {
    const int hh = i / (kHd / 8), ch = i % (kHd / 8);
    if (act & (1u << hh))
      *reinterpret_cast<u32x4*>(&sq[hh][ch * 8]) =
          ldg16(a.q + (int64_t)b * ldq + (int64_t)(hkv * a.qpk + hh) * kHd + ch * 8);
  }

  // Loads of one 64-key step: K and V tiles of 16 KB = 16 wave instructions
  // each; wave w issues K instructions 4w..4w+3 and V instructions 4w..4w+3.
  // token-major cache: row (b, key) holds all KV heads; head-major: the
  // (b, KV head) cache is one contiguous [L][128] block
  const int64_t ldk = a.head_major ? kHd : (int64_t)a.n_kv * kHd;
  const int64_t cache0 = a.head_major ? ((int64_t)b * a.n_kv + hkv) * a.L * kHd
                                      : (int64_t)b * a.L * ldk + hkv * kHd;
  auto issue = [&](int j0, int st) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int u = w * 4 + q;             // 4 rows of 256 bytes per instruction
      const int r = u * 4 + lane / 16;     // key row in the step
      const int lc = (lane & 15) ^ (r & 15);
      const int key = min(j0 + r, len - 1);  // rows past the end: any valid row (never used)
      const int64_t g = cache0 + key * ldk + lc * 8;
      __builtin_amdgcn_global_load_lds((gptr_t)(a.k + g), (lptr_t)(&sk[st][u * 4 * kHd]), 16, 0, 0);
      __builtin_amdgcn_global_load_lds((gptr_t)(a.v + g), (lptr_t)(&sv[st][u * 4 * kHd]), 16, 0, 0);
    }
  };

  // P.V layout: lane = (key slot ks = lane / 16, dim chunk dc = lane % 16);
  // the lane accumulates dims 8*dc .. 8*dc+7 over the keys = ks (mod 4).
  const int ks4 = lane >> 4, dc = lane & 15;
  float m[HPW], zl[HPW], acc[HPW][8];
#pragma unroll
  for (int i = 0; i < HPW; ++i) {
    m[i] = -INFINITY;
    zl[i] = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[i][e] = 0.0f;
  }
  const float sc = a.scale_log2;
  const int nsteps = (j_end - j_begin + kKeys - 1) / kKeys;
  issue(j_begin, 0);
  for (int s = 0; s < nsteps; ++s) {
    t256::wait_vm<0>();
    t256::stage_barrier();
    if (s + 1 < nsteps) issue(j_begin + (s + 1) * kKeys, (s + 1) & 1);
    const int j0 = j_begin + s * kKeys;
    const int nvalid = min(kKeys, j_end - j0);  // keys of this step inside [0, kv_len)
    const uint16_t* ks = sk[s & 1];
    const uint16_t* vs = sv[s & 1];
    // this lane's key row (lane = key)
    u32x4 kr[16];
#pragma unroll
    for (int ch = 0; ch < 16; ++ch) kr[ch] = *reinterpret_cast<const u32x4*>(&ks[dswz(lane, ch)]);
#pragma unroll
    for (int i = 0; i < HPW; ++i) {
      const int hh = w + 4 * i;
      if (hh >= a.qpk || !(act & (1u << hh))) continue;  // wave-uniform
      float sdot = 0.0f;
#pragma unroll
      for (int ch = 0; ch < 16; ++ch) {
        const u32x4 qv = *reinterpret_cast<const u32x4*>(&sq[hh][ch * 8]);
#pragma unroll
        for (int e = 0; e < 4; ++e) sdot = dot2(kr[ch][e], qv[e], sdot);
      }
      const float sv2 = lane < nvalid ? sdot * sc : -INFINITY;
      const float mnew = fmaxf(m[i], wave_max(sv2));  // finite: the step has a valid key
      const float alpha = __builtin_amdgcn_exp2f(m[i] - mnew);
      const float p = __builtin_amdgcn_exp2f(sv2 - mnew);
      m[i] = mnew;
      zl[i] = zl[i] * alpha + p;
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[i][e] *= alpha;
      // P.V over the 64 keys of the step, 16 per lane (rows past kv_len hold a
      // copy of a valid row and carry p = 0)
#pragma unroll
      for (int it = 0; it < kKeys / 4; ++it) {
        const int key = 4 * it + ks4;
        const float pj = __int_as_float(__builtin_amdgcn_ds_bpermute(key * 4, __float_as_int(p)));
        const u32x4 vv = *reinterpret_cast<const u32x4*>(&vs[dswz(key, dc)]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          acc[i][2 * e] = fmaf(pj, __uint_as_float(vv[e] << 16), acc[i][2 * e]);
          acc[i][2 * e + 1] = fmaf(pj, __uint_as_float(vv[e] & 0xffff0000u), acc[i][2 * e + 1]);
        }
      }
    }
  }
  // partials: (max, sum, o[128]) per (token, head, chunk)
#pragma unroll
  for (int i = 0; i < HPW; ++i) {
    const int hh = w + 4 * i;
    if (hh >= a.qpk || !(act & (1u << hh))) continue;
    const float z = wave_sum(zl[i]);
    float o8[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {  // add the four key slots
      float v = acc[i][e];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      o8[e] = v;
    }
    float* part = a.part + (((int64_t)b * a.n_q + hkv * a.qpk + hh) * a.n_chunks + c) * (kHd + 2);
    if (lane == 0) {
      part[0] = m[i];
      part[1] = z;
    }
    if (lane < 16) {
#pragma unroll
      for (int e = 0; e < 8; ++e) part[2 + 8 * lane + e] = o8[e];
    }
  }
}

// Merge of the chunks: one wave per (token, query head); lane = two dims.
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
  for (int c = 0; c < nc; ++c) mx = fmaxf(mx, part[c * (kHd + 2)]);
  float z = 0.0f, o0 = 0.0f, o1 = 0.0f;
  for (int c = 0; c < nc; ++c) {
    const float* pc = part + c * (kHd + 2);
    const float f = __builtin_amdgcn_exp2f(pc[0] - mx);
    z = fmaf(f, pc[1], z);
    o0 = fmaf(f, pc[2 + 2 * lane], o0);
    o1 = fmaf(f, pc[3 + 2 * lane], o1);
  }
  const float inv = 1.0f / z;
  *reinterpret_cast<uint32_t*>(orow) = pack_bf16x2_hw(o0 * inv, o1 * inv);
}

}  // namespace

int attn_decode_chunk(int B, int n_kv, int L) {
  int ch = 1024;
  while (ch > kKeys && (int64_t)B * n_kv * ((L + ch - 1) / ch) < 2048) ch /= 2;
  return ch;
}

hipError_t launch_attention_decode(AttnDecArgs a, hipStream_t s) {
  if (a.B == 0) return hipSuccess;
  const int hpw = (a.qpk + 3) / 4;
  const dim3 grid((unsigned)((int64_t)a.B * a.n_kv * a.n_chunks));
  if (hpw <= 1) WIDE_LAUNCH_NAMED("wide_attn_decode", (wide_attn_decode<1>), grid, dim3(kDT), 0, s, a);
  else if (hpw <= 2) WIDE_LAUNCH_NAMED("wide_attn_decode", (wide_attn_decode<2>), grid, dim3(kDT), 0, s, a);
  else if (hpw <= 4) WIDE_LAUNCH_NAMED("wide_attn_decode", (wide_attn_decode<4>), grid, dim3(kDT), 0, s, a);
  else WIDE_LAUNCH_NAMED("wide_attn_decode", (wide_attn_decode<8>), grid, dim3(kDT), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int waves = a.B * a.n_q;
  WIDE_LAUNCH(wide_attn_decode_merge, dim3((unsigned)((waves + 3) / 4)), dim3(kDT), 0, s, a);
  return hipGetLastError();
}

}  // namespace wide
