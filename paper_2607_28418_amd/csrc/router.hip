// Bottleneck router, inference form (WIDE Section 3.1, "Routing Components").
//
// R = X W1 W2 with W1 in R^{D x r} (r <= 32) and W2 in R^{r x 2 n_groups},
// read as n_groups (execute, skip) pairs; mask[t][g] = 1 when the argmax of
// the pair is class 0, i.e. R[t][2g] >= R[t][2g+1] (a tie executes).
//
// One workgroup (16 waves) per 32 tokens:
//   stage 1  H = X W1 for the 32 tokens with v_mfma_f32_32x32x16_bf16 (tokens
//            as rows, the r bottleneck units as columns, padded to 32);
//            d_model is streamed in chunks of 256 through a ring of four LDS
//            stages with direct-to-LDS loads (each wave's 1 KB load covers
//            two rows' 512 contiguous bytes: whole cache lines; reading the
//            MFMA operands straight from memory touched 32 lines per load
//            and ran 2-3x slower); wave w takes the 16-wide k step w of
//            every chunk, and the sixteen fp32 partials are added in LDS.
//            H stays fp32 (never rounded to bf16).
//   stage 2  eight threads per group (W2 staged through LDS as fp32, 128
//            groups at a time), each with the group's two W2 rows in
//            registers (fp32, zero beyond the rank) and every eighth token:
//            the pair logits in fp32 (terms in rank order), then the mask
//            byte and, if asked for, the logits.
// The work is a few GFLOP at prefill sizes and bound by reading X once.
#include "common.h"
#include "kernels.h"
#include "launch.h"
#include "tile256.h"

namespace wide {

namespace {
constexpr int kRT = 1024;         // threads (16 waves)
constexpr int kRW = kRT / kWave;
constexpr int kRTok = 32;         // tokens per workgroup
constexpr int kRPad = kRouterMaxRank + 1;
constexpr int kRChunk = 256;      // d_model elements per LDS stage (16 k steps of 16)
constexpr int kRRowB = kRChunk * 2;
constexpr int kRTileB = 32 * kRRowB;  // one operand's stage: 32 rows x 512 bytes
constexpr int kRNst = 4;          // ring stages
static_assert(kRChunk / 16 == kRW, "one k step of every chunk per wave");
static_assert(kRW * kRTok * kRPad * 4 <= kRNst * 2 * kRTileB, "partials fit in the ring");
static_assert(2 * (kRT / 8) * kRPad * 4 <= kRNst * 2 * kRTileB, "W2 rows fit in the ring");
}  // namespace

__global__ __launch_bounds__(kRT) void wide_router(RouterArgs a) {
  // The ring; after stage 1 the same bytes hold the waves' partials, then
  // stage 2's W2 rows.
  __shared__ __attribute__((aligned(16))) char s_ring[kRNst * 2 * kRTileB];  // 128 KB
  __shared__ float s_h[kRTok][kRPad];
  auto s_part = reinterpret_cast<float(*)[kRTok][kRPad]>(s_ring);
  auto s_w2 = reinterpret_cast<float(*)[kRPad]>(s_ring);
  const int tid = threadIdx.x, w = wave_id(), lane = lane_id();
  const int l32 = lane & 31, lhi = lane >> 5;
  const int64_t t0 = (int64_t)blockIdx.x * kRTok;
  const int D = a.D, r = a.r, ng = a.ng;

  // ---- stage 1: H = X W1.  Chunk c of a row sits in its stage as 32
  // 16-byte pieces, piece j at position j ^ (row % 32) so that the operand
  // reads (32 rows, one piece each) spread over the banks.  Wave w loads rows
  // 2w and 2w+1 of both operands: lane l writes position l % 32 of row
  // 2w + l / 32 and so fetches piece (l % 32) ^ row.  Every wave issues its
  // two loads for every chunk (uniform wait counts): token rows past M read
  // the last token, units past the rank the last unit (never used: H's
  // columns past the rank are zeroed below), pieces past d_model the row's
  // first piece (no wave reads them).
  const int rows = (int)min((int64_t)kRTok, a.M - t0);
  const int lrow = 2 * w + lhi, pos = l32;
  const int piece = pos ^ lrow;
  const char* xrow = reinterpret_cast<const char*>(a.x + (t0 + min(lrow, rows - 1)) * (int64_t)D);
  const char* wrow = reinterpret_cast<const char*>(a.w1 + (int64_t)min(lrow, r - 1) * D);
  const int nch = (D + kRChunk - 1) / kRChunk;
  auto issue = [&](int c) {
    const int st = c % kRNst;
    const int64_t off = (int64_t)c * kRRowB + (c * kRChunk + piece * 8 < D ? piece * 16 : 0);
    char* xs = s_ring + st * 2 * kRTileB + 2 * w * kRRowB;
    __builtin_amdgcn_global_load_lds((t256::gptr_t)(xrow + off), (t256::lptr_t)xs, 16, 0, 0);
    __builtin_amdgcn_global_load_lds((t256::gptr_t)(wrow + off), (t256::lptr_t)(xs + kRTileB), 16, 0, 0);
  };
  // This wave's k step in each chunk: pieces 2w (lane half 0) and 2w + 1.
  const int rd = l32 * kRRowB + (((2 * w + lhi) ^ l32) << 4);
  f32x16 acc = f32x16{};
  for (int c = 0; c < min(kRNst - 1, nch); ++c) issue(c);
  for (int c = 0; c < nch; ++c) {
    const int younger = min(kRNst - 2, nch - 1 - c);  // chunks issued after c
    if (younger >= 2) t256::wait_vm<4>();
    else if (younger == 1) t256::wait_vm<2>();
    else t256::wait_vm<0>();
    t256::stage_barrier();  // chunk c is in LDS; every wave is done with chunk c - 1
    if (c + kRNst - 1 < nch) issue(c + kRNst - 1);
    if (c * kRChunk + w * 16 < D) {
      const char* st = s_ring + (c % kRNst) * 2 * kRTileB;
      const u32x4 xa = *reinterpret_cast<const u32x4*>(st + rd);
      const u32x4 wb = *reinterpret_cast<const u32x4*>(st + kRTileB + rd);
      acc = mfma32(xa, wb, acc);
    }
  }
  t256::stage_barrier();  // the ring becomes the partials
  // accumulator element i: token row (i/4)*8 + lhi*4 + i%4, unit l32
#pragma unroll
  for (int i = 0; i < 16; ++i) s_part[w][(i >> 2) * 8 + lhi * 4 + (i & 3)][l32] = acc[i];
  __syncthreads();
  for (int i = tid; i < kRTok * kRouterMaxRank; i += kRT) {
    const int t = i / kRouterMaxRank, u = i % kRouterMaxRank;
    float s = 0.f;
#pragma unroll
    for (int q = 0; q < kRW; ++q) s += s_part[q][t][u];
    s_h[t][u] = u < r ? s : 0.f;  // units past the rank are exact zeros
  }

  // ---- stage 2: eight threads per group, each taking every eighth token.
  // The W2 rows of 128 groups at a time go to LDS as fp32 with coalesced
  // 16-byte loads (rows are contiguous), then each thread keeps its group's
  // two rows in registers.
  constexpr int kTPG = 8;
  constexpr int kGPP = kRT / kTPG;  // groups per pass
  const int nt = (int)min((int64_t)kRTok, a.M - t0);
  const int gl = tid % kGPP, tq = tid / kGPP;
  const bufview_t w2v = buf_view(a.w2, (uint32_t)(2 * ng * r) * 2);
  for (int g0 = 0; g0 < ng; g0 += kGPP) {
    const int gc = min(kGPP, ng - g0);
    __syncthreads();  // s_h complete; the previous pass is done with s_w2
    {
      const int elems = 2 * gc * r;                 // bf16 values of this pass
      const uint32_t base = (uint32_t)(2 * g0 * r) * 2;
      for (int e0 = tid * 8; e0 < elems; e0 += kRT * 8) {
        const u32x4 v = buf_ld16(w2v, base + (uint32_t)e0 * 2);  // past the end: zeros
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int e = e0 + i;
          if (e < elems) {
            const uint32_t word = v[i >> 1];
            s_w2[e / r][e % r] = bf16_to_f32((uint16_t)(i & 1 ? word >> 16 : word & 0xffffu));
          }
        }
      }
    }
    __syncthreads();
    if (gl >= gc) continue;
    const int g = g0 + gl;
    float w0[kRouterMaxRank], w1v[kRouterMaxRank];
#pragma unroll
    for (int u = 0; u < kRouterMaxRank; ++u) {  // units past the rank weigh zero
      w0[u] = u < r ? s_w2[2 * gl][u] : 0.f;
      w1v[u] = u < r ? s_w2[2 * gl + 1][u] : 0.f;
    }
    for (int t = tq; t < nt; t += kTPG) {
      float r0 = 0.f, r1 = 0.f;
#pragma unroll
      for (int u = 0; u < kRouterMaxRank; ++u) {  // terms past the rank add exact zeros
        r0 = fmaf(s_h[t][u], w0[u], r0);
        r1 = fmaf(s_h[t][u], w1v[u], r1);
      }
      const int64_t row = t0 + t;
      a.mask[row * ng + g] = r0 >= r1 ? 1 : 0;
      if (a.logits) {
        a.logits[row * 2 * ng + 2 * g] = r0;
        a.logits[row * 2 * ng + 2 * g + 1] = r1;
      }
    }
  }
}

hipError_t launch_router(const RouterArgs& a, hipStream_t s) {
  if (a.M == 0) return hipSuccess;
  const int64_t blocks = (a.M + kRTok - 1) / kRTok;
  WIDE_LAUNCH(wide_router, dim3((unsigned)blocks), dim3(kRT), 0, s, a);
  return hipGetLastError();
}

}  // namespace wide
