// Bottleneck router, inference form (WIDE Section 3.1, "Routing Components").
//
// R = X W1 W2 with W1 in R^{D x r} (r <= 32) and W2 in R^{r x 2 n_groups},
// read as n_groups (execute, skip) pairs; mask[t][g] = 1 when the argmax of
// the pair is class 0, i.e. R[t][2g] >= R[t][2g+1] (a tie executes).
//
// One workgroup (16 waves) per 32 tokens:
//   stage 1  H = X W1 for the 32 tokens with v_mfma_f32_32x32x16_bf16 (tokens
//            as rows, the r bottleneck units as columns, zero-padded to 32);
//            the 16-wide k steps of d_model are dealt round-robin to the
//            waves, each keeping eight steps of loads in flight, and the
//            sixteen fp32 partials are added in LDS.  H stays fp32 (never
//            rounded to bf16).
//   stage 2  eight threads per group (W2 staged through LDS as fp32, 128
//            groups at a time), each with the group's two W2 rows in
//            registers (fp32, zero beyond the rank) and every eighth token:
//            the pair logits in fp32 (terms in rank order), then the mask
//            byte and, if asked for, the logits.
// The work is a few GFLOP at prefill sizes and bound by reading X once.
#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace wide {

namespace {
constexpr int kRT = 1024;         // threads (16 waves)
constexpr int kRW = kRT / kWave;
constexpr int kRDepth = 8;        // k steps in flight per wave
constexpr int kRTok = 32;         // tokens per workgroup
constexpr int kRPad = kRouterMaxRank + 1;
}  // namespace

__global__ __launch_bounds__(kRT) void wide_router(RouterArgs a) {
  __shared__ float s_part[kRW][kRTok][kRPad];
  __shared__ float s_h[kRTok][kRPad];
  __shared__ float s_w2[2 * (kRT / 8)][kRPad];
  const int tid = threadIdx.x, w = wave_id(), lane = lane_id();
  const int l32 = lane & 31, lhi = lane >> 5;
  const int64_t t0 = (int64_t)blockIdx.x * kRTok;
  const int D = a.D, r = a.r, ng = a.ng;

  // ---- stage 1: H = X W1; wave w takes k steps w, w + 8, w + 16, ...
  // Tokens past M and bottleneck units past the rank read zeros (buffer views
  // of this workgroup's rows of X and of W1).
  const int rows = (int)min((int64_t)kRTok, a.M - t0);
  const bufview_t xv = buf_view(a.x + t0 * D, (uint32_t)rows * D * 2);
  const bufview_t wv = buf_view(a.w1, (uint32_t)r * D * 2);
  const uint32_t xo = l32 < rows ? (uint32_t)(l32 * D + lhi * 8) * 2 : kOffNone;
  const uint32_t wo = l32 < r ? (uint32_t)(l32 * D + lhi * 8) * 2 : kOffNone;
  const int nsteps = D / 16;
  const int my = nsteps > w ? (nsteps - w + kRW - 1) / kRW : 0;
  f32x16 acc = f32x16{};
  u32x4 xa[kRDepth], wb[kRDepth];
  // Steps past this wave's share load zeros (no memory access), so the
  // pipeline runs branch-free to a multiple of its depth: the extra MFMAs add 0.
  auto load = [&](int q, int j) {
    const uint32_t kb = (uint32_t)(w + q * kRW) * 32;  // byte offset of the k step
    xa[j] = buf_ld16(xv, (q < my && xo != kOffNone) ? xo + kb : kOffNone);
    wb[j] = buf_ld16(wv, (q < my && wo != kOffNone) ? wo + kb : kOffNone);
  };
#pragma unroll
  for (int j = 0; j < kRDepth; ++j) load(j, j);
  for (int q = 0; q < my; q += kRDepth) {
#pragma unroll
    for (int j = 0; j < kRDepth; ++j) {
      acc = mfma32(xa[j], wb[j], acc);
      load(q + j + kRDepth, j);
    }
  }
  // accumulator element i: token row (i/4)*8 + lhi*4 + i%4, unit l32
#pragma unroll
  for (int i = 0; i < 16; ++i) s_part[w][(i >> 2) * 8 + lhi * 4 + (i & 3)][l32] = acc[i];
  __syncthreads();
  for (int i = tid; i < kRTok * kRouterMaxRank; i += kRT) {
    const int t = i / kRouterMaxRank, u = i % kRouterMaxRank;
    float s = 0.f;
#pragma unroll
    for (int q = 0; q < kRW; ++q) s += s_part[q][t][u];
    s_h[t][u] = s;
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
