// Bottleneck router, inference form (WIDE Section 3.1, "Routing Components").
//
// R = X W1 W2 with W1 in R^{D x r} (r <= 32) and W2 in R^{r x 2 n_groups},
// read as n_groups (execute, skip) pairs; mask[t][g] = 1 when the argmax of
// the pair is class 0, i.e. R[t][2g] >= R[t][2g+1] (a tie executes).
//
// One workgroup (4 waves) per 32 tokens:
//   stage 1  H = X W1 for the 32 tokens with v_mfma_f32_32x32x16_bf16 (tokens
//            as rows, the r bottleneck units as columns, zero-padded to 32);
//            each wave takes a quarter of d_model, the four fp32 partials are
//            added in LDS.  H stays fp32 (never rounded to bf16).
//   stage 2  the pair logits in fp32 on the vector ALUs from H and W2 (staged
//            in LDS as fp32, 256 groups at a time), then the mask byte and,
//            if asked for, the logits.
// The work is a few GFLOP at prefill sizes and bound by reading X once.
#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace wide {

namespace {
constexpr int kRT = 256;          // threads (4 waves)
constexpr int kRTok = 32;         // tokens per workgroup
constexpr int kRChunk = 256;      // groups whose W2 rows sit in LDS at a time
constexpr int kRPad = kRouterMaxRank + 1;
}  // namespace

__global__ __launch_bounds__(kRT) void wide_router(RouterArgs a) {
  __shared__ float s_part[kRT / kWave][kRTok][kRPad];
  __shared__ float s_h[kRTok][kRPad];
  __shared__ float s_w2[2 * kRChunk][kRPad];
  const int tid = threadIdx.x, w = wave_id(), lane = lane_id();
  const int l32 = lane & 31, lhi = lane >> 5;
  const int64_t t0 = (int64_t)blockIdx.x * kRTok;
  const int D = a.D, r = a.r, ng = a.ng;

  // ---- stage 1: H = X W1 (this wave: d_model range [w*D/4, (w+1)*D/4))
  const int64_t tok = t0 + l32;
  const bool tok_ok = tok < a.M;
  const bool unit_ok = l32 < r;
  const uint16_t* xr = a.x + (tok_ok ? tok : 0) * (int64_t)D + lhi * 8;
  const uint16_t* wr = a.w1 + (int64_t)(unit_ok ? l32 : 0) * D + lhi * 8;
  const int kq = D / (kRT / kWave);
  const int kb = w * kq;
  f32x16 acc = f32x16{};
  const u32x4 zero = u32x4{0u, 0u, 0u, 0u};
  constexpr int U = 4;  // k steps of 16 in flight
  int k = 0;
  for (; k + 16 * U <= kq; k += 16 * U) {
    u32x4 xa[U], wb[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      xa[u] = tok_ok ? ldg16(xr + kb + k + 16 * u) : zero;
      wb[u] = unit_ok ? ldg16(wr + kb + k + 16 * u) : zero;
    }
#pragma unroll
    for (int u = 0; u < U; ++u) acc = mfma32(xa[u], wb[u], acc);
  }
  for (; k < kq; k += 16) {
    const u32x4 xa = tok_ok ? ldg16(xr + kb + k) : zero;
    const u32x4 wb = unit_ok ? ldg16(wr + kb + k) : zero;
    acc = mfma32(xa, wb, acc);
  }
  // accumulator element i: token row (i/4)*8 + lhi*4 + i%4, unit l32
#pragma unroll
  for (int i = 0; i < 16; ++i) s_part[w][(i >> 2) * 8 + lhi * 4 + (i & 3)][l32] = acc[i];
  __syncthreads();
  for (int i = tid; i < kRTok * kRouterMaxRank; i += kRT) {
    const int t = i / kRouterMaxRank, u = i % kRouterMaxRank;
    float s = 0.f;
#pragma unroll
    for (int q = 0; q < kRT / kWave; ++q) s += s_part[q][t][u];
    s_h[t][u] = s;
  }

  // ---- stage 2: pair logits and the mask, 256 groups at a time
  const int nt = (int)min((int64_t)kRTok, a.M - t0);
  for (int c0 = 0; c0 < ng; c0 += kRChunk) {
    const int gc = min(kRChunk, ng - c0);
    __syncthreads();  // s_h complete / previous chunk's s_w2 no longer read
    for (int i = tid; i < 2 * gc * r; i += kRT) {
      const int row = i / r, u = i % r;
      s_w2[row][u] = bf16_to_f32(a.w2[(int64_t)(2 * c0 + row) * r + u]);
    }
    __syncthreads();
    for (int p = tid; p < nt * gc; p += kRT) {
      const int t = p / gc, gl = p % gc;
      float r0 = 0.f, r1 = 0.f;
      for (int u = 0; u < r; ++u) {
        r0 = fmaf(s_h[t][u], s_w2[2 * gl][u], r0);
        r1 = fmaf(s_h[t][u], s_w2[2 * gl + 1][u], r1);
      }
      const int64_t row = t0 + t;
      const int g = c0 + gl;
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
