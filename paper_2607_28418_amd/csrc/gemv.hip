// Decode (small batch) masked projections, bf16 MFMA on gfx950.
//
// At decode the mask reorder is skipped and routing is checked per group
// directly (WIDE Appendix B: the GEMV variants of GEMM-MN and GEMM-K, and the
// decode note of the attention kernel).  The batch is B <= 64 tokens and the
// work is bound by streaming weights from HBM, so the aim is to read exactly
// the weight bytes of the groups some token of the batch uses (the union U)
// and nothing else, with full-cache-line 128-bit loads.
//
// gemv_n  (N-axis: gate/up + SwiGLU, Q; dense K/V).  A workgroup owns 16
//         output columns of one group and its 4 waves split the reduction
//         dimension K.  If no token of the batch is active in the group, the
//         workgroup writes +0 and exits before touching a weight byte.
//         Otherwise lane l streams 32 contiguous bytes of weight row l%16 per
//         64-wide k step (four lanes cover a full 128-byte line) and the
//         activations ride along as the other MFMA operand (16x16x32, tokens
//         as rows); both operands use the same permutation of k inside the
//         step, so the sum is unchanged.  Partial sums of the 4 waves meet in
//         LDS; inactive (token, group) outputs are +0.
//
// gemv_k  (K-axis: down, O).  A workgroup owns 16 output rows n and its 8
//         waves split the union groups; for each union group a wave reads the
//         2G-byte segment w[n, gG:(g+1)G] of its 16 rows and the matching
//         activations, masked per token (inactive blocks are not read).  No
//         atomics: the 8 partial sums meet in LDS.
#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace wide {

namespace {
constexpr int kTB = kDecodeMaxB / 16;   // token blocks of 16
}

template <bool SWIGLU>
__global__ __launch_bounds__(256) void wide_gemv_n(GVNArgs a) {
  constexpr int NW = 4;
  __shared__ float red[NW][2][kDecodeMaxB][16];
  __shared__ int any_active;

  int nb = blockIdx.x;
  GVRegion R = a.reg[0];
  if (a.n_regions > 1 && nb >= a.reg[0].n_blocks) {
    nb -= a.reg[0].n_blocks;
    R = a.reg[1];
    if (a.n_regions > 2 && nb >= a.reg[1].n_blocks) {
      nb -= a.reg[1].n_blocks;
      R = a.reg[2];
    }
  }
  const int n0 = nb * 16;
  const int g = n0 / a.G;
  const int tid = threadIdx.x;
  const int B = a.B, K = a.K;

  if (tid == 0) any_active = 0;
  __syncthreads();
  if (R.masked) {
    if (tid < B && a.mask[(int64_t)tid * a.n_groups + g] != 0) any_active = 1;
  } else if (tid == 0) {
    any_active = 1;
  }
  __syncthreads();
  if (!any_active) {
    // group unused by the whole batch: no weight reads, outputs +0
    for (int i = tid; i < B * 2; i += 256) {
      const int b = i / 2, h = i % 2;
      stg16(R.out + (int64_t)b * R.ldo + n0 + h * 8, u32x4{0, 0, 0, 0});
    }
    return;
  }

  const int w = wave_id(), lane = lane_id();
  const int ln = lane & 15, lq = lane >> 4;
  const int kw = K / NW;  // this wave's slice of K
  const int kb = w * kw;
  const uint16_t* wg = R.w0 + (int64_t)(n0 + ln) * K + kb + lq * 16;
  const uint16_t* wu = SWIGLU ? R.w1 + (int64_t)(n0 + ln) * K + kb + lq * 16 : nullptr;
  const int ntb = (B + 15) / 16;

  f32x4 ag[kTB], au[kTB];
#pragma unroll
  for (int i = 0; i < kTB; ++i) {
    ag[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    au[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  for (int k = 0; k < kw; k += 64) {
    const u32x4 g0 = ldg16(wg + k), g1 = ldg16(wg + k + 8);
    u32x4 u0 = {0, 0, 0, 0}, u1 = {0, 0, 0, 0};
    if (SWIGLU) {
      u0 = ldg16(wu + k);
      u1 = ldg16(wu + k + 8);
    }
#pragma unroll
    for (int tb = 0; tb < kTB; ++tb) {
      if (tb < ntb) {
        const int b = tb * 16 + ln;
        u32x4 x0 = {0, 0, 0, 0}, x1 = {0, 0, 0, 0};
        if (b < B) {
          const uint16_t* xp = a.x + (int64_t)b * K + kb + k + lq * 16;
          x0 = ldg16(xp);
          x1 = ldg16(xp + 8);
        }
        ag[tb] = mfma16(x0, g0, ag[tb]);
        ag[tb] = mfma16(x1, g1, ag[tb]);
        if (SWIGLU) {
          au[tb] = mfma16(x0, u0, au[tb]);
          au[tb] = mfma16(x1, u1, au[tb]);
        }
      }
    }
  }
  // C[row = token (lane/16)*4 + i][col = lane%16]
#pragma unroll
  for (int tb = 0; tb < kTB; ++tb) {
    if (tb < ntb) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int b = tb * 16 + lq * 4 + i;
        red[w][0][b][ln] = ag[tb][i];
        if (SWIGLU) red[w][1][b][ln] = au[tb][i];
      }
    }
  }
  __syncthreads();
  for (int i = tid; i < B * 16; i += 256) {
    const int b = i / 16, c = i % 16;
    float s0 = 0.f, s1 = 0.f;
#pragma unroll
    for (int v = 0; v < NW; ++v) {
      s0 += red[v][0][b][c];
      if (SWIGLU) s1 += red[v][1][b][c];
    }
    const bool on = !R.masked || a.mask[(int64_t)b * a.n_groups + g] != 0;
    const float o = on ? (SWIGLU ? silu(s0) * s1 : s0) : 0.f;
    R.out[(int64_t)b * R.ldo + n0 + c] = f32_to_bf16(o);
  }
}

__global__ __launch_bounds__(512) void wide_gemv_k(GVKArgs a) {
  constexpr int NW = 8;
  __shared__ float red[NW][kDecodeMaxB][16];
  __shared__ uint16_t ulist[4096];
  __shared__ int n_union;

  const int tid = threadIdx.x;
  const int B = a.B, K = a.K, G = a.G, ng = a.n_groups;
  const int n0 = blockIdx.x * 16;
  // Union of the batch's active groups, compacted in ascending order.
  if (tid == 0) n_union = 0;
  __syncthreads();
  for (int g0 = 0; g0 < ng; g0 += 512) {
    const int gg = g0 + tid;
    bool on = false;
    if (gg < ng)
      for (int b = 0; b < B && !on; ++b) on = a.mask[(int64_t)b * ng + gg] != 0;
    // block-wide ordered compaction: wave ballots then a serial prefix
    __shared__ int wc[NW];
    const uint64_t bal = __ballot(on);
    const int lane = lane_id(), w = wave_id();
    if (lane == 0) wc[w] = __popcll(bal);
    __syncthreads();
    int before = n_union;
    for (int i = 0; i < w; ++i) before += wc[i];
    if (on) {
      const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
      ulist[before + __popcll(bal & below)] = (uint16_t)gg;
    }
    __syncthreads();
    if (tid == 0) {
      int s = 0;
      for (int i = 0; i < NW; ++i) s += wc[i];
      n_union += s;
    }
    __syncthreads();
  }
  const int nu = n_union;

  const int w = wave_id(), lane = lane_id();
  const int ln = lane & 15, lq = lane >> 4;
  const int ntb = (B + 15) / 16;
  f32x4 acc[kTB];
#pragma unroll
  for (int i = 0; i < kTB; ++i) acc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
  const uint16_t* wrow = a.w + (int64_t)(n0 + ln) * K + lq * 16;

  for (int ui = w; ui < nu; ui += NW) {
    const int g = ulist[ui];
    const int kg = g * G;
    bool tok_on[kTB];
#pragma unroll
    for (int tb = 0; tb < kTB; ++tb) {
      const int b = tb * 16 + ln;
      tok_on[tb] = tb < ntb && b < B && a.mask[(int64_t)b * ng + g] != 0;
    }
    for (int k = kg; k < kg + G; k += 64) {
      const u32x4 w0 = ldg16(wrow + k), w1 = ldg16(wrow + k + 8);
#pragma unroll
      for (int tb = 0; tb < kTB; ++tb) {
        if (tb < ntb) {
          u32x4 x0 = {0, 0, 0, 0}, x1 = {0, 0, 0, 0};
          if (tok_on[tb]) {
            const uint16_t* xp = a.a + (int64_t)(tb * 16 + ln) * K + k + lq * 16;
            x0 = ldg16(xp);
            x1 = ldg16(xp + 8);
          }
          acc[tb] = mfma16(x0, w0, acc[tb]);
          acc[tb] = mfma16(x1, w1, acc[tb]);
        }
      }
    }
  }
#pragma unroll
  for (int tb = 0; tb < kTB; ++tb)
    if (tb < ntb)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[w][tb * 16 + lq * 4 + i][ln] = acc[tb][i];
  __syncthreads();
  for (int i = tid; i < B * 16; i += 512) {
    const int b = i / 16, c = i % 16;
    float s = 0.f;
#pragma unroll
    for (int v = 0; v < NW; ++v) s += red[v][b][c];
    a.y[(int64_t)b * a.N + n0 + c] = f32_to_bf16(s);
  }
}

hipError_t launch_gemv_n(const GVNArgs& a, bool swiglu, hipStream_t s) {
  int nb = 0;
  for (int i = 0; i < a.n_regions; ++i) nb += a.reg[i].n_blocks;
  if (nb == 0 || a.B == 0) return hipSuccess;
  if (swiglu)
    WIDE_LAUNCH((wide_gemv_n<true>), dim3(nb), dim3(256), 0, s, a);
  else
    WIDE_LAUNCH((wide_gemv_n<false>), dim3(nb), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gemv_k(const GVKArgs& a, hipStream_t s) {
  if (a.B == 0 || a.N == 0) return hipSuccess;
  WIDE_LAUNCH(wide_gemv_k, dim3(a.N / 16), dim3(512), 0, s, a);
  return hipGetLastError();
}

}  // namespace wide
