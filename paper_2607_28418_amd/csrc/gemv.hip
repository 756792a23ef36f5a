// Decode (small batch) masked projections, bf16 MFMA on gfx950.
//
// At decode the mask reorder is skipped and routing is checked per group
// directly (WIDE Appendix B: the GEMV variants of GEMM-MN and GEMM-K, and the
// decode note of the attention kernel).  The batch is B <= 64 tokens and the
// work is bound by streaming weights from HBM, so the aim is to read exactly
// the weight bytes of the groups some token of the batch uses (the union U)
// and nothing else, with full-cache-line 128-bit loads and many loads in
// flight per lane.
//
// gemv_n  (N-axis: gate/up + SwiGLU, Q; dense K/V).  A workgroup owns 16
//         output columns of one group; its 8 waves take turns over the
//         64-wide steps of the reduction dimension K.  If no token of the
//         batch is active in the group, the workgroup writes +0 and exits
//         before touching a weight byte.  Otherwise lane l streams 32
//         contiguous bytes of weight row l%16 per k step (four lanes cover a
//         128-byte line), four steps at a time together with the matching
//         activations, which ride along as the other MFMA operand (16x16x32,
//         tokens as rows); both operands use the same permutation of k inside
//         a step, so the sum is unchanged.  Inactive (token, group) outputs
//         are +0.
//
// gemv_k  (K-axis: down, O).  A workgroup owns 16 output rows n; its 8 waves
//         take turns over the k steps of the union groups; for each union
//         group a wave reads the 2G-byte segments w[n, gG:(g+1)G] of its 16
//         rows and the matching activations of the tokens active in the group
//         (inactive blocks are never read).  The batch's mask sits in LDS as
//         one 64-bit token set per group.  No atomics.
//
// Both reduce the 8 waves' partial sums through LDS in a fixed order, so the
// results are deterministic.  NTB (1, 2 or 4 blocks of 16 tokens) sizes the
// registers to the batch.
#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace wide {

namespace {
constexpr int NW = 8;                  // waves per workgroup
constexpr int NT = NW * kWave;
constexpr int U = 4;                   // k steps in flight per lane

// Sum 8 waves' [NTB*16 tokens][16 cols] partials: waves 4..7 park theirs,
// waves 0..3 add theirs on top, then out(b, c, sums) runs per output.
template <int NV, int NTB, class Out>
__device__ __forceinline__ void reduce_out(float (*red)[kDecodeMaxB][16], const f32x4 (&acc)[NV][NTB],
                                           int B, Out out) {
  const int w = wave_id(), lane = lane_id();
  const int ln = lane & 15, lq = lane >> 4;
  if (w >= NW / 2) {
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int tb = 0; tb < NTB; ++tb)
#pragma unroll
        for (int i = 0; i < 4; ++i) red[(w - NW / 2) * NV + v][tb * 16 + lq * 4 + i][ln] = acc[v][tb][i];
  }
  __syncthreads();
  if (w < NW / 2) {
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int tb = 0; tb < NTB; ++tb)
#pragma unroll
        for (int i = 0; i < 4; ++i) red[w * NV + v][tb * 16 + lq * 4 + i][ln] += acc[v][tb][i];
  }
  __syncthreads();
  for (int i = threadIdx.x; i < B * 16; i += NT) {
    const int b = i / 16, c = i % 16;
    float s[NV];
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      s[v] = 0.f;
#pragma unroll
      for (int q = 0; q < NW / 2; ++q) s[v] += red[q * NV + v][b][c];
    }
    out(b, c, s);
  }
}

// Loads of one k step: weights of NV row sets and activations of NTB token
// blocks.
template <int NV, int NTB>
struct StepRegs {
  u32x4 w[NV][2];
  u32x4 x[NTB][2];
};

template <int NV, int NTB>
__device__ __forceinline__ void step_mfma(const StepRegs<NV, NTB>& r, f32x4 (&acc)[NV][NTB]) {
#pragma unroll
  for (int tb = 0; tb < NTB; ++tb)
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      acc[v][tb] = mfma16(r.x[tb][0], r.w[v][0], acc[v][tb]);
      acc[v][tb] = mfma16(r.x[tb][1], r.w[v][1], acc[v][tb]);
    }
}
}  // namespace

template <bool SWIGLU, int NTB>
__global__ __launch_bounds__(NT) void wide_gemv_n(GVNArgs a) {
  constexpr int NV = SWIGLU ? 2 : 1;
  __shared__ float red[NW / 2 * NV][kDecodeMaxB][16];
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

  if (tid == 0) any_active = R.masked ? 0 : 1;
  __syncthreads();
  if (R.masked && tid < B && a.mask[(int64_t)tid * a.n_groups + g] != 0) any_active = 1;
  __syncthreads();
  if (!any_active) {
    // group unused by the whole batch: no weight reads, outputs +0
    for (int i = tid; i < B * 2; i += NT) {
      const int b = i / 2, h = i % 2;
      stg16(R.out + (int64_t)b * R.ldo + n0 + h * 8, u32x4{0, 0, 0, 0});
    }
    return;
  }

  const int w = wave_id(), lane = lane_id();
  const int ln = lane & 15, lq = lane >> 4;
  // The K/64 steps are dealt round-robin to the 8 waves.
  const int nsteps = K / 64;
  const int my_steps = nsteps > w ? (nsteps - w + NW - 1) / NW : 0;
  const uint16_t* wrow[NV];
  wrow[0] = R.w0 + (int64_t)(n0 + ln) * K + lq * 16;
  if (SWIGLU) wrow[NV - 1] = R.w1 + (int64_t)(n0 + ln) * K + lq * 16;
  const uint16_t* xrow[NTB];
  bool xon[NTB];
#pragma unroll
  for (int tb = 0; tb < NTB; ++tb) {
    const int b = tb * 16 + ln;
    xon[tb] = b < B;
    xrow[tb] = a.x + (int64_t)(xon[tb] ? b : 0) * K + lq * 16;
  }

  f32x4 acc[NV][NTB];
#pragma unroll
  for (int v = 0; v < NV; ++v)
#pragma unroll
    for (int i = 0; i < NTB; ++i) acc[v][i] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto load = [&](int k, StepRegs<NV, NTB>& r) {
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      r.w[v][0] = ldg16(wrow[v] + k);
      r.w[v][1] = ldg16(wrow[v] + k + 8);
    }
#pragma unroll
    for (int tb = 0; tb < NTB; ++tb) {
      r.x[tb][0] = xon[tb] ? ldg16(xrow[tb] + k) : u32x4{0, 0, 0, 0};
      r.x[tb][1] = xon[tb] ? ldg16(xrow[tb] + k + 8) : u32x4{0, 0, 0, 0};
    }
  };
  int q = 0;
  for (; q + U <= my_steps; q += U) {
    StepRegs<NV, NTB> r[U];
#pragma unroll
    for (int s = 0; s < U; ++s) load((w + (q + s) * NW) * 64, r[s]);
#pragma unroll
    for (int s = 0; s < U; ++s) step_mfma(r[s], acc);
  }
  for (; q < my_steps; ++q) {
    StepRegs<NV, NTB> r;
    load((w + q * NW) * 64, r);
    step_mfma(r, acc);
  }
  // C[row = token (lane/16)*4 + i][col = lane%16]
  reduce_out<NV, NTB>(red, acc, B, [&](int b, int c, const float (&s)[NV]) {
    const bool on = !R.masked || a.mask[(int64_t)b * a.n_groups + g] != 0;
    const float o = on ? (SWIGLU ? silu(s[0]) * s[NV - 1] : s[0]) : 0.f;
    R.out[(int64_t)b * R.ldo + n0 + c] = f32_to_bf16(o);
  });
}

template <int NTB>
__global__ __launch_bounds__(NT) void wide_gemv_k(GVKArgs a) {
  __shared__ float red[NW / 2][kDecodeMaxB][16];
  __shared__ unsigned long long s_act[4096];  // bit b: token b active in group g
  __shared__ uint16_t ulist[4096];
  __shared__ int wc[NW];
  __shared__ int n_union;

  const int tid = threadIdx.x;
  const int B = a.B, K = a.K, G = a.G, ng = a.n_groups;
  const int n0 = blockIdx.x * 16;
  const int w = wave_id(), lane = lane_id();
  for (int i = tid; i < ng; i += NT) s_act[i] = 0ull;
  __syncthreads();
  for (int i = tid; i < B * ng; i += NT)
    if (a.mask[i] != 0) atomicOr(&s_act[i % ng], 1ull << (i / ng));
  if (tid == 0) n_union = 0;
  __syncthreads();
  // Union of the batch's active groups, compacted in ascending order.
  for (int g0 = 0; g0 < ng; g0 += NT) {
    const int gg = g0 + tid;
    const bool on = gg < ng && s_act[gg] != 0ull;
    const uint64_t bal = __ballot(on);
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
  const int spg = G / 64;        // k steps per group
  const int nsteps = nu * spg;   // steps of the union, dealt round-robin to the waves
  const int my_steps = nsteps > w ? (nsteps - w + NW - 1) / NW : 0;

  const int ln = lane & 15, lq = lane >> 4;
  f32x4 acc[1][NTB];
#pragma unroll
  for (int i = 0; i < NTB; ++i) acc[0][i] = f32x4{0.f, 0.f, 0.f, 0.f};
  const uint16_t* wrow = a.w + (int64_t)(n0 + ln) * K + lq * 16;
  const uint16_t* xrow[NTB];
  int tok[NTB];
#pragma unroll
  for (int tb = 0; tb < NTB; ++tb) {
    tok[tb] = tb * 16 + ln;
    xrow[tb] = a.a + (int64_t)(tok[tb] < B ? tok[tb] : 0) * K + lq * 16;
  }

  auto load = [&](int q, StepRegs<1, NTB>& r) {
    const int s = w + q * NW;
    const int g = ulist[s / spg];
    const int k = g * G + (s % spg) * 64;
    const unsigned long long act = s_act[g];
    r.w[0][0] = ldg16(wrow + k);
    r.w[0][1] = ldg16(wrow + k + 8);
#pragma unroll
    for (int tb = 0; tb < NTB; ++tb) {
      const bool on = tok[tb] < B && ((act >> tok[tb]) & 1ull);  // inactive blocks are never read
      r.x[tb][0] = on ? ldg16(xrow[tb] + k) : u32x4{0, 0, 0, 0};
      r.x[tb][1] = on ? ldg16(xrow[tb] + k + 8) : u32x4{0, 0, 0, 0};
    }
  };
  int q = 0;
  for (; q + U <= my_steps; q += U) {
    StepRegs<1, NTB> r[U];
#pragma unroll
    for (int s = 0; s < U; ++s) load(q + s, r[s]);
#pragma unroll
    for (int s = 0; s < U; ++s) step_mfma(r[s], acc);
  }
  for (; q < my_steps; ++q) {
    StepRegs<1, NTB> r;
    load(q, r);
    step_mfma(r, acc);
  }
  reduce_out<1, NTB>(red, acc, B, [&](int b, int c, const float (&s)[1]) {
    a.y[(int64_t)b * a.N + n0 + c] = f32_to_bf16(s[0]);
  });
}

namespace {
template <bool SW>
hipError_t gemv_n_ntb(const GVNArgs& a, int nb, hipStream_t s) {
  const char* name = SW ? "wide_gemv_n<true>" : "wide_gemv_n<false>";
  if (a.B <= 16)
    WIDE_LAUNCH_NAMED(name, (wide_gemv_n<SW, 1>), dim3(nb), dim3(NT), 0, s, a);
  else if (a.B <= 32)
    WIDE_LAUNCH_NAMED(name, (wide_gemv_n<SW, 2>), dim3(nb), dim3(NT), 0, s, a);
  else
    WIDE_LAUNCH_NAMED(name, (wide_gemv_n<SW, 4>), dim3(nb), dim3(NT), 0, s, a);
  return hipGetLastError();
}
}  // namespace

hipError_t launch_gemv_n(const GVNArgs& a, bool swiglu, hipStream_t s) {
  int nb = 0;
  for (int i = 0; i < a.n_regions; ++i) nb += a.reg[i].n_blocks;
  if (nb == 0 || a.B == 0) return hipSuccess;
  return swiglu ? gemv_n_ntb<true>(a, nb, s) : gemv_n_ntb<false>(a, nb, s);
}

hipError_t launch_gemv_k(const GVKArgs& a, hipStream_t s) {
  if (a.B == 0 || a.N == 0) return hipSuccess;
  if (a.B <= 16)
    WIDE_LAUNCH_NAMED("wide_gemv_k", (wide_gemv_k<1>), dim3(a.N / 16), dim3(NT), 0, s, a);
  else if (a.B <= 32)
    WIDE_LAUNCH_NAMED("wide_gemv_k", (wide_gemv_k<2>), dim3(a.N / 16), dim3(NT), 0, s, a);
  else
    WIDE_LAUNCH_NAMED("wide_gemv_k", (wide_gemv_k<4>), dim3(a.N / 16), dim3(NT), 0, s, a);
  return hipGetLastError();
}

}  // namespace wide
