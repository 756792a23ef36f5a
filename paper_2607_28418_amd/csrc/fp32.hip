// fp32 masked projections (vector ALU, no reduced-precision matrix ops).
//
// The fp32 data path keeps every value in fp32 end to end.  Both kernels use
// a 16 x 16 output tile per 256-thread workgroup with 64-wide k slices staged
// in LDS.
//   f32_nproj  out[t, n] = x_t . w[n] for active (t, group of n), else +0
//              (optionally the SwiGLU pair: silu(x_t . w0[n]) * (x_t . w1[n]));
//              a tile whose 16 tokens are all inactive in its group exits
//              after writing +0.  (WIDE Section 3.1, equations (1) and (3).)
//   f32_kproj  y[t, n] = sum over active groups g of t of
//              sum_{k in g} a[t, k] w[n, k]; inactive (t, g) blocks are not
//              read (zero in LDS).  (Section 3.1 equations (2)-(3), the
//              GEMM-K sum of Appendix B.)
#include "common.h"
#include "kernels.h"
#include "launch.h"

namespace wide {

namespace {
constexpr int T = 16, KS = 64;
}

template <bool SWIGLU>
__global__ __launch_bounds__(256) void wide_f32_nproj(F32NArgs a) {
  __shared__ float xs[T][KS + 1];
  __shared__ float w0s[T][KS + 1];
  __shared__ float w1s[SWIGLU ? T : 1][KS + 1];
  const int m_tiles = (int)((a.M + T - 1) / T);
  const int mt = blockIdx.x % m_tiles, nt = blockIdx.x / m_tiles;
  const int64_t t0 = (int64_t)mt * T;
  const int n0 = nt * T;
  const int tid = threadIdx.x, ti = tid / T, ni = tid % T;
  const int64_t t = t0 + ti;
  const int g = n0 / a.G;
  const bool on = t < a.M && (!a.mask || a.mask[t * a.n_groups + g] != 0);
  if (!__syncthreads_or(on)) {
    if (t < a.M) a.out[t * a.ldo + n0 + ni] = 0.f;
    return;
  }
  float s0 = 0.f, s1 = 0.f;
  for (int k0 = 0; k0 < a.K; k0 += KS) {
    for (int i = tid; i < T * KS; i += 256) {
      const int r = i / KS, c = i % KS, k = k0 + c;
      const int64_t tr = t0 + r;
      xs[r][c] = (tr < a.M && k < a.K) ? a.x[tr * a.K + k] : 0.f;
      w0s[r][c] = (k < a.K) ? a.w0[(int64_t)(n0 + r) * a.K + k] : 0.f;
      if (SWIGLU) w1s[r][c] = (k < a.K) ? a.w1[(int64_t)(n0 + r) * a.K + k] : 0.f;
    }
    __syncthreads();
#pragma unroll 8
    for (int c = 0; c < KS; ++c) {
      s0 = fmaf(xs[ti][c], w0s[ni][c], s0);
      if (SWIGLU) s1 = fmaf(xs[ti][c], w1s[ni][c], s1);
    }
    __syncthreads();
  }
  if (t < a.M) {
    const float o = on ? (SWIGLU ? silu(s0) * s1 : s0) : 0.f;
    a.out[t * a.ldo + n0 + ni] = o;
  }
}

__global__ __launch_bounds__(256) void wide_f32_kproj(F32KArgs a) {
  __shared__ float as[T][KS + 1];
  __shared__ float ws[T][KS + 1];
  const int m_tiles = (int)((a.M + T - 1) / T);
  const int mt = blockIdx.x % m_tiles, nt = blockIdx.x / m_tiles;
  const int64_t t0 = (int64_t)mt * T;
  const int n0 = nt * T;
  const int tid = threadIdx.x, ti = tid / T, ni = tid % T;
  float s = 0.f;
  for (int k0 = 0; k0 < a.K; k0 += KS) {
    for (int i = tid; i < T * KS; i += 256) {
      const int r = i / KS, c = i % KS, k = k0 + c;
      const int64_t tr = t0 + r;
      const bool on = tr < a.M && k < a.K && a.mask[tr * a.n_groups + k / a.G] != 0;
      as[r][c] = on ? a.a[tr * a.K + k] : 0.f;
      ws[r][c] = (k < a.K) ? a.w[(int64_t)(n0 + r) * a.K + k] : 0.f;
    }
    __syncthreads();
#pragma unroll 8
    for (int c = 0; c < KS; ++c) s = fmaf(as[ti][c], ws[ni][c], s);
    __syncthreads();
  }
  const int64_t t = t0 + ti;
  if (t < a.M) a.y[t * a.N + n0 + ni] = s;
}

hipError_t launch_f32_nproj(const F32NArgs& a, bool swiglu, hipStream_t s) {
  const int64_t m_tiles = (a.M + T - 1) / T;
  const int64_t total = m_tiles * (a.N / T);
  if (total == 0) return hipSuccess;
  if (swiglu)
    WIDE_LAUNCH((wide_f32_nproj<true>), dim3((unsigned)total), dim3(256), 0, s, a);
  else
    WIDE_LAUNCH((wide_f32_nproj<false>), dim3((unsigned)total), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_f32_kproj(const F32KArgs& a, hipStream_t s) {
  const int64_t m_tiles = (a.M + T - 1) / T;
  const int64_t total = m_tiles * (a.N / T);
  if (total == 0) return hipSuccess;
  WIDE_LAUNCH(wide_f32_kproj, dim3((unsigned)total), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace wide
