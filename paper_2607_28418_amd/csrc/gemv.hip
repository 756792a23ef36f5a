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
// gemv_n  (N-axis: gate/up + SwiGLU, Q; dense K/V).  A workgroup owns 16*NCB
//         output columns of one group; its 8 waves take turns over the
//         64-wide steps of the reduction dimension K.  If no token of the
//         batch is active in the group, the workgroup writes +0 and exits
//         before touching a weight byte.  Otherwise, per 64-wide k step,
//         lane l reads two 16-byte pieces of weight row l%16, at bytes
//         16*(l/16) and 64 + 16*(l/16) of the row's 128-byte line, so each
//         load instruction covers whole 64-byte halves of 16 lines.  The
//         matching activations ride along as the other MFMA operand
//         (16x16x32, tokens as rows) with the same k order, so the sum is
//         unchanged.  Two register sets keep about two steps of NCB blocks in
//         flight per lane.  Inactive (token, group) outputs are +0.
//
// gemv_k  (K-axis: down, O).  A workgroup owns 16*NCB output rows n and a
//         share of the k steps of the union groups (k_split workgroups per row
//         block; their fp32 partial sums are added in a fixed order by a small
//         finishing kernel); its 8 waves take turns over those steps.  For
//         each union group a wave reads the 2G-byte segments w[n, gG:(g+1)G]
//         of its rows and the matching activations of the tokens active in
//         the group (inactive blocks are never read).  The batch's mask sits
//         in LDS as one 64-bit token set per group.  No atomics.
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

// The k loop of a wave is a software pipeline over D register sets and LDS
// slots: the loads of step q+D go out right after step q's MFMAs, so D steps
// stay in flight per lane for the whole loop (loading a few steps and then
// multiplying them drains the memory pipeline at every iteration).

__device__ __host__ __forceinline__ int gv_total_cols(const GVNArgs& a) {
  int n = 0;
  for (int i = 0; i < a.n_regions; ++i) n += a.reg[i].n_blocks * 16;
  return n;
}

// Activations go through LDS.  Loaded straight into MFMA operand registers,
// a 16-token block of one 64-wide k step is 16 rows x 64 bytes per load
// instruction, and such half-line loads cost the vector memory path as much
// as the weight stream itself (measured on MI355X: the down projection at
// B = 32 took 40 us with them, 25 us without).  Instead each wave moves a
// step's activations with whole-line direct-to-LDS loads (8 token rows x 128
// bytes per instruction, lane L landing at byte 16*L: row L/8, physical chunk
// L%8) into a ring of D slots of its own, and reads the fragments back from
// LDS.  Logical chunk c of row r sits at physical chunk c ^ xf(r), so the 16
// rows an MFMA fragment reads at one chunk fall in 16 distinct bank groups.
typedef const void __attribute__((address_space(1)))* gv_gptr;
typedef void __attribute__((address_space(3)))* gv_lptr;
__device__ __attribute__((aligned(16))) uint16_t g_gv_zero[8];  // 16 bytes, stays zero: never written

__device__ __forceinline__ int xf(int r) { return (r & 7) ^ ((r >> 3) & 1); }

// Pipeline depth for weight registers of `reg_dwords` per step and NTB token
// blocks of activations in LDS (8 waves x D slots x 2*NTB KB, at most
// LDS_KB), from 2 to 4.
template <int REG_DWORDS, int NTB, int LDS_KB = 130>
constexpr int gv_depth() {
  constexpr int by_regs = 160 / REG_DWORDS >= 4 ? 4 : 160 / REG_DWORDS >= 3 ? 3 : 2;
  constexpr int by_lds = LDS_KB / (NW * 2 * NTB);
  return by_regs < by_lds ? by_regs : (by_lds < 2 ? 2 : by_lds);
}

// Issue one step's activation loads into ring slot `slot` (2*NTB KB):
// token row r of the slot reads x[r][k0 .. k0+64) when rowok(r), else zeros.
template <int NTB, class RowOk>
__device__ __forceinline__ void x_to_lds(u32x4* slot, const uint16_t* x, int K, int k0, RowOk rowok) {
  const int lane = lane_id();
#pragma unroll
  for (int i = 0; i < 2 * NTB; ++i) {
    const int r = i * 8 + (lane >> 3);
    const int c = (lane & 7) ^ xf(r);
    const uint16_t* src = rowok(r) ? x + (int64_t)r * K + k0 + c * 8 : g_gv_zero;
    __builtin_amdgcn_global_load_lds((gv_gptr)src, (gv_lptr)(slot + i * 64), 16, 0, 0);
  }
}

// Token block tb's operand for half h (k 32h .. 32h+32 of the step): lane
// (ln, lq) holds row tb*16 + ln, logical chunk 4h + lq.
__device__ __forceinline__ u32x4 x_frag(const u32x4* slot, int tb, int h) {
  const int lane = lane_id(), r = tb * 16 + (lane & 15), c = h * 4 + (lane >> 4);
  return slot[(r >> 3) * 64 + ((r & 7) << 3) + (c ^ xf(r))];
}

// Wait until step q's loads (P per step) have landed, given that the steps
// after it up to q + D - 1 (or the last step n - 1) were issued after it.
template <int P, int D>
__device__ __forceinline__ void wait_step_loads(int q, int n) {
  static_assert((D - 1) * P <= 63, "vmcnt range");
  const int younger = min(D - 1, n - 1 - q);
  if (younger >= 3) __builtin_amdgcn_s_waitcnt(((3 * P) & 15) | (((3 * P) >> 4) << 14) | (7 << 4) | (15 << 8));
  else if (younger == 2) __builtin_amdgcn_s_waitcnt(((2 * P) & 15) | (((2 * P) >> 4) << 14) | (7 << 4) | (15 << 8));
  else if (younger == 1) __builtin_amdgcn_s_waitcnt((P & 15) | ((P >> 4) << 14) | (7 << 4) | (15 << 8));
  else __builtin_amdgcn_s_waitcnt((7 << 4) | (15 << 8));
}

}  // namespace

// Sum the k_split partials of every (token, column) in a fixed order, apply
// SwiGLU (gate/up pair) and the mask, store bf16.  A thread takes four
// adjacent columns (the column count is a multiple of 16, so they share a
// row, a region and a group); its k_split loads are all issued before the
// first add.
__device__ __forceinline__ f32x4 ld4f(const float* p) { return *reinterpret_cast<const f32x4*>(p); }
__device__ __forceinline__ void st4bf(uint16_t* p, f32x4 v) {
  const uint32_t lo = (uint32_t)f32_to_bf16(v[0]) | ((uint32_t)f32_to_bf16(v[1]) << 16);
  const uint32_t hi = (uint32_t)f32_to_bf16(v[2]) | ((uint32_t)f32_to_bf16(v[3]) << 16);
  *reinterpret_cast<uint2*>(p) = uint2{lo, hi};
}

template <bool SWIGLU, int KS>
__global__ __launch_bounds__(256) void wide_gemv_n_finish(GVNArgs a) {
  constexpr int NV = SWIGLU ? 2 : 1;
  const int ncols = gv_total_cols(a);
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i >= (int64_t)a.B * ncols) return;
  const int b = (int)(i / ncols);
  int col = (int)(i % ncols);
  GVRegion R = a.reg[0];
  if (a.n_regions > 1 && col >= a.reg[1].col0) R = a.reg[1];
  if (a.n_regions > 2 && col >= a.reg[2].col0) R = a.reg[2];
  const int lc = col - R.col0;
  const bool on = !R.masked || a.mask[(int64_t)b * a.n_groups + lc / a.G] != 0;
  f32x4 o = f32x4{0.f, 0.f, 0.f, 0.f};
  if (on) {
    f32x4 p[NV][KS];
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int q = 0; q < KS; ++q) p[v][q] = ld4f(a.part + (((int64_t)q * NV + v) * a.B + b) * ncols + col);
    f32x4 s[NV];
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      s[v] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int q = 0; q < KS; ++q) s[v] += p[v][q];
    }
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = SWIGLU ? silu(s[0][e]) * s[NV - 1][e] : s[0][e];
  }
  st4bf(R.out + (int64_t)b * R.ldo + lc, o);
}

template <bool SWIGLU, int NTB, int NCB>
__global__ __launch_bounds__(NT) void wide_gemv_n(GVNArgs a) {
  constexpr int NV = SWIGLU ? 2 : 1;
  constexpr int REG = NCB * NV * 2 * 4;        // weight dwords per step per lane
  constexpr int D = gv_depth<REG, NTB>();
  constexpr int P = NCB * NV * 2 + 2 * NTB;    // vector-memory instructions per step
  constexpr int RING = NW * D * 2 * NTB * 64;  // u32x4 of the activation rings
  constexpr int RED = NW / 2 * NV * kDecodeMaxB * 16;  // floats of the wave reduction
  // the reduction reuses the rings' bytes once the k loop is done
  __shared__ __attribute__((aligned(16))) u32x4 lds[RING > RED / 4 ? RING : RED / 4];
  float (*red)[kDecodeMaxB][16] = reinterpret_cast<float (*)[kDecodeMaxB][16]>(lds);
  __shared__ int any_active;
  __shared__ uint8_t s_on[kDecodeMaxB];  // token b runs group g (read once, used by the epilogue)

  const int kq = blockIdx.x % a.k_split;  // this workgroup's share of the k steps
  int nb = blockIdx.x / a.k_split;
  GVRegion R = a.reg[0];
  if (a.n_regions > 1 && nb >= a.reg[0].n_blocks / NCB) {
    nb -= a.reg[0].n_blocks / NCB;
    R = a.reg[1];
    if (a.n_regions > 2 && nb >= a.reg[1].n_blocks / NCB) {
      nb -= a.reg[1].n_blocks / NCB;
      R = a.reg[2];
    }
  }
  const int n0 = nb * 16 * NCB;  // the NCB blocks lie in one group (16*NCB divides G)
  const int g = n0 / a.G;
  const int tid = threadIdx.x;
  const int B = a.B, K = a.K;

  if (tid == 0) any_active = R.masked ? 0 : 1;
  __syncthreads();
  if (tid < B) {
    const bool on = !R.masked || a.mask[(int64_t)tid * a.n_groups + g] != 0;
    s_on[tid] = on;
    if (on && R.masked) any_active = 1;
  }
  __syncthreads();
  if (!any_active) {
    // group unused by the whole batch: no weight reads, outputs +0 (with a
    // k split the finishing kernel writes them)
    if (a.k_split > 1) return;
    for (int i = tid; i < B * 2 * NCB; i += NT) {
      const int b = i / (2 * NCB), h = i % (2 * NCB);
      stg16(R.out + (int64_t)b * R.ldo + n0 + h * 8, u32x4{0, 0, 0, 0});
    }
    return;
  }

  const int w = wave_id(), lane = lane_id();
  const int ln = lane & 15, lq = lane >> 4;
  // This workgroup's share of the K/64 steps, dealt round-robin to the 8 waves.
  const int all_steps = K / 64;
  const int s_beg = (int)((int64_t)all_steps * kq / a.k_split);
  const int nsteps = (int)((int64_t)all_steps * (kq + 1) / a.k_split) - s_beg;
  const int my_steps = nsteps > w ? (nsteps - w + NW - 1) / NW : 0;
  // Weights: a workgroup-uniform part plus one per-lane offset (row ln of a
  // block of 16, piece lq), raw buffer loads with the uniform part in a
  // scalar register.
  const uint32_t loff = (uint32_t)(ln * K + lq * 8) * 2u;
  const uint32_t slab = (uint32_t)(16 * NCB) * (uint32_t)K * 2u;
  bufview_t wv[NV];
  wv[0] = buf_view(R.w0 + (int64_t)n0 * K, slab);
  if (SWIGLU) wv[NV - 1] = buf_view(R.w1 + (int64_t)n0 * K, slab);
  u32x4* ring = lds + w * (D * 2 * NTB * 64);

  f32x4 acc[NCB][NV][NTB];
#pragma unroll
  for (int c = 0; c < NCB; ++c)
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int i = 0; i < NTB; ++i) acc[c][v][i] = f32x4{0.f, 0.f, 0.f, 0.f};

  struct Regs {
    u32x4 w[NCB][NV][2];
  };
  auto load = [&](int q, int slot, Regs& r) {
    const int k = (s_beg + w + q * NW) * 64;
#pragma unroll
    for (int c = 0; c < NCB; ++c)
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        r.w[c][v][0] = buf_ld16s(wv[v], loff, (uint32_t)(c * 16 * K + k) * 2u);
        r.w[c][v][1] = buf_ld16s(wv[v], loff, (uint32_t)(c * 16 * K + k + 32) * 2u);
      }
    x_to_lds<NTB>(ring + slot * (2 * NTB * 64), a.x, K, k, [&](int row) { return row < B; });
  };
  auto mma = [&](int q, int slot, const Regs& r) {
    wait_step_loads<P, D>(q, my_steps);
    const u32x4* sl = ring + slot * (2 * NTB * 64);
    u32x4 xr[NTB][2];
#pragma unroll
    for (int tb = 0; tb < NTB; ++tb) {
      xr[tb][0] = x_frag(sl, tb, 0);
      xr[tb][1] = x_frag(sl, tb, 1);
    }
#pragma unroll
    for (int tb = 0; tb < NTB; ++tb)
#pragma unroll
      for (int c = 0; c < NCB; ++c)
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          acc[c][v][tb] = mfma16(xr[tb][0], r.w[c][v][0], acc[c][v][tb]);
          acc[c][v][tb] = mfma16(xr[tb][1], r.w[c][v][1], acc[c][v][tb]);
        }
    asm volatile("" ::: "memory");  // the slot's reads stay ahead of its next loads
  };
  Regs rr[D];
#pragma unroll
  for (int j = 0; j < D; ++j)
    if (j < my_steps) load(j, j, rr[j]);
  for (int q = 0; q < my_steps; q += D) {
#pragma unroll
    for (int j = 0; j < D; ++j) {
      if (q + j < my_steps) {
        mma(q + j, j, rr[j]);
        if (q + j + D < my_steps) load(q + j + D, j, rr[j]);
      }
    }
  }
  __syncthreads();  // the reduction below reuses the rings' LDS
  // C[row = token (lane/16)*4 + i][col = lane%16], one column block at a time
#pragma unroll
  for (int c = 0; c < NCB; ++c) {
    reduce_out<NV, NTB>(red, acc[c], B, [&](int b, int cc, const float (&sm)[NV]) {
      if (a.k_split > 1) {  // fp32 partials, finished by wide_gemv_n_finish
        const int ncols = gv_total_cols(a);
#pragma unroll
        for (int v = 0; v < NV; ++v)
          a.part[(((int64_t)kq * NV + v) * B + b) * ncols + R.col0 + n0 + c * 16 + cc] = sm[v];
        return;
      }
      const bool on = s_on[b] != 0;
      const float o = on ? (SWIGLU ? silu(sm[0]) * sm[NV - 1] : sm[0]) : 0.f;
      R.out[(int64_t)b * R.ldo + n0 + c * 16 + cc] = f32_to_bf16(o);
    });
    __syncthreads();
  }
}

template <int NTB, int NCB>
__global__ __launch_bounds__(NT) void wide_gemv_k(GVKArgs a) {
  // Up to 32 tokens the activations go through per-wave LDS rings (see
  // x_to_lds); at 33..64 tokens the rings would not fit beside the group
  // tables, and the activations load straight into registers.
  constexpr bool XLDS = NTB <= 2;
  constexpr int REG = XLDS ? NCB * 2 * 4 : (NCB * 2 + NTB * 2) * 4;  // staged dwords per step
  constexpr int D = XLDS ? gv_depth<REG, NTB, 96>() : (160 / REG >= 4 ? 4 : 160 / REG >= 3 ? 3 : 2);
  constexpr int P = NCB * 2 + 2 * NTB;  // vector-memory instructions per step
  __shared__ __attribute__((aligned(16))) u32x4 xring[XLDS ? NW * D * 2 * NTB * 64 : 1];
  __shared__ float red[NW / 2][kDecodeMaxB][16];
  __shared__ unsigned long long s_act[4096];  // bit b: token b active in group g
  __shared__ uint16_t ulist[4096];
  __shared__ int wc[NW];
  __shared__ int n_union;

  const int tid = threadIdx.x;
  const int B = a.B, K = a.K, G = a.G, ng = a.n_groups;
  const int kq = blockIdx.x % a.k_split;            // this workgroup's share of the union steps
  const int n0 = (blockIdx.x / a.k_split) * 16 * NCB;
  const int w = wave_id(), lane = lane_id();
  // Token sets per group: lane b of a wave reads token b's mask bytes of
  // the wave's groups (every eighth), and one ballot per group collects
  // them.  (Groups narrower than 64 arrive merged: a.merge mask columns per
  // group of G; the inactive ones inside an active merged group hold exact
  // zeros.)
  const int rng = ng * a.merge;
  {
    constexpr int GB = 16;  // groups per wave whose loads are in flight together
    for (int g0 = w; g0 < ng; g0 += NW * GB) {
      uint32_t v[GB];
#pragma unroll
      for (int j = 0; j < GB; ++j) {
        const int g = g0 + j * NW;
        v[j] = 0;
        if (lane < B && g < ng)
          for (int m = 0; m < a.merge; ++m) v[j] |= a.mask[(int64_t)lane * rng + g * a.merge + m];
      }
#pragma unroll
      for (int j = 0; j < GB; ++j) {
        const uint64_t bal = __ballot(v[j] != 0);
        if (lane == 0 && g0 + j * NW < ng) s_act[g0 + j * NW] = bal;
      }
    }
  }
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
  const int spg = G / 64;  // k steps per group
  const int all_steps = nu * spg;
  const int s_beg = (int)((int64_t)all_steps * kq / a.k_split);
  const int s_end = (int)((int64_t)all_steps * (kq + 1) / a.k_split);
  const int nsteps = s_end - s_beg;  // dealt round-robin to the waves
  const int my_steps = nsteps > w ? (nsteps - w + NW - 1) / NW : 0;

  const int ln = lane & 15, lq = lane >> 4;
  f32x4 acc[NCB][NTB];
#pragma unroll
  for (int c = 0; c < NCB; ++c)
#pragma unroll
    for (int i = 0; i < NTB; ++i) acc[c][i] = f32x4{0.f, 0.f, 0.f, 0.f};
  // workgroup-uniform bases plus one per-lane offset shared by weights and
  // (in registers) activations, both of row stride K
  const uint32_t loff = (uint32_t)(ln * K + lq * 8) * 2u;
  const bufview_t wv = buf_view(a.w + (int64_t)n0 * K, (uint32_t)(16 * NCB) * (uint32_t)K * 2u);
  const bufview_t xv = buf_view(a.a, (uint32_t)B * (uint32_t)K * 2u);
  u32x4* ring = xring + (XLDS ? w * (D * 2 * NTB * 64) : 0);

  struct Regs {
    u32x4 w[NCB][2];
    u32x4 x[XLDS ? 1 : NTB][2];
  };
  auto load = [&](int q, int slot, Regs& r) {
    const int s = s_beg + w + q * NW;
    const int g = ulist[s / spg];
    const int k = g * G + (s % spg) * 64;
    const unsigned long long act = s_act[g];
#pragma unroll
    for (int c = 0; c < NCB; ++c) {
      r.w[c][0] = buf_ld16s(wv, loff, (uint32_t)(c * 16 * K + k) * 2u);
      r.w[c][1] = buf_ld16s(wv, loff, (uint32_t)(c * 16 * K + k + 32) * 2u);
    }
    // inactive (token, group) blocks are never read: they load zeros
    if constexpr (XLDS) {
      x_to_lds<NTB>(ring + slot * (2 * NTB * 64), a.a, K, k,
                    [&](int row) { return row < B && ((act >> row) & 1ull); });
    } else {
#pragma unroll
      for (int tb = 0; tb < NTB; ++tb) {
        const int tok = tb * 16 + ln;
        const bool on = tok < B && ((act >> tok) & 1ull);
        const uint32_t o = (uint32_t)(tb * 16 * K + k) * 2u + loff;
        r.x[tb][0] = buf_ld16(xv, on ? o : kOffNone);
        r.x[tb][1] = buf_ld16(xv, on ? o + 64u : kOffNone);
      }
    }
  };
  auto mma = [&](int q, int slot, const Regs& r) {
    u32x4 xr[NTB][2];
    if constexpr (XLDS) {
      wait_step_loads<P, D>(q, my_steps);
      const u32x4* sl = ring + slot * (2 * NTB * 64);
#pragma unroll
      for (int tb = 0; tb < NTB; ++tb) {
        xr[tb][0] = x_frag(sl, tb, 0);
        xr[tb][1] = x_frag(sl, tb, 1);
      }
    } else {
#pragma unroll
      for (int tb = 0; tb < NTB; ++tb) {
        xr[tb][0] = r.x[XLDS ? 0 : tb][0];
        xr[tb][1] = r.x[XLDS ? 0 : tb][1];
      }
    }
#pragma unroll
    for (int tb = 0; tb < NTB; ++tb)
#pragma unroll
      for (int c = 0; c < NCB; ++c) {
        acc[c][tb] = mfma16(xr[tb][0], r.w[c][0], acc[c][tb]);
        acc[c][tb] = mfma16(xr[tb][1], r.w[c][1], acc[c][tb]);
      }
    asm volatile("" ::: "memory");  // the slot's reads stay ahead of its next loads
  };
  Regs rr[D];
#pragma unroll
  for (int j = 0; j < D; ++j)
    if (j < my_steps) load(j, j, rr[j]);
  for (int q = 0; q < my_steps; q += D) {
#pragma unroll
    for (int j = 0; j < D; ++j) {
      if (q + j < my_steps) {
        mma(q + j, j, rr[j]);
        if (q + j + D < my_steps) load(q + j + D, j, rr[j]);
      }
    }
  }
#pragma unroll
  for (int c = 0; c < NCB; ++c) {
    f32x4 one[1][NTB];
#pragma unroll
    for (int tb = 0; tb < NTB; ++tb) one[0][tb] = acc[c][tb];
    reduce_out<1, NTB>(red, one, B, [&](int b, int cc, const float (&sm)[1]) {
      const int64_t o = (int64_t)b * a.N + n0 + c * 16 + cc;
      if (a.k_split == 1)
        a.y[o] = f32_to_bf16(sm[0]);
      else
        a.part[(int64_t)kq * B * a.N + o] = sm[0];  // summed in fixed order by gemv_k_finish
    });
    __syncthreads();
  }
}

// y = bf16(sum over the k_split partial sums), in a fixed order; four
// adjacent outputs per thread (n is a multiple of 16).
template <int KS>
__global__ __launch_bounds__(256) void wide_gemv_k_finish(const float* __restrict__ part, int64_t n,
                                                          uint16_t* __restrict__ y) {
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i >= n) return;
  f32x4 p[KS];
#pragma unroll
  for (int q = 0; q < KS; ++q) p[q] = ld4f(part + (int64_t)q * n + i);
  f32x4 s = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int q = 0; q < KS; ++q) s += p[q];
  st4bf(y + i, s);
}

namespace {
// Timing labels name the variant: "wide_gemv_n<true>/ntb2_ncb4" is
// wide_gemv_n<true, 2, 4> (queries of "wide_gemv_n<true>" cover them all).
constexpr int ncb_index(int ncb) { return ncb == 1 ? 0 : ncb == 2 ? 1 : ncb == 4 ? 2 : 3; }
constexpr int ntb_index(int ntb) { return ntb == 1 ? 0 : ntb == 2 ? 1 : 2; }
#define WIDE_GV_ROW(BASE, NTB) {BASE "/ntb" #NTB "_ncb1", BASE "/ntb" #NTB "_ncb2", BASE "/ntb" #NTB "_ncb4", BASE "/ntb" #NTB "_ncb8"}
#define WIDE_GV_TABLE(BASE) {WIDE_GV_ROW(BASE, 1), WIDE_GV_ROW(BASE, 2), WIDE_GV_ROW(BASE, 4)}
constexpr const char* kGemvNLabels[2][3][4] = {WIDE_GV_TABLE("wide_gemv_n<false>"), WIDE_GV_TABLE("wide_gemv_n<true>")};
constexpr const char* kGemvKLabels[3][4] = WIDE_GV_TABLE("wide_gemv_k");
#undef WIDE_GV_TABLE
#undef WIDE_GV_ROW

template <bool SW, int NTB, int NCB>
constexpr const char* gemv_n_label() { return kGemvNLabels[SW ? 1 : 0][ntb_index(NTB)][ncb_index(NCB)]; }
template <int NTB, int NCB>
constexpr const char* gemv_k_label() { return kGemvKLabels[ntb_index(NTB)][ncb_index(NCB)]; }

template <bool SW, int NCB>
hipError_t gemv_n_launch(const GVNArgs& a, int nb, hipStream_t s) {
  const int grid = nb / NCB * a.k_split;
  if constexpr (SW && NCB == 8)
    return hipErrorInvalidValue;  // not instantiated: gemv_n_ncb never picks it
  else if (a.B <= 16)
    WIDE_LAUNCH_NAMED((gemv_n_label<SW, 1, NCB>()), (wide_gemv_n<SW, 1, NCB>), dim3(grid), dim3(NT), 0, s, a);
  else if (a.B <= 32)
    WIDE_LAUNCH_NAMED((gemv_n_label<SW, 2, NCB>()), (wide_gemv_n<SW, 2, NCB>), dim3(grid), dim3(NT), 0, s, a);
  else if constexpr ((SW && NCB == 4) || NCB == 8)
    return hipErrorInvalidValue;  // not instantiated: gemv_n_ncb never picks it
  else
    WIDE_LAUNCH_NAMED((gemv_n_label<SW, 4, NCB>()), (wide_gemv_n<SW, 4, NCB>), dim3(grid), dim3(NT), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.k_split == 1) return e;
  const int64_t n = (int64_t)a.B * gv_total_cols(a) / 4;  // four columns per thread
  const dim3 fg((unsigned)((n + 255) / 256));
  if (a.k_split == 2)
    WIDE_LAUNCH_NAMED("wide_gemv_n_finish", (wide_gemv_n_finish<SW, 2>), fg, dim3(256), 0, s, a);
  else if (a.k_split == 4)
    WIDE_LAUNCH_NAMED("wide_gemv_n_finish", (wide_gemv_n_finish<SW, 4>), fg, dim3(256), 0, s, a);
  else if (a.k_split == 8)
    WIDE_LAUNCH_NAMED("wide_gemv_n_finish", (wide_gemv_n_finish<SW, 8>), fg, dim3(256), 0, s, a);
  else
    return hipErrorInvalidValue;  // the split is a power of two up to 8
  return hipGetLastError();
}

template <int NCB>
hipError_t gemv_k_launch(const GVKArgs& a, hipStream_t s) {
  const int grid = a.N / (16 * NCB) * a.k_split;
  if (a.B <= 16)
    WIDE_LAUNCH_NAMED((gemv_k_label<1, NCB>()), (wide_gemv_k<1, NCB>), dim3(grid), dim3(NT), 0, s, a);
  else if (a.B <= 32)
    WIDE_LAUNCH_NAMED((gemv_k_label<2, NCB>()), (wide_gemv_k<2, NCB>), dim3(grid), dim3(NT), 0, s, a);
  else if constexpr (NCB == 8)
    return hipErrorInvalidValue;  // not instantiated: gemv_k_ncb never picks it
  else
    WIDE_LAUNCH_NAMED((gemv_k_label<4, NCB>()), (wide_gemv_k<4, NCB>), dim3(grid), dim3(NT), 0, s, a);
  return hipGetLastError();
}
}  // namespace

DecodeTuning& decode_tuning() {
  static DecodeTuning t{0, 0, 0, 0};
  return t;
}

// Column blocks per workgroup: the most (4, 2 or 1) that divide every region
// into runs inside one group and still leave at least 160 runs, so that the
// chip is busy without a k split.  Measured on MI355X (Llama-3-8B and
// Llama-7B projections, weights read from HBM): at 17..64 tokens 64 columns
// per workgroup ran gate/up fastest even at 224 workgroups (activation
// re-reads fall with the run width), and Q/K/V at 32 columns and no split
// beat 64 columns with a split plus its finishing kernel.  With fewer tokens
// 16 columns per workgroup ran fastest -- gate/up up to 8 tokens (0-25%
// faster; at 16 tokens 3% slower on the Llama-3-8B shape), Q/K/V up to 16
// tokens (2-7%): the activations of one token block cost little, and narrow
// workgroups spread the active ones over more CUs.
int gemv_n_ncb(const GVNArgs& a) {
  const int forced = decode_tuning().n_ncb;
  if (!forced && a.B <= (a.swiglu ? 8 : 16)) return 1;
  int nb = 0;
  for (int i = 0; i < a.n_regions; ++i) nb += a.reg[i].n_blocks;
  for (int ncb : {8, 4, 2}) {
    if (forced ? ncb > forced : ncb == 8) continue;
    // eight blocks only for plain columns and up to 32 tokens; gate/up at
    // more than 32 tokens: four blocks would not fit the registers
    if (ncb == 8 && (a.swiglu || a.B > 32)) continue;
    if (ncb == 4 && a.swiglu && a.B > 32) continue;
    if ((a.G / 16) % ncb) continue;
    bool ok = true;
    for (int i = 0; i < a.n_regions; ++i) ok = ok && a.reg[i].n_blocks % ncb == 0;
    if (ok && (forced || nb / ncb >= 160)) return ncb;
  }
  return 1;
}

// Split of the k steps over workgroups.  A split costs a finishing kernel
// (about 4.5 us on MI355X inside a graph), which only pays when the column
// runs alone leave most CUs idle: split (at most 8 ways, at least 4 k steps
// per share) until there are 160 workgroups.
int gemv_n_split(const GVNArgs& a) {
  int nb = 0;
  for (int i = 0; i < a.n_regions; ++i) nb += a.reg[i].n_blocks;
  const int runs = nb / gemv_n_ncb(a);
  int ks = 1;
  const int forced = decode_tuning().n_split;
  if (forced) {
    while (ks < forced && a.K / 64 / (2 * ks) >= 1) ks *= 2;
    return ks;
  }
  while (runs * ks < 160 && ks < 8 && a.K / 64 / (2 * ks) >= 4) ks *= 2;
  return ks;
}

namespace {
// A long reduction (at least 128 k steps, as in a down projection) at more
// than 16 tokens: 64 rows per workgroup and a 4-way split.  Each workgroup
// then re-reads the activations once per 64 weight rows rather than per 16,
// and at 17..64 tokens that saved more than the finishing kernel costs
// (MI355X, Llama-3-8B and Llama-7B down at 32 and 64 tokens: 2..8%).  Short
// reductions (the O projection) do not win it back.
bool gemv_k_wide_rows(int N, int B, int K) {
  return B > 16 && K / 64 >= 128 && N % 64 == 0 && N / 64 * 4 >= 192;
}
}  // namespace

// Output rows per workgroup (16 * ncb): one block, unless that leaves fewer
// than 192 workgroups (or the long-reduction rule above applies).
int gemv_k_ncb(int N, int B, int K) {
  const int forced = decode_tuning().k_ncb;
  if (forced) {
    for (int ncb : {8, 4, 2})  // (eight blocks: up to 32 tokens)
      if (ncb <= forced && N % (16 * ncb) == 0 && (ncb < 8 || B <= 32)) return ncb;
    return 1;
  }
  if (gemv_k_wide_rows(N, B, K)) return 4;
  if (N / 16 >= 192) return 1;
  for (int ncb : {4, 2})
    if (N % (16 * ncb) == 0) return ncb;
  return 1;
}

// Split the union steps until there are 192 workgroups (at most 8 ways).
int gemv_k_split(int N, int B, int K) {
  const int forced = decode_tuning().k_split;
  if (forced) return forced;
  if (!decode_tuning().k_ncb && gemv_k_wide_rows(N, B, K)) return 4;
  const int row_blocks = N / (16 * gemv_k_ncb(N, B, K));
  int ks = 1;
  while (row_blocks * ks < 192 && ks < 8) ks *= 2;
  return ks;
}

size_t gemv_n_part_floats(const GVNArgs& a, bool swiglu) {
  const int ks = gemv_n_split(a);
  return ks > 1 ? (size_t)ks * (swiglu ? 2 : 1) * a.B * gv_total_cols(a) : 0;
}

hipError_t launch_gemv_n(const GVNArgs& a, bool swiglu, hipStream_t s) {
  int nb = 0;
  for (int i = 0; i < a.n_regions; ++i) nb += a.reg[i].n_blocks;
  if (nb == 0 || a.B == 0) return hipSuccess;
  const int ncb = gemv_n_ncb(a);
  if (swiglu)
    return ncb == 4 ? gemv_n_launch<true, 4>(a, nb, s)
                    : ncb == 2 ? gemv_n_launch<true, 2>(a, nb, s) : gemv_n_launch<true, 1>(a, nb, s);
  return ncb == 8   ? gemv_n_launch<false, 8>(a, nb, s)
         : ncb == 4 ? gemv_n_launch<false, 4>(a, nb, s)
         : ncb == 2 ? gemv_n_launch<false, 2>(a, nb, s)
                    : gemv_n_launch<false, 1>(a, nb, s);
}

hipError_t launch_gemv_k(const GVKArgs& a, hipStream_t s) {
  if (a.B == 0 || a.N == 0) return hipSuccess;
  // 16 * gemv_k_ncb output rows per workgroup, the union steps split over
  // k_split workgroups (chosen by the host, partials in a.part).
  const int ncb = gemv_k_ncb(a.N, a.B, a.K);
  hipError_t e = ncb == 8   ? gemv_k_launch<8>(a, s)
                 : ncb == 4 ? gemv_k_launch<4>(a, s)
                 : ncb == 2 ? gemv_k_launch<2>(a, s)
                            : gemv_k_launch<1>(a, s);
  if (e != hipSuccess || a.k_split == 1) return e;
  const int64_t n = (int64_t)a.B * a.N;
  const dim3 fg((unsigned)((n / 4 + 255) / 256));
  if (a.k_split == 2)
    WIDE_LAUNCH_NAMED("wide_gemv_k_finish", (wide_gemv_k_finish<2>), fg, dim3(256), 0, s, a.part, n, a.y);
  else if (a.k_split == 4)
    WIDE_LAUNCH_NAMED("wide_gemv_k_finish", (wide_gemv_k_finish<4>), fg, dim3(256), 0, s, a.part, n, a.y);
  else if (a.k_split == 8)
    WIDE_LAUNCH_NAMED("wide_gemv_k_finish", (wide_gemv_k_finish<8>), fg, dim3(256), 0, s, a.part, n, a.y);
  else
    return hipErrorInvalidValue;  // the split is a power of two up to 8
  return hipGetLastError();
}

}  // namespace wide
