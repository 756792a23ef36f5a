// C ABI of libwide: argument validation, workspace layout, dispatch.
//
// Every check runs on the host before anything is enqueued; on failure the
// call returns a status and leaves all outputs untouched.  Nothing here
// allocates device memory or synchronises with the device (timing queries
// excepted, which are measurement-only).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "wide.h"
#include "kernels.h"

namespace {

thread_local std::string g_last_error;

wide_status_t fail(wide_status_t st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

wide_status_t ok() {
  g_last_error.clear();
  return WIDE_OK;
}

wide_status_t hip_fail(hipError_t e, const char* where) {
  return fail(WIDE_ERR_HIP, "%s: %s", where, hipGetErrorString(e));
}

// ---- tunables (wide_set_option) ---------------------------------------------
// Process-wide; atomics so that a setting made on one host thread is read
// whole on another (a call still reads them at several points, so settings
// are meant to change between calls, not during them).
std::atomic<int64_t> g_decode_max_m{64};  // M <= this uses the decode (GEMV) kernels
std::atomic<int> g_k_path{0};             // 0 auto, 1 dense-masked, 2 scatter
std::atomic<int> g_big_tiles{1};          // 1: 256x256 tile kernels where the shape allows
std::atomic<int> g_mn_tail{1};            // 1: 256-tile N-axis launches split each XCD's last partial round along k
std::atomic<int> g_mn_order{7};           // bit 0: Q/K/V launch K and V before Q; bit 1: full tiles before partial ones;
                                          // bit 2: gate/up tiles m-tile by m-tile over each XCD's groups
std::atomic<int> g_kd_pattern{1};         // 1: dense-masked K axis reads rows in mask-pattern order (<= 8 groups)
std::atomic<int> g_ks_pack{1};            // scatter K axis (256 tiles): K-groups per workgroup

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool is_pow2(int64_t v) { return v > 0 && (v & (v - 1)) == 0; }

constexpr size_t kAlign = 256;
size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// Bump allocator over the caller's workspace.
struct Carve {
  char* base;
  size_t off = 0;
  explicit Carve(void* b) : base(static_cast<char*>(b)) {}
  template <class T>
  T* take(size_t count) {
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += align_up(count * sizeof(T));
    return p;
  }
};

bool use_decode(wide_dtype_t dt, int64_t M) {
  return dt == WIDE_BF16 && M <= g_decode_max_m && M <= wide::kDecodeMaxB;
}

int k_path_for(int G) {
  const int kp = g_k_path;
  if (kp == 1 || kp == 2) return kp;
  // fp32 atomics ran at ~1 TB/s on MI355X, which makes the scatter schedule
  // slower than the dense-masked one unless G is very large.
  return G >= 2048 ? 2 : 1;
}

// With one group (G = K, the M-axis case) the K axis runs as a row-gathered
// N-axis GEMM over the whole output width; it needs the reorder.
bool kaxis_row_gathered(int K, int N, int G) {
  return G == K && g_big_tiles && N % wide::kT256 == 0 && K % 64 == 0;
}

// Workspace pieces of a prefill reorder held internally.
struct ReorderWS {
  int32_t* idx = nullptr;
  int32_t* cnt = nullptr;
  int32_t* chunk_cnt = nullptr;
  int32_t* chunk_off = nullptr;
};

void carve_reorder(Carve& c, int64_t M, int ng, bool need_idx, ReorderWS& r) {
  if (need_idx) {
    r.idx = c.take<int32_t>((size_t)ng * (size_t)M);
    r.cnt = c.take<int32_t>((size_t)ng);
  }
  const size_t sc = std::max<size_t>(wide::reorder_scratch_ints(M, ng), 1);
  r.chunk_cnt = c.take<int32_t>(sc);
  r.chunk_off = c.take<int32_t>(sc);
}

// K-axis scratch (fp32 accumulation or per-tile group union), worst case of
// both schedules when `path` is 0.
struct KWS {
  float* acc32 = nullptr;
  uint8_t* tu = nullptr;
  int32_t* perm = nullptr;  // tokens ordered by mask pattern (dense-masked, few groups)
  int32_t* pat = nullptr;   // scratch of that ordering
};

// The dense-masked 256-tile schedule reads its rows in mask-pattern order
// when there are few groups (2..8): tiles then skip the groups none of their
// rows uses.
bool kaxis_pattern_order(int N, int ng, int path) {
  return g_kd_pattern && path != 2 && ng > 1 && ng <= wide::kPatternMaxGroups && g_big_tiles &&
         N % wide::kT256 == 0;
}

void carve_kaxis(Carve& c, int64_t M, int N, int ng, int path, KWS& k) {
  if (ng == 1 && g_big_tiles && N % wide::kT256 == 0) return;  // row-gathered single group: no scratch
  if (path == 0 || path == 2) k.acc32 = c.take<float>((size_t)M * (size_t)N);
  if (path == 0 || path == 1) k.tu = c.take<uint8_t>(wide::tile_union_bytes(M, ng));
  if (kaxis_pattern_order(N, ng, path)) {
    k.perm = c.take<int32_t>((size_t)M);
    k.pat = c.take<int32_t>(wide::pattern_scratch_ints(M));
  }
}

// ---- argument checks ----------------------------------------------------------
wide_status_t check_ptr(const void* p, const char* name, bool need16 = true) {
  if (!p) return fail(WIDE_ERR_INVALID_ARG, "%s is NULL", name);
  if (need16 && !aligned16(p)) return fail(WIDE_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
  return WIDE_OK;
}

#define CHECK(expr)                          \
  do {                                       \
    wide_status_t st_ = (expr);              \
    if (st_ != WIDE_OK) return st_;          \
  } while (0)

wide_status_t check_ws(void* ws, size_t ws_bytes, size_t need) {
  if (need == 0) return WIDE_OK;
  if (!ws) return fail(WIDE_ERR_WORKSPACE, "workspace is NULL but %zu bytes are needed", need);
  if (reinterpret_cast<uintptr_t>(ws) % kAlign)
    return fail(WIDE_ERR_INVALID_ARG, "workspace is not 256-byte aligned");
  if (ws_bytes < need)
    return fail(WIDE_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, need);
  return WIDE_OK;
}

wide_status_t check_common(wide_dtype_t dt, int64_t M) {
  if (dt != WIDE_F32 && dt != WIDE_BF16) return fail(WIDE_ERR_INVALID_ARG, "unknown dtype %d", (int)dt);
  if (M < 0 || M >= (int64_t(1) << 31)) return fail(WIDE_ERR_INVALID_ARG, "M=%lld out of range", (long long)M);
  return WIDE_OK;
}


// Decode-path argument blocks (pointers may be null when only sizes are needed).
wide::GVNArgs ffn_gvn(int64_t M, int D, int Dff, int G, const uint8_t* mask, const void* x, const void* wg,
                      const void* wu, uint16_t* h) {
  wide::GVNArgs na{};
  na.x = static_cast<const uint16_t*>(x);
  na.mask = mask;
  na.B = (int)M;
  na.K = D;
  na.G = G;
  na.n_groups = Dff / G;
  na.n_regions = 1;
  na.reg[0] = wide::GVRegion{static_cast<const uint16_t*>(wg), static_cast<const uint16_t*>(wu), h, Dff,
                             Dff / 16, 1, 0};
  na.swiglu = 1;
  na.k_split = wide::gemv_n_split(na);
  return na;
}

// ---- FFN -------------------------------------------------------------------------
wide_status_t ffn_shape(wide_dtype_t dt, int64_t M, int D, int Dff, int G) {
  CHECK(check_common(dt, M));
  if (D <= 0 || Dff <= 0) return fail(WIDE_ERR_INVALID_ARG, "d_model and d_ff must be positive");
  // G = d_ff is one group for the whole FFN (the M-axis case, App. A: a
  // token runs the FFN or skips it); otherwise G is in {2^k, k >= 4}.
  if ((!is_pow2(G) || G < 16) && G != Dff)
    return fail(WIDE_ERR_INVALID_ARG, "group_size=%d must be a power of two >= 16 (or d_ff)", G);
  if (Dff % G) return fail(WIDE_ERR_INVALID_ARG, "group_size=%d does not divide d_ff=%d", G, Dff);
  if (D % 8 || Dff % 8) return fail(WIDE_ERR_INVALID_ARG, "d_model and d_ff must be multiples of 8");
  if (Dff / G > 4096) return fail(WIDE_ERR_UNSUPPORTED, "more than 4096 groups");
  if (dt == WIDE_F32) {
    if (D % 16 || Dff % 16) return fail(WIDE_ERR_UNSUPPORTED, "fp32 path needs d_model, d_ff multiples of 16");
  } else {
    if (D % 256) return fail(WIDE_ERR_UNSUPPORTED, "bf16 path needs d_model %% 256 == 0 (got %d)", D);
    if (G < wide::kKMergeWidth && (Dff % 128 || Dff / wide::kKMergeWidth > wide::kKd256MaxGroups))
      return fail(WIDE_ERR_UNSUPPORTED, "bf16 path with group_size < 64 needs d_ff %% 128 == 0 and d_ff <= %d",
                  wide::kKd256MaxGroups * wide::kKMergeWidth);
    if (G == Dff && !is_pow2(G) && G % 128)
      return fail(WIDE_ERR_UNSUPPORTED, "bf16 single-group path needs d_ff %% 128 == 0 (got %d)", G);
  }
  return WIDE_OK;
}

// Groups narrower than the K axis's 64-wide k step (bf16 prefill): the
// N axis runs on 256-row tiles in token order and stores +0 for inactive
// (token, group) blocks; the K axis then works on 64-wide merged blocks (a
// block is active for a token when any of its groups is, and the inactive
// groups inside it contribute the zeros H holds).
bool small_groups(wide_dtype_t dt, int G) { return dt == WIDE_BF16 && G < wide::kKMergeWidth; }

size_t ffn_ws_bytes(wide_dtype_t dt, int64_t M, int D, int Dff, int G, bool need_idx, bool need_h,
                    int kpath) {
  Carve c(nullptr);
  const int ng = Dff / G;
  if (dt == WIDE_F32) {
    if (need_h) c.take<float>((size_t)M * Dff);
    return c.off;
  }
  if (need_h) c.take<uint16_t>((size_t)M * Dff);
  if (use_decode(dt, M)) {
    const size_t pn = wide::gemv_n_part_floats(ffn_gvn(M, D, Dff, G, nullptr, nullptr, nullptr, nullptr, nullptr), true);
    if (pn) c.take<float>(pn);
    const int ks = wide::gemv_k_split(D, (int)M, Dff);
    if (ks > 1) c.take<float>((size_t)ks * M * D);
  } else if (small_groups(dt, G)) {
    const int nm = Dff / wide::kKMergeWidth;
    c.take<uint8_t>((size_t)M * nm);  // merged mask
    KWS k;
    carve_kaxis(c, M, D, nm, 1, k);
  } else {
    ReorderWS r;
    carve_reorder(c, M, ng, need_idx, r);
    KWS k;
    carve_kaxis(c, M, D, ng, kpath, k);
  }
  return c.off;
}

// ---- attention ----------------------------------------------------------------------
struct AttnDims {
  int D, nq, nkv, hd, G, Nq, Nkv, ng;
};

wide_status_t attn_shape(wide_dtype_t dt, int64_t M, int D, int nq, int nkv, int hd, int G,
                         AttnDims& d) {
  CHECK(check_common(dt, M));
  if (D <= 0 || nq <= 0 || nkv <= 0 || hd <= 0 || G <= 0)
    return fail(WIDE_ERR_INVALID_ARG, "dimensions must be positive");
  if (nq % nkv) return fail(WIDE_ERR_INVALID_ARG, "n_q_heads=%d not a multiple of n_kv_heads=%d", nq, nkv);
  if (G % hd) return fail(WIDE_ERR_INVALID_ARG, "group_size=%d not a multiple of head_dim=%d", G, hd);
  const int Nq = nq * hd, Nkv = nkv * hd;
  if (Nq % G) return fail(WIDE_ERR_INVALID_ARG, "group_size=%d does not divide n_q*head_dim=%d", G, Nq);
  if (D % 8 || Nq % 8 || Nkv % 8) return fail(WIDE_ERR_INVALID_ARG, "row lengths must be multiples of 8");
  if (Nq / G > 4096) return fail(WIDE_ERR_UNSUPPORTED, "more than 4096 groups");
  if (dt == WIDE_F32) {
    if (D % 16 || Nkv % 16 || G % 16)
      return fail(WIDE_ERR_UNSUPPORTED, "fp32 path needs d_model, n_kv*head_dim, group_size multiples of 16");
  } else {
    if (D % 256) return fail(WIDE_ERR_UNSUPPORTED, "bf16 path needs d_model %% 256 == 0");
    if (G == 64) {  // Q on token-order 256-wide tiles
      if (Nq % 256 || Nkv % 256)
        return fail(WIDE_ERR_UNSUPPORTED, "bf16 path with group_size 64 needs n_q*head_dim and n_kv*head_dim %% 256 == 0");
    } else if (G % 128) {
      return fail(WIDE_ERR_UNSUPPORTED, "bf16 path needs group_size 64 or a multiple of 128");
    }
    if (Nkv % 128) return fail(WIDE_ERR_UNSUPPORTED, "bf16 path needs n_kv*head_dim %% 128 == 0");
  }
  d = AttnDims{D, nq, nkv, hd, G, Nq, Nkv, Nq / G};
  return WIDE_OK;
}


wide::GVNArgs qkv_gvn(int64_t M, const AttnDims& d, const uint8_t* mask, const void* x, const void* wq,
                      const void* wk, const void* wv, void* q, void* k, void* v) {
  wide::GVNArgs na{};
  na.x = static_cast<const uint16_t*>(x);
  na.mask = mask;
  na.B = (int)M;
  na.K = d.D;
  na.G = d.G;
  na.n_groups = d.ng;
  na.n_regions = 3;
  na.reg[0] = wide::GVRegion{static_cast<const uint16_t*>(wq), nullptr, static_cast<uint16_t*>(q), d.Nq,
                             d.Nq / 16, 1, 0};
  na.reg[1] = wide::GVRegion{static_cast<const uint16_t*>(wk), nullptr, static_cast<uint16_t*>(k), d.Nkv,
                             d.Nkv / 16, 0, d.Nq};
  na.reg[2] = wide::GVRegion{static_cast<const uint16_t*>(wv), nullptr, static_cast<uint16_t*>(v), d.Nkv,
                             d.Nkv / 16, 0, d.Nq + d.Nkv};
  na.swiglu = 0;
  na.k_split = wide::gemv_n_split(na);
  return na;
}

// Q groups narrower than 128 columns: Q runs on 256-wide tiles in token order
// (every output computed, +0 stored where the group is inactive).
bool qkv_token_order(const AttnDims& d) { return d.G < 128; }
// Q/K/V on 256x256 tiles (else the 128-tile kernel)
bool qkv_big(const AttnDims& d) {
  return qkv_token_order(d) || (g_big_tiles && d.G % wide::kT256 == 0 && d.Nkv % wide::kT256 == 0);
}

size_t attn_ws_bytes(wide_phase_t ph, wide_dtype_t dt, int64_t M, const AttnDims& d, bool need_idx,
                     int kpath) {
  Carve c(nullptr);
  if (dt == WIDE_F32) return 0;
  if (use_decode(dt, M)) {
    if (ph == WIDE_PHASE_QKV) {
      // d.Nkv < 0: sizing query without n_kv; bound the split (<= 8) and the
      // columns (n_kv <= n_q, so at most 3 * n_q * head_dim).
      const size_t pn = d.Nkv < 0 ? (size_t)8 * M * 3 * d.Nq
                                  : wide::gemv_n_part_floats(qkv_gvn(M, d, nullptr, nullptr, nullptr, nullptr,
                                                                     nullptr, nullptr, nullptr, nullptr),
                                                             false);
      if (pn) c.take<float>(pn);
    } else {
      const int ks = wide::gemv_k_split(d.D, (int)M, d.Nq);
      if (ks > 1) c.take<float>((size_t)ks * M * d.D);
    }
    return c.off;
  }
  if (ph == WIDE_PHASE_QKV) {
    ReorderWS r;
    if (need_idx) carve_reorder(c, M, d.ng, true, r);
    // Q/K/V tail tiles (a sizing query without n_kv assumes the 256 tiles)
    if (d.Nkv < 0 ? d.G < 128 || (g_big_tiles && d.G % wide::kT256 == 0) : qkv_big(d))
      c.take<float>(wide::kMN256TailFloats);
  } else {
    ReorderWS r;
    const int path = kpath;
    if (need_idx && (path == 0 || path == 2 || kaxis_row_gathered(d.Nq, d.D, d.G)))
      carve_reorder(c, M, d.ng, true, r);
    KWS k;
    carve_kaxis(c, M, d.D, d.ng, path, k);
  }
  return c.off;
}

// K-axis product for down / O on the bf16 prefill path.
wide_status_t run_kaxis(const uint16_t* a, const uint16_t* w, const uint8_t* mask,
                        const int32_t* idx, const int32_t* cnt, uint16_t* y, int64_t M, int K,
                        int N, int G, int path, const KWS& kws, hipStream_t s) {
  wide::KArgs ka{};
  ka.a = a;
  ka.w = w;
  ka.mask = mask;
  ka.idx = idx;
  ka.cnt = cnt;
  ka.acc32 = kws.acc32;
  ka.y = y;
  ka.tile_union = kws.tu;
  ka.M = M;
  ka.K = K;
  ka.N = N;
  ka.G = G;
  ka.pack = g_ks_pack;
  hipError_t e;
  const bool big = g_big_tiles && N % wide::kT256 == 0;
  if (kaxis_row_gathered(K, N, G)) {
    if (!idx || !cnt) return fail(WIDE_ERR_INVALID_ARG, "single-group K axis without a reorder");
    // One group (the M-axis case): every output row takes one contribution,
    // so the active rows run as a row-gathered N-axis GEMM over the whole
    // output width, and the rows of inactive tokens are written +0; neither
    // atomics nor dense-masked FLOPs are needed.
    wide::MN256Args ma{};
    ma.order = (g_mn_order >> 1) & 1;
    ma.x = a;
    ma.M = M;
    ma.K = K;
    ma.idx = idx;
    ma.cnt = cnt;
    ma.m_tiles = (int)((M + wide::kT256 - 1) / wide::kT256);
    ma.n_regions = 1;
    ma.reg[0] = wide::MN256Region{w, nullptr, y, N, N, 1, ma.m_tiles * (N / wide::kT256)};
    if ((e = wide::launch_mn256(ma, false, s)) != hipSuccess) return hip_fail(e, "mn256 single-group K axis");
    return WIDE_OK;
  }
  if (path == 2) {
    if ((e = wide::launch_zero_f32(kws.acc32, M * (int64_t)N, s)) != hipSuccess) return hip_fail(e, "zero");
    e = big ? wide::launch_ks256(ka, s) : wide::launch_gemm_k_scatter(ka, s);
    if (e != hipSuccess) return hip_fail(e, "gemm_k scatter");
    if ((e = wide::launch_f32_to_bf16(kws.acc32, y, M * (int64_t)N, s)) != hipSuccess)
      return hip_fail(e, "f32_to_bf16");
  } else {
    const bool use256 = big && K / G <= wide::kKd256MaxGroups;
    if (use256 && kaxis_pattern_order(N, K / G, path) && kws.perm) {
      if ((e = wide::launch_pattern_order(mask, M, K / G, kws.perm, kws.pat, s)) != hipSuccess)
        return hip_fail(e, "pattern order");
      ka.perm = kws.perm;
    }
    e = use256 ? wide::launch_kd256(ka, s) : wide::launch_gemm_k_dense_masked(ka, s);
    if (e != hipSuccess) return hip_fail(e, "gemm_k dense-masked");
  }
  return WIDE_OK;
}

// ---- timing ----------------------------------------------------------------------------
struct TimingRec {
  int name;
  hipEvent_t start, stop;
};

std::mutex g_tmu;
std::atomic<bool> g_timing{false};  // read unlocked by every launch
std::vector<TimingRec> g_pool;
size_t g_used = 0;
std::vector<std::string> g_names;
std::string g_timing_filter;  // only launches whose label it matches are timed ("": every launch)

// `label` is `want` exactly, or `want` followed by a template argument list or
// a "/variant" suffix.
bool label_matches(const std::string& label, const std::string& want) {
  return label.compare(0, want.size(), want) == 0 &&
         (label.size() == want.size() || label[want.size()] == '<' || label[want.size()] == '/');
}

int name_id(const char* n) {
  for (size_t i = 0; i < g_names.size(); ++i)
    if (g_names[i] == n) return (int)i;
  g_names.emplace_back(n);
  return (int)g_names.size() - 1;
}

}  // namespace

namespace wide {

int timing_begin(const char* name, hipStream_t s) {
  if (!g_timing) return -1;
  std::lock_guard<std::mutex> lk(g_tmu);
  if (!g_timing || g_used >= g_pool.size()) return -1;
  if (!g_timing_filter.empty() && !label_matches(name, g_timing_filter)) return -1;
  const int slot = (int)g_used++;
  g_pool[slot].name = name_id(name);
  (void)hipEventRecord(g_pool[slot].start, s);
  return slot;
}

void timing_end(int slot, hipStream_t s) {
  if (slot < 0) return;
  (void)hipEventRecord(g_pool[slot].stop, s);
}

}  // namespace wide

extern "C" {

const char* wide_last_error(void) { return g_last_error.c_str(); }

wide_status_t wide_set_option(const char* key, int64_t value) {
  if (!key) return fail(WIDE_ERR_INVALID_ARG, "key is NULL");
  if (!strcmp(key, "decode_max_m")) {
    if (value < 0) return fail(WIDE_ERR_INVALID_ARG, "decode_max_m must be >= 0");
    g_decode_max_m = value;
    return ok();
  }
  if (!strcmp(key, "k_path")) {
    if (value < 0 || value > 2) return fail(WIDE_ERR_INVALID_ARG, "k_path must be 0, 1 or 2");
    g_k_path = (int)value;
    return ok();
  }
  if (!strcmp(key, "big_tiles")) {
    if (value < 0 || value > 1) return fail(WIDE_ERR_INVALID_ARG, "big_tiles must be 0 or 1");
    g_big_tiles = (int)value;
    return ok();
  }
  for (const char* k : {"gemv_n_ncb", "gemv_k_ncb"})
    if (!strcmp(key, k)) {
      if (value != 0 && value != 1 && value != 2 && value != 4 && value != 8)
        return fail(WIDE_ERR_INVALID_ARG, "%s must be 0, 1, 2, 4 or 8", key);
      (key[5] == 'n' ? wide::decode_tuning().n_ncb : wide::decode_tuning().k_ncb) = (int)value;
      return ok();
    }
  for (const char* k : {"gemv_n_split", "gemv_k_split"})
    if (!strcmp(key, k)) {
      if (value != 0 && value != 1 && value != 2 && value != 4 && value != 8)
        return fail(WIDE_ERR_INVALID_ARG, "%s must be 0, 1, 2, 4 or 8", key);
      (key[5] == 'n' ? wide::decode_tuning().n_split : wide::decode_tuning().k_split) = (int)value;
      return ok();
    }
  if (!strcmp(key, "mn_tail")) {
    if (value < 0 || value > 1) return fail(WIDE_ERR_INVALID_ARG, "mn_tail must be 0 or 1");
    g_mn_tail = (int)value;
    return ok();
  }
  if (!strcmp(key, "mn_order")) {
    if (value < 0 || value > 7) return fail(WIDE_ERR_INVALID_ARG, "mn_order must be 0..7");
    g_mn_order = (int)value;
    return ok();
  }
  if (!strcmp(key, "ks_pack")) {
    if (value < 1 || value > 4096) return fail(WIDE_ERR_INVALID_ARG, "ks_pack must be 1..4096");
    g_ks_pack = (int)value;
    return ok();
  }
  if (!strcmp(key, "kd_pattern")) {
    if (value < 0 || value > 1) return fail(WIDE_ERR_INVALID_ARG, "kd_pattern must be 0 or 1");
    g_kd_pattern = (int)value;
    return ok();
  }
  if (!strcmp(key, "attn_split_rounds")) {
    if (value < 1 || value > 8) return fail(WIDE_ERR_INVALID_ARG, "attn_split_rounds must be 1..8");
    wide::g_attn_split_rounds = (int)value;
    return ok();
  }
  if (!strcmp(key, "attn_split")) {
    if (value < 0 || value > wide::kAttnMaxSplitTiles)
      return fail(WIDE_ERR_INVALID_ARG, "attn_split must be 0..%d", wide::kAttnMaxSplitTiles);
    wide::g_attn_split = (int)value;
    return ok();
  }
  return fail(WIDE_ERR_INVALID_ARG, "unknown option '%s'", key);
}

wide_status_t wide_get_option(const char* key, int64_t* value) {
  if (!key || !value) return fail(WIDE_ERR_INVALID_ARG, "NULL argument");
  if (!strcmp(key, "decode_max_m")) *value = g_decode_max_m;
  else if (!strcmp(key, "k_path")) *value = g_k_path;
  else if (!strcmp(key, "big_tiles")) *value = g_big_tiles;
  else if (!strcmp(key, "gemv_n_ncb")) *value = wide::decode_tuning().n_ncb;
  else if (!strcmp(key, "gemv_n_split")) *value = wide::decode_tuning().n_split;
  else if (!strcmp(key, "gemv_k_ncb")) *value = wide::decode_tuning().k_ncb;
  else if (!strcmp(key, "gemv_k_split")) *value = wide::decode_tuning().k_split;
  else if (!strcmp(key, "kd_pattern")) *value = g_kd_pattern;
  else if (!strcmp(key, "ks_pack")) *value = g_ks_pack;
  else if (!strcmp(key, "mn_order")) *value = g_mn_order;
  else if (!strcmp(key, "mn_tail")) *value = g_mn_tail;
  else if (!strcmp(key, "attn_split")) *value = wide::g_attn_split;
  else if (!strcmp(key, "attn_split_rounds")) *value = wide::g_attn_split_rounds;
  else return fail(WIDE_ERR_INVALID_ARG, "unknown option '%s'", key);
  return ok();
}

size_t wide_workspace_size(wide_op_t op, wide_dtype_t dt, int64_t M, int32_t d_model,
                           int32_t d_inner, int32_t group_size) {
  switch (op) {
    case WIDE_OP_REORDER: {
      if (M < 0 || M >= (int64_t(1) << 31) || d_inner < 1 || d_inner > 4096) return SIZE_MAX;
      Carve c(nullptr);
      ReorderWS r;
      carve_reorder(c, M, d_inner, false, r);
      return c.off;
    }
    case WIDE_OP_FFN:
      if (ffn_shape(dt, M, d_model, d_inner, group_size) != WIDE_OK) return SIZE_MAX;
      return ffn_ws_bytes(dt, M, d_model, d_inner, group_size, true, true, 0);
    case WIDE_OP_ROUTER: {
      if (check_common(dt, M) != WIDE_OK || dt != WIDE_BF16 || d_model <= 0 || d_model % 64 ||
          group_size < 1 || group_size > wide::kRouterMaxRank || d_inner < 1 || d_inner > 4096)
        return SIZE_MAX;
      Carve c(nullptr);
      ReorderWS r;
      carve_reorder(c, M, d_inner, false, r);
      return c.off;
    }
    case WIDE_OP_QKV:
    case WIDE_OP_O: {
      // The size depends on M, d_model and the number of groups only.
      if (check_common(dt, M) != WIDE_OK || d_model <= 0 || group_size <= 0 || d_inner <= 0 ||
          d_inner % group_size || d_inner / group_size > 4096)
        return SIZE_MAX;
      AttnDims d{d_model, 0, 0, 0, group_size, d_inner, -1, d_inner / group_size};
      return attn_ws_bytes(op == WIDE_OP_QKV ? WIDE_PHASE_QKV : WIDE_PHASE_O, dt, M, d, true, 0);
    }
  }
  return SIZE_MAX;
}

wide_status_t wide_mask_reorder(const uint8_t* mask, int64_t M, int32_t n_groups, int32_t* idx,
                                int32_t* counts, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (M < 0 || M >= (int64_t(1) << 31)) return fail(WIDE_ERR_INVALID_ARG, "M out of range");
  if (n_groups < 1 || n_groups > 4096) return fail(WIDE_ERR_INVALID_ARG, "n_groups must be in [1, 4096]");
  CHECK(check_ptr(counts, "counts", false));
  if (M > 0) {
    CHECK(check_ptr(mask, "mask"));
    CHECK(check_ptr(idx, "idx", false));
  }
  Carve c0(nullptr);
  ReorderWS r0;
  carve_reorder(c0, M, n_groups, false, r0);
  CHECK(check_ws(ws, ws_bytes, M == 0 ? 0 : c0.off));
  Carve c(ws);
  ReorderWS r;
  carve_reorder(c, M, n_groups, false, r);
  hipError_t e = wide::launch_reorder(mask, M, n_groups, idx, counts, r.chunk_cnt, r.chunk_off, stream);
  if (e != hipSuccess) return hip_fail(e, "reorder");
  return ok();
}

wide_status_t wide_router(wide_dtype_t dt, int64_t M, int32_t d_model, int32_t rank,
                          int32_t n_groups, const void* x, const void* w1, const void* w2,
                          uint8_t* mask, float* logits, int32_t* idx, int32_t* counts,
                          void* ws, size_t ws_bytes, hipStream_t stream) {
  CHECK(check_common(dt, M));
  if (dt != WIDE_BF16) return fail(WIDE_ERR_UNSUPPORTED, "the router runs on bf16 inputs only");
  if (d_model <= 0 || d_model % 64) return fail(WIDE_ERR_INVALID_ARG, "d_model must be a positive multiple of 64");
  if (rank < 1 || rank > wide::kRouterMaxRank) return fail(WIDE_ERR_INVALID_ARG, "rank must be in [1, 32]");
  if (n_groups < 1 || n_groups > 4096) return fail(WIDE_ERR_INVALID_ARG, "n_groups must be in [1, 4096]");
  // (with M == 0 the index array is empty and may be NULL)
  if (M > 0 && (idx == nullptr) != (counts == nullptr))
    return fail(WIDE_ERR_INVALID_ARG, "idx and counts must both be given or both be NULL");
  CHECK(check_ptr(w1, "w1"));
  CHECK(check_ptr(w2, "w2"));
  if (M == 0) {  // nothing to route; a requested reorder still reports zero counts
    if (!counts) return ok();
    CHECK(check_ptr(counts, "counts", false));
    const hipError_t e = wide::launch_reorder(mask, 0, n_groups, idx, counts, nullptr, nullptr, stream);
    return e == hipSuccess ? ok() : hip_fail(e, "router counts");
  }
  CHECK(check_ptr(x, "x"));
  CHECK(check_ptr(mask, "mask"));
  if (logits) CHECK(check_ptr(logits, "logits", false));
  if (idx) {
    CHECK(check_ptr(idx, "idx", false));
    CHECK(check_ptr(counts, "counts", false));
    Carve c0(nullptr);
    ReorderWS r0;
    carve_reorder(c0, M, n_groups, false, r0);
    CHECK(check_ws(ws, ws_bytes, c0.off));
  }
  wide::RouterArgs ra{static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(w1),
                      static_cast<const uint16_t*>(w2), mask, logits, M, d_model, rank, n_groups};
  hipError_t e = wide::launch_router(ra, stream);
  if (e != hipSuccess) return hip_fail(e, "router");
  if (idx) {
    Carve c(ws);
    ReorderWS r;
    carve_reorder(c, M, n_groups, false, r);
    e = wide::launch_reorder(mask, M, n_groups, idx, counts, r.chunk_cnt, r.chunk_off, stream);
    if (e != hipSuccess) return hip_fail(e, "router reorder");
  }
  return ok();
}

wide_status_t wide_ffn_masked(wide_dtype_t dt, int64_t M, int32_t d_model, int32_t d_ff,
                              int32_t group_size, const uint8_t* mask, const int32_t* idx,
                              const int32_t* counts, const void* x, const void* w_gate,
                              const void* w_up, const void* w_down, void* h_out, void* y,
                              void* ws, size_t ws_bytes, hipStream_t stream) {
  CHECK(ffn_shape(dt, M, d_model, d_ff, group_size));
  if ((idx == nullptr) != (counts == nullptr))
    return fail(WIDE_ERR_INVALID_ARG, "idx and counts must both be given or both be NULL");
  CHECK(check_ptr(w_gate, "w_gate"));
  CHECK(check_ptr(w_up, "w_up"));
  CHECK(check_ptr(w_down, "w_down"));
  if (h_out) CHECK(check_ptr(h_out, "h_out"));
  if (M == 0) return ok();
  CHECK(check_ptr(mask, "mask"));
  CHECK(check_ptr(x, "x"));
  CHECK(check_ptr(y, "y"));
  if (idx) {
    CHECK(check_ptr(idx, "idx", false));
    CHECK(check_ptr(counts, "counts", false));
  }
  const int D = d_model, Dff = d_ff, G = group_size, ng = Dff / G;
  const bool decode = use_decode(dt, M);
  const int kpath = k_path_for(G);
  CHECK(check_ws(ws, ws_bytes, ffn_ws_bytes(dt, M, D, Dff, G, idx == nullptr, h_out == nullptr, kpath)));

  Carve c(ws);
  hipError_t e;
  if (dt == WIDE_F32) {
    float* h = h_out ? static_cast<float*>(h_out) : c.take<float>((size_t)M * Dff);
    wide::F32NArgs na{static_cast<const float*>(x), static_cast<const float*>(w_gate),
                      static_cast<const float*>(w_up), h, mask, M, D, Dff, Dff, G, ng};
    if ((e = wide::launch_f32_nproj(na, true, stream)) != hipSuccess) return hip_fail(e, "f32 gate/up");
    wide::F32KArgs ka{h, static_cast<const float*>(w_down), mask, static_cast<float*>(y), M, Dff, D, G, ng};
    if ((e = wide::launch_f32_kproj(ka, stream)) != hipSuccess) return hip_fail(e, "f32 down");
    return ok();
  }

  uint16_t* h = h_out ? static_cast<uint16_t*>(h_out) : c.take<uint16_t>((size_t)M * Dff);
  if (decode) {
    wide::GVNArgs na = ffn_gvn(M, D, Dff, G, mask, x, w_gate, w_up, h);
    const size_t pn = wide::gemv_n_part_floats(na, true);
    na.part = pn ? c.take<float>(pn) : nullptr;
    if ((e = wide::launch_gemv_n(na, true, stream)) != hipSuccess) return hip_fail(e, "gemv gate/up");
    const int ks = wide::gemv_k_split(D, (int)M, Dff);
    float* part = ks > 1 ? c.take<float>((size_t)ks * M * D) : nullptr;
    // groups narrower than 64 are walked as merged 64-wide groups
    const int mg = std::max(1, wide::kKMergeWidth / G);
    wide::GVKArgs ka{h, static_cast<const uint16_t*>(w_down), mask, static_cast<uint16_t*>(y),
                     (int)M, Dff, D, G * mg, ng / mg, ks, part, mg};
    if ((e = wide::launch_gemv_k(ka, stream)) != hipSuccess) return hip_fail(e, "gemv down");
    return ok();
  }

  if (small_groups(dt, G)) {
    const int nm = Dff / wide::kKMergeWidth;
    uint8_t* merged = c.take<uint8_t>((size_t)M * nm);
    KWS kws;
    carve_kaxis(c, M, D, nm, 1, kws);
    wide::MN256Args ma{};
    ma.x = static_cast<const uint16_t*>(x);
    ma.M = M;
    ma.K = D;
    ma.m_tiles = (int)((M + wide::kT256 - 1) / wide::kT256);
    ma.n_regions = 1;
    ma.mask = mask;
    ma.mask_ng = ng;
    ma.mask_G = G;
    // every H block is written (+0 where inactive): the merged K axis reads them
    ma.reg[0] = wide::MN256Region{static_cast<const uint16_t*>(w_gate), static_cast<const uint16_t*>(w_up), h,
                                  Dff, Dff, wide::kMN256TokenOrder, ma.m_tiles * (Dff / 128), 0};
    if ((e = wide::launch_mn256(ma, true, stream)) != hipSuccess) return hip_fail(e, "mn256 gate/up");
    if ((e = wide::launch_mask_merge(mask, M, ng, wide::kKMergeWidth / G, merged, stream)) != hipSuccess)
      return hip_fail(e, "mask merge");
    CHECK(run_kaxis(h, static_cast<const uint16_t*>(w_down), merged, nullptr, nullptr, static_cast<uint16_t*>(y), M,
                    Dff, D, wide::kKMergeWidth, 1, kws, stream));
    return ok();
  }
  ReorderWS r;
  carve_reorder(c, M, ng, idx == nullptr, r);
  KWS kws;
  carve_kaxis(c, M, D, ng, kpath, kws);
  const int32_t* ix = idx;
  const int32_t* ct = counts;
  if (!idx) {
    if ((e = wide::launch_reorder(mask, M, ng, r.idx, r.cnt, r.chunk_cnt, r.chunk_off, stream)) != hipSuccess)
      return hip_fail(e, "reorder");
    ix = r.idx;
    ct = r.cnt;
  }
  if (g_big_tiles && G % 128 == 0) {
    wide::MN256Args ma{};
    ma.order = (g_mn_order >> 1) & 1;
    ma.mblock = (g_mn_order >> 2) & 1;
    ma.x = static_cast<const uint16_t*>(x);
    ma.M = M;
    ma.K = D;
    ma.idx = ix;
    ma.cnt = ct;
    ma.m_tiles = (int)((M + wide::kT256 - 1) / wide::kT256);
    ma.n_regions = 1;
    // An H kept in the workspace is read only through its active blocks by
    // every K-axis schedule, so its inactive blocks need no zeros.
    ma.reg[0] = wide::MN256Region{static_cast<const uint16_t*>(w_gate), static_cast<const uint16_t*>(w_up), h,
                                  Dff, G, 1, ng * ma.m_tiles * (G / 128), h_out == nullptr ? 1 : 0};
    // (no tail split for gate/up: over seven rounds of tiles the chunks and
    // their finishing kernel cost about what the last partial round saves)
    if ((e = wide::launch_mn256(ma, true, stream)) != hipSuccess) return hip_fail(e, "mn256 gate/up");
  } else {
    wide::MNArgs ma{};
    ma.x = static_cast<const uint16_t*>(x);
    ma.M = M;
    ma.K = D;
    ma.idx = ix;
    ma.cnt = ct;
    ma.G = G;
    ma.m_tiles = (int)((M + wide::kMNTileM - 1) / wide::kMNTileM);
    ma.n_regions = 1;
    ma.reg[0] = wide::MNRegion{static_cast<const uint16_t*>(w_gate), static_cast<const uint16_t*>(w_up), h,
                               Dff, Dff / wide::kMNTileNSwiglu, 1};
    if ((e = wide::launch_gemm_mn(ma, true, stream)) != hipSuccess) return hip_fail(e, "gemm_mn gate/up");
  }
  CHECK(run_kaxis(h, static_cast<const uint16_t*>(w_down), mask, ix, ct, static_cast<uint16_t*>(y), M, Dff,
                  D, G, kpath, kws, stream));
  return ok();
}

// ---- allocation-free FFN ------------------------------------------------------------
// For callers that cannot allocate (graph capture, serving loops): the
// workspace of wide_ffn_masked lives in a file-scope device array instead of
// the caller's buffer.  Host code never uses the array's name as an address
// (it is a host-side stand-in there): each device's address comes from
// hipGetSymbolAddress, looked up once per device with that device current.
namespace {
constexpr size_t kStaticScratchBytes = size_t(32) << 20;
__device__ __align__(256) unsigned char scratch[kStaticScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};  // device address of `scratch`, per device

wide_status_t scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices) return fail(WIDE_ERR_UNSUPPORTED, "device ordinal %d out of range", dev);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p) return fail(WIDE_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_dev[dev] = p;
  }
  *out = g_scratch_dev[dev];
  return WIDE_OK;
}
}  // namespace

size_t wide_static_scratch_bytes(void) { return kStaticScratchBytes; }

wide_status_t wide_ffn_masked_noalloc(wide_dtype_t dt, int64_t M, int32_t d_model, int32_t d_ff,
                                      int32_t group_size, const uint8_t* mask, const int32_t* idx,
                                      const int32_t* counts, const void* x, const void* w_gate, const void* w_up,
                                      const void* w_down, void* h_out, void* y, hipStream_t stream) {
  CHECK(ffn_shape(dt, M, d_model, d_ff, group_size));
  if ((idx == nullptr) != (counts == nullptr))
    return fail(WIDE_ERR_INVALID_ARG, "idx and counts must both be given or both be NULL");
  const size_t need = ffn_ws_bytes(dt, M, d_model, d_ff, group_size, idx == nullptr, h_out == nullptr,
                                   k_path_for(group_size));
  if (need > kStaticScratchBytes)
    return fail(WIDE_ERR_WORKSPACE,
                "this call needs %zu bytes of scratch; the static scratch holds %zu (pass h_out, or use "
                "wide_ffn_masked with a workspace)", need, kStaticScratchBytes);
  if (M == 0) return wide_ffn_masked(dt, M, d_model, d_ff, group_size, mask, idx, counts, x, w_gate, w_up,
                                     w_down, h_out, y, nullptr, 0, stream);
  void* ws = nullptr;
  if (need) CHECK(scratch_address(&ws));
  return wide_ffn_masked(dt, M, d_model, d_ff, group_size, mask, idx, counts, x, w_gate, w_up, w_down, h_out, y,
                         ws, need ? kStaticScratchBytes : 0, stream);
}

wide_status_t wide_qkvo_masked(wide_phase_t phase, wide_dtype_t dt, int64_t M, int32_t d_model,
                               int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                               int32_t group_size, const uint8_t* mask, const int32_t* idx,
                               const int32_t* counts, const void* in, const void* w_q,
                               const void* w_k, const void* w_v, const void* w_o, void* q, void* k,
                               void* v, void* y, void* ws, size_t ws_bytes, hipStream_t stream) {
  if (phase != WIDE_PHASE_QKV && phase != WIDE_PHASE_O)
    return fail(WIDE_ERR_INVALID_ARG, "unknown phase %d", (int)phase);
  AttnDims d;
  CHECK(attn_shape(dt, M, d_model, n_q_heads, n_kv_heads, head_dim, group_size, d));
  if ((idx == nullptr) != (counts == nullptr))
    return fail(WIDE_ERR_INVALID_ARG, "idx and counts must both be given or both be NULL");
  if (phase == WIDE_PHASE_QKV) {
    CHECK(check_ptr(w_q, "w_q"));
    CHECK(check_ptr(w_k, "w_k"));
    CHECK(check_ptr(w_v, "w_v"));
  } else {
    CHECK(check_ptr(w_o, "w_o"));
  }
  if (M == 0) return ok();
  CHECK(check_ptr(mask, "mask"));
  CHECK(check_ptr(in, "in"));
  if (phase == WIDE_PHASE_QKV) {
    CHECK(check_ptr(q, "q"));
    CHECK(check_ptr(k, "k"));
    CHECK(check_ptr(v, "v"));
  } else {
    CHECK(check_ptr(y, "y"));
  }
  if (idx) {
    CHECK(check_ptr(idx, "idx", false));
    CHECK(check_ptr(counts, "counts", false));
  }
  const int kpath = k_path_for(d.G);
  CHECK(check_ws(ws, ws_bytes, attn_ws_bytes(phase, dt, M, d, idx == nullptr, kpath)));
  Carve c(ws);
  hipError_t e;
  const int ng = d.ng;

  if (dt == WIDE_F32) {
    const float* x = static_cast<const float*>(in);
    if (phase == WIDE_PHASE_QKV) {
      wide::F32NArgs qa{x, static_cast<const float*>(w_q), nullptr, static_cast<float*>(q), mask, M, d.D, d.Nq,
                        d.Nq, d.G, ng};
      if ((e = wide::launch_f32_nproj(qa, false, stream)) != hipSuccess) return hip_fail(e, "f32 q");
      wide::F32NArgs ka{x, static_cast<const float*>(w_k), nullptr, static_cast<float*>(k), nullptr, M, d.D,
                        d.Nkv, d.Nkv, d.Nkv, 1};
      if ((e = wide::launch_f32_nproj(ka, false, stream)) != hipSuccess) return hip_fail(e, "f32 k");
      ka.w0 = static_cast<const float*>(w_v);
      ka.out = static_cast<float*>(v);
      if ((e = wide::launch_f32_nproj(ka, false, stream)) != hipSuccess) return hip_fail(e, "f32 v");
    } else {
      wide::F32KArgs oa{x, static_cast<const float*>(w_o), mask, static_cast<float*>(y), M, d.Nq, d.D, d.G, ng};
      if ((e = wide::launch_f32_kproj(oa, stream)) != hipSuccess) return hip_fail(e, "f32 o");
    }
    return ok();
  }

  const uint16_t* x = static_cast<const uint16_t*>(in);
  if (use_decode(dt, M)) {
    if (phase == WIDE_PHASE_QKV) {
      wide::GVNArgs na = qkv_gvn(M, d, mask, x, w_q, w_k, w_v, q, k, v);
      const size_t pn = wide::gemv_n_part_floats(na, false);
      na.part = pn ? c.take<float>(pn) : nullptr;
      if ((e = wide::launch_gemv_n(na, false, stream)) != hipSuccess) return hip_fail(e, "gemv qkv");
    } else {
      const int ks = wide::gemv_k_split(d.D, (int)M, d.Nq);
      float* part = ks > 1 ? c.take<float>((size_t)ks * M * d.D) : nullptr;
      wide::GVKArgs ka{x, static_cast<const uint16_t*>(w_o), mask, static_cast<uint16_t*>(y), (int)M, d.Nq,
                       d.D, d.G, ng, ks, part, 1};
      if ((e = wide::launch_gemv_k(ka, stream)) != hipSuccess) return hip_fail(e, "gemv o");
    }
    return ok();
  }

  const bool rows_k = phase == WIDE_PHASE_O && kaxis_row_gathered(d.Nq, d.D, d.G);
  const bool need_reorder =
      idx == nullptr && ((phase == WIDE_PHASE_QKV && !qkv_token_order(d)) || kpath == 2 || rows_k);
  ReorderWS r;
  float* tail_ws = nullptr;
  if (phase == WIDE_PHASE_QKV) {
    if (idx == nullptr) carve_reorder(c, M, ng, true, r);
    if (qkv_big(d)) tail_ws = c.take<float>(wide::kMN256TailFloats);
  } else if (idx == nullptr && (kpath == 0 || kpath == 2 || rows_k)) {
    carve_reorder(c, M, ng, true, r);
  }
  const int32_t* ix = idx;
  const int32_t* ct = counts;
  if (need_reorder) {
    if ((e = wide::launch_reorder(mask, M, ng, r.idx, r.cnt, r.chunk_cnt, r.chunk_off, stream)) != hipSuccess)
      return hip_fail(e, "reorder");
    ix = r.idx;
    ct = r.cnt;
  }
  if (phase == WIDE_PHASE_QKV) {
    const uint16_t* wq = static_cast<const uint16_t*>(w_q);
    const uint16_t* wk = static_cast<const uint16_t*>(w_k);
    const uint16_t* wv = static_cast<const uint16_t*>(w_v);
    if (qkv_big(d)) {
      wide::MN256Args ma{};
    ma.order = (g_mn_order >> 1) & 1;
      ma.x = x;
      ma.M = M;
      ma.K = d.D;
      ma.idx = ix;
      ma.cnt = ct;
      ma.m_tiles = (int)((M + wide::kT256 - 1) / wide::kT256);
      ma.n_regions = 3;
      const int T = wide::kT256;
      // K and V first: the masked Q tiles, whose last m-tiles are partial
      // or empty, then end each XCD's run of tiles.
      const int iq = (g_mn_order & 1) ? 2 : 0, ik = iq ? 0 : 1;
      ma.reg[ik] = wide::MN256Region{wk, nullptr, static_cast<uint16_t*>(k), d.Nkv, d.Nkv, 0,
                                     ma.m_tiles * (d.Nkv / T)};
      ma.reg[ik + 1] = wide::MN256Region{wv, nullptr, static_cast<uint16_t*>(v), d.Nkv, d.Nkv, 0,
                                         ma.m_tiles * (d.Nkv / T)};
      if (qkv_token_order(d)) {
        ma.mask = mask;
        ma.mask_ng = ng;
        ma.mask_G = d.G;
        ma.reg[iq] = wide::MN256Region{wq, nullptr, static_cast<uint16_t*>(q), d.Nq, d.Nq, wide::kMN256TokenOrder,
                                       ma.m_tiles * (d.Nq / T)};
      } else {
        ma.reg[iq] = wide::MN256Region{wq, nullptr, static_cast<uint16_t*>(q), d.Nq, d.G, wide::kMN256Sorted,
                                       ng * ma.m_tiles * (d.G / T)};
      }
      ma.tail = g_mn_tail && wide::mn256_tail_ok(ma, 256) ? 1 : 0;
      ma.tail_ws = tail_ws;
      if ((e = wide::launch_mn256(ma, false, stream)) != hipSuccess) return hip_fail(e, "mn256 qkv");
      return ok();
    }
    wide::MNArgs ma{};
    ma.x = x;
    ma.M = M;
    ma.K = d.D;
    ma.idx = ix;
    ma.cnt = ct;
    ma.G = d.G;
    ma.m_tiles = (int)((M + wide::kMNTileM - 1) / wide::kMNTileM);
    ma.n_regions = 3;
    const int T = wide::kMNTileNPlain;
    ma.reg[0] = wide::MNRegion{wq, nullptr, static_cast<uint16_t*>(q), d.Nq, d.Nq / T, 1};
    ma.reg[1] = wide::MNRegion{wk, nullptr, static_cast<uint16_t*>(k), d.Nkv, d.Nkv / T, 0};
    ma.reg[2] = wide::MNRegion{wv, nullptr, static_cast<uint16_t*>(v), d.Nkv, d.Nkv / T, 0};
    if ((e = wide::launch_gemm_mn(ma, false, stream)) != hipSuccess) return hip_fail(e, "gemm_mn qkv");
    return ok();
  }
  KWS kws;
  carve_kaxis(c, M, d.D, ng, kpath, kws);
  CHECK(run_kaxis(x, static_cast<const uint16_t*>(w_o), mask, ix, ct, static_cast<uint16_t*>(y), M, d.Nq, d.D,
                  d.G, kpath, kws, stream));
  return ok();
}

wide_status_t wide_timing_enable(int enable) {
  std::lock_guard<std::mutex> lk(g_tmu);
  if (enable && g_pool.empty()) {
    g_pool.resize(16384);
    for (auto& r : g_pool) {
      hipError_t e1 = hipEventCreate(&r.start);
      hipError_t e2 = hipEventCreate(&r.stop);
      if (e1 != hipSuccess || e2 != hipSuccess) {
        g_pool.clear();
        return hip_fail(e1 != hipSuccess ? e1 : e2, "hipEventCreate");
      }
    }
  }
  g_timing = enable != 0;
  return ok();
}

wide_status_t wide_timing_filter(const char* name) {
  std::lock_guard<std::mutex> lk(g_tmu);
  g_timing_filter = name ? name : "";
  return ok();
}

wide_status_t wide_timing_reset(void) {
  std::lock_guard<std::mutex> lk(g_tmu);
  g_used = 0;
  return ok();
}

wide_status_t wide_timing_query(const char* name, double* total_ms, int64_t* launches) {
  if (!name || !total_ms || !launches) return fail(WIDE_ERR_INVALID_ARG, "NULL argument");
  std::lock_guard<std::mutex> lk(g_tmu);
  const std::string want(name);
  double tot = 0.0;
  int64_t n = 0;
  for (size_t i = 0; i < g_used; ++i) {
    if (!label_matches(g_names[g_pool[i].name], want)) continue;
    hipError_t e = hipEventSynchronize(g_pool[i].stop);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, g_pool[i].start, g_pool[i].stop);
    if (e != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
    tot += ms;
    ++n;
  }
  *total_ms = tot;
  *launches = n;
  return ok();
}

}  // extern "C"

// ---- masked attention (prefill) -------------------------------------------------
namespace {

struct AttnShape {
  int64_t M = 0, Mk = 0;
  int T_kp = 0, ng = 0, hpg = 0, qpk = 0;
  int T_q = 0, T_k = 0, n_q = 0;
};

wide_status_t attention_shape(wide_dtype_t dt, int64_t n_seq, int T_q, int T_k, int nq, int nkv,
                              int hd, int G, int causal, AttnShape& s) {
  if (dt != WIDE_F32 && dt != WIDE_BF16) return fail(WIDE_ERR_INVALID_ARG, "unknown dtype %d", (int)dt);
  if (n_seq < 0 || T_q < 0 || T_k < 0) return fail(WIDE_ERR_INVALID_ARG, "n_seq, T_q and T_k must be >= 0");
  if (nq <= 0 || nkv <= 0 || hd <= 0 || G <= 0)
    return fail(WIDE_ERR_INVALID_ARG, "head counts, head_dim and group_size must be positive");
  if (nq % nkv) return fail(WIDE_ERR_INVALID_ARG, "n_q_heads=%d not a multiple of n_kv_heads=%d", nq, nkv);
  if (G % hd) return fail(WIDE_ERR_INVALID_ARG, "group_size=%d not a multiple of head_dim=%d", G, hd);
  if ((int64_t)nq * hd % G) return fail(WIDE_ERR_INVALID_ARG, "group_size=%d does not divide n_q*head_dim", G);
  if (causal != 0 && causal != 1) return fail(WIDE_ERR_INVALID_ARG, "causal must be 0 or 1");
  s.M = n_seq * (int64_t)T_q;
  s.Mk = n_seq * (int64_t)T_k;
  if (s.M >= (int64_t(1) << 31) || s.Mk >= (int64_t(1) << 31))
    return fail(WIDE_ERR_INVALID_ARG, "n_seq*T_q and n_seq*T_k must be < 2^31");
  if (s.M > 0 && T_k == 0) return fail(WIDE_ERR_INVALID_ARG, "queries with no keys (T_k = 0)");
  if (causal && T_k < T_q)
    return fail(WIDE_ERR_INVALID_ARG, "causal attention needs T_k >= T_q (queries are the last T_q positions)");
  s.ng = (int)((int64_t)nq * hd / G);
  if (s.ng > 4096) return fail(WIDE_ERR_UNSUPPORTED, "more than 4096 groups");
  if (dt != WIDE_BF16) return fail(WIDE_ERR_UNSUPPORTED, "attention runs on bf16 only");
  if (hd != wide::kAttnHeadDim) return fail(WIDE_ERR_UNSUPPORTED, "attention needs head_dim 128 (got %d)", hd);
  s.T_kp = (int)((T_k + 63) / 64 * 64);
  s.hpg = G / hd;
  s.qpk = nq / nkv;
  s.T_q = T_q;
  s.T_k = T_k;
  s.n_q = nq;
  return WIDE_OK;
}

struct AttnWS {
  ReorderWS r;
  uint16_t* vt = nullptr;
  int32_t* seq_off = nullptr;
  int split_tiles = 0;  // key-range split (0: none)
  int32_t* sched = nullptr;
  float* part = nullptr;
};

void carve_attention(Carve& c, int64_t n_seq, int nkv, const AttnShape& s, bool need_idx, AttnWS& w) {
  if (need_idx) carve_reorder(c, s.M, s.ng, true, w.r);
  w.vt = c.take<uint16_t>((size_t)n_seq * nkv * wide::kAttnHeadDim * (size_t)s.T_kp);
  w.seq_off = c.take<int32_t>((size_t)s.ng * (size_t)(n_seq + 1));
  w.split_tiles = wide::attn_split_tiles(n_seq, s.T_q, s.T_k, s.n_q, s.hpg, s.qpk);
  if (w.split_tiles > 0) {
    w.sched = c.take<int32_t>(wide::attn_sched_ints(w.split_tiles));
    w.part = c.take<float>(wide::attn_part_floats());
  }
}

}  // namespace

size_t wide_attention_workspace_size(int64_t n_seq, int32_t T_q, int32_t T_k, int32_t n_q_heads,
                                     int32_t n_kv_heads, int32_t head_dim, int32_t group_size,
                                     int32_t with_reorder) {
  AttnShape s;
  const std::string keep = g_last_error;
  const bool bad = attention_shape(WIDE_BF16, n_seq, T_q, T_k, n_q_heads, n_kv_heads, head_dim, group_size,
                                   0, s) != WIDE_OK;
  g_last_error = keep;
  if (bad) return SIZE_MAX;
  if (s.M == 0) return 0;
  Carve c(nullptr);
  AttnWS w;
  carve_attention(c, n_seq, n_kv_heads, s, with_reorder != 0, w);
  return c.off;
}

wide_status_t wide_attention_masked(wide_dtype_t dt, int64_t n_seq, int32_t T_q, int32_t T_k,
                                    int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                    int32_t group_size, int32_t causal, const int32_t* leftpad,
                                    const uint8_t* mask, const int32_t* idx, const int32_t* counts,
                                    const void* q, const void* k, const void* v, void* o, void* ws,
                                    size_t ws_bytes, hipStream_t stream) {
  AttnShape s;
  CHECK(attention_shape(dt, n_seq, T_q, T_k, n_q_heads, n_kv_heads, head_dim, group_size, causal, s));
  if ((idx == nullptr) != (counts == nullptr))
    return fail(WIDE_ERR_INVALID_ARG, "idx and counts must both be given or both be NULL");
  if (s.M == 0) return ok();
  CHECK(check_ptr(mask, "mask"));
  CHECK(check_ptr(q, "q"));
  CHECK(check_ptr(k, "k"));
  CHECK(check_ptr(v, "v"));
  CHECK(check_ptr(o, "o"));
  if (idx) {
    CHECK(check_ptr(idx, "idx", false));
    CHECK(check_ptr(counts, "counts", false));
  }
  if (leftpad) CHECK(check_ptr(leftpad, "leftpad", false));
  {
    Carve c0(nullptr);
    AttnWS w0;
    carve_attention(c0, n_seq, n_kv_heads, s, idx == nullptr, w0);
    CHECK(check_ws(ws, ws_bytes, c0.off));
  }
  Carve c(ws);
  AttnWS w;
  carve_attention(c, n_seq, n_kv_heads, s, idx == nullptr, w);
  hipError_t e;
  if (!idx) {
    if ((e = wide::launch_reorder(mask, s.M, s.ng, w.r.idx, w.r.cnt, w.r.chunk_cnt, w.r.chunk_off, stream)) !=
        hipSuccess)
      return hip_fail(e, "attention reorder");
    idx = w.r.idx;
    counts = w.r.cnt;
  }
  wide::AttnArgs a{};
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.vt = w.vt;
  a.o = static_cast<uint16_t*>(o);
  a.idx = idx;
  a.cnt = counts;
  a.M = s.M;
  a.n_seq = (int)n_seq;
  a.T_q = T_q;
  a.T_k = T_k;
  a.T_kp = s.T_kp;
  a.n_q = n_q_heads;
  a.n_kv = n_kv_heads;
  a.ng = s.ng;
  a.hpg = s.hpg;
  a.qpk = s.qpk;
  a.causal = causal;
  a.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)head_dim));
  a.sched = w.sched;
  a.part = w.part;
  a.split_tiles = w.split_tiles;
  a.leftpad = leftpad;
  if ((e = wide::launch_attention(a, static_cast<const uint16_t*>(v), w.seq_off, stream)) != hipSuccess)
    return hip_fail(e, "attention");
  return ok();
}

// ---- masked attention (decode) ----------------------------------------------------
namespace {

wide_status_t attention_decode_shape(wide_dtype_t dt, int64_t B, int32_t L, int nq, int nkv, int hd, int G,
                                     AttnShape& s) {
  if (dt != WIDE_F32 && dt != WIDE_BF16) return fail(WIDE_ERR_INVALID_ARG, "unknown dtype %d", (int)dt);
  if (B < 0 || B >= (int64_t(1) << 31) || L < 0) return fail(WIDE_ERR_INVALID_ARG, "batch and L must be >= 0");
  if (nq <= 0 || nkv <= 0 || hd <= 0 || G <= 0)
    return fail(WIDE_ERR_INVALID_ARG, "head counts, head_dim and group_size must be positive");
  if (nq % nkv) return fail(WIDE_ERR_INVALID_ARG, "n_q_heads=%d not a multiple of n_kv_heads=%d", nq, nkv);
  if (G % hd) return fail(WIDE_ERR_INVALID_ARG, "group_size=%d not a multiple of head_dim=%d", G, hd);
  if ((int64_t)nq * hd % G) return fail(WIDE_ERR_INVALID_ARG, "group_size=%d does not divide n_q*head_dim", G);
  if (B > 0 && L == 0) return fail(WIDE_ERR_INVALID_ARG, "a key cache of length 0");
  if (B * (int64_t)L >= (int64_t(1) << 31)) return fail(WIDE_ERR_INVALID_ARG, "batch*L must be < 2^31");
  s.ng = (int)((int64_t)nq * hd / G);
  if (s.ng > 4096) return fail(WIDE_ERR_UNSUPPORTED, "more than 4096 groups");
  if (dt != WIDE_BF16) return fail(WIDE_ERR_UNSUPPORTED, "attention runs on bf16 only");
  if (hd != wide::kAttnHeadDim) return fail(WIDE_ERR_UNSUPPORTED, "attention needs head_dim 128 (got %d)", hd);
  if (nq / nkv > 16) return fail(WIDE_ERR_UNSUPPORTED, "more than 16 query heads per KV head");
  s.M = B;
  s.Mk = B * (int64_t)L;
  s.hpg = G / hd;
  s.qpk = nq / nkv;
  return WIDE_OK;
}

size_t attention_decode_ws(int64_t B, int L, int nq, int nkv) {
  if (B == 0) return 0;
  const int ch = wide::attn_decode_chunk((int)B, nkv, L);
  const int nc = (L + ch - 1) / ch;
  return align_up((size_t)B * nq * nc * (wide::kAttnHeadDim + 2) * sizeof(float));
}

}  // namespace

size_t wide_attention_decode_workspace_size(int64_t batch, int32_t L, int32_t n_q_heads, int32_t n_kv_heads,
                                            int32_t head_dim, int32_t group_size) {
  AttnShape s;
  const std::string keep = g_last_error;
  const bool bad =
      attention_decode_shape(WIDE_BF16, batch, L, n_q_heads, n_kv_heads, head_dim, group_size, s) != WIDE_OK;
  g_last_error = keep;
  return bad ? SIZE_MAX : attention_decode_ws(batch, L, n_q_heads, n_kv_heads);
}

wide_status_t wide_attention_decode(wide_dtype_t dt, int64_t batch, int32_t L, int32_t n_q_heads,
                                    int32_t n_kv_heads, int32_t head_dim, int32_t group_size,
                                    const uint8_t* mask, const int32_t* kv_len, int32_t kv_layout,
                                    const void* q, const void* k_cache, const void* v_cache, void* o,
                                    void* ws, size_t ws_bytes, hipStream_t stream) {
  AttnShape s;
  CHECK(attention_decode_shape(dt, batch, L, n_q_heads, n_kv_heads, head_dim, group_size, s));
  if (kv_layout != WIDE_KV_TOKEN_MAJOR && kv_layout != WIDE_KV_HEAD_MAJOR)
    return fail(WIDE_ERR_INVALID_ARG, "kv_layout must be WIDE_KV_TOKEN_MAJOR or WIDE_KV_HEAD_MAJOR");
  if (batch == 0) return ok();
  CHECK(check_ptr(mask, "mask"));
  if (kv_len) CHECK(check_ptr(kv_len, "kv_len", false));
  CHECK(check_ptr(q, "q"));
  CHECK(check_ptr(k_cache, "k_cache"));
  CHECK(check_ptr(v_cache, "v_cache"));
  CHECK(check_ptr(o, "o"));
  CHECK(check_ws(ws, ws_bytes, attention_decode_ws(batch, L, n_q_heads, n_kv_heads)));
  wide::AttnDecArgs a{};
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k_cache);
  a.v = static_cast<const uint16_t*>(v_cache);
  a.o = static_cast<uint16_t*>(o);
  a.mask = mask;
  a.kv_len = kv_len;
  a.part = static_cast<float*>(ws);
  a.B = (int)batch;
  a.L = L;
  a.n_q = n_q_heads;
  a.n_kv = n_kv_heads;
  a.ng = s.ng;
  a.hpg = s.hpg;
  a.qpk = s.qpk;
  a.head_major = kv_layout == WIDE_KV_HEAD_MAJOR;
  a.chunk = wide::attn_decode_chunk(a.B, n_kv_heads, L);
  a.n_chunks = (L + a.chunk - 1) / a.chunk;
  a.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)head_dim));
  const hipError_t e = wide::launch_attention_decode(a, stream);
  if (e != hipSuccess) return hip_fail(e, "attention decode");
  return ok();
}
