/*
 * WIDE masked-projection oracle: plain, slow, fp64 CPU reference.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may call, link or
 * load this file; only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark use it.  It shares no code with the HIP library.
 *
 * What it computes (WIDE, "Token-level Dynamic Width Pruning"):
 *   - the per-group stable sort of the routing mask (Section 3.3, the SortDesc
 *     equation; Appendix B, Algorithm 1);
 *   - N-axis masked projections: Q and the SwiGLU gate/up pair, pruned over
 *     their out-features (Section 3.1, equations (1)-(3), Figure 1 caption);
 *   - K-axis masked projections: W_o and W_down, pruned over their
 *     in-features (Section 3.1 equations (2)-(3); Appendix B, the masked
 *     K-axis sum that defines GEMM-K);
 *   - the complete masked SwiGLU FFN of equation (3);
 *   - the bottleneck router in its inference form (Section 3.1, "Routing
 *     Components"): logits X W1 W2 read as n_groups pairs, and the mask bit
 *     "class 0 (execute) wins the pair";
 *   - head-group masked attention at prefill (Section 3.1 equations (1)-(2);
 *     Appendix B, Algorithm 4): an active (token, head group) attends as in
 *     standard scaled dot-product attention, an inactive one outputs zeros.
 *
 * Every floating-point input is widened exactly to fp64 (bf16 bit patterns or
 * fp32 values) and every sum is accumulated in fp64 in natural index order,
 * token by token, over the active groups only.  When `round_bf16` is set the
 * oracle rounds to bf16 (round-to-nearest-even, straight from fp64) at the
 * points where the bf16 data path stores a tensor: the FFN intermediate H,
 * and every output.  Parallelised with OpenMP over tokens only; each token's
 * arithmetic is sequential and identical to the serial loop.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ---- input widening --------------------------------------------------- */

/* dtype 0: fp32 array; dtype 1: bf16 bit patterns (uint16). */
static inline double load_elem(const void* p, int dtype, int64_t i) {
  if (dtype == 1) {
    uint32_t bits = ((uint32_t)((const uint16_t*)p)[i]) << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
  }
  return (double)((const float*)p)[i];
}

/* ---- bf16 rounding ------------------------------------------------------ */

/* Round an fp64 value to the nearest bf16 value (8 significant bits,
 * exponent range of fp32), ties to even, in one step from fp64 (no
 * intermediate fp32 rounding).  Returns the rounded value as fp64. */
double oracle_bf16_round(double v) {
  if (isnan(v) || isinf(v) || v == 0.0) return v;
  int e;
  frexp(v, &e);               /* v = f * 2^e, 0.5 <= |f| < 1 */
  if (e < -125) e = -125;     /* below the normal range the quantum is fixed */
  double q = ldexp(1.0, e - 8);  /* spacing of bf16 values in this binade */
  double r = nearbyint(v / q) * q;  /* v/q exact; nearbyint: ties to even */
  const double bf16_max = 3.3895313892515355e38; /* 0x7F7F */
  if (fabs(r) > bf16_max) r = copysign(INFINITY, v);
  return r;
}

static inline double store_round(double v, int round_bf16) {
  return round_bf16 ? oracle_bf16_round(v) : v;
}

static inline double silu(double a) { return a / (1.0 + exp(-a)); }

/* ---- mask reordering (Section 3.3 SortDesc; Algorithm 1) -------------- */

/* For each routing column g: idx[g*M + 0 .. cnt[g]) lists the tokens t with
 * mask[t*n_groups+g] != 0 in ascending order, followed by the remaining
 * tokens in ascending order; cnt[g] counts the active ones.  A descending
 * sort of a 0/1 column whose ties keep token order. */
void oracle_mask_reorder(const uint8_t* mask, int64_t M, int32_t n_groups,
                         int32_t* idx, int32_t* cnt) {
  for (int32_t g = 0; g < n_groups; ++g) {
    int32_t* out = idx + (int64_t)g * M;
    int64_t j = 0;
    for (int64_t t = 0; t < M; ++t)
      if (mask[t * n_groups + g] != 0) out[j++] = (int32_t)t;
    cnt[g] = (int32_t)j;
    for (int64_t t = 0; t < M; ++t)
      if (mask[t * n_groups + g] == 0) out[j++] = (int32_t)t;
  }
}

/* ---- dense projection --------------------------------------------------- */

/* out[t, n] = sum_k x[t, k] * w[n, k]   (x: [M][K], w: [N][K], nn.Linear
 * layout).  Used for the unpruned K and V projections (equation (1)). */
void oracle_linear(int dtype, int round_bf16, int64_t M, int32_t K, int32_t N,
                   const void* x, const void* w, double* out) {
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t t = 0; t < M; ++t) {
    for (int32_t n = 0; n < N; ++n) {
      double acc = 0.0;
      for (int32_t k = 0; k < K; ++k)
        acc += load_elem(x, dtype, t * K + k) * load_elem(w, dtype, (int64_t)n * K + k);
      out[t * N + n] = store_round(acc, round_bf16);
    }
  }
}

/* ---- N-axis masked projection (Q; Section 3.1, Figure 1) ---------------- */

/* The out-feature axis N is cut into n_groups = N / G contiguous groups.
 * out[t, n] = sum_k x[t,k] w[n,k] when group n/G is active for token t,
 * and exactly zero otherwise. */
void oracle_nproj(int dtype, int round_bf16, int64_t M, int32_t K, int32_t N,
                  int32_t G, const uint8_t* mask, const void* x, const void* w,
                  double* out) {
  const int32_t n_groups = N / G;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t t = 0; t < M; ++t) {
    for (int32_t n = 0; n < N; ++n) out[t * N + n] = 0.0;
    for (int32_t g = 0; g < n_groups; ++g) {
      if (mask[t * n_groups + g] == 0) continue;
      for (int32_t n = g * G; n < (g + 1) * G; ++n) {
        double acc = 0.0;
        for (int32_t k = 0; k < K; ++k)
          acc += load_elem(x, dtype, t * K + k) * load_elem(w, dtype, (int64_t)n * K + k);
        out[t * N + n] = store_round(acc, round_bf16);
      }
    }
  }
}

/* ---- K-axis masked projection (W_o, W_down; Appendix B GEMM-K sum) ------ */

/* The in-feature (reduction) axis K is cut into n_groups = K / G groups.
 * out[t, n] = sum over active groups g of sum_{k in group g} a[t,k] w[n,k]:
 * inactive groups contribute nothing, whatever a holds there. */
void oracle_kproj(int dtype, int round_bf16, int64_t M, int32_t K, int32_t N,
                  int32_t G, const uint8_t* mask, const void* a, const void* w,
                  double* out) {
  const int32_t n_groups = K / G;
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t t = 0; t < M; ++t) {
    for (int32_t n = 0; n < N; ++n) {
      double acc = 0.0;
      for (int32_t g = 0; g < n_groups; ++g) {
        if (mask[t * n_groups + g] == 0) continue;
        for (int32_t k = g * G; k < (g + 1) * G; ++k)
          acc += load_elem(a, dtype, t * K + k) * load_elem(w, dtype, (int64_t)n * K + k);
      }
      out[t * N + n] = store_round(acc, round_bf16);
    }
  }
}

/* ---- masked SwiGLU FFN (Section 3.1, equation (3)) ---------------------- */

/* x: [M][D]; w_gate, w_up: [Dff][D]; w_down: [D][Dff]; mask: [M][Dff/G].
 * For each token, for each active group g and each channel j of that group:
 *   h_j = silu(x . w_gate[j]) * (x . w_up[j])   (rounded to bf16 if asked)
 *   y  += h_j * w_down[:, j]
 * then y is rounded to bf16 if asked.  h (optional, [M][Dff]) receives the
 * stored intermediate, zero at inactive groups. */
void oracle_ffn(int dtype, int round_bf16, int64_t M, int32_t D, int32_t Dff,
                int32_t G, const uint8_t* mask, const void* x,
                const void* w_gate, const void* w_up, const void* w_down,
                double* h, double* y) {
  const int32_t n_groups = Dff / G;
#pragma omp parallel
  {
    double* acc = (double*)malloc(sizeof(double) * (size_t)D);
#pragma omp for schedule(dynamic, 1)
    for (int64_t t = 0; t < M; ++t) {
      for (int32_t n = 0; n < D; ++n) acc[n] = 0.0;
      if (h)
        for (int32_t j = 0; j < Dff; ++j) h[t * Dff + j] = 0.0;
      for (int32_t g = 0; g < n_groups; ++g) {
        if (mask[t * n_groups + g] == 0) continue;
        for (int32_t j = g * G; j < (g + 1) * G; ++j) {
          double a = 0.0, b = 0.0;
          for (int32_t k = 0; k < D; ++k) {
            double xv = load_elem(x, dtype, t * D + k);
            a += xv * load_elem(w_gate, dtype, (int64_t)j * D + k);
            b += xv * load_elem(w_up, dtype, (int64_t)j * D + k);
          }
          double hj = store_round(silu(a) * b, round_bf16);
          if (h) h[t * Dff + j] = hj;
          for (int32_t n = 0; n < D; ++n)
            acc[n] += hj * load_elem(w_down, dtype, (int64_t)n * Dff + j);
        }
      }
      for (int32_t n = 0; n < D; ++n) y[t * D + n] = store_round(acc[n], round_bf16);
    }
    free(acc);
  }
}

/* ---- bottleneck router (Section 3.1, Routing Components) --------------- */

/* Inference form of the router: R = X W1 W2 with W1 in R^{D x r} and W2 in
 * R^{r x 2 n_groups}, reshaped to [M][n_groups][2]; the mask bit of group g
 * is 1 when the argmax over the pair is class 0 (execution).  argmax returns
 * the first maximal index, so a tie executes.
 *
 * The weights are passed transposed, as linear-layer weights: w1 is
 * [r][D] (row i = column i of W1) and w2 is [2 n_groups][r] (row j = column
 * j of W2).  The bottleneck activation is kept in fp64, unrounded.
 * logits: [M][2 n_groups] fp64 out; mask: [M][n_groups] out. */
void oracle_router(int dtype, int64_t M, int32_t D, int32_t r, int32_t n_groups,
                   const void* x, const void* w1, const void* w2, double* logits,
                   uint8_t* mask) {
  const int32_t J = 2 * n_groups;
#pragma omp parallel
  {
    double* h = (double*)malloc(sizeof(double) * (size_t)(r > 0 ? r : 1));
#pragma omp for schedule(static)
    for (int64_t t = 0; t < M; ++t) {
      for (int32_t i = 0; i < r; ++i) {
        double acc = 0.0;
        for (int32_t k = 0; k < D; ++k)
          acc += load_elem(x, dtype, t * D + k) * load_elem(w1, dtype, (int64_t)i * D + k);
        h[i] = acc;
      }
      for (int32_t j = 0; j < J; ++j) {
        double acc = 0.0;
        for (int32_t i = 0; i < r; ++i) acc += h[i] * load_elem(w2, dtype, (int64_t)j * r + i);
        logits[t * J + j] = acc;
      }
      for (int32_t g = 0; g < n_groups; ++g)
        mask[t * n_groups + g] = logits[t * J + 2 * g] >= logits[t * J + 2 * g + 1] ? 1 : 0;
    }
    free(h);
  }
}

/* ---- head-group masked attention, prefill (Section 3.1; Algorithm 4) --- */

/* n_seq sequences, T_q queries and T_k keys each (query row t = b*T_q + p,
 * key row b*T_k + j).  Query head h belongs to head group h / (n_q / n_groups)
 * and reads KV head h / (n_q / n_kv).  For an active (t, group):
 * o[t][h] = sum_j softmax_j(q[t][h] . k[j][hkv] / sqrt(d)) v[j][hkv] over the
 * keys of sequence b, and with causal masking only those with
 * j <= p + (T_k - T_q) (queries are the last T_q positions of the sequence);
 * for an inactive one o[t][h] = 0.  With left padding (leftpad not NULL,
 * Algorithm 4's first key j_min = leftpad(b)) the keys j < leftpad[b] of
 * sequence b are not visible either; a query that sees no key gets o = 0.
 * The softmax is the textbook one: subtract the row maximum, exponentiate,
 * divide by the sum, all in fp64.  Layouts: q/o [n_seq*T_q][n_q*d],
 * k/v [n_seq*T_k][n_kv*d], mask [n_seq*T_q][n_groups], leftpad [n_seq]. */
void oracle_attention(int dtype, int round_bf16, int64_t n_seq, int32_t T_q, int32_t T_k,
                      int32_t n_q, int32_t n_kv, int32_t d, int32_t n_groups, int causal,
                      const uint8_t* mask, const void* q, const void* k, const void* v,
                      const int32_t* leftpad, double* o) {
  const int64_t M = n_seq * T_q;
  const int32_t hpg = n_q / n_groups, qpk = n_q / n_kv;
  const int64_t delta = (int64_t)T_k - T_q;
  const double scale = 1.0 / sqrt((double)d);
#pragma omp parallel
  {
    double* s = (double*)malloc(sizeof(double) * (size_t)(T_k > 0 ? T_k : 1));
    double* acc = (double*)malloc(sizeof(double) * (size_t)(d > 0 ? d : 1));
#pragma omp for schedule(static)
    for (int64_t t = 0; t < M; ++t) {
      const int64_t b = t / T_q, p = t % T_q;
      const int64_t nk = causal ? p + delta + 1 : T_k; /* keys j0 .. nk-1 are visible */
      const int64_t j0 = leftpad ? leftpad[b] : 0;
      const int64_t kr0 = b * T_k;                     /* first key row of sequence b */
      for (int32_t h = 0; h < n_q; ++h) {
        double* out = o + t * (int64_t)n_q * d + (int64_t)h * d;
        if (mask[t * n_groups + h / hpg] == 0 || j0 >= nk) {
          for (int32_t e = 0; e < d; ++e) out[e] = 0.0;
          continue;
        }
        const int32_t hk = h / qpk;
        double mx = -INFINITY;
        for (int64_t j = j0; j < nk; ++j) {
          double dot = 0.0;
          for (int32_t e = 0; e < d; ++e)
            dot += load_elem(q, dtype, t * (int64_t)n_q * d + (int64_t)h * d + e) *
                   load_elem(k, dtype, (kr0 + j) * (int64_t)n_kv * d + (int64_t)hk * d + e);
          s[j] = dot * scale;
          if (s[j] > mx) mx = s[j];
        }
        double z = 0.0;
        for (int64_t j = j0; j < nk; ++j) {
          s[j] = exp(s[j] - mx);
          z += s[j];
        }
        for (int32_t e = 0; e < d; ++e) acc[e] = 0.0;
        for (int64_t j = j0; j < nk; ++j)
          for (int32_t e = 0; e < d; ++e)
            acc[e] += s[j] * load_elem(v, dtype, (kr0 + j) * (int64_t)n_kv * d + (int64_t)hk * d + e);
        for (int32_t e = 0; e < d; ++e) out[e] = store_round(acc[e] / z, round_bf16);
      }
    }
    free(s);
    free(acc);
  }
}

/* Number of OpenMP threads the oracle runs with (for reporting). */
int oracle_num_threads(void) {
  int n = 1;
#pragma omp parallel
  {
#pragma omp single
    {
#ifdef _OPENMP
      extern int omp_get_num_threads(void);
      n = omp_get_num_threads();
#endif
    }
  }
  return n;
}
