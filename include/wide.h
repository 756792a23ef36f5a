/*
 * libwide: token-level dynamic-width masked projections on MI355X (gfx950).
 *
 * Implements the inference hot path of WIDE ("Token-level Dynamic Width
 * Pruning"): every token executes only the FFN channel groups and attention
 * head groups that its binary routing mask selects.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - All pointers except `ws_bytes`-sized host scalars are DEVICE pointers to
 *    memory on the current HIP device.  All tensors are row-major and
 *    contiguous; weights use the nn.Linear layout [out_features][in_features].
 *  - Floating-point tensors are fp32 (WIDE_F32) or bf16 (WIDE_BF16, stored as
 *    16-bit patterns).  On the bf16 path products accumulate in fp32 and every
 *    stored tensor (the FFN intermediate H, Q/K/V, y) is rounded to bf16,
 *    nearest-even.  On the fp32 path everything stays fp32.
 *  - A routing mask is uint8 [M][n_groups], token-major; any nonzero byte
 *    means "execute this group for this token" (class 0 of the router in
 *    Section 3.1), zero means "skip".
 *  - Pointers must be 16-byte aligned and row lengths (d_model, d_ff,
 *    n_heads*head_dim) multiples of 8 elements, so every row starts on a
 *    128-bit boundary; otherwise WIDE_ERR_INVALID_ARG.
 *  - The caller owns every buffer, including the workspace `ws` (device
 *    memory of at least wide_workspace_size() bytes, 256-byte aligned).  The
 *    library allocates nothing per call, never synchronises the host with the
 *    device, and only enqueues work on `stream` (0 = the null stream); calls
 *    can be captured into a HIP graph.  Calls that share a workspace must be
 *    ordered on one stream.
 *  - Validation happens on the host before anything is enqueued.  On any
 *    non-OK status no output has been touched and wide_last_error() describes
 *    the problem.  No entry point throws or aborts.
 *  - M == 0 is a valid no-op.
 *  - Every output element is written: skipped (inactive) N-axis blocks are
 *    +0, and a token whose mask row is all zero gets an all-zero output row.
 *  - Only idx/counts are bit-reproducible run to run; some prefill K-axis
 *    paths reduce with fp32 atomics whose order varies.
 */
#ifndef WIDE_H
#define WIDE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  WIDE_KV_TOKEN_MAJOR = 0, /* cache [batch][L][n_kv_heads*head_dim]  */
  WIDE_KV_HEAD_MAJOR = 1   /* cache [batch][n_kv_heads][L][head_dim] */
} wide_kv_layout_t;

typedef enum {
  WIDE_OK = 0,
  WIDE_ERR_INVALID_ARG = 1, /* bad pointer, shape, alignment or enum       */
  WIDE_ERR_UNSUPPORTED = 2, /* valid per the paper but not implemented here */
  WIDE_ERR_WORKSPACE = 3,   /* ws NULL or smaller than required             */
  WIDE_ERR_HIP = 4          /* a HIP launch or runtime call failed          */
} wide_status_t;

typedef enum { WIDE_F32 = 0, WIDE_BF16 = 1 } wide_dtype_t;

typedef enum { WIDE_PHASE_QKV = 0, WIDE_PHASE_O = 1 } wide_phase_t;

typedef enum {
  WIDE_OP_REORDER = 0,
  WIDE_OP_FFN = 1,
  WIDE_OP_QKV = 2,
  WIDE_OP_O = 3,
  WIDE_OP_ROUTER = 4
} wide_op_t;

/*
 * Mask reordering (WIDE Section 3.3, the per-column SortDesc; Appendix B,
 * Algorithm 1).  For every routing column g in [0, n_groups):
 *   idx[g*M + 0 .. counts[g])  = tokens t with mask[t*n_groups+g] != 0,
 *                                in ascending order,
 *   idx[g*M + counts[g] .. M)  = the remaining tokens, ascending,
 *   counts[g]                  = number of active tokens.
 * This is the descending sort of a 0/1 column with ties kept in token order,
 * so the result is unique and bit-exact.
 *   mask    [M][n_groups] uint8, read only.
 *   idx     [n_groups][M] int32, written.      counts [n_groups] int32, written.
 *   ws      workspace of wide_workspace_size(WIDE_OP_REORDER, ., M, 0,
 *           n_groups, 1) bytes (per-chunk counts).
 * Limits: 0 <= M < 2^31, 1 <= n_groups <= 4096.
 */
wide_status_t wide_mask_reorder(const uint8_t* mask, int64_t M, int32_t n_groups,
                                int32_t* idx, int32_t* counts, void* ws,
                                size_t ws_bytes, hipStream_t stream);

/*
 * Masked SwiGLU FFN (WIDE Section 3.1, equation (3), with phi = SiLU):
 *   h[t, j] = silu(x_t . w_gate[j]) * (x_t . w_up[j])  if group j/G is active
 *             for token t, else +0;
 *   y[t]    = sum over active groups g of h[t, gG:(g+1)G] . w_down[:, gG:(g+1)G]^T.
 * W_gate and W_up are pruned over their out-features (N-axis), W_down over its
 * in-features (K-axis); one mask covers the whole FFN.
 *   dt          WIDE_BF16 or WIDE_F32 (applies to x, weights, h_out, y).
 *   M           tokens (B*T flattened).
 *   d_model, d_ff, group_size (G): G must be a power of two >= 16 dividing
 *               d_ff (Section 3.1: the tile-size set {2^k, k >= 4}), or d_ff
 *               itself: one group, so each token runs the whole FFN or none
 *               of it (the M-axis case of Appendix A).  d_model and d_ff are
 *               multiples of 8 and there are at most 4096 groups
 *               (WIDE_ERR_INVALID_ARG / WIDE_ERR_UNSUPPORTED otherwise).
 *               Limits of the kernels (WIDE_ERR_UNSUPPORTED): bf16 needs
 *               d_model % 256 == 0; with G = 16 or 32 also d_ff % 128 == 0
 *               and d_ff <= 32768; with G = d_ff not a power of two, d_ff %
 *               128 == 0.  fp32 needs d_model and d_ff multiples of 16.
 *   mask        [M][d_ff/G] uint8.
 *   idx, counts optional reorder of `mask` from wide_mask_reorder (reusable by
 *               every operator under the same routing decision, Appendix B);
 *               both NULL => computed internally into the workspace.  Passing
 *               a reorder that does not match `mask` is undefined behaviour.
 *   x           [M][d_model];  w_gate, w_up [d_ff][d_model];
 *   w_down      [d_model][d_ff].
 *   h_out       optional [M][d_ff] output of the intermediate (inactive
 *               blocks +0); NULL => kept in the workspace.
 *   y           [M][d_model] output.
 *   ws          workspace, >= wide_workspace_size(WIDE_OP_FFN, dt, M, d_model,
 *               d_ff, G) bytes.
 */
wide_status_t wide_ffn_masked(wide_dtype_t dt, int64_t M, int32_t d_model,
                              int32_t d_ff, int32_t group_size,
                              const uint8_t* mask, const int32_t* idx,
                              const int32_t* counts, const void* x,
                              const void* w_gate, const void* w_up,
                              const void* w_down, void* h_out, void* y,
                              void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * wide_ffn_masked without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  Same arguments, semantics and errors as
 * wide_ffn_masked minus ws/ws_bytes; the scratch it needs (the reorder, H
 * when h_out is NULL, the K-axis scratch) lives in a device array inside the
 * library of wide_static_scratch_bytes() bytes (32 MiB) per GPU, held from the
 * first call on that GPU until the process ends.  A call needing more scratch
 * than that (wide_workspace_size(WIDE_OP_FFN, ...) > 32 MiB, e.g. a long
 * prefill with h_out NULL) returns WIDE_ERR_WORKSPACE before enqueuing
 * anything.  Nothing is allocated and no library routine that allocates is
 * called.  The first call on a device looks up the array's address on that
 * device (make it outside graph capture, with that device current).
 * Every call on one GPU shares that GPU's scratch: calls that overlap on one
 * GPU (concurrent streams, other host threads) race and must be ordered by
 * the caller (e.g. issued on one stream).
 */
wide_status_t wide_ffn_masked_noalloc(wide_dtype_t dt, int64_t M, int32_t d_model,
                                      int32_t d_ff, int32_t group_size,
                                      const uint8_t* mask, const int32_t* idx,
                                      const int32_t* counts, const void* x,
                                      const void* w_gate, const void* w_up,
                                      const void* w_down, void* h_out, void* y,
                                      hipStream_t stream);

/* Bytes of the per-GPU scratch of wide_ffn_masked_noalloc (32 MiB). */
size_t wide_static_scratch_bytes(void);

/*
 * Head-group masked attention projections (WIDE Section 3.1, equations
 * (1)-(2) and Figure 1): W_q is pruned over its out-features and W_o over its
 * in-features in groups of G = group_size features (whole heads, contiguous:
 * group g holds q-heads [g*G/head_dim, (g+1)*G/head_dim)); W_k and W_v stay
 * dense so the KV cache is never pruned.
 *
 * phase WIDE_PHASE_QKV:
 *   q[t, gG:(g+1)G] = x_t . w_q[gG:(g+1)G]^T if group g is active, else +0;
 *   k = x w_k^T and v = x w_v^T, dense.
 *   in = x [M][d_model]; w_q [n_q*hd][d_model]; w_k, w_v [n_kv*hd][d_model];
 *   q [M][n_q*hd]; k, v [M][n_kv*hd].  w_o and y are ignored (may be NULL).
 * phase WIDE_PHASE_O:
 *   y[t] = sum over active g of in[t, gG:(g+1)G] . w_o[:, gG:(g+1)G]^T
 *   (the attention output gated by the mask before W_o, equation (2)).
 *   in = attention output [M][n_q*hd]; w_o [d_model][n_q*hd]; y [M][d_model].
 *   Inactive blocks of `in` are never read.  w_q/w_k/w_v/q/k/v are ignored.
 * Shapes: n_q a multiple of n_kv; G a multiple of head_dim dividing n_q*hd
 * (the paper's default is (n_q/n_kv)*head_dim, one KV head per group); at
 * most 4096 groups.  Limits of the kernels (WIDE_ERR_UNSUPPORTED): bf16
 * needs d_model % 256 == 0, n_kv*hd % 128 == 0 and G = 64 (then n_q*hd and
 * n_kv*hd % 256 == 0) or a multiple of 128; fp32 needs d_model, n_kv*hd and
 * G multiples of 16.
 * mask [M][n_q*hd/G]; idx/counts as for wide_ffn_masked (same routing
 * decision for both phases, Appendix B).
 * ws >= wide_workspace_size(phase == QKV ? WIDE_OP_QKV : WIDE_OP_O, dt, M,
 *       d_model, n_q*hd, G) bytes.
 */
wide_status_t wide_qkvo_masked(wide_phase_t phase, wide_dtype_t dt, int64_t M,
                               int32_t d_model, int32_t n_q_heads,
                               int32_t n_kv_heads, int32_t head_dim,
                               int32_t group_size, const uint8_t* mask,
                               const int32_t* idx, const int32_t* counts,
                               const void* in, const void* w_q,
                               const void* w_k, const void* w_v,
                               const void* w_o, void* q, void* k, void* v,
                               void* y, void* ws, size_t ws_bytes,
                               hipStream_t stream);

/*
 * Bottleneck router, inference form (WIDE Section 3.1, "Routing Components").
 * R = X W1 W2 is read as n_groups pairs (class 0 = execute, class 1 = skip);
 * mask[t][g] = 1 when class 0 wins the pair, i.e. R[t][2g] >= R[t][2g+1]
 * (argmax returns the first maximal class, so a tie executes), else 0.
 *   x        [M][d_model] bf16.
 *   w1       [rank][d_model] bf16: W1 transposed (linear-layer layout),
 *            1 <= rank <= 32.
 *   w2       [2*n_groups][rank] bf16: W2 transposed; rows 2g and 2g+1 are
 *            group g's execute and skip logits.
 *   mask     [M][n_groups] uint8 out (1 execute, 0 skip).
 *   logits   optional [M][2*n_groups] fp32 out (R); NULL skips it.
 *   idx, counts  optional, both or neither: the reorder of the new mask, as
 *            wide_mask_reorder computes it (with M == 0 only counts is
 *            written, all zero, and idx may be NULL).
 *   ws       workspace of wide_workspace_size(WIDE_OP_ROUTER, WIDE_BF16, M,
 *            d_model, n_groups, rank) bytes (used by the reorder).
 * Arithmetic: X W1 with bf16 products summed in fp32 and kept in fp32 (not
 * rounded to bf16); R in fp32; the decision is taken on the fp32 R.
 * Limits: bf16 only (WIDE_ERR_UNSUPPORTED otherwise); d_model % 64 == 0;
 * 1 <= n_groups <= 4096; 0 <= M < 2^31.
 */
wide_status_t wide_router(wide_dtype_t dt, int64_t M, int32_t d_model, int32_t rank,
                          int32_t n_groups, const void* x, const void* w1, const void* w2,
                          uint8_t* mask, float* logits, int32_t* idx, int32_t* counts,
                          void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Head-group masked attention, prefill (WIDE Section 3.1, equations (1)-(2);
 * Appendix B, Algorithm 4).  For query token t = b*T_q + p of sequence b and
 * query head h in head group g = h / (group_size/head_dim):
 *   o[t, h] = sum_j softmax_j(q[t, h] . k[b*T_k + j, h_kv] / sqrt(head_dim))
 *             v[b*T_k + j, h_kv]     if mask[t][g] != 0, else +0,
 * with h_kv = h / (n_q_heads/n_kv_heads), over the keys j of sequence b;
 * with causal = 1 only keys j <= p + (T_k - T_q) (the queries are the last
 * T_q of the sequence's T_k positions, as after a cached prefix), and with
 * left padding only keys j >= leftpad[b] (Algorithm 4's first key
 * leftpad(b)); a query that sees no key at all gets +0.
 *   dt        WIDE_BF16 (WIDE_ERR_UNSUPPORTED otherwise).
 *   n_seq, T_q, T_k   sequences and their query / key lengths; causal needs
 *             T_k >= T_q, and T_k >= 1 whenever there are queries.
 *   leftpad   optional int32 [n_seq] (device): the first non-padding key of
 *             each sequence, in [0, T_k] (values outside are clamped); NULL
 *             means no padding.  With padding the key-range split is off.
 *   n_q_heads, n_kv_heads, head_dim (128 only, else WIDE_ERR_UNSUPPORTED),
 *   group_size  as for wide_qkvo_masked (a multiple of head_dim dividing
 *             n_q_heads*head_dim; group g holds contiguous heads).
 *   mask      [n_seq*T_q][n_q_heads*head_dim/group_size] uint8.
 *   idx, counts  optional reorder of `mask` (wide_mask_reorder over the
 *             n_seq*T_q tokens: the same routing decision as the Q and O
 *             projections, Appendix B); both NULL => computed internally.
 *   q         [n_seq*T_q][n_q_heads*head_dim]; k, v [n_seq*T_k][n_kv_heads*head_dim].
 *   o         [n_seq*T_q][n_q_heads*head_dim] out; every element is written
 *             (inactive (token, group) rows +0).
 *   ws        >= wide_attention_workspace_size(...) bytes (a transposed copy
 *             of V, per-sequence offsets, the reorder when idx is NULL, and,
 *             for one sequence with 8..1024 key tiles of 64 while the
 *             "attn_split" option is on, the key-range split's schedule and
 *             fp32 partials: 138 MB).
 * With few active query tiles (one causal sequence, at most "attn_split"
 * tiles of 32 rows x a head block) the tiles' causal key ranges are cut into
 * chunks run by separate workgroups; a third kernel combines each tile's
 * chunks in chunk order (the result is deterministic, and differs from the
 * unsplit run only in fp32 summation order).
 * Arithmetic: scores as fp32 sums of bf16 products; softmax in fp32 (online,
 * one running maximum and sum per query); the probabilities are rounded to
 * bf16 for the P.V product, which accumulates in fp32; o is rounded to bf16.
 * n_seq*T_q == 0 is a valid no-op.
 */
wide_status_t wide_attention_masked(wide_dtype_t dt, int64_t n_seq, int32_t T_q, int32_t T_k,
                                    int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                    int32_t group_size, int32_t causal, const int32_t* leftpad,
                                    const uint8_t* mask, const int32_t* idx,
                                    const int32_t* counts, const void* q, const void* k,
                                    const void* v, void* o, void* ws, size_t ws_bytes,
                                    hipStream_t stream);

/*
 * Head-group masked attention, decode (WIDE Section 3.1, equations (1)-(2);
 * Appendix B: at decode the reorder is bypassed and the routing is checked
 * per block).  One query token per sequence b attends to its cached keys:
 *   o[b, h] = sum_{j < len_b} softmax_j(q[b, h] . k[b, j, h_kv] / sqrt(head_dim))
 *             v[b, j, h_kv]      if mask[b][g(h)] != 0, else +0,
 * with g(h) = h / (group_size/head_dim), h_kv = h / (n_q_heads/n_kv_heads)
 * and len_b = min(kv_len[b], L) (L when kv_len is NULL; len_b <= 0 gives +0).
 * A (sequence, KV head) none of whose query heads is active reads nothing of
 * the cache.
 *   dt        WIDE_BF16 (WIDE_ERR_UNSUPPORTED otherwise).
 *   batch, L  sequences and the cache capacity (rows per sequence).
 *   n_q_heads, n_kv_heads (at most 16 query heads per KV head), head_dim (128
 *             only), group_size as for wide_qkvo_masked.
 *   mask      [batch][n_q_heads*head_dim/group_size] uint8.
 *   kv_len    optional int32 [batch] (device).
 *   kv_layout WIDE_KV_TOKEN_MAJOR: k_cache, v_cache [batch][L][n_kv_heads*head_dim]
 *             (rows as the K/V projections write them); WIDE_KV_HEAD_MAJOR:
 *             [batch][n_kv_heads][L][head_dim] (one KV head's cache contiguous,
 *             so skipping a KV head skips a contiguous block).
 *   q         [batch][n_q_heads*head_dim]; o [batch][n_q_heads*head_dim] out.
 *   ws        >= wide_attention_decode_workspace_size(...) bytes (per-chunk
 *             partial maxima, sums and outputs).
 * Arithmetic: scores from bf16 pairs with fp32 sums; softmax and P.V in fp32
 * (probabilities are not rounded); partial results over key chunks are merged
 * in fp32; o is rounded to bf16.
 */
wide_status_t wide_attention_decode(wide_dtype_t dt, int64_t batch, int32_t L, int32_t n_q_heads,
                                    int32_t n_kv_heads, int32_t head_dim, int32_t group_size,
                                    const uint8_t* mask, const int32_t* kv_len, int32_t kv_layout,
                                    const void* q, const void* k_cache, const void* v_cache, void* o,
                                    void* ws, size_t ws_bytes, hipStream_t stream);

/* Workspace bytes for wide_attention_decode (SIZE_MAX for rejected shapes). */
size_t wide_attention_decode_workspace_size(int64_t batch, int32_t L, int32_t n_q_heads,
                                            int32_t n_kv_heads, int32_t head_dim,
                                            int32_t group_size);

/*
 * Workspace bytes for wide_attention_masked (with_reorder != 0: idx/counts
 * will be NULL and the reorder is held in the workspace).  SIZE_MAX for
 * shapes wide_attention_masked would reject (causal-only checks aside).
 */
size_t wide_attention_workspace_size(int64_t n_seq, int32_t T_q, int32_t T_k,
                                     int32_t n_q_heads, int32_t n_kv_heads,
                                     int32_t head_dim, int32_t group_size,
                                     int32_t with_reorder);

/*
 * Workspace bytes needed by one call (0 is a valid answer).
 *   op = WIDE_OP_REORDER: d_inner = n_groups, group_size = 1, d_model unused.
 *   op = WIDE_OP_FFN:     d_inner = d_ff.
 *   op = WIDE_OP_QKV/O:   d_inner = n_q*head_dim.
 *   op = WIDE_OP_ROUTER:  d_inner = n_groups, group_size = rank.
 * Returns SIZE_MAX for arguments the matching entry point would reject.
 */
size_t wide_workspace_size(wide_op_t op, wide_dtype_t dt, int64_t M,
                           int32_t d_model, int32_t d_inner,
                           int32_t group_size);

/*
 * Process-wide tuning knobs (not part of the paper's interface; every value
 * gives the same result up to fp32 summation order).  Keys:
 *   "decode_max_m"  bf16 calls with M <= value (and M <= 64) use the decode
 *                   kernels, which skip the mask reorder; default 64.
 *   "k_path"        schedule of the prefill K-axis product (down, O):
 *                   0 automatic (default), 1 dense-masked (no atomics),
 *                   2 scatter (the paper's GEMM-K with fp32 atomics).
 *   "mn_order"      tile order of the 256x256 N-axis kernels, three bits
 *                   (default 7).  Bit 2: in the FFN call, each XCD runs the
 *                   gate/up tiles of its groups m-tile by m-tile (m-tile 0
 *                   of every group, then m-tile 1, ...); it takes precedence
 *                   over bit 1 there.  Bit 1: each XCD runs the full tiles
 *                   of its groups first, then their partial last m-tiles,
 *                   then the empty ones.  Bit 0: the Q/K/V call puts the
 *                   dense K and V tiles before the masked Q tiles, so the
 *                   partial Q tiles come last.  Outputs are identical for
 *                   all values.
 *   "mn_tail"       1 (default): in the Q/K/V call, each XCD's last partial
 *                   round of 256x256 tiles is cut along k into chunks run by
 *                   extra workgroups (fp32 partial tiles in the workspace,
 *                   added in a fixed order by a short second kernel); 0 runs
 *                   those tiles whole.  Results differ only in fp32
 *                   summation order.
 *   "kd_pattern"    1 (default): before the dense-masked K-axis schedule on
 *                   256x256 tiles with 2..8 groups (attention's O projection),
 *                   three small kernels order the tokens by mask pattern so a
 *                   tile skips every group none of its rows uses; 0 keeps
 *                   token order.  Outputs are bitwise equal either way.
 *   "ks_pack"       scatter schedule on 256x256 tiles: K-groups one workgroup
 *                   runs in turn (Appendix B, Algorithm 3's outer loop; default
 *                   1); the column tiles are dealt so that all adds into one
 *                   256-column slab come from one XCD.
 *   "big_tiles"     1 (default): prefill GEMMs use 256x256 tiles where the
 *                   shape allows; 0: always the 128x128 tiles.
 *   "gemv_n_ncb", "gemv_k_ncb"
 *                   decode: at most this many blocks of 16 output columns
 *                   (N-axis) or rows (K-axis) per workgroup: 1, 2, 4 or 8
 *                   (8: up to 32 tokens, and for the N axis plain columns
 *                   only); 0 (default) chooses by shape.
 *   "gemv_n_split", "gemv_k_split"
 *                   decode: workgroups sharing one block's reduction: 1, 2, 4
 *                   or 8; 0 (default) chooses by shape.  A split above one
 *                   adds a small kernel that sums the partial results.
 *                   Workspace sizes depend on these four options: query
 *                   wide_workspace_size after setting them.
 *   "attn_split"    prefill attention key-range split: split when at most
 *                   this many query tiles are active (0..1024, default 1024;
 *                   0 never splits).  Changes the
 *                   workspace size: query it again after setting this.
 *   "attn_split_rounds"  chunks per resident workgroup slot the split aims at
 *                   (1..8, default 1: the chunk length is the mean work per
 *                   slot, so only the longer key ranges split).
 * Process-wide settings, stored atomically; a call reads them at several
 * points, so change them between calls, not while calls run on other host
 * threads.
 */
wide_status_t wide_set_option(const char* key, int64_t value);
wide_status_t wide_get_option(const char* key, int64_t* value);

/* Thread-local description of the last non-OK status ("" if none). */
const char* wide_last_error(void);

/*
 * Kernel timing for measurement (not needed for correctness).  When enabled,
 * every kernel launch is bracketed by two HIP events recorded on the launch
 * stream; the events come from a pool created by wide_timing_enable(1) (the
 * only call here that creates HIP objects) and recording stops silently when
 * the pool is exhausted.  wide_timing_query() synchronises on the recorded
 * events and returns, for kernels whose label is `name` -- exactly, or
 * followed by a template argument list or a "/variant" suffix ("wide_mn256"
 * covers "wide_mn256<true>/bk64", not "wide_mn256_x") -- the total elapsed
 * milliseconds and the number of launches.  Do not enable timing while
 * capturing a graph.
 */
wide_status_t wide_timing_enable(int enable);
/*
 * Restrict timing to launches whose label matches `name` (the same rule as
 * wide_timing_query); NULL or "" times every launch again.  Each timed
 * launch adds two event records to its stream, and between short kernels
 * they lengthen the stream by several microseconds each; a measurement of a
 * whole pass can time just the kernel it needs.  Takes effect for launches
 * issued after the call; the recorded events are kept.
 */
wide_status_t wide_timing_filter(const char* name);
wide_status_t wide_timing_reset(void);
wide_status_t wide_timing_query(const char* name, double* total_ms,
                                int64_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* WIDE_H */
