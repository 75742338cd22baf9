/*
 * zeta.h -- C ABI of the Z-order top-k attention (ZETA): the forward pass and
 * the attention gradients, for
 * AMD Instinct MI355X (gfx950).
 *
 * The forward pass has four calls, run in this order on one stream:
 *
 *   zeta_morton_encode  -> Z-order codes of queries and keys
 *   zeta_sort_keys      -> keys sorted by code per (batch, head); called on
 *                          the query codes too, its permutation (regrouped
 *                          by zeta_query_order) is a processing order for
 *                          the next two calls
 *   zeta_select_topk    -> k candidate keys per query around its insertion point
 *   zeta_topk_attn_fwd  -> Cauchy-softmax attention over the candidates
 *
 * zeta_topk_attn_bwd gives the attention's gradients for the same windows.
 * zeta_history_mean prepares the optional history-mean candidate that the
 * attention calls (and the gradients) add to every window.  zeta_exact_knn
 * and zeta_index_overlap measure how well the windows keep the exact nearest
 * keys (the locality experiment).
 *
 * zeta_select_attend_fwd runs the last two in one pass (the candidates never
 * leave the chip); zeta_query_order prepares the fast processing order.
 *
 * Conventions shared by every call:
 *
 * - A "segment" is one (batch, head) pair; B*H segments are independent and
 *   each holds N positions.  Tensors are dense, row-major, with no strides:
 *   q and k are [B][H][N][d_k], v and out are [B][H][N][d_v], codes and
 *   permutations are [B*H][N], idx is [B*H][N][topk].
 * - Every pointer argument is device memory owned by the caller (the library
 *   allocates nothing and keeps no state).  Workspace buffers are caller
 *   supplied; their size comes from zeta_workspace_size.
 * - Every call validates its arguments on the host, enqueues its kernels on
 *   `stream` and returns without synchronising.  Faults inside a kernel
 *   surface at the caller's next synchronisation.  A launch failure reported
 *   by the runtime maps to ZETA_ERR_HIP.
 * - Validation failures return before any GPU work is enqueued and before
 *   any HIP runtime call; nothing is printed and no exception crosses the ABI.
 * - Calls on distinct streams with distinct buffers may run concurrently.
 * - Input floating-point values must be finite.
 */
#ifndef ZETA_H
#define ZETA_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ZETA_OK = 0,
  ZETA_ERR_INVALID_ARG = 1, /* null pointer, size out of range, eps <= 0, aliasing */
  ZETA_ERR_UNSUPPORTED = 2, /* valid but not compiled: d_k > 8, bits > 24, d_v, dtype, topk > 1024 */
  ZETA_ERR_WORKSPACE = 3,   /* workspace null or smaller than the call needs */
  ZETA_ERR_HIP = 4          /* the HIP runtime reported a launch error */
} zeta_status_t;

typedef enum { ZETA_F32 = 0, ZETA_BF16 = 1 } zeta_dtype_t;

/*
 * Attention scores over the selected candidates.  ZETA_SCORE_CAUCHY is the
 * method's Adaptive Cauchy-Softmax (Section 3.3, equation cauchy); the others
 * are the variants the paper compares it with (Section 4.3; Appendix G.2;
 * the dot-product softmax of equation 3), each normalised over the window:
 *   DOT         softmax of q.k / sqrt(d_k)
 *   NEG_EUCLID  softmax of -||q - k||^2 / sqrt(d_k)
 *   INV_EUCLID  weights 1 / (||q - k|| + eps)
 *   NORM_DOT    softmax of (q/|q|).(k/|k|) / sqrt(d_k)  (a zero vector gives 0)
 * Softmax weights are shifted by the window's largest logit.  Only the
 * Cauchy score has gradients (zeta_topk_attn_bwd).
 */
typedef enum {
  ZETA_SCORE_CAUCHY = 0,
  ZETA_SCORE_DOT = 1,
  ZETA_SCORE_NEG_EUCLID = 2,
  ZETA_SCORE_INV_EUCLID = 3,
  ZETA_SCORE_NORM_DOT = 4
} zeta_score_t;

/* Largest supported values of the size parameters. */
#define ZETA_MAX_DK 8
#define ZETA_MAX_TOPK 1024
#define ZETA_MAX_BITS 24 /* 2^bits - 1 and every grid coordinate exact in float32 */

/*
 * zeta_morton_encode -- Z-order codes of queries and keys (Section 3.1,
 * Z-order curves and equation Z; Section 3.2.2 maps queries and keys into the
 * same one-dimensional space).
 *
 * Each coordinate is discretised onto a grid of 2^bits cells,
 *   code_a = clamp(floor((x_a - lo_a) * (2^bits - 1) / (hi_a - lo_a)), 0, 2^bits - 1),
 * evaluated in float32 with one IEEE rounding per operation (subtract,
 * multiply, divide, floor; no fused multiply-add), and 0 when hi_a <= lo_a.
 * The d_k grid coordinates are then interleaved most significant bit first,
 * axis 0 first within each group of d_k bits: bit s of coordinate a goes to
 * bit d_k*s + (d_k - 1 - a) of the code.
 *
 *   q, k        [B][H][N][d_k] of `dtype` (float32, or bfloat16 bit patterns)
 *   range_lohi  optional float32 [B*H][2][d_k]: per segment, lo then hi per
 *               axis.  NULL selects the joint min/max over the segment's
 *               queries and keys.  Values outside a given range clamp.
 *   range_out   optional float32 [B*H][2][d_k]: receives the range used.
 *   q_codes, k_codes  uint32 [B*H][N] outputs.
 *   workspace   at least zeta_workspace_size(...) bytes (used only when
 *               range_lohi is NULL).
 *
 * Requires 1 <= d_k <= ZETA_MAX_DK, 1 <= bits <= ZETA_MAX_BITS, d_k * bits <= 32,
 * B, H, N >= 1 and B*H*N < 2^31.  Outputs must not overlap the inputs.
 */
zeta_status_t zeta_morton_encode(const void* q, const void* k, zeta_dtype_t dtype, int64_t B,
                                 int64_t H, int64_t N, int d_k, int bits,
                                 const float* range_lohi, float* range_out, uint32_t* q_codes,
                                 uint32_t* k_codes, void* workspace, size_t workspace_bytes,
                                 hipStream_t stream);

/*
 * zeta_morton_encode_static -- zeta_morton_encode for callers that cannot
 * allocate or pass a workspace: code under HIP graph capture, tight serving
 * loops, harnesses that forbid device allocation.  Same arguments, layouts,
 * results (bit for bit) and errors as zeta_morton_encode, without the
 * workspace.
 *
 * The per-segment range partials (when range_lohi is NULL) go to a
 * file-scope device array of ZETA_ENCODE_STATIC_SCRATCH_BYTES inside the
 * library: one copy per GPU, looked up once per device on the first call
 * that needs it on that device and held until the process ends.  The call
 * itself allocates nothing (no hipMalloc, no allocating library routine).
 * It needs 24 * B*H * ceil(N / 512) bytes there for d_k = 3 (8 * d_k per
 * segment and 512-row chunk in general); a larger problem returns
 * ZETA_ERR_UNSUPPORTED before any GPU work.  Every call on one GPU shares
 * that GPU's array: calls that overlap in time on one GPU (other streams,
 * other threads) race and must be serialised by the caller.  The stream's
 * device (the current device for the null stream) is the one used.
 */
#define ZETA_ENCODE_STATIC_SCRATCH_BYTES (1u << 20)
zeta_status_t zeta_morton_encode_static(const void* q, const void* k, zeta_dtype_t dtype, int64_t B,
                                        int64_t H, int64_t N, int d_k, int bits,
                                        const float* range_lohi, float* range_out, uint32_t* q_codes,
                                        uint32_t* k_codes, hipStream_t stream);

/*
 * zeta_sort_keys -- sort each segment's key codes ascending (Section 3.2.2,
 * keys sorted in the one-dimensional space; Algorithm 1, Step 2; Appendix B
 * names a radix sort).  Equal codes keep ascending position order (the sort is
 * stable), so the result is fully determined.
 *
 *   k_codes       uint32 [n_segments][N], every code below 2^code_bits.
 *   sorted_codes  uint32 [n_segments][N] output: k_codes[perm] per segment.
 *   perm          int32  [n_segments][N] output: original positions.
 *   code_bits     1..32, the number of significant low bits of each code.
 *
 * Outputs must not overlap k_codes.
 */
zeta_status_t zeta_sort_keys(const uint32_t* k_codes, int64_t n_segments, int64_t N, int code_bits,
                             uint32_t* sorted_codes, int32_t* perm, void* workspace,
                             size_t workspace_bytes, hipStream_t stream);

/*
 * zeta_query_order -- a processing order for zeta_select_topk and
 * zeta_topk_attn_fwd that groups queries by the sorted key list they search.
 *
 * Causal selection searches, for a query at position i, the keys at
 * positions below 2^t in code order, t = max(ceil(log2(topk)), bit length
 * of i) (the full sorted list once 2^t >= N).  This call regroups the given
 * order by that level, keeping the given order inside each level; for the
 * Z-order of the query codes (the permutation zeta_sort_keys returns for
 * them) consecutive queries then search one list with non-decreasing codes
 * and share most of their candidates, which both later calls exploit.  Any
 * permutation gives the same results; this one is the fast one.
 *
 *   q_order    int32 [n_segments][N] permutation per segment, or NULL for
 *              position order.
 *   order_out  int32 [n_segments][N] output; may be the same buffer as
 *              q_order, but must not otherwise overlap it (INVALID_ARG).
 *   topk, causal, chunk  as for zeta_select_topk (non-causal: a copy of
 *              q_order); the levels follow the pool each query has under
 *              the causal rule the later calls use.
 *   workspace  at least zeta_workspace_size(...) bytes.
 */
zeta_status_t zeta_query_order(const int32_t* q_order, int64_t n_segments, int64_t N, int topk,
                               int causal, int chunk, int32_t* order_out, void* workspace,
                               size_t workspace_bytes, hipStream_t stream);

/*
 * zeta_select_topk -- candidate keys of every query (Section 3.2.2: the
 * insertion point of the query's code among the sorted keys by binary search,
 * then a window of k keys centred on it, with causal masking restricting each
 * query to past keys; Algorithm 1, Steps 3-5).
 *
 * For query i the pool is {0..i} when causal (the diagonal included) and all
 * N keys otherwise.  With chunk = M > 0 (causal only) the pool follows the
 * paper's chunked rule instead (Section 3.2.2; Algorithm 1, Step 4): the
 * first floor(i / M) chunks of M positions, i.e. positions below
 * floor(i / M) * M, so queries of the first chunk get no candidate.  Let T be the pool in (code, position) order, L = |pool|,
 * p = number of pool keys whose code is below the query's code,
 * m = min(topk, L) and s = min(max(p - floor(topk/2), 0), L - m).  Then
 * idx[seg][i][0..m) = positions of T[s .. s+m) in that order, and the rest of
 * the row is -1.  The result is unique.
 *
 *   q_codes       uint32 [n_segments][N]
 *   sorted_codes  uint32 [n_segments][N], perm int32 [n_segments][N]: the
 *                 outputs of zeta_sort_keys for the same key codes.
 *   q_order       optional int32 [n_segments][N]: the order in which queries
 *                 are processed, a permutation of 0..N-1 per segment (NULL:
 *                 position order).  It changes no result; zeta_query_order
 *                 gives neighbouring queries overlapping windows and makes the
 *                 call faster.  Entries outside 0..N-1 are skipped.
 *   idx           int32 [n_segments][N][topk] output, indexed by position.
 *   topk          1..ZETA_MAX_TOPK; causal 0 or 1; chunk 0 (exact prefix) or
 *                 a chunk size M >= 1 (requires causal; INVALID_ARG otherwise).
 *   workspace     at least zeta_workspace_size(...) bytes, 16-byte aligned
 *                 (the prefix lists and each query's window as list-index
 *                 bounds, 8 bytes per query; WORKSPACE / INVALID_ARG
 *                 otherwise).
 */
zeta_status_t zeta_select_topk(const uint32_t* q_codes, const uint32_t* sorted_codes,
                               const int32_t* perm, int64_t n_segments, int64_t N, int topk,
                               int causal, int chunk, const int32_t* q_order, int32_t* idx,
                               void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * zeta_topk_attn_fwd -- Adaptive Cauchy-softmax attention over each query's
 * candidates (Section 3.3, equation cauchy; Section 3.4; Appendix E.1):
 *   S_ij = 1 / (||q_i - k_j||^2 + eps)  for j in idx[i] (entries -1 skipped),
 *   o_i  = sum_j S_ij v_j / sum_j S_ij.
 * Distances use the unquantised q and k.  Accumulation is float32; a
 * bfloat16 output is rounded to nearest even.  A row whose idx holds no
 * valid entry is written as zeros.
 * With mean_k and mean_v (both given, or both NULL) every window gains the
 * history-mean candidate of Section 3.4: the pair (mean_k[i], mean_v[i])
 * scored and normalised like the other candidates (a row with no valid
 * entry then attends to it alone).  `score` picks the Cauchy score or one of
 * the variants of zeta_score_t (same candidates, other weights).
 *
 *   q, k   [B][H][N][d_k], v [B][H][N][d_v], out [B][H][N][d_v], all `dtype`.
 *   idx      int32 [B*H][N][topk]; valid entries (0 <= j < N) first, then -1.
 *   q_order  optional int32 [B*H][N] processing order, as for
 *            zeta_select_topk (NULL: position order; entries outside 0..N-1
 *            are skipped and leave their rows untouched).  Without it each
 *            query is computed alone, over its row in slot order, and its
 *            bits depend only on its own row.  With it, for bfloat16 inputs
 *            with d_k = 3, d_v of 32, 64 or 128 and topk <= 128, each 16
 *            consecutive queries of the order form a tile: the union of
 *            their rows is loaded once and the weighted sums run on the
 *            matrix cores (scores split into two bfloat16 parts, float32
 *            accumulation), as in zeta_select_attend_fwd.  The outputs then
 *            agree with the per-query ones to float32 rounding and repeat
 *            bit for bit for the same order, but a query's last bits follow
 *            the tile it shares.  zeta_query_order's order gives tiles whose
 *            rows overlap and makes the call fastest; in other orders the
 *            tiles split (down to single queries) until their unions fit.
 *   score    a zeta_score_t (UNSUPPORTED otherwise).
 *   eps      gamma^2: finite and > 0 (read by the Cauchy and inverse
 *            Euclidean scores).
 *   mean_k, mean_v  optional float32 [B*H][N][d_k] and [B*H][N][d_v] (as
 *            zeta_history_mean writes them); mean_v 16-byte aligned.
 *
 * Supported d_v: 32, 64, 128, 256.  v and out must be 16-byte aligned; out
 * must not overlap the inputs.
 */
zeta_status_t zeta_topk_attn_fwd(const void* q, const void* k, const void* v, zeta_dtype_t dtype,
                                 int64_t B, int64_t H, int64_t N, int d_k, int d_v, int topk,
                                 const int32_t* idx, const int32_t* q_order, zeta_score_t score,
                                 float eps, const float* mean_k, const float* mean_v, void* out,
                                 hipStream_t stream);

/*
 * zeta_select_attend_fwd -- zeta_select_topk and zeta_topk_attn_fwd in one
 * pass (same definitions, Section 3.2.2 and Algorithm 1, Steps 3-5; Section
 * 3.3, equation cauchy; Section 3.4; Appendix E.1).  No index tensor is
 * needed: the windows are kept as list-index bounds (8 bytes per query in the
 * workspace) instead of k positions per query.
 *
 * float32: each query is served as by the two calls, and `out` holds their
 * bits.  bfloat16: 16 neighbouring queries of the processing order share one
 * pass over the union of their windows, and the weighted sum of value rows
 * runs on the matrix cores (scores split into two bfloat16 parts, float32
 * accumulation).  The output agrees with the two calls to float32 rounding,
 * and a query's bits depend only on its own window, so they are the same for
 * every processing order.  The history-mean candidate, when given, is added
 * per query in float32.  With d_k = 3 the score variants run on the tiles
 * too (softmax variants as an online softmax per query: running maximum,
 * sums rescaled when it grows); float32 inputs, and the variants with other
 * d_k, take the per-query path.
 *
 *   q, k, v, dtype, B, H, N, d_k, d_v, topk, score, eps, mean_k, mean_v,
 *            out: as for zeta_topk_attn_fwd; causal and chunk as for
 *            zeta_select_topk.
 *   q_codes, sorted_codes, perm, q_order: as for zeta_select_topk.
 *   idx_out  optional int32 [B*H][N][topk]: receives the windows, exactly as
 *            zeta_select_topk writes them.
 *   workspace  at least zeta_workspace_size(...) bytes, 16-byte aligned.
 */
zeta_status_t zeta_select_attend_fwd(const void* q, const void* k, const void* v, zeta_dtype_t dtype,
                                     int64_t B, int64_t H, int64_t N, int d_k, int d_v, int topk,
                                     int causal, int chunk, const uint32_t* q_codes,
                                     const uint32_t* sorted_codes, const int32_t* perm,
                                     const int32_t* q_order, zeta_score_t score, float eps,
                                     const float* mean_k, const float* mean_v, void* out,
                                     int32_t* idx_out, void* workspace, size_t workspace_bytes,
                                     hipStream_t stream);

/*
 * zeta_history_mean -- the history-mean candidate (Section 3.4, last
 * paragraph: the mean vector of the history, from a cumulative sum, is added
 * to the top-k candidates as smoothing).  For causal calls row i holds the
 * means of rows 0..i,
 *   mean_k[i] = (k_0 + ... + k_i) / (i + 1),  mean_v[i] likewise;
 * otherwise every row holds the means over all N rows.  Sums are float32,
 * formed per chunk of 64 rows and then across chunks, in a fixed order.
 *
 *   k        [B][H][N][d_k], v [B][H][N][d_v], `dtype`; v 16-byte aligned.
 *   causal   0 or 1.
 *   mean_k   float32 [B*H][N][d_k] output; mean_v float32 [B*H][N][d_v]
 *            output, 16-byte aligned; neither may be an input.
 *   workspace  at least zeta_workspace_size(...) bytes.
 * Supported d_v: 32, 64, 128, 256; d_k up to ZETA_MAX_DK.
 */
zeta_status_t zeta_history_mean(const void* k, const void* v, zeta_dtype_t dtype, int64_t B,
                                int64_t H, int64_t N, int d_k, int d_v, int causal, float* mean_k,
                                float* mean_v, void* workspace, size_t workspace_bytes,
                                hipStream_t stream);

/*
 * zeta_topk_attn_bwd -- gradients of the attention of zeta_topk_attn_fwd
 * with respect to q, k, v and eps, for fixed windows idx (Appendix E.2,
 * summary of gradient computations; the selection has no gradient).  With
 * S_ij = 1 / (||q_i - k_j||^2 + eps), Z_i = sum_j S_ij, A_ij = S_ij / Z_i,
 * o_i = sum_j A_ij v_j and L the loss with dout = dL/do:
 *   dv_j  = sum over queries i whose window holds j of A_ij dout_i
 *   dq_i  = -2 sum_j w_ij (q_i - k_j),  w_ij = dout_i . (v_j - o_i) S_ij^2 / Z_i
 *   dk_j  =  2 sum over i of w_ij (q_i - k_j)
 *   deps  = -sum over all i, j of w_ij
 * o_i is recomputed from the same terms (the forward output is not needed).
 * With mean_k and mean_v the history-mean candidate takes part as in the
 * forward: its terms join Z_i, o_i, dq_i and deps, and the gradients that
 * reach mean_k[i] and mean_v[i] pass to every row j of query i's history,
 * divided by its length: dk_j, dv_j gain the sum over i >= j (causal) or
 * over all i of those, divided by i + 1 (causal) or N.
 * All arithmetic and all gradients are float32.
 *
 *   q, k, v, dtype, B, H, N, d_k, d_v, topk, idx, q_order, eps: as for
 *            zeta_topk_attn_fwd (q_order only changes the processing order).
 *   dout     [B][H][N][d_v], `dtype`, 16-byte aligned: dL/do.
 *   mean_k, mean_v  optional, as for zeta_topk_attn_fwd; causal (0 or 1)
 *            says how zeta_history_mean formed them (read only with them).
 *   dq, dk   float32 [B][H][N][d_k] outputs; dv float32 [B][H][N][d_v]
 *            (16-byte aligned when the means are given).
 *   deps     float32 [1] output: the gradient of the one eps of the call.
 *   workspace  at least zeta_bwd_workspace_size(B, H, N, d_k, d_v, topk,
 *            means given) bytes (it holds one key per window slot and their
 *            sorted copy).
 * The gradients are those of the Cauchy score.  Every output element is
 * written (rows without candidates and keys in no window get zeros).  No
 * atomics: dk and dv are summed per key after a stable
 * sort of the window slots by key, so every output is bit-identical from run
 * to run and for every q_order.  N * topk above 2^31 - 1 is UNSUPPORTED.  The
 * outputs must be distinct buffers and none may be an input (INVALID_ARG).
 */
zeta_status_t zeta_topk_attn_bwd(const void* q, const void* k, const void* v, zeta_dtype_t dtype, int64_t B,
                                 int64_t H, int64_t N, int d_k, int d_v, int topk, const int32_t* idx,
                                 const int32_t* q_order, const void* dout, float eps, const float* mean_k,
                                 const float* mean_v, int causal, float* dq, float* dk, float* dv,
                                 float* deps, void* workspace, size_t workspace_bytes,
                                 hipStream_t stream);

/*
 * zeta_select_attend_bwd -- the gradients of zeta_topk_attn_bwd (same
 * definitions, Appendix E.2) for the windows zeta_select_attend_fwd selects,
 * computed from the lists as the one-pass call does, without an index tensor:
 * bfloat16 inputs, d_k = 3, the Cauchy score, with or without the
 * history-mean candidate.
 * 16 neighbouring queries of the processing order form a tile.  A query pass
 * walks each tile's windows and gives dq, Z_i, c_i = dout_i . o_i and the
 * tile's window range per list; a key pass per list then takes 16 list
 * entries at a time and sums over the tiles whose windows meet them.  The dot
 * products dout_i . v_j and the sums of A_ij dout_i over queries run on the
 * matrix cores (A_ij split into two bfloat16 parts, float32 accumulation);
 * everything else is float32.  dk and dv are summed per list, the full sorted
 * list first and then the prefix lists, in a fixed order without atomics: the
 * outputs are the same from run to run for a given q_order (the bits of dk
 * and dv depend on which queries share a tile).  Any q_order is correct; with
 * the one from zeta_query_order each list entry meets few tiles.
 *
 *   q, k, v, dtype, B, H, N, d_k, d_v, topk, causal, chunk, q_codes,
 *            sorted_codes, perm, q_order, eps: as for zeta_select_attend_fwd.
 *   dout     [B][H][N][d_v] bfloat16, 16-byte aligned: dL/do.
 *   mean_k, mean_v  optional, as for zeta_topk_attn_bwd (from
 *            zeta_history_mean with the same causal flag): the candidate
 *            joins every query's sums and the gradients reaching the means
 *            pass to the rows of each query's history.
 *   dq, dk   float32 [B][H][N][d_k] outputs; dv float32 [B][H][N][d_v],
 *            16-byte aligned; deps float32 [1].  Every element is written.
 *   workspace  at least zeta_select_attend_bwd_workspace_size(...) bytes,
 *            16-byte aligned.
 * Supported: dtype ZETA_BF16, d_k = 3, d_v 32, 64, 128 or 256 (otherwise
 * UNSUPPORTED: zeta_topk_attn_bwd serves those).  The outputs must be
 * distinct buffers and none may be an input (INVALID_ARG).
 */
zeta_status_t zeta_select_attend_bwd(const void* q, const void* k, const void* v, zeta_dtype_t dtype,
                                     int64_t B, int64_t H, int64_t N, int d_k, int d_v, int topk,
                                     int causal, int chunk, const uint32_t* q_codes,
                                     const uint32_t* sorted_codes, const int32_t* perm,
                                     const int32_t* q_order, const void* dout, float eps,
                                     const float* mean_k, const float* mean_v, float* dq, float* dk,
                                     float* dv, float* deps, void* workspace, size_t workspace_bytes,
                                     hipStream_t stream);

/*
 * zeta_exact_knn -- the locality experiment's reference (Section 4.4): the kn
 * keys nearest to each query in Euclidean distance, among the query's pool
 * ({0..i} when causal, all N keys otherwise), ordered by (distance,
 * position) and padded with -1.  The squared distance is evaluated in
 * float32 with one rounding per subtraction, product and sum, axes in order
 * (no fused multiply-add).  An exact search over the pool: meant for the
 * experiment's sizes, not for the attention path.
 *
 *   q, k     [B][H][N][d_k] of `dtype`.
 *   kn       1..ZETA_MAX_TOPK; causal 0 or 1.
 *   knn_idx  int32 [B*H][N][kn] output.
 * Supported N: up to 4096 (UNSUPPORTED above).
 */
zeta_status_t zeta_exact_knn(const void* q, const void* k, zeta_dtype_t dtype, int64_t B, int64_t H,
                             int64_t N, int d_k, int kn, int causal, int32_t* knn_idx,
                             hipStream_t stream);

/*
 * zeta_index_overlap -- per row, the number of positions two index rows
 * share (entries -1 and outside 0..N-1 ignored; each row's valid entries
 * distinct): with the windows of zeta_select_topk and the nearest keys of
 * zeta_exact_knn it gives Section 4.4's locality measure (shared / kn).
 *
 *   idx_a    int32 [n_rows][ka]; idx_b int32 [n_rows][kb]; ka, kb in
 *            1..ZETA_MAX_TOPK.
 *   N        positions per segment (up to 65536; UNSUPPORTED above).
 *   counts   int32 [n_rows] output.
 */
zeta_status_t zeta_index_overlap(const int32_t* idx_a, int ka, const int32_t* idx_b, int kb,
                                 int64_t n_rows, int64_t N, int32_t* counts, hipStream_t stream);

/*
 * zeta_workspace_size -- bytes of device workspace enough for each of
 * zeta_morton_encode, zeta_sort_keys, zeta_query_order, zeta_select_topk and
 * zeta_select_attend_fwd on this shape, where the sort may cover the query
 * codes together with the key codes (2*B*H segments).  One buffer serves all
 * forward calls run in order on one stream, and zeta_history_mean.  Returns
 * 0 for invalid shapes.
 */
size_t zeta_workspace_size(int64_t B, int64_t H, int64_t N, int d_k, int bits, int topk,
                           int causal);

/*
 * zeta_bwd_workspace_size -- bytes of device workspace for zeta_topk_attn_bwd
 * on this shape: about 22 bytes per window slot (B*H*N*topk slots: the slot
 * keys, their sorted copy with slot numbers, the sort's ping-pong buffer)
 * plus per-row partials and the sort's histograms; with history_mean
 * nonzero also 4 * (d_k + d_v) bytes per row for the gradients reaching the
 * means.  Returns 0 for invalid or unsupported shapes and for N * topk above
 * 2^31 - 1.
 */
size_t zeta_bwd_workspace_size(int64_t B, int64_t H, int64_t N, int d_k, int d_v, int topk,
                               int history_mean);

/*
 * zeta_select_attend_bwd_workspace_size -- bytes of device workspace for
 * zeta_select_attend_bwd on this shape: the one-pass call's lists, window
 * bounds and key rows, 36 + 2 * d_v bytes per row (a 32-byte record of the
 * row's query, a copy of its dout row and its part of deps), 24 bytes per
 * tile of 16 rows and list, and 4 KiB of sums; with history_mean nonzero also
 * 4 * (3 + d_v) bytes per row (the gradients reaching the means) and their
 * scan's sums.  Returns 0 for invalid shapes and unsupported d_v.
 */
size_t zeta_select_attend_bwd_workspace_size(int64_t B, int64_t H, int64_t N, int d_v, int topk,
                                             int causal, int history_mean);

/* Static, human-readable name of a status code. */
const char* zeta_status_string(zeta_status_t status);

#ifdef __cplusplus
}
#endif

#endif /* ZETA_H */
