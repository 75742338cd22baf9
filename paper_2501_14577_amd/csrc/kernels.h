// Kernel launchers (one translation unit per step).  Each enqueues its kernels
// on `stream` and returns the runtime's launch status.  Arguments have already
// been validated by the C ABI layer.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace zeta {

// Attention scores: the method's Cauchy score and the variants compared with
// it (the values match zeta_score_t).
enum ScoreMode : int { kScoreCauchy = 0, kScoreDot = 1, kScoreNegEuclid = 2, kScoreInvEuclid = 3, kScoreNormDot = 4 };
__host__ __device__ constexpr bool score_is_softmax(int mode) {
  return mode == kScoreDot || mode == kScoreNegEuclid || mode == kScoreNormDot;
}

// The history-mean candidate (optional): float32 mean keys [S][N][d_k] and
// mean values [S][N][d_v], row i holding query i's; both NULL when off.
struct HistMean {
  const float* k;
  const float* v;
};

// History means of k and v (causal: rows 0..i; else all N rows) into
// mean_k and mean_v.  Workspace: hist_ws(S, N, dk + dv).
hipError_t launch_history_mean(const void* k, const void* v, bool is_bf16, int64_t S, int64_t N, int dk, int dv,
                               bool causal, float* mean_k, float* mean_v, void* workspace, hipStream_t stream);

// For two float32 matrices ([S][N][Da] and [S][N][Db]) at once: adds to
// out[j] the sum of x[i] over i >= j (causal) or over all i, per segment and
// column.  Workspace: hist_ws(S, N, Da + Db).
hipError_t launch_history_spread(const float* xa, float* outa, int Da, const float* xb, float* outb, int Db, int64_t S,
                                 int64_t N, bool causal, void* workspace, hipStream_t stream);

// Encode: optional joint-range reduction, then quantise + interleave.
// is_bf16: q and k hold bfloat16 bit patterns, else float32.
hipError_t launch_encode(const void* q, const void* k, bool is_bf16, int64_t S, int64_t N, int dk,
                         int bits, const float* range_lohi, float* range_out, uint32_t* q_codes,
                         uint32_t* k_codes, void* workspace, hipStream_t stream);

// launch_encode with the range partials in the library's own per-GPU
// scratch array (kEncStaticScratchBytes) instead of a caller workspace; the
// caller has checked that they fit.
hipError_t launch_encode_static(const void* q, const void* k, bool is_bf16, int64_t S, int64_t N, int dk, int bits,
                                const float* range_lohi, float* range_out, uint32_t* q_codes, uint32_t* k_codes,
                                hipStream_t stream);

// Stable LSD radix sort of each segment's codes.
hipError_t launch_sort(const uint32_t* k_codes, int64_t S, int64_t N, int code_bits,
                       uint32_t* sorted_codes, int32_t* perm, void* workspace, hipStream_t stream);

// One stable radix pass whose digit is the prefix-list level class of each
// carried value (a query position; vals NULL: the positions 0..N-1) under the
// causal rule `chunk` (0: exact prefix): a stable partition of each segment
// by list level.  hist holds S * (ceil(N / kLevelTile) + 1) * kRadixMax words.
// vals_out must not alias vals.
hipError_t launch_level_partition(const int32_t* vals, int64_t S, int64_t N, int t0, int t_hi, int levels, int chunk,
                                  int32_t* vals_out, uint32_t* hist, hipStream_t stream);

// Regroup a processing order (NULL: position order) by the list level each
// query searches in select, keeping the given order inside each level.
hipError_t launch_query_order(const int32_t* q_order, int64_t S, int64_t N, int topk, bool causal, int chunk,
                              int32_t* order_out, void* workspace, hipStream_t stream);

// Causal prefix lists (when needed) and the window of every query.  chunk:
// 0 for the exact causal prefix, M for the paper's chunked rule.  q_order:
// optional processing order (a permutation of 0..N-1 per segment).
hipError_t launch_select(const uint32_t* q_codes, const uint32_t* sorted_codes, const int32_t* perm,
                         int64_t S, int64_t N, int topk, bool causal, int chunk, const int32_t* q_order, int32_t* idx,
                         void* workspace, hipStream_t stream);

// Doubling prefix lists of causal selection in the workspace (none when
// every query searches the full list: *list_codes stays NULL).  With k_rows
// (bfloat16 keys, d_k = 3) the same pass writes the key rows of the full
// sorted lists and of the prefix lists in list order, as the tiles read them.
hipError_t launch_prefix_lists(const uint32_t* sorted_codes, const int32_t* perm, int64_t S, int64_t N, int topk,
                               void* workspace, hipStream_t stream, const uint32_t** list_codes,
                               const int32_t** list_pos, const uint16_t* k_rows = nullptr,
                               uint2* keys_full = nullptr, uint2* keys_list = nullptr);

// bfloat16 one-pass select and attend on the matrix cores, 16 queries per
// wavefront (the prefix lists already built when causal): window bounds per
// processing-order slot into `bounds` (S*N entries); for d_k = 3 the lists'
// key rows in list order into keys_full (S*N) and keys_list (S*cap); then the
// tiles.
bool tile_supports(int dv);
// The attend call on the matrix-core tiles (bfloat16, d_k = 3, d_v 32, 64 or
// 128, topk <= kIdxTileMaxTopk, a processing order given): each wavefront
// takes 16 consecutive queries of q_order and the union of their index rows.
hipError_t launch_attend_idx_tile(const void* q, const void* k, const void* v, int64_t S, int64_t N, int dv, int topk,
                                  const int32_t* idx, const int32_t* q_order, int score, float eps, HistMean hm,
                                  void* out, hipStream_t stream);
// The tiles' inputs alone: key rows in list order (d_k = 3) and the window
// bounds of every processing-order slot (idx_out optional).
hipError_t launch_tile_windows(const void* k, int64_t S, int64_t N, int dk, int topk, bool causal, int chunk,
                               const uint32_t* q_codes, const uint32_t* sorted_codes, const int32_t* perm,
                               const uint32_t* list_codes, const int32_t* list_pos, const int32_t* q_order,
                               int32_t* idx_out, int2* bounds, uint2* keys_full, uint2* keys_list,
                               bool keys_built, hipStream_t stream);
hipError_t launch_select_attend_tile(const void* q, const void* k, const void* v, int64_t S, int64_t N, int dk, int dv,
                                     int topk, bool causal, int chunk, const uint32_t* q_codes,
                                     const uint32_t* sorted_codes,
                                     const int32_t* perm, const uint32_t* list_codes, const int32_t* list_pos,
                                     const int32_t* q_order, int score, float eps, HistMean hm, void* out,
                                     int32_t* idx_out, int2* bounds, uint2* keys_full, uint2* keys_list,
                                     bool keys_built, hipStream_t stream);

// Gradients of the bfloat16 one-pass attention (d_k = 3, Cauchy score) over
// its windows, with the optional history-mean candidate: prefix lists, window
// bounds, query pass, envelopes, key passes, the means' spread and the deps
// sum; dq, dk, dv and deps float32.
hipError_t launch_select_attend_bwd(const void* q, const void* k, const void* v, const void* dout, int64_t S,
                                    int64_t N, int dk_, int dv_, int topk, bool causal, int chunk,
                                    const uint32_t* q_codes, const uint32_t* sorted_codes, const int32_t* perm,
                                    const int32_t* q_order, float eps, HistMean hm, float* dq, float* dk,
                                    float* dv, float* deps, void* workspace, hipStream_t stream);

// Select and attend in one pass (idx_out optional); score: a ScoreMode (the
// matrix-core tiles serve bfloat16 inputs: the Cauchy score, and every score
// when d_k = 3).
hipError_t launch_select_attend(const void* q, const void* k, const void* v, bool is_bf16, int64_t S, int64_t N,
                                int dk, int dv, int topk, bool causal, int chunk, const uint32_t* q_codes,
                                const uint32_t* sorted_codes, const int32_t* perm, const int32_t* q_order,
                                int score, float eps, HistMean hm, void* out, int32_t* idx_out, void* workspace,
                                hipStream_t stream);

// Cauchy-softmax attention over the selected rows (and the history-mean
// candidate when hm is given).
hipError_t launch_attend(const void* q, const void* k, const void* v, bool is_bf16, int64_t S,
                         int64_t N, int dk, int dv, int topk, const int32_t* idx, const int32_t* q_order,
                         int score, float eps, HistMean hm, void* out, hipStream_t stream);

bool attend_supports(int dv);

// Attention gradients for fixed windows (dq, dk, dv written, deps = one
// float); with hm, the history-mean candidate's share too, passed back to the
// history's rows (causal: rows 0..i of query i).  Workspace:
// bwd_ws(S, N, topk, dk, dv, hm given).
hipError_t launch_attend_bwd(const void* q, const void* k, const void* v, const void* dout, bool is_bf16, int64_t S,
                             int64_t N, int dk, int dv, int topk, const int32_t* idx, const int32_t* q_order,
                             float eps, HistMean hm, bool causal, float* dq, float* dkg, float* dvg, float* deps,
                             void* workspace, hipStream_t stream);

// The locality experiment: the kn keys nearest to each query in Euclidean
// distance within its pool (N <= kKnnMaxN), ordered by (distance, position),
// -1 padded; and per row the number of entries two index rows share
// (N <= kOverlapMaxN).
hipError_t launch_exact_knn(const void* q, const void* k, bool is_bf16, int64_t S, int64_t N, int dk, int kn,
                            bool causal, int32_t* out, hipStream_t stream);
hipError_t launch_index_overlap(const int32_t* a, int ka, const int32_t* b, int kb, int64_t rows, int64_t N,
                                int32_t* counts, hipStream_t stream);

}  // namespace zeta
