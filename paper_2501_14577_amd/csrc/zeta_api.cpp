// C ABI of the Z-order top-k attention and its gradients: argument
// validation on the host, then the kernel launchers.  Validation touches no HIP runtime call, so
// every error path can be exercised without a GPU.
#include <math.h>

#include "../../include/zeta.h"
#include "kernels.h"
#include "layout.h"

static_assert(ZETA_MAX_DK == zeta::kMaxDk, "d_k limit mismatch");
static_assert(ZETA_MAX_TOPK == zeta::kMaxTopk, "topk limit mismatch");
static_assert(ZETA_MAX_BITS == zeta::kMaxBits, "bits limit mismatch");
static_assert(ZETA_ENCODE_STATIC_SCRATCH_BYTES == zeta::kEncStaticScratchBytes, "static scratch size mismatch");
static_assert(int(ZETA_SCORE_CAUCHY) == zeta::kScoreCauchy && int(ZETA_SCORE_DOT) == zeta::kScoreDot &&
                  int(ZETA_SCORE_NEG_EUCLID) == zeta::kScoreNegEuclid &&
                  int(ZETA_SCORE_INV_EUCLID) == zeta::kScoreInvEuclid &&
                  int(ZETA_SCORE_NORM_DOT) == zeta::kScoreNormDot,
              "score mode mismatch");

namespace {

constexpr int64_t kMaxElems = (int64_t(1) << 31) - 1;  // B*H*N limit (int32 positions, grid sizes)

bool shape_ok(int64_t S, int64_t N) { return S >= 1 && N >= 1 && N <= kMaxElems && S <= kMaxElems / N; }

bool dtype_known(zeta_dtype_t d) { return d == ZETA_F32 || d == ZETA_BF16; }

bool score_known(zeta_score_t s) { return int(s) >= int(ZETA_SCORE_CAUCHY) && int(s) <= int(ZETA_SCORE_NORM_DOT); }

// The causal mode and the chunked rule's chunk size: 0 (exact prefix) or a
// positive chunk size, the latter only for causal calls.
bool bad_pool(int causal, int chunk) { return (causal != 0 && causal != 1) || chunk < 0 || (chunk > 0 && !causal); }

zeta_status_t hip_status(hipError_t e) { return e == hipSuccess ? ZETA_OK : ZETA_ERR_HIP; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// True when [a, a + bytes) and [b, b + bytes) share a byte.
bool overlaps(const void* a, const void* b, size_t bytes) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + bytes && y < x + bytes;
}

// Window slots per segment that the gradient's key sort can index (int32).
constexpr int64_t zeta_max_bwd_slots() { return (int64_t(1) << 31) - 1; }

bool bad_count(int64_t B, int64_t H, int64_t N) {
  if (B < 1 || H < 1 || N < 1) return true;
  if (B > kMaxElems / H) return true;
  return !shape_ok(B * H, N);
}

// The history-mean rows are given together or not at all; mean values are
// read with 16-byte loads.
bool bad_means(const float* mean_k, const float* mean_v) {
  if ((mean_k == nullptr) != (mean_v == nullptr)) return true;
  return mean_v != nullptr && !aligned16(mean_v);
}

// Argument checks shared by both encode entry points.
zeta_status_t encode_args(const void* q, const void* k, zeta_dtype_t dtype, int64_t B, int64_t H, int64_t N, int d_k,
                          int bits, const uint32_t* q_codes, const uint32_t* k_codes) {
  if (!q || !k || !q_codes || !k_codes) return ZETA_ERR_INVALID_ARG;
  if (bad_count(B, H, N)) return ZETA_ERR_INVALID_ARG;
  if (d_k < 1 || bits < 1 || int64_t(d_k) * bits > 32) return ZETA_ERR_INVALID_ARG;
  if (q_codes == k_codes) return ZETA_ERR_INVALID_ARG;
  if (!dtype_known(dtype)) return ZETA_ERR_UNSUPPORTED;
  if (d_k > zeta::kMaxDk || bits > zeta::kMaxBits) return ZETA_ERR_UNSUPPORTED;
  return ZETA_OK;
}

}  // namespace

extern "C" {

zeta_status_t zeta_morton_encode(const void* q, const void* k, zeta_dtype_t dtype, int64_t B, int64_t H,
                                 int64_t N, int d_k, int bits, const float* range_lohi, float* range_out,
                                 uint32_t* q_codes, uint32_t* k_codes, void* workspace,
                                 size_t workspace_bytes, hipStream_t stream) {
  const zeta_status_t st = encode_args(q, k, dtype, B, H, N, d_k, bits, q_codes, k_codes);
  if (st != ZETA_OK) return st;
  const int64_t S = B * H;
  if (range_lohi == nullptr) {
    const zeta::EncodeWs ws = zeta::encode_ws(S, N, d_k);
    if (workspace == nullptr || workspace_bytes < ws.bytes) return ZETA_ERR_WORKSPACE;
  }
  return hip_status(zeta::launch_encode(q, k, dtype == ZETA_BF16, S, N, d_k, bits, range_lohi, range_out,
                                        q_codes, k_codes, workspace, stream));
}

zeta_status_t zeta_morton_encode_static(const void* q, const void* k, zeta_dtype_t dtype, int64_t B, int64_t H,
                                        int64_t N, int d_k, int bits, const float* range_lohi, float* range_out,
                                        uint32_t* q_codes, uint32_t* k_codes, hipStream_t stream) {
  const zeta_status_t st = encode_args(q, k, dtype, B, H, N, d_k, bits, q_codes, k_codes);
  if (st != ZETA_OK) return st;
  const int64_t S = B * H;
  if (range_lohi == nullptr && zeta::encode_ws(S, N, d_k).bytes > zeta::kEncStaticScratchBytes)
    return ZETA_ERR_UNSUPPORTED;
  return hip_status(zeta::launch_encode_static(q, k, dtype == ZETA_BF16, S, N, d_k, bits, range_lohi, range_out,
                                               q_codes, k_codes, stream));
}

zeta_status_t zeta_sort_keys(const uint32_t* k_codes, int64_t n_segments, int64_t N, int code_bits,
                             uint32_t* sorted_codes, int32_t* perm, void* workspace,
                             size_t workspace_bytes, hipStream_t stream) {
  if (!k_codes || !sorted_codes || !perm) return ZETA_ERR_INVALID_ARG;
  if (!shape_ok(n_segments, N)) return ZETA_ERR_INVALID_ARG;
  if (code_bits < 1 || code_bits > 32) return ZETA_ERR_INVALID_ARG;
  if (static_cast<const void*>(k_codes) == static_cast<const void*>(sorted_codes) ||
      static_cast<const void*>(k_codes) == static_cast<const void*>(perm) ||
      static_cast<const void*>(sorted_codes) == static_cast<const void*>(perm))
    return ZETA_ERR_INVALID_ARG;
  const zeta::SortWs ws = zeta::sort_ws(n_segments, N, code_bits);
  if (workspace == nullptr || workspace_bytes < ws.bytes) return ZETA_ERR_WORKSPACE;
  return hip_status(zeta::launch_sort(k_codes, n_segments, N, code_bits, sorted_codes, perm, workspace, stream));
}

zeta_status_t zeta_query_order(const int32_t* q_order, int64_t n_segments, int64_t N, int topk, int causal,
                               int chunk, int32_t* order_out, void* workspace, size_t workspace_bytes,
                               hipStream_t stream) {
  if (!order_out) return ZETA_ERR_INVALID_ARG;
  if (!shape_ok(n_segments, N)) return ZETA_ERR_INVALID_ARG;
  if (topk < 1 || bad_pool(causal, chunk)) return ZETA_ERR_INVALID_ARG;
  if (topk > zeta::kMaxTopk) return ZETA_ERR_UNSUPPORTED;
  // In place is allowed; a partial overlap is not.
  if (q_order != nullptr && q_order != order_out &&
      overlaps(q_order, order_out, size_t(n_segments) * size_t(N) * sizeof(int32_t)))
    return ZETA_ERR_INVALID_ARG;
  const zeta::ListPlan lp = zeta::list_plan(N, topk);
  if (causal && lp.levels > 0) {
    const zeta::QueryOrderWs ws = zeta::query_order_ws(n_segments, N);
    if (workspace == nullptr || workspace_bytes < ws.bytes) return ZETA_ERR_WORKSPACE;
  }
  return hip_status(
      zeta::launch_query_order(q_order, n_segments, N, topk, causal != 0, chunk, order_out, workspace, stream));
}

zeta_status_t zeta_select_topk(const uint32_t* q_codes, const uint32_t* sorted_codes, const int32_t* perm,
                               int64_t n_segments, int64_t N, int topk, int causal, int chunk,
                               const int32_t* q_order, int32_t* idx, void* workspace, size_t workspace_bytes,
                               hipStream_t stream) {
  if (!q_codes || !sorted_codes || !perm || !idx) return ZETA_ERR_INVALID_ARG;
  if (!shape_ok(n_segments, N)) return ZETA_ERR_INVALID_ARG;
  if (topk < 1 || bad_pool(causal, chunk)) return ZETA_ERR_INVALID_ARG;
  if (topk > zeta::kMaxTopk) return ZETA_ERR_UNSUPPORTED;
  const zeta::SelectWs ws = zeta::select_ws(n_segments, N, topk, causal);
  if (workspace == nullptr || workspace_bytes < ws.call_bytes) return ZETA_ERR_WORKSPACE;
  if (!aligned16(workspace)) return ZETA_ERR_INVALID_ARG;
  return hip_status(zeta::launch_select(q_codes, sorted_codes, perm, n_segments, N, topk, causal != 0, chunk,
                                        q_order, idx, workspace, stream));
}

zeta_status_t zeta_history_mean(const void* k, const void* v, zeta_dtype_t dtype, int64_t B, int64_t H, int64_t N,
                                int d_k, int d_v, int causal, float* mean_k, float* mean_v, void* workspace,
                                size_t workspace_bytes, hipStream_t stream) {
  if (!k || !v || !mean_k || !mean_v) return ZETA_ERR_INVALID_ARG;
  if (bad_count(B, H, N)) return ZETA_ERR_INVALID_ARG;
  if (d_k < 1 || d_v < 1 || (causal != 0 && causal != 1)) return ZETA_ERR_INVALID_ARG;
  if (!aligned16(v) || !aligned16(mean_v)) return ZETA_ERR_INVALID_ARG;
  if (mean_k == mean_v || static_cast<const void*>(mean_k) == k || static_cast<const void*>(mean_v) == v)
    return ZETA_ERR_INVALID_ARG;
  if (!dtype_known(dtype)) return ZETA_ERR_UNSUPPORTED;
  if (d_k > zeta::kMaxDk || !zeta::attend_supports(d_v)) return ZETA_ERR_UNSUPPORTED;
  const int64_t S = B * H;
  const zeta::HistWs ws = zeta::hist_ws(S, N, d_k + d_v);
  if (workspace == nullptr || workspace_bytes < ws.bytes) return ZETA_ERR_WORKSPACE;
  return hip_status(zeta::launch_history_mean(k, v, dtype == ZETA_BF16, S, N, d_k, d_v, causal != 0, mean_k, mean_v,
                                              workspace, stream));
}

zeta_status_t zeta_topk_attn_fwd(const void* q, const void* k, const void* v, zeta_dtype_t dtype, int64_t B,
                                 int64_t H, int64_t N, int d_k, int d_v, int topk, const int32_t* idx,
                                 const int32_t* q_order, zeta_score_t score, float eps, const float* mean_k,
                                 const float* mean_v, void* out, hipStream_t stream) {
  if (!q || !k || !v || !idx || !out) return ZETA_ERR_INVALID_ARG;
  if (bad_count(B, H, N)) return ZETA_ERR_INVALID_ARG;
  if (d_k < 1 || d_v < 1 || topk < 1) return ZETA_ERR_INVALID_ARG;
  if (!(isfinite(eps) && eps > 0.0f)) return ZETA_ERR_INVALID_ARG;
  if (!aligned16(v) || !aligned16(out)) return ZETA_ERR_INVALID_ARG;
  if (out == q || out == k || out == v) return ZETA_ERR_INVALID_ARG;
  if (bad_means(mean_k, mean_v)) return ZETA_ERR_INVALID_ARG;
  if (!dtype_known(dtype)) return ZETA_ERR_UNSUPPORTED;
  if (d_k > zeta::kMaxDk || topk > zeta::kMaxTopk || !zeta::attend_supports(d_v)) return ZETA_ERR_UNSUPPORTED;
  if (!score_known(score)) return ZETA_ERR_UNSUPPORTED;
  return hip_status(zeta::launch_attend(q, k, v, dtype == ZETA_BF16, B * H, N, d_k, d_v, topk, idx, q_order,
                                        int(score), eps, zeta::HistMean{mean_k, mean_v}, out, stream));
}

zeta_status_t zeta_select_attend_fwd(const void* q, const void* k, const void* v, zeta_dtype_t dtype, int64_t B,
                                     int64_t H, int64_t N, int d_k, int d_v, int topk, int causal, int chunk,
                                     const uint32_t* q_codes, const uint32_t* sorted_codes, const int32_t* perm,
                                     const int32_t* q_order, zeta_score_t score, float eps, const float* mean_k,
                                     const float* mean_v, void* out, int32_t* idx_out, void* workspace,
                                     size_t workspace_bytes,
                                     hipStream_t stream) {
  if (!q || !k || !v || !out || !q_codes || !sorted_codes || !perm) return ZETA_ERR_INVALID_ARG;
  if (bad_count(B, H, N)) return ZETA_ERR_INVALID_ARG;
  if (d_k < 1 || d_v < 1 || topk < 1 || bad_pool(causal, chunk)) return ZETA_ERR_INVALID_ARG;
  if (!(isfinite(eps) && eps > 0.0f)) return ZETA_ERR_INVALID_ARG;
  if (!aligned16(v) || !aligned16(out)) return ZETA_ERR_INVALID_ARG;
  if (out == q || out == k || out == v) return ZETA_ERR_INVALID_ARG;
  if (bad_means(mean_k, mean_v)) return ZETA_ERR_INVALID_ARG;
  if (!dtype_known(dtype)) return ZETA_ERR_UNSUPPORTED;
  if (d_k > zeta::kMaxDk || topk > zeta::kMaxTopk || !zeta::attend_supports(d_v)) return ZETA_ERR_UNSUPPORTED;
  if (!score_known(score)) return ZETA_ERR_UNSUPPORTED;
  const int64_t S = B * H;
  if (zeta::tile_path(dtype == ZETA_BF16, d_v, score == ZETA_SCORE_CAUCHY, d_k)) {
    // Lists, per-slot window bounds and (d_k = 3) key rows in list order.
    const zeta::FusedWs ws = zeta::fused_ws(S, N, topk, causal);
    if (workspace == nullptr || workspace_bytes < ws.bytes) return ZETA_ERR_WORKSPACE;
    if (!aligned16(workspace)) return ZETA_ERR_INVALID_ARG;
  } else {
    const zeta::SelectWs ws = zeta::select_ws(S, N, topk, causal);
    if (ws.bytes > 0 && (workspace == nullptr || workspace_bytes < ws.bytes)) return ZETA_ERR_WORKSPACE;
  }
  return hip_status(zeta::launch_select_attend(q, k, v, dtype == ZETA_BF16, S, N, d_k, d_v, topk, causal != 0, chunk,
                                               q_codes, sorted_codes, perm, q_order, int(score), eps,
                                               zeta::HistMean{mean_k, mean_v}, out, idx_out, workspace, stream));
}

zeta_status_t zeta_topk_attn_bwd(const void* q, const void* k, const void* v, zeta_dtype_t dtype, int64_t B, int64_t H,
                                 int64_t N, int d_k, int d_v, int topk, const int32_t* idx, const int32_t* q_order,
                                 const void* dout, float eps, const float* mean_k, const float* mean_v, int causal,
                                 float* dq, float* dk, float* dv, float* deps, void* workspace,
                                 size_t workspace_bytes, hipStream_t stream) {
  if (!q || !k || !v || !idx || !dout || !dq || !dk || !dv || !deps) return ZETA_ERR_INVALID_ARG;
  if (bad_count(B, H, N)) return ZETA_ERR_INVALID_ARG;
  if (d_k < 1 || d_v < 1 || topk < 1 || (causal != 0 && causal != 1)) return ZETA_ERR_INVALID_ARG;
  if (!(isfinite(eps) && eps > 0.0f)) return ZETA_ERR_INVALID_ARG;
  if (!aligned16(v) || !aligned16(dout)) return ZETA_ERR_INVALID_ARG;
  if (bad_means(mean_k, mean_v)) return ZETA_ERR_INVALID_ARG;
  const bool history = mean_k != nullptr;
  if (history && !aligned16(dv)) return ZETA_ERR_INVALID_ARG;
  // Outputs are distinct buffers, none of them an input.
  const void* outs[4] = {dq, dk, dv, deps};
  const void* ins[8] = {q, k, v, dout, idx, q_order, mean_k, mean_v};
  for (int a = 0; a < 4; ++a) {
    for (int b = a + 1; b < 4; ++b)
      if (outs[a] == outs[b]) return ZETA_ERR_INVALID_ARG;
    for (int b = 0; b < 8; ++b)
      if (ins[b] != nullptr && outs[a] == ins[b]) return ZETA_ERR_INVALID_ARG;
  }
  if (!dtype_known(dtype)) return ZETA_ERR_UNSUPPORTED;
  if (d_k > zeta::kMaxDk || topk > zeta::kMaxTopk || !zeta::attend_supports(d_v)) return ZETA_ERR_UNSUPPORTED;
  const int64_t S = B * H;
  if (N > zeta_max_bwd_slots() / topk) return ZETA_ERR_UNSUPPORTED;
  const zeta::BwdWs ws = zeta::bwd_ws(S, N, topk, d_k, d_v, history);
  if (workspace == nullptr || workspace_bytes < ws.bytes) return ZETA_ERR_WORKSPACE;
  return hip_status(zeta::launch_attend_bwd(q, k, v, dout, dtype == ZETA_BF16, S, N, d_k, d_v, topk, idx, q_order, eps,
                                            zeta::HistMean{mean_k, mean_v}, causal != 0, dq, dk, dv, deps, workspace,
                                            stream));
}

zeta_status_t zeta_exact_knn(const void* q, const void* k, zeta_dtype_t dtype, int64_t B, int64_t H, int64_t N,
                             int d_k, int kn, int causal, int32_t* knn_idx, hipStream_t stream) {
  if (!q || !k || !knn_idx) return ZETA_ERR_INVALID_ARG;
  if (bad_count(B, H, N)) return ZETA_ERR_INVALID_ARG;
  if (d_k < 1 || kn < 1 || (causal != 0 && causal != 1)) return ZETA_ERR_INVALID_ARG;
  if (!dtype_known(dtype)) return ZETA_ERR_UNSUPPORTED;
  if (d_k > zeta::kMaxDk || kn > zeta::kMaxTopk || N > zeta::kKnnMaxN) return ZETA_ERR_UNSUPPORTED;
  return hip_status(zeta::launch_exact_knn(q, k, dtype == ZETA_BF16, B * H, N, d_k, kn, causal != 0, knn_idx, stream));
}

zeta_status_t zeta_index_overlap(const int32_t* idx_a, int ka, const int32_t* idx_b, int kb, int64_t n_rows,
                                 int64_t N, int32_t* counts, hipStream_t stream) {
  if (!idx_a || !idx_b || !counts) return ZETA_ERR_INVALID_ARG;
  if (ka < 1 || kb < 1 || n_rows < 1 || N < 1 || n_rows > kMaxElems) return ZETA_ERR_INVALID_ARG;
  if (ka > zeta::kMaxTopk || kb > zeta::kMaxTopk || N > zeta::kOverlapMaxN) return ZETA_ERR_UNSUPPORTED;
  return hip_status(zeta::launch_index_overlap(idx_a, ka, idx_b, kb, n_rows, N, counts, stream));
}

zeta_status_t zeta_select_attend_bwd(const void* q, const void* k, const void* v, zeta_dtype_t dtype, int64_t B,
                                     int64_t H, int64_t N, int d_k, int d_v, int topk, int causal, int chunk,
                                     const uint32_t* q_codes, const uint32_t* sorted_codes, const int32_t* perm,
                                     const int32_t* q_order, const void* dout, float eps, const float* mean_k,
                                     const float* mean_v, float* dq, float* dk, float* dv, float* deps,
                                     void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!q || !k || !v || !dout || !q_codes || !sorted_codes || !perm || !dq || !dk || !dv || !deps)
    return ZETA_ERR_INVALID_ARG;
  if (bad_count(B, H, N)) return ZETA_ERR_INVALID_ARG;
  if (d_k < 1 || d_v < 1 || topk < 1 || bad_pool(causal, chunk)) return ZETA_ERR_INVALID_ARG;
  if (!(isfinite(eps) && eps > 0.0f)) return ZETA_ERR_INVALID_ARG;
  if (!aligned16(v) || !aligned16(dout) || !aligned16(dv)) return ZETA_ERR_INVALID_ARG;
  if (bad_means(mean_k, mean_v)) return ZETA_ERR_INVALID_ARG;
  // Outputs are distinct buffers, none of them an input.
  const void* outs[4] = {dq, dk, dv, deps};
  const void* ins[10] = {q, k, v, dout, q_codes, sorted_codes, perm, q_order, mean_k, mean_v};
  for (int a = 0; a < 4; ++a) {
    for (int b = a + 1; b < 4; ++b)
      if (outs[a] == outs[b]) return ZETA_ERR_INVALID_ARG;
    for (int b = 0; b < 10; ++b)
      if (ins[b] != nullptr && outs[a] == ins[b]) return ZETA_ERR_INVALID_ARG;
  }
  if (!dtype_known(dtype)) return ZETA_ERR_UNSUPPORTED;
  if (dtype != ZETA_BF16 || d_k != 3 || !zeta::tile_supports(d_v) || topk > zeta::kMaxTopk)
    return ZETA_ERR_UNSUPPORTED;
  const int64_t S = B * H;
  const zeta::TileBwdWs ws = zeta::tile_bwd_ws(S, N, d_v, topk, causal, mean_k != nullptr);
  if (workspace == nullptr || workspace_bytes < ws.bytes) return ZETA_ERR_WORKSPACE;
  if (!aligned16(workspace)) return ZETA_ERR_INVALID_ARG;
  return hip_status(zeta::launch_select_attend_bwd(q, k, v, dout, S, N, d_k, d_v, topk, causal != 0, chunk, q_codes,
                                                   sorted_codes, perm, q_order, eps,
                                                   zeta::HistMean{mean_k, mean_v}, dq, dk, dv, deps, workspace,
                                                   stream));
}

size_t zeta_select_attend_bwd_workspace_size(int64_t B, int64_t H, int64_t N, int d_v, int topk, int causal,
                                             int history_mean) {
  if (bad_count(B, H, N) || topk < 1 || (causal != 0 && causal != 1) || !zeta::tile_supports(d_v)) return 0;
  return zeta::tile_bwd_ws(B * H, N, d_v, topk, causal, history_mean != 0).bytes;
}

size_t zeta_workspace_size(int64_t B, int64_t H, int64_t N, int d_k, int bits, int topk, int causal) {
  if (bad_count(B, H, N) || d_k < 1 || bits < 1 || int64_t(d_k) * bits > 32 || topk < 1) return 0;
  const int64_t S = B * H;
  size_t bytes = zeta::encode_ws(S, N, d_k).bytes;
  // Room to sort the query codes together with the key codes (2*B*H segments).
  const size_t sb = zeta::sort_ws(2 * S, N, d_k * bits).bytes;
  const size_t lb = zeta::select_ws(S, N, topk, causal ? 1 : 0).call_bytes;
  const size_t ob = zeta::query_order_ws(S, N).bytes;
  const size_t fb = zeta::fused_ws(S, N, topk, causal ? 1 : 0).bytes;
  const size_t hb = zeta::hist_ws(S, N, zeta::kHistMaxCols).bytes;
  if (fb > bytes) bytes = fb;
  if (hb > bytes) bytes = hb;
  if (sb > bytes) bytes = sb;
  if (lb > bytes) bytes = lb;
  if (ob > bytes) bytes = ob;
  return bytes;
}

size_t zeta_bwd_workspace_size(int64_t B, int64_t H, int64_t N, int d_k, int d_v, int topk, int history_mean) {
  if (bad_count(B, H, N) || topk < 1 || topk > zeta::kMaxTopk) return 0;
  if (d_k < 1 || d_k > zeta::kMaxDk || !zeta::attend_supports(d_v)) return 0;
  if (N > zeta_max_bwd_slots() / topk) return 0;
  return zeta::bwd_ws(B * H, N, topk, d_k, d_v, history_mean != 0).bytes;
}

const char* zeta_status_string(zeta_status_t status) {
  switch (status) {
    case ZETA_OK:
      return "ZETA_OK";
    case ZETA_ERR_INVALID_ARG:
      return "ZETA_ERR_INVALID_ARG";
    case ZETA_ERR_UNSUPPORTED:
      return "ZETA_ERR_UNSUPPORTED";
    case ZETA_ERR_WORKSPACE:
      return "ZETA_ERR_WORKSPACE";
    case ZETA_ERR_HIP:
      return "ZETA_ERR_HIP";
  }
  return "ZETA_ERR_UNKNOWN";
}

}  // extern "C"
