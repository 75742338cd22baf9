// Candidate selection and Cauchy-softmax attention in one pass (Section
// 3.2.2 and Algorithm 1, Steps 3-5, for the window; Section 3.3, equation
// cauchy, Section 3.4 and Appendix E.1 for the attention).
//
// The select and attend entry points meet through the index tensor: select
// writes k positions per query and attend reads them back.  Here the window
// stays in LDS: a wavefront serves a run of consecutive queries of the
// processing order, and for each it searches the query's list (galloping from
// the previous query's insertion point), collects the window into LDS, then
// scores the candidates and gathers their value rows exactly as the attend
// kernel does (same lane mapping, same fused multiply-adds), so the output
// bits equal those of select followed by attend.  The index row is written
// only when the caller asks for it.  The score variants (Section 4.3;
// Appendix G.2) run here for both dtypes.
#include "attend_device.h"
#include "device_common.h"
#include "kernels.h"
#include "layout.h"
#include "select_device.h"

namespace zeta {
namespace {

constexpr int kFusedWaves = 8;  // wavefronts per block
constexpr int kFusedRun = 8;    // consecutive processing-order slots per wavefront

template <typename T, int DV, int DK, bool kOff32, bool kVariants>
__global__ void __launch_bounds__(kFusedWaves * 64)
    select_attend_kernel(const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
                         const uint32_t* __restrict__ q_codes, const uint32_t* __restrict__ sorted_codes,
                         const int32_t* __restrict__ perm, const uint32_t* __restrict__ list_codes,
                         const int32_t* __restrict__ list_pos, const int32_t* __restrict__ order, int64_t total,
                         int64_t N, int dk_rt, int topk, int causal, int chunk, int t0, int t_hi, int64_t cap,
                         int score_rt, float eps, const float* __restrict__ mk, const float* __restrict__ mv,
                         T* __restrict__ out, int32_t* __restrict__ idx_out) {
  constexpr int kE = Vec16<T>::kElems;
  constexpr int kLpr = DV / kE;
  constexpr int kGroups = 64 / kLpr;
  constexpr int kUnroll = 4;  // rows in flight per lane (measured best here)
  constexpr int kRowBytes = DV * int(sizeof(T));
  static_assert(kLpr >= 1 && kLpr <= 64 && 64 % kLpr == 0, "row must split evenly over lanes");
  using Off = typename RowOff<kOff32>::type;
  constexpr int KD = DK > 0 ? DK : kMaxDk;
  const int dk = DK > 0 ? DK : dk_rt;
  // The Cauchy instantiation (kVariants false) carries none of the variants' code.
  const int score = kVariants ? score_rt : int(kScoreCauchy);
  const float rsd = 1.0f / sqrtf(float(dk));
  const bool softmax = score_is_softmax(score);

  extern __shared__ unsigned char s_raw[];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  // Per wave: window halves (2*topk positions), then row offsets and scores.
  int32_t* lbuf = reinterpret_cast<int32_t*>(s_raw) + size_t(wave) * 2 * topk;
  int32_t* rbuf = lbuf + topk;
  Off* s_off = reinterpret_cast<Off*>(s_raw + size_t(kFusedWaves) * 2 * topk * 4) + size_t(wave) * topk;
  float* s_w = reinterpret_cast<float*>(s_raw + size_t(kFusedWaves) * topk * (8 + sizeof(Off))) + size_t(wave) * topk;
  const int grp = lane / kLpr;
  const int sub = lane - grp * kLpr;
  const int64_t runs = (total + kFusedRun - 1) / kFusedRun;
  const int64_t nb = gridDim.x;

  for (int64_t blk = xcd_contiguous_block(blockIdx.x, nb); blk * kFusedWaves < runs; blk += nb) {
    const int64_t run = blk * kFusedWaves + wave;
    if (run >= runs) continue;
    const int64_t slot0 = run * kFusedRun;
    int32_t my_i = -1;
    uint32_t my_key = 0;
    {
      const int64_t sl = slot0 + lane;
      if (lane < kFusedRun && sl < total) {
        const int64_t sg = sl / N;
        const int64_t ii = order != nullptr ? int64_t(order[sl]) : sl - sg * N;
        if (ii >= 0 && ii < N) {
          my_i = int32_t(ii);
          my_key = q_codes[sg * N + ii];
        }
      }
    }
    const uint32_t* prev_codes = nullptr;
    uint32_t prev_key = 0;
    int32_t prev_p = 0;
    for (int u = 0; u < kFusedRun; ++u) {
      const int64_t slot = slot0 + u;
      if (slot >= total) break;
      const int32_t i = __builtin_amdgcn_readlane(my_i, u);
      const uint32_t key = uint32_t(__builtin_amdgcn_readlane(int32_t(my_key), u));
      if (i < 0) continue;  // not a permutation entry: nothing to do
      const int64_t seg = slot / N;
      const int64_t g = seg * N + i;

      // Window.
      const QueryList L =
          query_list(sorted_codes, perm, list_codes, list_pos, seg, N, i, causal, t0, t_hi, cap, chunk);
      int got_l = 0, got_r = 0;
      if (L.n > 0) {  // an empty pool (the chunked rule's first chunk) selects nothing
        const int32_t p = (L.codes == prev_codes && key >= prev_key)
                              ? wave_lower_bound_near(L.codes, prev_p, L.n, key, lane)
                              : wave_lower_bound(L.codes, 0, L.n, key, lane);
        prev_codes = L.codes;
        prev_key = key;
        prev_p = p;
        select_window(L, p, topk, lbuf, rbuf, lane, got_l, got_r);
      }
      wave_lds_sync();
      const int m = got_l + got_r;
      if (idx_out != nullptr) {
        int32_t* row = idx_out + g * topk;
        for (int c = lane; c < topk; c += 64) {
          int32_t jv = -1;
          if (c < got_l)
            jv = lbuf[topk - got_l + c];
          else if (c < m)
            jv = rbuf[c - got_l];
          row[c] = jv;
        }
      }

      // Scores, with the attend kernel's lane mapping (slot pairs 2l, 2l+1).
      const T* kseg = k + seg * N * dk;
      const unsigned char* vseg = reinterpret_cast<const unsigned char*>(v + seg * N * DV);
      float qv[DK > 0 ? DK : kMaxDk];
      if constexpr (DK == 3) {
        Row3<T>::load(q, g, total, qv);
      } else {
#pragma unroll
        for (int a = 0; a < (DK > 0 ? DK : kMaxDk); ++a) qv[a] = a < dk ? Elem<T>::load(q + g * dk + a) : 0.0f;
      }
      const float qn = score == kScoreNormDot ? row_norm<KD>(qv, dk) : 0.0f;
      float zsum = 0.0f;
      float zloc = -INFINITY;
      uint32_t okmask = 0u;
      int bit = 0;
      for (int c0 = 2 * lane; c0 < topk; c0 += 128) {
#pragma unroll
        for (int h = 0; h < 2; ++h, ++bit) {
          const int c = c0 + h;
          const bool ok = c < m;
          float s = 0.0f;
          int32_t j = 0;
          if (ok) {
            j = c < got_l ? lbuf[topk - got_l + c] : rbuf[c - got_l];
            float kv[DK > 0 ? DK : kMaxDk];
            if constexpr (DK == 3) {
              Row3<T>::load(k, seg * N + j, total, kv);
            } else {
#pragma unroll
              for (int a = 0; a < (DK > 0 ? DK : kMaxDk); ++a)
                kv[a] = a < dk ? Elem<T>::load(kseg + int64_t(j) * dk + a) : 0.0f;
            }
            if (score == kScoreCauchy) {
              float d2 = 0.0f;
#pragma unroll
              for (int a = 0; a < (DK > 0 ? DK : kMaxDk); ++a) {
                if (a < dk) {
                  const float diff = qv[a] - kv[a];
                  d2 = fmaf(diff, diff, d2);
                }
              }
              s = 1.0f / (d2 + eps);
            } else {
              s = variant_term<KD>(score, qv, kv, dk, eps, rsd, qn);
              zloc = fmaxf(zloc, s);
              okmask |= 1u << bit;
            }
          }
          if (c < topk) {
            s_off[c] = Off(j) * Off(kRowBytes);
            s_w[c] = s;
          }
          zsum += s;
        }
      }
      float s_mean = 0.0f;
      if (!softmax) {
        zsum = wave_sum(zsum);
        if (mk != nullptr) {
          if (score == kScoreCauchy) {
            s_mean = mean_score<KD>(mk, g, dk, qv, eps);
          } else {
            float mkv[KD];
#pragma unroll
            for (int a = 0; a < KD; ++a) mkv[a] = a < dk ? mk[g * dk + a] : 0.0f;
            s_mean = variant_term<KD>(score, qv, mkv, dk, eps, rsd, qn);
          }
          zsum += s_mean;
        }
      } else {
        if (mk != nullptr) {
          float mkv[KD];
#pragma unroll
          for (int a = 0; a < KD; ++a) mkv[a] = a < dk ? mk[g * dk + a] : 0.0f;
          s_mean = variant_term<KD>(score, qv, mkv, dk, eps, rsd, qn);
        }
        zsum = softmax_weights(s_w, topk, lane, okmask, zloc, mk != nullptr, s_mean);
      }
      wave_lds_sync();

      // Weighted gather of value rows.
      float acc[kE];
#pragma unroll
      for (int e = 0; e < kE; ++e) acc[e] = 0.0f;
      const Off lane_off = Off(sub * 16);
      int c = grp;
      for (; c + (kUnroll - 1) * kGroups < m; c += kUnroll * kGroups) {
        uint4 raw[kUnroll];
        float wv[kUnroll];
#pragma unroll
        for (int uu = 0; uu < kUnroll; ++uu) {
          const int cc = c + uu * kGroups;
          wv[uu] = s_w[cc];
          raw[uu] = *reinterpret_cast<const uint4*>(vseg + (s_off[cc] + lane_off));
        }
#pragma unroll
        for (int uu = 0; uu < kUnroll; ++uu) {
          float f[kE];
          Vec16<T>::widen(raw[uu], f);
#pragma unroll
          for (int e = 0; e < kE; ++e) acc[e] = fmaf(wv[uu], f[e], acc[e]);
        }
      }
      for (; c < m; c += kGroups) {
        float f[kE];
        const float w = s_w[c];
        Vec16<T>::widen(*reinterpret_cast<const uint4*>(vseg + (s_off[c] + lane_off)), f);
#pragma unroll
        for (int e = 0; e < kE; ++e) acc[e] = fmaf(w, f[e], acc[e]);
      }
#pragma unroll
      for (int off = kLpr; off < 64; off <<= 1)
#pragma unroll
        for (int e = 0; e < kE; ++e) acc[e] += __shfl_xor(acc[e], off, 64);
      if (grp == 0) {
        if (mv != nullptr) add_mean_value<kE>(mv + g * DV + sub * kE, s_mean, acc);
        const float inv = zsum > 0.0f ? 1.0f / zsum : 0.0f;
#pragma unroll
        for (int e = 0; e < kE; ++e) acc[e] *= inv;
        Vec16<T>::store(out + g * DV + sub * kE, acc);
      }
      wave_lds_sync();
    }
  }
}

template <typename T, int DV, int DK>
hipError_t launch_t(const void* q, const void* k, const void* v, int64_t S, int64_t N, int dk, int topk, bool causal,
                    int chunk, const uint32_t* q_codes, const uint32_t* sorted_codes, const int32_t* perm,
                    const uint32_t* list_codes, const int32_t* list_pos, const int32_t* q_order, int score, float eps,
                    HistMean hm, void* out, int32_t* idx_out, hipStream_t stream) {
  const ListPlan lp = list_plan(N, topk);
  const int64_t total = S * N;
  const int64_t runs = ceil_div(total, kFusedRun);
  const int64_t want = ceil_div(runs, kFusedWaves);
  const unsigned blocks = unsigned(want < (int64_t(1) << 20) ? want : (int64_t(1) << 20));
  const bool off32 = N * int64_t(DV) * int64_t(sizeof(T)) <= int64_t(0xFFFFFFFFu) - int64_t(DV) * int64_t(sizeof(T));
  const size_t lds = size_t(kFusedWaves) * topk * (8 + (off32 ? 4 : 8) + 4);
#define ZETA_FUSED_LAUNCH(OFF, VAR)                                                                            \
  hipLaunchKernelGGL((select_attend_kernel<T, DV, DK, OFF, VAR>), dim3(blocks), dim3(kFusedWaves * 64), lds, stream, \
                     static_cast<const T*>(q), static_cast<const T*>(k), static_cast<const T*>(v), q_codes,          \
                     sorted_codes, perm, list_codes, list_pos, q_order, total, N, dk, topk, causal ? 1 : 0, chunk,  \
                     lp.t0, lp.t_hi, lp.cap, score, eps, hm.k, hm.v, static_cast<T*>(out), idx_out)
  const bool var = score != kScoreCauchy;
  if (off32) {
    if (var)
      ZETA_FUSED_LAUNCH(true, true);
    else
      ZETA_FUSED_LAUNCH(true, false);
  } else {
    if (var)
      ZETA_FUSED_LAUNCH(false, true);
    else
      ZETA_FUSED_LAUNCH(false, false);
  }
#undef ZETA_FUSED_LAUNCH
  return hipGetLastError();
}

template <typename T, int DV>
hipError_t launch_dk(const void* q, const void* k, const void* v, int64_t S, int64_t N, int dk, int topk, bool causal,
                     int chunk, const uint32_t* q_codes, const uint32_t* sorted_codes, const int32_t* perm,
                     const uint32_t* list_codes, const int32_t* list_pos, const int32_t* q_order, int score, float eps,
                     HistMean hm, void* out, int32_t* idx_out, hipStream_t stream) {
  if (dk == 3)
    return launch_t<T, DV, 3>(q, k, v, S, N, dk, topk, causal, chunk, q_codes, sorted_codes, perm, list_codes,
                              list_pos, q_order, score, eps, hm, out, idx_out, stream);
  return launch_t<T, DV, 0>(q, k, v, S, N, dk, topk, causal, chunk, q_codes, sorted_codes, perm, list_codes, list_pos,
                            q_order, score, eps, hm, out, idx_out, stream);
}

}  // namespace

hipError_t launch_select_attend(const void* q, const void* k, const void* v, bool is_bf16, int64_t S, int64_t N,
                                int dk, int dv, int topk, bool causal, int chunk, const uint32_t* q_codes,
                                const uint32_t* sorted_codes, const int32_t* perm, const int32_t* q_order,
                                int score, float eps, HistMean hm, void* out, int32_t* idx_out, void* workspace,
                                hipStream_t stream) {
  const uint32_t* list_codes = nullptr;
  const int32_t* list_pos = nullptr;
  const bool tile = tile_path(is_bf16, dv, score == kScoreCauchy, dk);
  const FusedWs fw = fused_ws(S, N, topk, causal ? 1 : 0);
  char* wsb = static_cast<char*>(workspace);
  uint2* keys_full = reinterpret_cast<uint2*>(wsb + fw.keys_full_off);
  uint2* keys_list = reinterpret_cast<uint2*>(wsb + fw.keys_list_off);
  // The tiles' key rows in list order come with the prefix lists (d_k = 3).
  const bool rows_with_lists = tile && dk == 3;
  if (causal) {
    const hipError_t e =
        launch_prefix_lists(sorted_codes, perm, S, N, topk, workspace, stream, &list_codes, &list_pos,
                            rows_with_lists ? static_cast<const uint16_t*>(k) : nullptr, keys_full, keys_list);
    if (e != hipSuccess) return e;
  }
  if (tile) {
    int2* bounds = reinterpret_cast<int2*>(wsb + fw.bounds_off);
    return launch_select_attend_tile(q, k, v, S, N, dk, dv, topk, causal, chunk, q_codes, sorted_codes, perm,
                                     list_codes, list_pos, q_order, score, eps, hm, out, idx_out, bounds, keys_full,
                                     keys_list, rows_with_lists && list_codes != nullptr, stream);
  }
#define ZETA_FUSED_CASE(DVV)                                                                                       \
  case DVV:                                                                                                        \
    return is_bf16 ? launch_dk<uint16_t, DVV>(q, k, v, S, N, dk, topk, causal, chunk, q_codes, sorted_codes, perm, \
                                              list_codes, list_pos, q_order, score, eps, hm, out, idx_out, stream) \
                   : launch_dk<float, DVV>(q, k, v, S, N, dk, topk, causal, chunk, q_codes, sorted_codes, perm,    \
                                           list_codes, list_pos, q_order, score, eps, hm, out, idx_out, stream);
  switch (dv) {
    ZETA_FUSED_CASE(32)
    ZETA_FUSED_CASE(64)
    ZETA_FUSED_CASE(128)
    ZETA_FUSED_CASE(256)
    default:
      return hipErrorInvalidValue;
  }
#undef ZETA_FUSED_CASE
}

}  // namespace zeta
