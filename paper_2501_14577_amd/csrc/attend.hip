// Adaptive Cauchy-softmax attention over each query's selected keys
// (Section 3.3, equation cauchy; Section 3.4; Appendix E.1 steps 1-4):
//   S_ij = 1 / (||q_i - k_j||^2 + eps),  o_i = sum_j S_ij v_j / sum_j S_ij,
// or one of the score variants the paper compares it with (Section 4.3;
// Appendix G.2): the same weighted sum with other weights.
//
// One wavefront per query.  d_k is 3, so scores are a handful of scalar FMAs
// per candidate and there is no dense contraction for the matrix cores: the
// kernel is a gather of k value rows per query.
//   Phase 1: lane l takes candidate slots 2l and 2l+1 (and every 128th
//            after): one 8-byte load reads both indices, one load per key row
//            gathers its coordinates; S_ij is computed in float32 and the pair
//            (byte offset of the value row, S_ij) staged in LDS; wavefront
//            reductions give the normaliser and the number of valid slots.
//   Phase 2: the wavefront splits into groups of LPR lanes, LPR = bytes per
//            value row / 16, so one 16-byte load per lane moves 64/LPR whole
//            rows per instruction; groups stride over the candidates with
//            eight rows in flight per lane, accumulating in float32.  Loads
//            address the segment's values through a wave-uniform base and a
//            32-bit per-lane offset.
//   Phase 3: xor-shuffles fold the groups; the first group adds the
//            history-mean candidate when given (its score joins the
//            normaliser), scales by the normaliser and stores the row
//            (bfloat16 rounded to nearest even).
// Distances and the accumulation use explicit fused multiply-adds.
//
// Queries are taken in an optional processing order (a permutation per
// segment).  Walking queries in Z-order makes neighbouring wavefronts gather
// overlapping rows; the logical blocks of each XCD are contiguous, so those
// wavefronts share one L2.  The order never changes a result of this kernel.
// Given an order, bfloat16 calls with d_k = 3, d_v <= 128 and k <= 128 run on
// the matrix-core tiles instead (tile.hip), which share each 16 queries'
// rows.
#include "attend_device.h"
#include "device_common.h"
#include "kernels.h"
#include "layout.h"

namespace zeta {
namespace {

template <typename T, int DV, int DK, bool kOff32, bool kVariants>
__global__ void __launch_bounds__(kAttWavesPerBlock * 64)
    attend_kernel(const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
                  const int32_t* __restrict__ idx, const int32_t* __restrict__ q_order, int64_t total,
                  int64_t N, int dk_rt, int topk, int score_rt, float eps, const float* __restrict__ mk,
                  const float* __restrict__ mv, T* __restrict__ out) {
  constexpr int kE = Vec16<T>::kElems;  // elements per lane load
  constexpr int kLpr = DV / kE;         // lanes per value row
  constexpr int kGroups = 64 / kLpr;    // rows per wavefront load
  constexpr int kUnroll = 8;            // rows in flight per lane
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
  // Per wave: topk row offsets, then (after every wave's offsets) topk scores.
  Off* s_off = reinterpret_cast<Off*>(s_raw) + size_t(wave) * topk;
  float* s_w = reinterpret_cast<float*>(s_raw + size_t(kAttWavesPerBlock) * topk * sizeof(Off)) + size_t(wave) * topk;
  const int grp = lane / kLpr;
  const int sub = lane - grp * kLpr;
  const int64_t nb = gridDim.x;

  for (int64_t blk = xcd_contiguous_block(blockIdx.x, nb); blk * kAttWavesPerBlock < total; blk += nb) {
    const int64_t slot = blk * kAttWavesPerBlock + wave;
    if (slot >= total) continue;
    const int64_t seg = slot / N;
    int64_t i = slot - seg * N;
    if (q_order != nullptr) {
      i = q_order[slot];
      if (i < 0 || i >= N) continue;  // not a permutation entry: nothing to do
    }
    const int64_t g = seg * N + i;
    const T* kseg = k + seg * N * dk;
    const unsigned char* vseg = reinterpret_cast<const unsigned char*>(v + seg * N * DV);

    float qv[DK > 0 ? DK : kMaxDk];
    if constexpr (DK == 3) {
      Row3<T>::load(q, g, total, qv);
    } else {
#pragma unroll
      for (int a = 0; a < (DK > 0 ? DK : kMaxDk); ++a) qv[a] = a < dk ? Elem<T>::load(q + g * dk + a) : 0.0f;
    }

    // Phase 1: scores.  Lane l takes the slot pair (2l, 2l+1) of every block
    // of 128 slots, reading both indices with one 8-byte load when the row
    // is 8-byte aligned (even topk).  The softmax variants store logits here
    // and exponentiate once the window's largest is known.
    const float qn = score == kScoreNormDot ? row_norm<KD>(qv, dk) : 0.0f;
    float zsum = 0.0f;
    float zloc = -INFINITY;
    uint32_t okmask = 0u;
    int bit = 0;
    int m = 0;  // one past the last valid slot
    const int32_t* irow = idx + g * topk;
    for (int c0 = 2 * lane; c0 < topk; c0 += 128) {
      int32_t jj[2];
      if ((topk & 1) == 0) {
        const Words2 w = *reinterpret_cast<const Words2*>(irow + c0);
        jj[0] = int32_t(w.a);
        jj[1] = int32_t(w.b);
      } else {
        jj[0] = irow[c0];
        jj[1] = c0 + 1 < topk ? irow[c0 + 1] : -1;
      }
#pragma unroll
      for (int h = 0; h < 2; ++h, ++bit) {
        const int c = c0 + h;
        const int32_t j = jj[h];
        const bool ok = c < topk && j >= 0 && j < N;
        float s = 0.0f;
        if (ok) {
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
          m = c + 1;
        }
        if (c < topk) {
          s_off[c] = ok ? Off(j) * Off(kRowBytes) : Off(0);
          s_w[c] = s;
        }
        zsum += s;
      }
    }
    m = wave_max(m);
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

    // Phase 2: weighted gather of value rows.
    float acc[kE];
#pragma unroll
    for (int e = 0; e < kE; ++e) acc[e] = 0.0f;
    const Off lane_off = Off(sub * 16);
    int c = grp;
    for (; c + (kUnroll - 1) * kGroups < m; c += kUnroll * kGroups) {
      uint4 raw[kUnroll];
      float wv[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int cc = c + u * kGroups;
        wv[u] = s_w[cc];
        raw[u] = *reinterpret_cast<const uint4*>(vseg + (s_off[cc] + lane_off));
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        float f[kE];
        Vec16<T>::widen(raw[u], f);
#pragma unroll
        for (int e = 0; e < kE; ++e) acc[e] = fmaf(wv[u], f[e], acc[e]);
      }
    }
    for (; c < m; c += kGroups) {
      float f[kE];
      const float w = s_w[c];
      Vec16<T>::widen(*reinterpret_cast<const uint4*>(vseg + (s_off[c] + lane_off)), f);
#pragma unroll
      for (int e = 0; e < kE; ++e) acc[e] = fmaf(w, f[e], acc[e]);
    }

    // Phase 3: fold the groups and store.
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

template <typename T, int DV, int DK>
hipError_t launch_attend_t(const void* q, const void* k, const void* v, int64_t S, int64_t N, int dk,
                           int topk, const int32_t* idx, const int32_t* q_order, int score, float eps, HistMean hm,
                           void* out, hipStream_t stream) {
  const int64_t total = S * N;
  const int64_t want = ceil_div(total, kAttWavesPerBlock);
  const unsigned blocks = unsigned(want < (int64_t(1) << 20) ? want : (int64_t(1) << 20));
  const bool off32 = N * int64_t(DV) * int64_t(sizeof(T)) <= int64_t(0xFFFFFFFFu) - int64_t(DV) * int64_t(sizeof(T));
  const size_t lds = size_t(kAttWavesPerBlock) * topk * ((off32 ? 4 : 8) + 4);
#define ZETA_ATTEND_LAUNCH(OFF, VAR)                                                                         \
  hipLaunchKernelGGL((attend_kernel<T, DV, DK, OFF, VAR>), dim3(blocks), dim3(kAttWavesPerBlock * 64), lds, stream, \
                     static_cast<const T*>(q), static_cast<const T*>(k), static_cast<const T*>(v), idx, q_order,   \
                     total, N, dk, topk, score, eps, hm.k, hm.v, static_cast<T*>(out))
  const bool var = score != kScoreCauchy;
  if (off32) {
    if (var)
      ZETA_ATTEND_LAUNCH(true, true);
    else
      ZETA_ATTEND_LAUNCH(true, false);
  } else {
    if (var)
      ZETA_ATTEND_LAUNCH(false, true);
    else
      ZETA_ATTEND_LAUNCH(false, false);
  }
#undef ZETA_ATTEND_LAUNCH
  return hipGetLastError();
}

template <typename T, int DV>
hipError_t launch_attend_dk(const void* q, const void* k, const void* v, int64_t S, int64_t N, int dk,
                            int topk, const int32_t* idx, const int32_t* q_order, int score, float eps, HistMean hm,
                            void* out, hipStream_t stream) {
  if (dk == 3) return launch_attend_t<T, DV, 3>(q, k, v, S, N, dk, topk, idx, q_order, score, eps, hm, out, stream);
  return launch_attend_t<T, DV, 0>(q, k, v, S, N, dk, topk, idx, q_order, score, eps, hm, out, stream);
}

}  // namespace

bool attend_supports(int dv) { return dv == 32 || dv == 64 || dv == 128 || dv == 256; }

hipError_t launch_attend(const void* q, const void* k, const void* v, bool is_bf16, int64_t S,
                         int64_t N, int dk, int dv, int topk, const int32_t* idx, const int32_t* q_order,
                         int score, float eps, HistMean hm, void* out, hipStream_t stream) {
  if (idx_tile_path(is_bf16, dk, dv, topk, q_order != nullptr))
    return launch_attend_idx_tile(q, k, v, S, N, dv, topk, idx, q_order, score, eps, hm, out, stream);
#define ZETA_ATTEND_CASE(DVV)                                                                            \
  case DVV:                                                                                              \
    return is_bf16                                                                                       \
               ? launch_attend_dk<uint16_t, DVV>(q, k, v, S, N, dk, topk, idx, q_order, score, eps, hm, out, \
                                                 stream)                                                 \
               : launch_attend_dk<float, DVV>(q, k, v, S, N, dk, topk, idx, q_order, score, eps, hm, out, stream);
  switch (dv) {
    ZETA_ATTEND_CASE(32)
    ZETA_ATTEND_CASE(64)
    ZETA_ATTEND_CASE(128)
    ZETA_ATTEND_CASE(256)
    default:
      return hipErrorInvalidValue;
  }
#undef ZETA_ATTEND_CASE
}

}  // namespace zeta
