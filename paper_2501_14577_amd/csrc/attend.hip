// Adaptive Cauchy-softmax attention over each query's selected keys
// (Section 3.3, equation cauchy; Section 3.4; Appendix E.1 steps 1-4):
//   S_ij = 1 / (||q_i - k_j||^2 + eps),  o_i = sum_j S_ij v_j / sum_j S_ij.
//
// One wavefront per query.  d_k is 3, so scores are a handful of scalar FMAs
// per candidate and there is no dense contraction for the matrix cores: the
// kernel is a gather of k value rows per query.
//   Phase 1: lane c takes candidates c, c+64, ...: reads the index, gathers
//            the key row, computes S_ij in float32 and stages the pair (byte
//            offset of the value row, S_ij) in LDS; wavefront reductions give
//            the normaliser and the number of valid slots.
//   Phase 2: the wavefront splits into groups of LPR lanes, LPR = bytes per
//            value row / 16, so one 16-byte load per lane moves 64/LPR whole
//            rows per instruction; groups stride over the candidates with
//            eight rows in flight per lane, accumulating in float32.  Loads
//            address the segment's values through a wave-uniform base and a
//            32-bit per-lane offset.
//   Phase 3: xor-shuffles fold the groups; the first group scales by the
//            normaliser and stores the row (bfloat16 rounded to nearest even).
//
// Queries are taken in an optional processing order (a permutation per
// segment).  Walking queries in Z-order makes neighbouring wavefronts gather
// overlapping rows; the logical blocks of each XCD are contiguous, so those
// wavefronts share one L2.  The order never changes any result.
#include "device_common.h"
#include "kernels.h"
#include "layout.h"

namespace zeta {
namespace {

template <typename T>
struct Vec16;  // one 16-byte lane load of a value row, widened to float32

template <>
struct Vec16<float> {
  static constexpr int kElems = 4;
  __device__ __forceinline__ static void widen(const uint4& x, float* f) {
    f[0] = __uint_as_float(x.x);
    f[1] = __uint_as_float(x.y);
    f[2] = __uint_as_float(x.z);
    f[3] = __uint_as_float(x.w);
  }
  __device__ __forceinline__ static void store(float* p, const float* f) {
    *reinterpret_cast<float4*>(p) = make_float4(f[0], f[1], f[2], f[3]);
  }
};

template <>
struct Vec16<uint16_t> {
  static constexpr int kElems = 8;
  __device__ __forceinline__ static void widen(const uint4& x, float* f) {
    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = __uint_as_float(w[i] << 16);
      f[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  }
  __device__ __forceinline__ static void store(uint16_t* p, const float* f) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = uint32_t(float_to_bf16_bits(f[2 * i])) | (uint32_t(float_to_bf16_bits(f[2 * i + 1])) << 16);
    *reinterpret_cast<uint4*>(p) = make_uint4(w[0], w[1], w[2], w[3]);
  }
};

// Byte offset of a value row inside its segment: 32-bit when the segment's
// values span less than 4 GiB, else 64-bit.
template <bool kOff32>
struct RowOff {
  using type = int64_t;
};
template <>
struct RowOff<true> {
  using type = uint32_t;
};

template <typename T, int DV, int DK, bool kOff32>
__global__ void __launch_bounds__(kAttWavesPerBlock * 64)
    attend_kernel(const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
                  const int32_t* __restrict__ idx, const int32_t* __restrict__ q_order, int64_t total,
                  int64_t N, int dk_rt, int topk, float eps, T* __restrict__ out) {
  constexpr int kE = Vec16<T>::kElems;  // elements per lane load
  constexpr int kLpr = DV / kE;         // lanes per value row
  constexpr int kGroups = 64 / kLpr;    // rows per wavefront load
  constexpr int kUnroll = 8;            // rows in flight per lane
  constexpr int kRowBytes = DV * int(sizeof(T));
  static_assert(kLpr >= 1 && kLpr <= 64 && 64 % kLpr == 0, "row must split evenly over lanes");
  using Off = typename RowOff<kOff32>::type;
  const int dk = DK > 0 ? DK : dk_rt;

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
#pragma unroll
    for (int a = 0; a < (DK > 0 ? DK : kMaxDk); ++a) qv[a] = a < dk ? Elem<T>::load(q + g * dk + a) : 0.0f;

    // Phase 1: scores.
    float zsum = 0.0f;
    int m = 0;  // one past the last valid slot
    const int32_t* irow = idx + g * topk;
    for (int c = lane; c < topk; c += 64) {
      const int32_t j = irow[c];
      const bool ok = j >= 0 && j < N;
      float s = 0.0f;
      if (ok) {
        const T* kr = kseg + int64_t(j) * dk;
        float d2 = 0.0f;
#pragma unroll
        for (int a = 0; a < (DK > 0 ? DK : kMaxDk); ++a) {
          if (a < dk) {
            const float diff = qv[a] - Elem<T>::load(kr + a);
            d2 += diff * diff;
          }
        }
        s = 1.0f / (d2 + eps);
        m = c + 1;
      }
      s_off[c] = ok ? Off(j) * Off(kRowBytes) : Off(0);
      s_w[c] = s;
      zsum += s;
    }
    zsum = wave_sum(zsum);
    m = wave_max(m);
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
        for (int e = 0; e < kE; ++e) acc[e] += wv[u] * f[e];
      }
    }
    for (; c < m; c += kGroups) {
      float f[kE];
      const float w = s_w[c];
      Vec16<T>::widen(*reinterpret_cast<const uint4*>(vseg + (s_off[c] + lane_off)), f);
#pragma unroll
      for (int e = 0; e < kE; ++e) acc[e] += w * f[e];
    }

    // Phase 3: fold the groups and store.
#pragma unroll
    for (int off = kLpr; off < 64; off <<= 1)
#pragma unroll
      for (int e = 0; e < kE; ++e) acc[e] += __shfl_xor(acc[e], off, 64);
    if (grp == 0) {
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
                           int topk, const int32_t* idx, const int32_t* q_order, float eps, void* out,
                           hipStream_t stream) {
  const int64_t total = S * N;
  const int64_t want = ceil_div(total, kAttWavesPerBlock);
  const unsigned blocks = unsigned(want < (int64_t(1) << 20) ? want : (int64_t(1) << 20));
  const bool off32 = N * int64_t(DV) * int64_t(sizeof(T)) <= int64_t(0xFFFFFFFFu) - int64_t(DV) * int64_t(sizeof(T));
  const size_t lds = size_t(kAttWavesPerBlock) * topk * ((off32 ? 4 : 8) + 4);
  if (off32)
    hipLaunchKernelGGL((attend_kernel<T, DV, DK, true>), dim3(blocks), dim3(kAttWavesPerBlock * 64), lds, stream,
                       static_cast<const T*>(q), static_cast<const T*>(k), static_cast<const T*>(v), idx,
                       q_order, total, N, dk, topk, eps, static_cast<T*>(out));
  else
    hipLaunchKernelGGL((attend_kernel<T, DV, DK, false>), dim3(blocks), dim3(kAttWavesPerBlock * 64), lds, stream,
                       static_cast<const T*>(q), static_cast<const T*>(k), static_cast<const T*>(v), idx,
                       q_order, total, N, dk, topk, eps, static_cast<T*>(out));
  return hipGetLastError();
}

template <typename T, int DV>
hipError_t launch_attend_dk(const void* q, const void* k, const void* v, int64_t S, int64_t N, int dk,
                            int topk, const int32_t* idx, const int32_t* q_order, float eps, void* out,
                            hipStream_t stream) {
  if (dk == 3) return launch_attend_t<T, DV, 3>(q, k, v, S, N, dk, topk, idx, q_order, eps, out, stream);
  return launch_attend_t<T, DV, 0>(q, k, v, S, N, dk, topk, idx, q_order, eps, out, stream);
}

}  // namespace

bool attend_supports(int dv) { return dv == 32 || dv == 64 || dv == 128 || dv == 256; }

hipError_t launch_attend(const void* q, const void* k, const void* v, bool is_bf16, int64_t S,
                         int64_t N, int dk, int dv, int topk, const int32_t* idx, const int32_t* q_order,
                         float eps, void* out, hipStream_t stream) {
#define ZETA_ATTEND_CASE(DVV)                                                                            \
  case DVV:                                                                                              \
    return is_bf16                                                                                       \
               ? launch_attend_dk<uint16_t, DVV>(q, k, v, S, N, dk, topk, idx, q_order, eps, out, stream) \
               : launch_attend_dk<float, DVV>(q, k, v, S, N, dk, topk, idx, q_order, eps, out, stream);
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
