// The locality experiment of Section 4.4: how many of a query's kn nearest
// keys in Euclidean distance its Z-order window of kn keys also holds.
//
//   exact_knn: one workgroup per query.  The squared distance to every key
//     of the query's pool is computed in float32 (one rounding per
//     subtraction, product and sum, axes in order: no fused multiply-add, so
//     that ties and near-ties are decided as a plain float32 evaluation
//     decides them), packed with the key's position into a 64-bit word
//     (distance bits above, position below; non-negative floats order as
//     their bits), and the words of up to 4096 keys are sorted in LDS by a
//     bitonic network.  The first kn positions are the answer, ordered by
//     (distance, position); a pool smaller than kn is padded with -1.
//   index_overlap: one wavefront per row marks row b's entries in an LDS
//     bit set of the segment's positions, counts row a's marked entries, and
//     clears its marks again.
// Both are small experiments (N up to 4096 keys per query for the exact
// search), not part of the attention's hot path.
#include "attend_device.h"
#include "device_common.h"
#include "kernels.h"
#include "layout.h"

namespace zeta {
namespace {

constexpr int kKnnThreads = 256;
constexpr int kOvWaves = 4;

// Squared distance of a query to key row kr, in float32 with one rounding
// per subtraction, product and sum, axes in order (no contraction into
// fused multiply-adds).
template <typename T, int KD>
__device__ __forceinline__ float plain_d2(const float* qv, const T* __restrict__ kr, int dk) {
#pragma clang fp contract(off)
  float d2 = 0.0f;
#pragma unroll
  for (int a = 0; a < KD; ++a) {
    if (a < dk) {
      const float diff = qv[a] - Elem<T>::load(kr + a);
      d2 = d2 + diff * diff;
    }
  }
  return d2;
}

template <typename T, int DK>
__global__ void __launch_bounds__(kKnnThreads)
    exact_knn_kernel(const T* __restrict__ q, const T* __restrict__ k, int64_t N, int dk_rt, int kn, int causal,
                     int P, int32_t* __restrict__ out) {
  constexpr int KD = DK > 0 ? DK : kMaxDk;
  const int dk = DK > 0 ? DK : dk_rt;
  __shared__ uint64_t s_key[kKnnMaxN];
  const int64_t row = blockIdx.x;  // segment * N + query position
  const int64_t seg = row / N;
  const int64_t i = row - seg * N;
  const int64_t end = causal ? i + 1 : N;  // pool: keys 0 .. end - 1
  float qv[KD];
#pragma unroll
  for (int a = 0; a < KD; ++a) qv[a] = a < dk ? Elem<T>::load(q + row * dk + a) : 0.0f;
  const T* kseg = k + seg * N * dk;
  for (int j = threadIdx.x; j < P; j += kKnnThreads) {
    uint64_t key = ~uint64_t(0);
    if (j < end) {
      const float d2 = plain_d2<T, KD>(qv, kseg + int64_t(j) * dk, dk);
      key = (uint64_t(__float_as_uint(d2)) << 32) | uint32_t(j);
    }
    s_key[j] = key;
  }
  __syncthreads();
  // Bitonic sort of the P words, ascending.
  for (int size = 2; size <= P; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int t = threadIdx.x; t < P; t += kKnnThreads) {
        const int u = t ^ stride;
        if (u > t) {
          const uint64_t x = s_key[t], y = s_key[u];
          const bool up = (t & size) == 0;
          if ((x > y) == up) {
            s_key[t] = y;
            s_key[u] = x;
          }
        }
      }
      __syncthreads();
    }
  }
  const int64_t m = end < kn ? end : kn;
  for (int c = threadIdx.x; c < kn; c += kKnnThreads)
    out[row * kn + c] = c < m ? int32_t(uint32_t(s_key[c] & 0xFFFFFFFFu)) : -1;
}

__global__ void __launch_bounds__(kOvWaves * 64)
    index_overlap_kernel(const int32_t* __restrict__ a, int ka, const int32_t* __restrict__ b, int kb, int64_t rows,
                         int64_t N, int32_t* __restrict__ counts) {
  __shared__ uint32_t s_bits[kOvWaves][kOverlapMaxN / 32];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int words = int((N + 31) / 32);
  for (int w = lane; w < words; w += 64) s_bits[wave][w] = 0u;
  wave_lds_sync();
  for (int64_t r = int64_t(blockIdx.x) * kOvWaves + wave; r < rows; r += int64_t(gridDim.x) * kOvWaves) {
    const int32_t* br = b + r * kb;
    const int32_t* ar = a + r * ka;
    for (int c = lane; c < kb; c += 64) {
      const int32_t j = br[c];
      if (j >= 0 && j < N) atomicOr(&s_bits[wave][j >> 5], 1u << (j & 31));
    }
    wave_lds_sync();
    int cnt = 0;
    for (int c = lane; c < ka; c += 64) {
      const int32_t j = ar[c];
      if (j >= 0 && j < N && ((s_bits[wave][j >> 5] >> (j & 31)) & 1u) != 0u) ++cnt;
    }
    cnt = int(wave_sum(float(cnt)));
    if (lane == 0) counts[r] = cnt;
    wave_lds_sync();
    for (int c = lane; c < kb; c += 64) {
      const int32_t j = br[c];
      if (j >= 0 && j < N) atomicAnd(&s_bits[wave][j >> 5], ~(1u << (j & 31)));
    }
    wave_lds_sync();
  }
}

template <typename T>
hipError_t knn_t(const void* q, const void* k, int64_t S, int64_t N, int dk, int kn, bool causal, int32_t* out,
                 hipStream_t stream) {
  int P = 1;
  while (P < N) P <<= 1;
  const dim3 grid(unsigned(S * N)), block(kKnnThreads);
  if (dk == 3)
    hipLaunchKernelGGL((exact_knn_kernel<T, 3>), grid, block, 0, stream, static_cast<const T*>(q),
                       static_cast<const T*>(k), N, dk, kn, causal ? 1 : 0, P, out);
  else
    hipLaunchKernelGGL((exact_knn_kernel<T, 0>), grid, block, 0, stream, static_cast<const T*>(q),
                       static_cast<const T*>(k), N, dk, kn, causal ? 1 : 0, P, out);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_exact_knn(const void* q, const void* k, bool is_bf16, int64_t S, int64_t N, int dk, int kn,
                            bool causal, int32_t* out, hipStream_t stream) {
  if (is_bf16) return knn_t<uint16_t>(q, k, S, N, dk, kn, causal, out, stream);
  return knn_t<float>(q, k, S, N, dk, kn, causal, out, stream);
}

hipError_t launch_index_overlap(const int32_t* a, int ka, const int32_t* b, int kb, int64_t rows, int64_t N,
                                int32_t* counts, hipStream_t stream) {
  const int64_t want = ceil_div(rows, kOvWaves);
  const unsigned blocks = unsigned(want < 4096 ? want : 4096);
  hipLaunchKernelGGL(index_overlap_kernel, dim3(blocks), dim3(kOvWaves * 64), 0, stream, a, ka, b, kb, rows, N,
                     counts);
  return hipGetLastError();
}

}  // namespace zeta
