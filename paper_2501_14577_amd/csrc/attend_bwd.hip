// Gradients of the top-k Cauchy-softmax attention (Appendix E.2, summary of
// gradient computations) for fixed windows idx.  With S_ij = 1 / delta_ij,
// delta_ij = ||q_i - k_j||^2 + eps, Z_i = sum_j S_ij, A_ij = S_ij / Z_i,
// o_i = sum_j A_ij v_j and g_ij = dout_i . (v_j - o_i):
//   dv_j += A_ij dout_i                      (every query i whose window holds j)
//   dq_i  = -2 sum_j w_ij (q_i - k_j)        w_ij = g_ij S_ij^2 / Z_i
//   dk_j += 2 w_ij (q_i - k_j)
//   deps  = -sum_ij w_ij
// o_i is not read: dout_i . o_i = sum_j A_ij (dout_i . v_j), from the same
// per-pair dot products.
//
// One wavefront per query, 4 per block:
//   phase 1: scores S_ij (lane pairs as in the forward kernel), Z_i;
//   phase 2: groups of d_v*s/16 lanes take one value row each with 16-byte
//            loads, form dout_i . v_j (group reduction) and add A_ij dout_i to
//            dv_j (float32 atomics, one per element);
//   phase 3: one lane per pair: w_ij, dq accumulated in registers, dk_j
//            updated with float32 atomics; the wavefront's sum of w_ij goes to
//            a per-query partial, reduced afterwards in a fixed order.
// dq, dk, dv and the partials are cleared by a fill kernel first (no
// memset), so every output element is defined.  dk and dv are sums of
// atomics: their last bits depend on the order in which they land.
#include "attend_device.h"
#include "device_common.h"
#include "kernels.h"
#include "layout.h"

namespace zeta {
namespace {

constexpr int kBwdWaves = 4;

__global__ void __launch_bounds__(256) fill_zero_kernel(float* __restrict__ p, int64_t n) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t t = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; t < n; t += stride) p[t] = 0.0f;
}

template <typename T, int DV, int DK>
__global__ void __launch_bounds__(kBwdWaves * 64)
    attend_bwd_kernel(const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
                      const T* __restrict__ dout, const int32_t* __restrict__ idx, const int32_t* __restrict__ q_order,
                      int64_t total, int64_t N, int dk_rt, int topk, float eps, float* __restrict__ dq,
                      float* __restrict__ dk, float* __restrict__ dv, float* __restrict__ deps_part) {
  constexpr int kE = Vec16<T>::kElems;  // elements per lane load
  constexpr int kLpr = DV / kE;         // lanes per value row
  constexpr int kGroups = 64 / kLpr;    // rows per wavefront load
  constexpr int kUnroll = 4;            // rows in flight per lane
  constexpr int KD = DK > 0 ? DK : kMaxDk;
  static_assert(kLpr >= 1 && kLpr <= 64 && 64 % kLpr == 0, "row must split evenly over lanes");
  const int dk_n = DK > 0 ? DK : dk_rt;

  extern __shared__ unsigned char s_raw[];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  // Per wave: topk key positions, then topk scores, then topk dot products.
  int32_t* s_j = reinterpret_cast<int32_t*>(s_raw) + size_t(wave) * topk;
  float* s_s = reinterpret_cast<float*>(s_raw) + size_t(kBwdWaves) * topk + size_t(wave) * topk;
  float* s_g = reinterpret_cast<float*>(s_raw) + size_t(2 * kBwdWaves) * topk + size_t(wave) * topk;
  const int grp = lane / kLpr;
  const int sub = lane - grp * kLpr;
  const int64_t nb = gridDim.x;

  for (int64_t blk = xcd_contiguous_block(blockIdx.x, nb); blk * kBwdWaves < total; blk += nb) {
    const int64_t slot = blk * kBwdWaves + wave;
    if (slot >= total) continue;
    const int64_t seg = slot / N;
    int64_t i = slot - seg * N;
    if (q_order != nullptr) {
      i = q_order[slot];
      if (i < 0 || i >= N) continue;  // not a permutation entry: nothing to do
    }
    const int64_t g = seg * N + i;
    const T* kseg = k + seg * N * dk_n;
    const T* vseg = v + seg * N * DV;
    float* dkseg = dk + seg * N * dk_n;
    float* dvseg = dv + seg * N * DV;

    float qv[KD];
    if constexpr (DK == 3) {
      Row3<T>::load(q, g, total, qv);
    } else {
#pragma unroll
      for (int a = 0; a < KD; ++a) qv[a] = a < dk_n ? Elem<T>::load(q + g * dk_n + a) : 0.0f;
    }

    // Phase 1: scores.
    float zsum = 0.0f;
    int m = 0;  // one past the last valid slot
    const int32_t* irow = idx + g * topk;
    for (int c = lane; c < topk; c += 64) {
      const int32_t j = irow[c];
      const bool ok = j >= 0 && j < N;
      float s = 0.0f;
      if (ok) {
        float kv[KD];
        if constexpr (DK == 3) {
          Row3<T>::load(k, seg * N + j, total, kv);
        } else {
#pragma unroll
          for (int a = 0; a < KD; ++a) kv[a] = a < dk_n ? Elem<T>::load(kseg + int64_t(j) * dk_n + a) : 0.0f;
        }
        float d2 = 0.0f;
#pragma unroll
        for (int a = 0; a < KD; ++a) {
          if (a < dk_n) {
            const float diff = qv[a] - kv[a];
            d2 = fmaf(diff, diff, d2);
          }
        }
        s = 1.0f / (d2 + eps);
        m = c + 1;
      }
      s_j[c] = ok ? j : -1;
      s_s[c] = s;
      zsum += s;
    }
    zsum = wave_sum(zsum);
    m = wave_max(m);
    const float inv_z = zsum > 0.0f ? 1.0f / zsum : 0.0f;
    wave_lds_sync();

    // Phase 2: dout_i . v_j per pair, and dv_j += A_ij dout_i.
    float du[kE];
    Vec16<T>::widen(*reinterpret_cast<const uint4*>(dout + g * DV + sub * kE), du);
    for (int c0 = grp; c0 < m; c0 += kUnroll * kGroups) {
      uint4 raw[kUnroll];
      int32_t jj[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int c = c0 + u * kGroups;
        jj[u] = c < m ? s_j[c] : -1;
        raw[u] = *reinterpret_cast<const uint4*>(vseg + int64_t(jj[u] >= 0 ? jj[u] : 0) * DV + sub * kE);
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int c = c0 + u * kGroups;
        float f[kE];
        Vec16<T>::widen(raw[u], f);
        float part = 0.0f;
#pragma unroll
        for (int e = 0; e < kE; ++e) part = fmaf(du[e], f[e], part);
#pragma unroll
        for (int off = 1; off < kLpr; off <<= 1) part += __shfl_xor(part, off, 64);
        if (jj[u] >= 0) {
          if (sub == 0) s_g[c] = part;
          const float a = s_s[c] * inv_z;
          float* dst = dvseg + int64_t(jj[u]) * DV + sub * kE;
#pragma unroll
          for (int e = 0; e < kE; ++e) atomicAdd(dst + e, a * du[e]);
        } else if (c < m && sub == 0) {
          s_g[c] = 0.0f;
        }
      }
    }
    wave_lds_sync();

    // dout_i . o_i = sum_j A_ij (dout_i . v_j).
    float cdot = 0.0f;
    for (int c = lane; c < m; c += 64) cdot = fmaf(s_s[c], s_g[c], cdot);
    cdot = wave_sum(cdot) * inv_z;

    // Phase 3: w_ij, dq, dk, deps.
    float dqa[KD];
#pragma unroll
    for (int a = 0; a < KD; ++a) dqa[a] = 0.0f;
    float wsum = 0.0f;
    for (int c = lane; c < m; c += 64) {
      const int32_t j = s_j[c];
      if (j < 0) continue;
      const float s = s_s[c];
      const float w = (s_g[c] - cdot) * s * s * inv_z;
      float kv[KD];
      if constexpr (DK == 3) {
        Row3<T>::load(k, seg * N + j, total, kv);
      } else {
#pragma unroll
        for (int a = 0; a < KD; ++a) kv[a] = a < dk_n ? Elem<T>::load(kseg + int64_t(j) * dk_n + a) : 0.0f;
      }
#pragma unroll
      for (int a = 0; a < KD; ++a) {
        if (a < dk_n) {
          const float diff = qv[a] - kv[a];
          dqa[a] = fmaf(w, diff, dqa[a]);
          atomicAdd(dkseg + int64_t(j) * dk_n + a, 2.0f * w * diff);
        }
      }
      wsum += w;
    }
#pragma unroll
    for (int a = 0; a < KD; ++a) dqa[a] = wave_sum(dqa[a]);
    wsum = wave_sum(wsum);
    if (lane == 0) {
#pragma unroll
      for (int a = 0; a < KD; ++a)
        if (a < dk_n) dq[g * dk_n + a] = -2.0f * dqa[a];
      deps_part[g] = -wsum;
    }
    wave_lds_sync();
  }
}

// deps = sum of the per-query partials, in a fixed order: each of up to
// kRedBlocks blocks sums a contiguous range (threads strided, then a tree in
// LDS), then one block sums the block results.
constexpr int kRedBlocks = 256;

__global__ void __launch_bounds__(256)
    reduce_partials_kernel(const float* __restrict__ part, int64_t n, float* __restrict__ block_sums) {
  __shared__ float s_sum[256];
  const int64_t per = (n + gridDim.x - 1) / gridDim.x;
  const int64_t b0 = int64_t(blockIdx.x) * per;
  const int64_t b1 = b0 + per < n ? b0 + per : n;
  float acc = 0.0f;
  for (int64_t t = b0 + threadIdx.x; t < b1; t += 256) acc += part[t];
  s_sum[threadIdx.x] = acc;
  __syncthreads();
  for (int w = 128; w >= 1; w >>= 1) {
    if (int(threadIdx.x) < w) s_sum[threadIdx.x] += s_sum[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) block_sums[blockIdx.x] = s_sum[0];
}

__global__ void __launch_bounds__(256)
    reduce_final_kernel(const float* __restrict__ block_sums, int nblocks, float* __restrict__ out) {
  __shared__ float s_sum[256];
  s_sum[threadIdx.x] = int(threadIdx.x) < nblocks ? block_sums[threadIdx.x] : 0.0f;
  __syncthreads();
  for (int w = 128; w >= 1; w >>= 1) {
    if (int(threadIdx.x) < w) s_sum[threadIdx.x] += s_sum[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) out[0] = s_sum[0];
}

void fill_zero(float* p, int64_t n, hipStream_t stream) {
  if (n <= 0) return;
  const int64_t want = (n + 255) / 256;
  const unsigned blocks = unsigned(want < 4096 ? want : 4096);
  hipLaunchKernelGGL(fill_zero_kernel, dim3(blocks), dim3(256), 0, stream, p, n);
}

template <typename T, int DV>
hipError_t launch_bwd_t(const T* q, const T* k, const T* v, const T* dout, int64_t S, int64_t N, int dk, int topk,
                        const int32_t* idx, const int32_t* q_order, float eps, float* dq, float* dkg, float* dv,
                        float* deps, float* part, float* block_sums, hipStream_t stream) {
  const int64_t total = S * N;
  fill_zero(dq, total * dk, stream);
  fill_zero(dkg, total * dk, stream);
  fill_zero(dv, total * DV, stream);
  fill_zero(part, total, stream);
  const int64_t want = ceil_div(total, kBwdWaves);
  const unsigned blocks = unsigned(want < (int64_t(1) << 20) ? want : (int64_t(1) << 20));
  const size_t lds = size_t(kBwdWaves) * topk * 12;
  if (dk == 3)
    hipLaunchKernelGGL((attend_bwd_kernel<T, DV, 3>), dim3(blocks), dim3(kBwdWaves * 64), lds, stream, q, k, v, dout,
                       idx, q_order, total, N, dk, topk, eps, dq, dkg, dv, part);
  else
    hipLaunchKernelGGL((attend_bwd_kernel<T, DV, 0>), dim3(blocks), dim3(kBwdWaves * 64), lds, stream, q, k, v, dout,
                       idx, q_order, total, N, dk, topk, eps, dq, dkg, dv, part);
  const int nred = int(total < kRedBlocks ? total : kRedBlocks);
  hipLaunchKernelGGL(reduce_partials_kernel, dim3(unsigned(nred)), dim3(256), 0, stream, part, total, block_sums);
  hipLaunchKernelGGL(reduce_final_kernel, dim3(1), dim3(256), 0, stream, block_sums, nred, deps);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_bwd_dv(const void* q, const void* k, const void* v, const void* dout, int64_t S, int64_t N, int dk,
                         int dv, int topk, const int32_t* idx, const int32_t* q_order, float eps, float* dq,
                         float* dkg, float* dvg, float* deps, float* part, float* block_sums, hipStream_t stream) {
  const T* qq = static_cast<const T*>(q);
  const T* kk = static_cast<const T*>(k);
  const T* vv = static_cast<const T*>(v);
  const T* dd = static_cast<const T*>(dout);
  switch (dv) {
    case 32:
      return launch_bwd_t<T, 32>(qq, kk, vv, dd, S, N, dk, topk, idx, q_order, eps, dq, dkg, dvg, deps, part,
                                 block_sums, stream);
    case 64:
      return launch_bwd_t<T, 64>(qq, kk, vv, dd, S, N, dk, topk, idx, q_order, eps, dq, dkg, dvg, deps, part,
                                 block_sums, stream);
    case 128:
      return launch_bwd_t<T, 128>(qq, kk, vv, dd, S, N, dk, topk, idx, q_order, eps, dq, dkg, dvg, deps, part,
                                  block_sums, stream);
    case 256:
      return launch_bwd_t<T, 256>(qq, kk, vv, dd, S, N, dk, topk, idx, q_order, eps, dq, dkg, dvg, deps, part,
                                  block_sums, stream);
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_attend_bwd(const void* q, const void* k, const void* v, const void* dout, bool is_bf16, int64_t S,
                             int64_t N, int dk, int dv, int topk, const int32_t* idx, const int32_t* q_order,
                             float eps, float* dq, float* dkg, float* dvg, float* deps, void* workspace,
                             hipStream_t stream) {
  const BwdWs ws = bwd_ws(S, N);
  char* wsb = static_cast<char*>(workspace);
  float* part = reinterpret_cast<float*>(wsb + ws.part_off);
  float* block_sums = reinterpret_cast<float*>(wsb + ws.block_off);
  if (is_bf16)
    return launch_bwd_dv<uint16_t>(q, k, v, dout, S, N, dk, dv, topk, idx, q_order, eps, dq, dkg, dvg, deps, part,
                                   block_sums, stream);
  return launch_bwd_dv<float>(q, k, v, dout, S, N, dk, dv, topk, idx, q_order, eps, dq, dkg, dvg, deps, part,
                              block_sums, stream);
}

}  // namespace zeta
