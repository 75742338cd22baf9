// Gradients of the top-k Cauchy-softmax attention (Appendix E.2, summary of
// gradient computations) for fixed windows idx.  With S_ij = 1 / delta_ij,
// delta_ij = ||q_i - k_j||^2 + eps, Z_i = sum_j S_ij, A_ij = S_ij / Z_i,
// o_i = sum_j A_ij v_j and g_ij = dout_i . (v_j - o_i):
//   dv_j  = sum over queries i whose window holds j of A_ij dout_i
//   dq_i  = -2 sum_j w_ij (q_i - k_j)        w_ij = g_ij S_ij^2 / Z_i
//   dk_j  = 2 sum over those i of w_ij (q_i - k_j)
//   deps  = -sum_ij w_ij
// o_i is not read: c_i = dout_i . o_i = sum_j A_ij (dout_i . v_j), from the
// same per-pair dot products.
//
// No atomics.  Sums over a key's queries are formed by the key's own
// wavefront after the (query, key) pairs are regrouped by key:
//   1. query pass, one wavefront per query: S_ij and Z_i (lane per pair);
//      dout_i . v_j (groups of d_v*s/16 lanes per value row, 16-byte loads,
//      group reduction); c_i; w_ij, dq_i and the query's part of deps.  It
//      stores (Z_i, c_i) and, for every window slot, the key index (N for an
//      empty slot) in query-major order;
//   2. the library's stable radix sort orders those slots by key per segment;
//      the sort's permutation gives each slot's query (slot / k);
//   3. run bounds: the first and last sorted slot of every key;
//   4. key pass, one wavefront per key: for each of its queries, S_ij, A_ij,
//      w_ij from (Z_i, c_i) and dout_i . v_j (the query's dout row gathered
//      with 16-byte loads against the key's value row held in registers);
//      dv_j and dk_j accumulate in registers and are written once.
// deps is the fixed-order sum of the per-query parts.  Every sum runs in a
// fixed order, so all gradients are bit-reproducible.
//
// With the history-mean candidate (Section 3.4, last paragraph) each window
// also holds the pair (mean_k[i], mean_v[i]); the query pass treats it like
// any candidate for Z_i, c_i, dq_i and deps, and writes the gradients that
// reach mean_k[i] and mean_v[i], divided by the history's length.  A reverse
// scan then adds to every row j the sum of those over the queries whose
// history holds j (i >= j when causal, all i otherwise).
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

__global__ void __launch_bounds__(256) fill_u32_kernel(uint32_t* __restrict__ p, int64_t n, uint32_t val) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t t = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; t < n; t += stride) p[t] = val;
}

template <typename T, int DV, int DK>
__global__ void __launch_bounds__(kBwdWaves * 64)
    bwd_query_kernel(const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
                     const T* __restrict__ dout, const int32_t* __restrict__ idx, const int32_t* __restrict__ q_order,
                     int64_t total, int64_t N, int dk_rt, int topk, float eps, const float* __restrict__ mk,
                     const float* __restrict__ mv, int causal, float* __restrict__ dq,
                     float* __restrict__ deps_part, float2* __restrict__ zc, uint32_t* __restrict__ slot_keys,
                     float* __restrict__ hk, float* __restrict__ hv) {
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
      slot_keys[g * topk + c] = ok ? uint32_t(j) : uint32_t(N);
      zsum += s;
    }
    zsum = wave_sum(zsum);
    m = wave_max(m);
    float s_mean = 0.0f;  // the history-mean candidate's score
    if (mk != nullptr) {
      s_mean = mean_score<KD>(mk, g, dk_n, qv, eps);
      zsum += s_mean;
    }
    const float inv_z = zsum > 0.0f ? 1.0f / zsum : 0.0f;
    wave_lds_sync();

    // Phase 2: dout_i . v_j per pair (and dout_i . mean_v[i]).
    float du[kE];
    Vec16<T>::widen(*reinterpret_cast<const uint4*>(dout + g * DV + sub * kE), du);
    float dot_mean = 0.0f;
    if (mv != nullptr) {
      const float* mrow = mv + g * DV + sub * kE;
#pragma unroll
      for (int e = 0; e < kE; ++e) dot_mean = fmaf(du[e], mrow[e], dot_mean);
#pragma unroll
      for (int off = 1; off < kLpr; off <<= 1) dot_mean += __shfl_xor(dot_mean, off, 64);
    }
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
        if (c < m && sub == 0) s_g[c] = jj[u] >= 0 ? part : 0.0f;
      }
    }
    wave_lds_sync();

    // dout_i . o_i = sum_j A_ij (dout_i . v_j).
    float cdot = 0.0f;
    for (int c = lane; c < m; c += 64) cdot = fmaf(s_s[c], s_g[c], cdot);
    cdot = fmaf(s_mean, dot_mean, wave_sum(cdot)) * inv_z;

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
      for (int a = 0; a < KD; ++a)
        if (a < dk_n) dqa[a] = fmaf(w, qv[a] - kv[a], dqa[a]);
      wsum += w;
    }
#pragma unroll
    for (int a = 0; a < KD; ++a) dqa[a] = wave_sum(dqa[a]);
    wsum = wave_sum(wsum);
    if (mk != nullptr) {
      // The history-mean candidate's terms, and the gradients reaching
      // mean_k[i] and mean_v[i] divided by the history's length.
      const float w = (dot_mean - cdot) * s_mean * s_mean * inv_z;
      const float inv_cnt = 1.0f / float(causal ? i + 1 : N);
      float diff[KD];
#pragma unroll
      for (int a = 0; a < KD; ++a) {
        diff[a] = a < dk_n ? qv[a] - mk[g * dk_n + a] : 0.0f;
        dqa[a] = fmaf(w, diff[a], dqa[a]);
      }
      wsum += w;
      if (lane == 0) {
#pragma unroll
        for (int a = 0; a < KD; ++a)
          if (a < dk_n) hk[g * dk_n + a] = 2.0f * w * diff[a] * inv_cnt;
      }
      if (grp == 0) {
        const float am = s_mean * inv_z * inv_cnt;
        float hvv[kE];
#pragma unroll
        for (int e = 0; e < kE; ++e) hvv[e] = am * du[e];
#pragma unroll
        for (int e = 0; e < kE; e += 4)
          *reinterpret_cast<float4*>(hv + g * DV + sub * kE + e) =
              make_float4(hvv[e], hvv[e + 1], hvv[e + 2], hvv[e + 3]);
      }
    }
    if (lane == 0) {
#pragma unroll
      for (int a = 0; a < KD; ++a)
        if (a < dk_n) dq[g * dk_n + a] = -2.0f * dqa[a];
      deps_part[g] = -wsum;
      zc[g] = make_float2(zsum, cdot);
    }
    wave_lds_sync();
  }
}

// First and last sorted slot of every key that has one (others keep the
// cleared (0, 0)).  Sorted slot keys are N for empty window slots.
__global__ void __launch_bounds__(256)
    key_runs_kernel(const uint32_t* __restrict__ sorted_keys, int64_t S, int64_t M, int64_t N,
                    int2* __restrict__ runs) {
  const int64_t t = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= S * M) return;
  const int64_t seg = t / M;
  const int64_t e = t - seg * M;
  const uint32_t key = sorted_keys[t];
  if (key >= uint32_t(N)) return;
  int2* r = runs + seg * N + key;
  if (e == 0 || sorted_keys[t - 1] != key) r->x = int32_t(e);
  if (e == M - 1 || sorted_keys[t + 1] != key) r->y = int32_t(e + 1);
}

// One wavefront per key: dv_j and dk_j over the key's queries, in sorted
// (query, slot) order, 256 pairs at a time staged in LDS.
constexpr int kKeyChunk = 256;

template <typename T, int DV, int DK>
__global__ void __launch_bounds__(kBwdWaves * 64)
    bwd_key_kernel(const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
                   const T* __restrict__ dout, int64_t total, int64_t N, int dk_rt, int topk, float eps,
                   const int32_t* __restrict__ sorted_slot, const int2* __restrict__ runs,
                   const float2* __restrict__ zc, float* __restrict__ dkg, float* __restrict__ dvg) {
  constexpr int kE = Vec16<T>::kElems;
  constexpr int kLpr = DV / kE;
  constexpr int kGroups = 64 / kLpr;
  constexpr int kUnroll = 4;
  constexpr int KD = DK > 0 ? DK : kMaxDk;
  const int dk_n = DK > 0 ? DK : dk_rt;

  __shared__ int32_t s_i[kBwdWaves][kKeyChunk];    // query position
  __shared__ float s_a[kBwdWaves][kKeyChunk];      // A_ij
  __shared__ float s_w2[kBwdWaves][kKeyChunk];     // S_ij^2 / Z_i
  __shared__ float s_c[kBwdWaves][kKeyChunk];      // c_i
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int grp = lane / kLpr;
  const int sub = lane - grp * kLpr;
  const int64_t nb = gridDim.x;

  for (int64_t blk = xcd_contiguous_block(blockIdx.x, nb); blk * kBwdWaves < total; blk += nb) {
    const int64_t key = blk * kBwdWaves + wave;  // seg * N + j
    if (key >= total) continue;
    const int64_t seg = key / N;
    const int2 run = runs[key];
    const int32_t* sl = sorted_slot + seg * N * topk;

    float kv[KD];
    if constexpr (DK == 3) {
      Row3<T>::load(k, key, total, kv);
    } else {
#pragma unroll
      for (int a = 0; a < KD; ++a) kv[a] = a < dk_n ? Elem<T>::load(k + key * dk_n + a) : 0.0f;
    }
    float vj[kE];
    Vec16<T>::widen(*reinterpret_cast<const uint4*>(v + key * DV + sub * kE), vj);

    float dva[kE];
#pragma unroll
    for (int e = 0; e < kE; ++e) dva[e] = 0.0f;
    float dka[KD];
#pragma unroll
    for (int a = 0; a < KD; ++a) dka[a] = 0.0f;

    for (int32_t e0 = run.x; e0 < run.y; e0 += kKeyChunk) {
      const int n = run.y - e0 < kKeyChunk ? run.y - e0 : kKeyChunk;
      // Pairs of this chunk: query, weights, and (q_i - k_j) folded into dk later.
      for (int c = lane; c < n; c += 64) {
        const int32_t i = sl[e0 + c] / topk;
        const int64_t gi = seg * N + i;
        float qv[KD];
        if constexpr (DK == 3) {
          Row3<T>::load(q, gi, total, qv);
        } else {
#pragma unroll
          for (int a = 0; a < KD; ++a) qv[a] = a < dk_n ? Elem<T>::load(q + gi * dk_n + a) : 0.0f;
        }
        float d2 = 0.0f;
#pragma unroll
        for (int a = 0; a < KD; ++a) {
          if (a < dk_n) {
            const float diff = qv[a] - kv[a];
            d2 = fmaf(diff, diff, d2);
          }
        }
        const float s = 1.0f / (d2 + eps);
        const float2 z = zc[gi];
        const float inv_z = z.x > 0.0f ? 1.0f / z.x : 0.0f;
        s_i[wave][c] = i;
        s_a[wave][c] = s * inv_z;
        s_w2[wave][c] = s * s * inv_z;
        s_c[wave][c] = z.y;
      }
      wave_lds_sync();
      // dout_i . v_j and dv_j += A_ij dout_i, one query row per lane group.
      for (int c0 = grp; c0 < n; c0 += kUnroll * kGroups) {
        uint4 raw[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          const int c = c0 + u * kGroups;
          const int64_t gi = seg * N + (c < n ? s_i[wave][c] : 0);
          raw[u] = *reinterpret_cast<const uint4*>(dout + gi * DV + sub * kE);
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          const int c = c0 + u * kGroups;
          float f[kE];
          Vec16<T>::widen(raw[u], f);
          const float a = c < n ? s_a[wave][c] : 0.0f;
          float part = 0.0f;
#pragma unroll
          for (int e = 0; e < kE; ++e) {
            part = fmaf(f[e], vj[e], part);
            dva[e] = fmaf(a, f[e], dva[e]);
          }
#pragma unroll
          for (int off = 1; off < kLpr; off <<= 1) part += __shfl_xor(part, off, 64);
          // w_ij = (dout_i . v_j - c_i) S_ij^2 / Z_i, kept where the score was.
          if (c < n && sub == 0) s_w2[wave][c] = (part - s_c[wave][c]) * s_w2[wave][c];
        }
      }
      wave_lds_sync();
      // dk_j += 2 w_ij (q_i - k_j).
      for (int c = lane; c < n; c += 64) {
        const int64_t gi = seg * N + s_i[wave][c];
        float qv[KD];
        if constexpr (DK == 3) {
          Row3<T>::load(q, gi, total, qv);
        } else {
#pragma unroll
          for (int a = 0; a < KD; ++a) qv[a] = a < dk_n ? Elem<T>::load(q + gi * dk_n + a) : 0.0f;
        }
        const float w = s_w2[wave][c];
#pragma unroll
        for (int a = 0; a < KD; ++a)
          if (a < dk_n) dka[a] = fmaf(w, qv[a] - kv[a], dka[a]);
      }
      wave_lds_sync();
    }

    // Fold the lane groups of dv, the lanes of dk, and store.
#pragma unroll
    for (int off = kLpr; off < 64; off <<= 1)
#pragma unroll
      for (int e = 0; e < kE; ++e) dva[e] += __shfl_xor(dva[e], off, 64);
    if (grp == 0) {
      float* dst = dvg + key * DV + sub * kE;
#pragma unroll
      for (int e = 0; e < kE; ++e) dst[e] = dva[e];
    }
#pragma unroll
    for (int a = 0; a < KD; ++a) dka[a] = wave_sum(dka[a]);
    if (lane == 0) {
#pragma unroll
      for (int a = 0; a < KD; ++a)
        if (a < dk_n) dkg[key * dk_n + a] = 2.0f * dka[a];
    }
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
                        const int32_t* idx, const int32_t* q_order, float eps, HistMean hm, bool causal, float* dq,
                        float* dkg, float* dv, float* deps, const BwdWs& ws, char* wsb, hipStream_t stream) {
  const int64_t total = S * N;
  const int64_t M = N * topk;  // window slots per segment
  float* part = reinterpret_cast<float*>(wsb + ws.part_off);
  float* block_sums = reinterpret_cast<float*>(wsb + ws.block_off);
  float2* zc = reinterpret_cast<float2*>(wsb + ws.zc_off);
  uint32_t* slot_keys = reinterpret_cast<uint32_t*>(wsb + ws.keys_off);
  uint32_t* sorted_keys = reinterpret_cast<uint32_t*>(wsb + ws.sorted_off);
  int32_t* sorted_slot = reinterpret_cast<int32_t*>(wsb + ws.slot_off);
  int2* runs = reinterpret_cast<int2*>(wsb + ws.runs_off);
  float* hk = reinterpret_cast<float*>(wsb + ws.hist_k_off);
  float* hv = reinterpret_cast<float*>(wsb + ws.hist_v_off);
  const bool history = hm.k != nullptr;
  fill_zero(dq, total * dk, stream);
  if (history && q_order != nullptr) {  // rows absent from q_order pass nothing back
    fill_zero(hk, total * dk, stream);
    fill_zero(hv, total * DV, stream);
  }
  fill_zero(part, total, stream);
  fill_zero(reinterpret_cast<float*>(zc), total * 2, stream);
  fill_zero(reinterpret_cast<float*>(runs), total * 2, stream);
  // Slots of queries absent from q_order keep the "empty" key N.
  if (q_order != nullptr) {
    const int64_t want = ceil_div(S * M, 256);
    hipLaunchKernelGGL(fill_u32_kernel, dim3(unsigned(want < 65536 ? want : 65536)), dim3(256), 0, stream,
                       slot_keys, S * M, uint32_t(N));
  }
  {
    const int64_t want = ceil_div(total, kBwdWaves);
    const unsigned blocks = unsigned(want < (int64_t(1) << 20) ? want : (int64_t(1) << 20));
    const size_t lds = size_t(kBwdWaves) * topk * 12;
    if (dk == 3)
      hipLaunchKernelGGL((bwd_query_kernel<T, DV, 3>), dim3(blocks), dim3(kBwdWaves * 64), lds, stream, q, k, v,
                         dout, idx, q_order, total, N, dk, topk, eps, hm.k, hm.v, causal ? 1 : 0, dq, part, zc,
                         slot_keys, hk, hv);
    else
      hipLaunchKernelGGL((bwd_query_kernel<T, DV, 0>), dim3(blocks), dim3(kBwdWaves * 64), lds, stream, q, k, v,
                         dout, idx, q_order, total, N, dk, topk, eps, hm.k, hm.v, causal ? 1 : 0, dq, part, zc,
                         slot_keys, hk, hv);
  }
  hipError_t e = launch_sort(slot_keys, S, M, ws.key_bits, sorted_keys, sorted_slot, wsb + ws.sort_off, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(key_runs_kernel, dim3(unsigned(ceil_div(S * M, 256))), dim3(256), 0, stream, sorted_keys, S, M,
                     N, runs);
  {
    const int64_t want = ceil_div(total, kBwdWaves);
    const unsigned blocks = unsigned(want < (int64_t(1) << 20) ? want : (int64_t(1) << 20));
    if (dk == 3)
      hipLaunchKernelGGL((bwd_key_kernel<T, DV, 3>), dim3(blocks), dim3(kBwdWaves * 64), 0, stream, q, k, v, dout,
                         total, N, dk, topk, eps, sorted_slot, runs, zc, dkg, dv);
    else
      hipLaunchKernelGGL((bwd_key_kernel<T, DV, 0>), dim3(blocks), dim3(kBwdWaves * 64), 0, stream, q, k, v, dout,
                         total, N, dk, topk, eps, sorted_slot, runs, zc, dkg, dv);
  }
  if (history) {
    e = launch_history_spread(hv, dv, DV, hk, dkg, dk, S, N, causal, wsb + ws.hist_scan_off, stream);
    if (e != hipSuccess) return e;
  }
  const int nred = int(total < kRedBlocks ? total : kRedBlocks);
  hipLaunchKernelGGL(reduce_partials_kernel, dim3(unsigned(nred)), dim3(256), 0, stream, part, total, block_sums);
  hipLaunchKernelGGL(reduce_final_kernel, dim3(1), dim3(256), 0, stream, block_sums, nred, deps);
  return hipGetLastError();
}

template <typename T>
hipError_t launch_bwd_dv(const void* q, const void* k, const void* v, const void* dout, int64_t S, int64_t N, int dk,
                         int dv, int topk, const int32_t* idx, const int32_t* q_order, float eps, HistMean hm,
                         bool causal, float* dq, float* dkg, float* dvg, float* deps, const BwdWs& ws, char* wsb,
                         hipStream_t stream) {
  const T* qq = static_cast<const T*>(q);
  const T* kk = static_cast<const T*>(k);
  const T* vv = static_cast<const T*>(v);
  const T* dd = static_cast<const T*>(dout);
  switch (dv) {
    case 32:
      return launch_bwd_t<T, 32>(qq, kk, vv, dd, S, N, dk, topk, idx, q_order, eps, hm, causal, dq, dkg, dvg, deps,
                                  ws, wsb, stream);
    case 64:
      return launch_bwd_t<T, 64>(qq, kk, vv, dd, S, N, dk, topk, idx, q_order, eps, hm, causal, dq, dkg, dvg, deps,
                                  ws, wsb, stream);
    case 128:
      return launch_bwd_t<T, 128>(qq, kk, vv, dd, S, N, dk, topk, idx, q_order, eps, hm, causal, dq, dkg, dvg, deps,
                                  ws, wsb, stream);
    case 256:
      return launch_bwd_t<T, 256>(qq, kk, vv, dd, S, N, dk, topk, idx, q_order, eps, hm, causal, dq, dkg, dvg, deps,
                                  ws, wsb, stream);
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_attend_bwd(const void* q, const void* k, const void* v, const void* dout, bool is_bf16, int64_t S,
                             int64_t N, int dk, int dv, int topk, const int32_t* idx, const int32_t* q_order,
                             float eps, HistMean hm, bool causal, float* dq, float* dkg, float* dvg, float* deps,
                             void* workspace, hipStream_t stream) {
  const BwdWs ws = bwd_ws(S, N, topk, dk, dv, hm.k != nullptr);
  char* wsb = static_cast<char*>(workspace);
  if (is_bf16)
    return launch_bwd_dv<uint16_t>(q, k, v, dout, S, N, dk, dv, topk, idx, q_order, eps, hm, causal, dq, dkg, dvg,
                                   deps, ws, wsb, stream);
  return launch_bwd_dv<float>(q, k, v, dout, S, N, dk, dv, topk, idx, q_order, eps, hm, causal, dq, dkg, dvg, deps,
                              ws, wsb, stream);
}

}  // namespace zeta
