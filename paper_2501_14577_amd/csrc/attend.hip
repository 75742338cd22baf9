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
#include <stdlib.h>
#include <string.h>

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

// ---------------------------------------------------------------------------
// Tiled variant.  A workgroup takes a tile of consecutive queries of the
// processing order.  In the order that select produces (list level, then
// Z-order) consecutive queries draw on the same stretch of one sorted list,
// so a tile of 16 queries (2048 candidate slots at k = 128) names only a few
// hundred distinct value rows.  The workgroup
//   1. files every candidate's global row into an LDS hash table (open
//      addressing with compare-and-swap; the table has at least as many slots
//      as candidates, so every insertion finds a slot),
//   2. numbers the distinct rows with one block-wide scan,
//   3. stages the first `rmax` distinct value rows (and key rows, widened to
//      float32) in LDS with coalesced 16-byte loads,
//   4. lets each wavefront run its queries as in the per-query kernel, reading
//      staged rows from LDS and any others from global memory.
// The gather then moves a tile's union of rows instead of every candidate of
// every query.  Scores, weights and the float32 accumulation are the same
// operations as in the per-query kernel (their order may differ).
struct TiledLayout {
  int tileq;      // queries per tile
  int hash_log2;  // hash slots = 2^hash_log2 >= tileq * topk
  int rmax;       // value rows staged per tile
  size_t hkey, cidx, ref, uniq, kst, vst, wref, ww, gq, misc, bytes;
};

constexpr int kTiledThreads = 256;
constexpr size_t kTiledLdsBudget = 80 * 1024;  // two workgroups per CU

inline TiledLayout tiled_layout(int topk, int dk, int row_bytes) {
  TiledLayout L{};
  L.tileq = 2048 / topk;
  if (L.tileq > 16) L.tileq = 16;
  if (L.tileq < 1) L.tileq = 1;
  const int refs = L.tileq * topk;
  L.hash_log2 = 8;  // at least one slot per thread
  while ((1 << L.hash_log2) < refs) ++L.hash_log2;
  const size_t H = size_t(1) << L.hash_log2;
  size_t off = 0;
  auto take = [&off](size_t bytes) {
    const size_t at = off;
    off = (off + bytes + 15) / 16 * 16;
    return at;
  };
  L.hkey = take(H * 4);
  L.cidx = take(H * 2);
  L.ref = take(size_t(refs) * 2);
  L.wref = take(size_t(kAttWavesPerBlock) * topk * 4);
  L.ww = take(size_t(kAttWavesPerBlock) * topk * 4);
  L.gq = take(size_t(L.tileq) * 8);
  L.misc = take(64);
  const size_t fixed = off;
  const size_t per_row = size_t(row_bytes) + size_t(dk) * 4 + 4;
  L.rmax = fixed + 16 * per_row > kTiledLdsBudget ? 0 : int((kTiledLdsBudget - fixed - 64) / per_row);
  L.uniq = take(size_t(L.rmax) * 4);
  L.kst = take(size_t(L.rmax) * dk * 4);
  L.vst = take(size_t(L.rmax) * row_bytes);
  L.bytes = off;
  return L;
}

template <typename T, int DV, int DK>
__global__ void __launch_bounds__(kTiledThreads)
    attend_tiled_kernel(const T* __restrict__ q, const T* __restrict__ k, const T* __restrict__ v,
                        const int32_t* __restrict__ idx, const int32_t* __restrict__ q_order, int64_t total,
                        int64_t N, int dk_rt, int topk, float eps, T* __restrict__ out, TiledLayout L) {
  constexpr int kE = Vec16<T>::kElems;
  constexpr int kLpr = DV / kE;
  constexpr int kGroups = 64 / kLpr;
  constexpr int kUnroll = 8;
  constexpr int kRowBytes = DV * int(sizeof(T));
  constexpr uint16_t kNone = 0xFFFF;
  static_assert(kLpr >= 1 && kLpr <= 64 && 64 % kLpr == 0, "row must split evenly over lanes");
  const int dk = DK > 0 ? DK : dk_rt;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int grp = lane / kLpr;
  const int sub = lane - grp * kLpr;
  const int H = 1 << L.hash_log2;
  const int refs = L.tileq * topk;

  extern __shared__ unsigned char s_raw[];
  int32_t* s_hkey = reinterpret_cast<int32_t*>(s_raw + L.hkey);
  uint16_t* s_cidx = reinterpret_cast<uint16_t*>(s_raw + L.cidx);
  uint16_t* s_ref = reinterpret_cast<uint16_t*>(s_raw + L.ref);
  int32_t* s_uniq = reinterpret_cast<int32_t*>(s_raw + L.uniq);
  float* s_kst = reinterpret_cast<float*>(s_raw + L.kst);
  unsigned char* s_vst = s_raw + L.vst;
  int32_t* s_wref = reinterpret_cast<int32_t*>(s_raw + L.wref) + wave * topk;
  float* s_ww = reinterpret_cast<float*>(s_raw + L.ww) + wave * topk;
  int64_t* s_gq = reinterpret_cast<int64_t*>(s_raw + L.gq);
  uint32_t* s_misc = reinterpret_cast<uint32_t*>(s_raw + L.misc);

  const int64_t tiles = (total + L.tileq - 1) / L.tileq;
  const int64_t nb = gridDim.x;
  for (int64_t tile = xcd_contiguous_block(blockIdx.x, nb); tile < tiles; tile += nb) {
    const int64_t slot0 = tile * L.tileq;
    const int nq = int(total - slot0 < L.tileq ? total - slot0 : L.tileq);

    // 1. The tile's query rows; an empty hash table.
    for (int h = tid; h < H; h += kTiledThreads) s_hkey[h] = -1;
    if (tid < nq) {
      const int64_t slot = slot0 + tid;
      const int64_t seg = slot / N;
      int64_t i = slot - seg * N;
      if (q_order != nullptr) i = q_order[slot];
      s_gq[tid] = (i >= 0 && i < N) ? seg * N + i : int64_t(-1);
    }
    __syncthreads();

    // 2. File every candidate's global row (segment base + position).
    for (int r = tid; r < nq * topk; r += kTiledThreads) {
      const int qi = r / topk;
      const int64_t g = s_gq[qi];
      uint16_t slot = kNone;
      if (g >= 0) {
        const int32_t j = idx[g * topk + (r - qi * topk)];
        if (j >= 0 && j < N) {
          const int32_t key = int32_t(g - g % N + j);
          uint32_t h = (uint32_t(key) * 2654435769u) >> (32 - L.hash_log2);
          for (int probe = 0; probe < H; ++probe) {
            const int32_t old = atomicCAS(&s_hkey[h], -1, key);
            if (old == -1 || old == key) break;
            h = (h + 1) & uint32_t(H - 1);
          }
          slot = uint16_t(h);
        }
      }
      s_ref[r] = slot;
    }
    __syncthreads();

    // 3. Number the distinct rows in table order.
    {
      const int per = H / kTiledThreads;
      const int h0 = tid * per;
      uint32_t cnt = 0;
      for (int h = h0; h < h0 + per; ++h) cnt += s_hkey[h] >= 0 ? 1u : 0u;
      uint32_t ci = block256_exclusive_scan(cnt, s_misc);
      for (int h = h0; h < h0 + per; ++h) {
        const int32_t key = s_hkey[h];
        if (key >= 0) {
          s_cidx[h] = uint16_t(ci < uint32_t(L.rmax) ? ci : uint32_t(L.rmax));
          if (ci < uint32_t(L.rmax)) s_uniq[ci] = key;
          ++ci;
        }
      }
      if (tid == kTiledThreads - 1) s_misc[4] = ci;  // distinct rows in the tile
    }
    __syncthreads();

    // 4. Stage value rows (16-byte chunks) and key rows (float32).
    const int rows = int(s_misc[4] < uint32_t(L.rmax) ? s_misc[4] : uint32_t(L.rmax));
    for (int ch = tid; ch < rows * kLpr; ch += kTiledThreads) {
      const int row = ch / kLpr;
      const int part = ch - row * kLpr;
      *reinterpret_cast<uint4*>(s_vst + row * kRowBytes + part * 16) =
          *reinterpret_cast<const uint4*>(v + int64_t(s_uniq[row]) * DV + part * kE);
    }
    for (int row = tid; row < rows; row += kTiledThreads) {
      const T* kr = k + int64_t(s_uniq[row]) * dk;
      for (int a = 0; a < dk; ++a) s_kst[row * dk + a] = Elem<T>::load(kr + a);
    }
    __syncthreads();

    // 5. Each wavefront runs its queries.
    for (int qi = wave; qi < nq; qi += kAttWavesPerBlock) {
      const int64_t g = s_gq[qi];
      if (g < 0) continue;
      float qv[DK > 0 ? DK : kMaxDk];
#pragma unroll
      for (int a = 0; a < (DK > 0 ? DK : kMaxDk); ++a) qv[a] = a < dk ? Elem<T>::load(q + g * dk + a) : 0.0f;

      // Scores; staged candidates are listed from the front of the wave's
      // buffer (LDS row offsets), the others from the back (global rows).
      float zsum = 0.0f;
      int n_lds = 0, n_glb = 0;
      for (int c0 = 0; c0 < topk; c0 += 64) {
        const int c = c0 + lane;
        bool ok = false, staged = false;
        int32_t ref = 0;
        float s = 0.0f;
        if (c < topk) {
          const uint16_t h = s_ref[qi * topk + c];
          if (h != kNone) {
            ok = true;
            const int ci = s_cidx[h];
            staged = ci < L.rmax;
            const int32_t key = s_hkey[h];
            float d2 = 0.0f;
            if (staged) {
#pragma unroll
              for (int a = 0; a < (DK > 0 ? DK : kMaxDk); ++a)
                if (a < dk) {
                  const float diff = qv[a] - s_kst[ci * dk + a];
                  d2 += diff * diff;
                }
              ref = ci * kRowBytes;
            } else {
              const T* kr = k + int64_t(key) * dk;
#pragma unroll
              for (int a = 0; a < (DK > 0 ? DK : kMaxDk); ++a)
                if (a < dk) {
                  const float diff = qv[a] - Elem<T>::load(kr + a);
                  d2 += diff * diff;
                }
              ref = key;
            }
            s = 1.0f / (d2 + eps);
          }
        }
        const uint64_t b_lds = wave_ballot(ok && staged);
        const uint64_t b_glb = wave_ballot(ok && !staged);
        if (ok && staged) {
          const int at = n_lds + int(lanes_below(b_lds));
          s_wref[at] = ref;
          s_ww[at] = s;
        } else if (ok) {
          const int at = topk - 1 - (n_glb + int(lanes_below(b_glb)));
          s_wref[at] = ref;
          s_ww[at] = s;
        }
        n_lds += __popcll(b_lds);
        n_glb += __popcll(b_glb);
        zsum += s;
      }
      zsum = wave_sum(zsum);
      wave_lds_sync();

      float acc[kE];
#pragma unroll
      for (int e = 0; e < kE; ++e) acc[e] = 0.0f;
      const int lane_off = sub * 16;
      int c = grp;
      for (; c + (kUnroll - 1) * kGroups < n_lds; c += kUnroll * kGroups) {
        uint4 raw[kUnroll];
        float wv[kUnroll];
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          const int cc = c + u * kGroups;
          wv[u] = s_ww[cc];
          raw[u] = *reinterpret_cast<const uint4*>(s_vst + s_wref[cc] + lane_off);
        }
#pragma unroll
        for (int u = 0; u < kUnroll; ++u) {
          float f[kE];
          Vec16<T>::widen(raw[u], f);
#pragma unroll
          for (int e = 0; e < kE; ++e) acc[e] += wv[u] * f[e];
        }
      }
      for (; c < n_lds; c += kGroups) {
        float f[kE];
        const float w = s_ww[c];
        Vec16<T>::widen(*reinterpret_cast<const uint4*>(s_vst + s_wref[c] + lane_off), f);
#pragma unroll
        for (int e = 0; e < kE; ++e) acc[e] += w * f[e];
      }
      for (int cg = grp; cg < n_glb; cg += kGroups) {
        const int at = topk - 1 - cg;
        float f[kE];
        const float w = s_ww[at];
        Vec16<T>::widen(*reinterpret_cast<const uint4*>(v + int64_t(s_wref[at]) * DV + sub * kE), f);
#pragma unroll
        for (int e = 0; e < kE; ++e) acc[e] += w * f[e];
      }

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
    __syncthreads();
  }
}

template <typename T, int DV, int DK>
hipError_t launch_attend_tiled_t(const void* q, const void* k, const void* v, int64_t S, int64_t N, int dk,
                                 int topk, const int32_t* idx, const int32_t* q_order, float eps, void* out,
                                 const TiledLayout& L, hipStream_t stream) {
  const int64_t total = S * N;
  const int64_t tiles = ceil_div(total, L.tileq);
  const unsigned blocks = unsigned(tiles < (int64_t(1) << 20) ? tiles : (int64_t(1) << 20));
  auto kern = attend_tiled_kernel<T, DV, DK>;
  hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, int(L.bytes));
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(blocks), dim3(kTiledThreads), L.bytes, stream, static_cast<const T*>(q),
                     static_cast<const T*>(k), static_cast<const T*>(v), idx, q_order, total, N, dk, topk, eps,
                     static_cast<T*>(out), L);
  return hipGetLastError();
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

// The tiled kernel is used when its LDS plan stages a useful number of rows;
// ZETA_ATTEND=direct in the environment selects the per-query kernel.
inline bool want_tiled() {
  const char* e = getenv("ZETA_ATTEND");
  return !(e != nullptr && strcmp(e, "direct") == 0);
}

template <typename T, int DV>
hipError_t launch_attend_dk(const void* q, const void* k, const void* v, int64_t S, int64_t N, int dk,
                            int topk, const int32_t* idx, const int32_t* q_order, float eps, void* out,
                            hipStream_t stream) {
  const TiledLayout L = tiled_layout(topk, dk, DV * int(sizeof(T)));
  if (want_tiled() && L.rmax >= 32) {
    if (dk == 3)
      return launch_attend_tiled_t<T, DV, 3>(q, k, v, S, N, dk, topk, idx, q_order, eps, out, L, stream);
    return launch_attend_tiled_t<T, DV, 0>(q, k, v, S, N, dk, topk, idx, q_order, eps, out, L, stream);
  }
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
