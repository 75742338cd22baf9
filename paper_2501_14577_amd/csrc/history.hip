// The history-mean candidate (Section 3.4, last paragraph): the mean key and
// the mean value of each query's history, obtained from cumulative sums,
// which the attention calls can add to every window as one more candidate.
// Causal: row i holds the mean of rows 0..i; otherwise every row holds the
// mean of all N rows.  The gradients that reach those means go back to the
// history's rows through the reverse sums (suffix sums).
//
// Both directions are a segmented scan over [S][N][D] matrices (the values
// and the keys together, so each kernel is launched once), in three kernels:
//   1. chunk sums: a group of G lanes (VEC columns each, G * VEC = D) walks
//      one chunk of kHistRows consecutive rows and writes its column sums;
//   2. chunk offsets: one wavefront per (segment, column) turns the chunk
//      sums into exclusive prefix sums (or suffix sums): each lane scans a
//      run of consecutive chunks, one lane scan joins the runs, and the
//      segment's total is written;
//   3. apply: each lane group walks its chunk again in scan order from the
//      chunk's offset.  Forward it writes the running mean (sum times the
//      reciprocal of the count) in float32; backward it adds the running
//      suffix sum into the gradient.
// Rows are read with 16-byte lane loads where the row allows it.  Every sum
// runs in a fixed order, so results are bit-reproducible.  The matrices are
// HBM-bound streams: each pass reads the input once (twice in all) and the
// forward writes the means once.
#include "attend_device.h"
#include "device_common.h"
#include "kernels.h"
#include "layout.h"

namespace zeta {
namespace {

constexpr int kHistWaves = 4;
constexpr int kOffBatch = 16;  // chunk sums loaded per lane before they are scanned

// VEC consecutive elements of a row: one load into a raw register value,
// widened to float32 where it is used.
template <typename T, int VEC>
struct RowVec;

template <typename T>
struct RowVec<T, 1> {
  using Raw = float;
  __device__ __forceinline__ static Raw raw(const T* p) { return Elem<T>::load(p); }
  __device__ __forceinline__ static void widen(Raw x, float* f) { f[0] = x; }
  __device__ __forceinline__ static void load(const T* p, float* f) { f[0] = Elem<T>::load(p); }
};

template <typename T, int VEC>
struct RowVec16 {
  using Raw = uint4;
  __device__ __forceinline__ static Raw raw(const T* p) { return *reinterpret_cast<const uint4*>(p); }
  __device__ __forceinline__ static void widen(const Raw& x, float* f) { Vec16<T>::widen(x, f); }
  __device__ __forceinline__ static void load(const T* p, float* f) { Vec16<T>::widen(raw(p), f); }
};

template <>
struct RowVec<float, 4> : RowVec16<float, 4> {};

template <>
struct RowVec<uint16_t, 8> : RowVec16<uint16_t, 8> {};

// Rows of a chunk loaded per batch (16-byte raw values kept in registers).
constexpr int kRowBatch = 16;

template <int VEC>
__device__ __forceinline__ void store_f32(float* p, const float* f) {
  if constexpr (VEC % 4 == 0) {
#pragma unroll
    for (int e = 0; e < VEC; e += 4)
      *reinterpret_cast<float4*>(p + e) = make_float4(f[e], f[e + 1], f[e + 2], f[e + 3]);
  } else {
#pragma unroll
    for (int e = 0; e < VEC; ++e) p[e] = f[e];
  }
}

// One matrix of a scan: S segments of N rows of D elements of T, VEC
// columns per lane; float32 output rows; chunk sums [S][D][nch] (turned into
// offsets in place; each column's chunks contiguous, for the offsets scan)
// and segment totals [S][D] in the workspace.
template <typename T, int VEC>
struct ScanMat {
  using ElemT = T;
  static constexpr int kVec = VEC;
  const T* x;
  float* out;
  int D;
  int64_t wave_tasks;
  float* sums;
  float* totals;
};

// The chunk and column group of a lane: chunks are taken 64 / G per
// wavefront; lanes past the last whole group idle (chunk -1).
struct ChunkLane {
  int64_t chunk;  // segment * nch + chunk index
  int col;        // first column
};

__device__ __forceinline__ ChunkLane chunk_lane(int64_t wave_task, int lane, int G, int VEC, int64_t chunks) {
  const int cpw = 64 / G;
  const int cl = lane / G;
  ChunkLane r;
  r.col = (lane - cl * G) * VEC;
  r.chunk = wave_task * cpw + cl;
  if (cl >= cpw || r.chunk >= chunks) r.chunk = -1;
  return r;
}

template <class M>
__device__ __forceinline__ void chunk_sums_task(const M& m, int64_t t, int lane, int64_t N, int64_t nch,
                                                int64_t chunks) {
  constexpr int VEC = M::kVec;
  const ChunkLane cl = chunk_lane(t, lane, m.D / VEC, VEC, chunks);
  if (cl.chunk < 0) return;
  const int64_t seg = cl.chunk / nch;
  const int64_t r0 = (cl.chunk - seg * nch) * kHistRows;
  const int64_t r1 = r0 + kHistRows < N ? r0 + kHistRows : N;
  const typename M::ElemT* p = m.x + (seg * N) * m.D + cl.col;
  float acc[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) acc[e] = 0.0f;
  // kRowBatch rows in flight at once (rows past the segment's end re-read
  // its last row and add nothing).
  using RV = RowVec<typename M::ElemT, VEC>;
  for (int b = 0; b < kHistRows; b += kRowBatch) {
    typename RV::Raw x[kRowBatch];
#pragma unroll
    for (int u = 0; u < kRowBatch; ++u) {
      const int64_t r = r0 + b + u < r1 ? r0 + b + u : r1 - 1;
      x[u] = RV::raw(p + r * m.D);
    }
#pragma unroll
    for (int u = 0; u < kRowBatch; ++u) {
      float f[VEC];
      RV::widen(x[u], f);
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[e] += r0 + b + u < r1 ? f[e] : 0.0f;
    }
  }
  const int64_t c = cl.chunk - seg * nch;
#pragma unroll
  for (int e = 0; e < VEC; ++e) m.sums[(seg * m.D + cl.col + e) * nch + c] = acc[e];
}

template <class MA, class MB>
__global__ void __launch_bounds__(kHistWaves * 64)
    hist_chunk_sums_kernel(MA a, MB b, int64_t N, int64_t nch, int64_t chunks) {
  const int lane = threadIdx.x & 63;
  const int64_t tasks = a.wave_tasks + b.wave_tasks;
  for (int64_t t = int64_t(blockIdx.x) * kHistWaves + (threadIdx.x >> 6); t < tasks;
       t += int64_t(gridDim.x) * kHistWaves) {
    if (t < a.wave_tasks)
      chunk_sums_task(a, t, lane, N, nch, chunks);
    else
      chunk_sums_task(b, t - a.wave_tasks, lane, N, nch, chunks);
  }
}

// One wavefront per (matrix, segment, column): exclusive prefix sums of the
// chunk sums (suffix sums when `reverse`), in place, and the segment total.
__global__ void __launch_bounds__(kHistWaves * 64)
    hist_chunk_offsets_kernel(float* __restrict__ sums_a, float* __restrict__ totals_a, int Da,
                              float* __restrict__ sums_b, float* __restrict__ totals_b, int Db, int64_t S,
                              int64_t nch, int reverse) {
  const int lane = threadIdx.x & 63;
  const int64_t tasks = S * (Da + Db);
  for (int64_t t = int64_t(blockIdx.x) * kHistWaves + (threadIdx.x >> 6); t < tasks;
       t += int64_t(gridDim.x) * kHistWaves) {
    const bool in_a = t < S * Da;
    const int D = in_a ? Da : Db;
    const int64_t tt = in_a ? t : t - S * Da;
    float* sums = in_a ? sums_a : sums_b;
    float* totals = in_a ? totals_a : totals_b;
    const int64_t seg = tt / D;
    const int col = int(tt - seg * D);
    // Lane l scans scan positions b0 + l*kOffBatch .. + kOffBatch - 1 in
    // order; one lane scan of the lanes' totals joins them.
    float carry = 0.0f;
    for (int64_t b0 = 0; b0 < nch; b0 += 64 * kOffBatch) {
      float xs[kOffBatch];
#pragma unroll
      for (int u = 0; u < kOffBatch; ++u) {
        const int64_t n = b0 + int64_t(lane) * kOffBatch + u;  // scan position
        const int64_t c = reverse ? nch - 1 - n : n;
        xs[u] = n < nch ? sums[(seg * D + col) * nch + c] : 0.0f;
      }
      float run = 0.0f;
#pragma unroll
      for (int u = 0; u < kOffBatch; ++u) {
        const float x = xs[u];
        xs[u] = run;  // exclusive within the lane
        run += x;
      }
      float incl = run;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const float y = __shfl_up(incl, off, 64);
        if (lane >= off) incl += y;
      }
      float excl = __shfl_up(incl, 1, 64);
      if (lane == 0) excl = 0.0f;
      const float base = carry + excl;
#pragma unroll
      for (int u = 0; u < kOffBatch; ++u) {
        const int64_t n = b0 + int64_t(lane) * kOffBatch + u;
        if (n < nch) sums[(seg * D + col) * nch + (reverse ? nch - 1 - n : n)] = base + xs[u];
      }
      carry += __shfl(incl, 63, 64);
    }
    if (lane == 0) totals[seg * D + col] = carry;
  }
}

// Forward: running means of a chunk's rows from the chunk's offset, or the
// segment mean in every row when not causal.
template <class M>
__device__ __forceinline__ void mean_task(const M& m, int64_t t, int lane, int64_t N, int64_t nch, int64_t chunks,
                                          int causal) {
  constexpr int VEC = M::kVec;
  const ChunkLane cl = chunk_lane(t, lane, m.D / VEC, VEC, chunks);
  if (cl.chunk < 0) return;
  const int64_t seg = cl.chunk / nch;
  const int64_t r0 = (cl.chunk - seg * nch) * kHistRows;
  const int64_t r1 = r0 + kHistRows < N ? r0 + kHistRows : N;
  const typename M::ElemT* p = m.x + (seg * N) * m.D + cl.col;
  float* o = m.out + (seg * N) * m.D + cl.col;
  if (!causal) {
    float mm[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) mm[e] = m.totals[seg * m.D + cl.col + e] / float(N);
    for (int64_t r = r0; r < r1; ++r) store_f32<VEC>(o + r * m.D, mm);
    return;
  }
  float acc[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) acc[e] = m.sums[(seg * m.D + cl.col + e) * nch + (cl.chunk - seg * nch)];
  using RV = RowVec<typename M::ElemT, VEC>;
  for (int b = 0; b < kHistRows; b += kRowBatch) {
    typename RV::Raw x[kRowBatch];
#pragma unroll
    for (int u = 0; u < kRowBatch; ++u) {
      const int64_t r = r0 + b + u < r1 ? r0 + b + u : r1 - 1;
      x[u] = RV::raw(p + r * m.D);
    }
#pragma unroll
    for (int u = 0; u < kRowBatch; ++u) {
      const int64_t r = r0 + b + u;
      if (r >= r1) break;
      float f[VEC];
      RV::widen(x[u], f);
      const float inv_cnt = 1.0f / float(r + 1);
      float mm[VEC];
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        acc[e] += f[e];
        mm[e] = acc[e] * inv_cnt;
      }
      store_f32<VEC>(o + r * m.D, mm);
    }
  }
}

template <class MA, class MB>
__global__ void __launch_bounds__(kHistWaves * 64)
    hist_mean_kernel(MA a, MB b, int64_t N, int64_t nch, int64_t chunks, int causal) {
  const int lane = threadIdx.x & 63;
  const int64_t tasks = a.wave_tasks + b.wave_tasks;
  for (int64_t t = int64_t(blockIdx.x) * kHistWaves + (threadIdx.x >> 6); t < tasks;
       t += int64_t(gridDim.x) * kHistWaves) {
    if (t < a.wave_tasks)
      mean_task(a, t, lane, N, nch, chunks, causal);
    else
      mean_task(b, t - a.wave_tasks, lane, N, nch, chunks, causal);
  }
}

// Backward: out[j] += the sum of x[i] over i >= j within the segment (each
// chunk walked from its last row, starting at the sum of the later chunks),
// or the segment total in every row when not causal.
template <class M>
__device__ __forceinline__ void spread_task(const M& m, int64_t t, int lane, int64_t N, int64_t nch,
                                            int64_t chunks, int causal) {
  constexpr int VEC = M::kVec;
  const ChunkLane cl = chunk_lane(t, lane, m.D / VEC, VEC, chunks);
  if (cl.chunk < 0) return;
  const int64_t seg = cl.chunk / nch;
  const int64_t r0 = (cl.chunk - seg * nch) * kHistRows;
  const int64_t r1 = r0 + kHistRows < N ? r0 + kHistRows : N;
  const float* p = m.x + (seg * N) * m.D + cl.col;
  float* o = m.out + (seg * N) * m.D + cl.col;
  if (!causal) {
    float tv[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) tv[e] = m.totals[seg * m.D + cl.col + e];
    for (int64_t r = r0; r < r1; ++r) {
      float f[VEC];
      RowVec<float, VEC>::load(o + r * m.D, f);
#pragma unroll
      for (int e = 0; e < VEC; ++e) f[e] += tv[e];
      store_f32<VEC>(o + r * m.D, f);
    }
    return;
  }
  float acc[VEC];
#pragma unroll
  for (int e = 0; e < VEC; ++e) acc[e] = m.sums[(seg * m.D + cl.col + e) * nch + (cl.chunk - seg * nch)];
#pragma unroll 8
  for (int64_t r = r1 - 1; r >= r0; --r) {
    float f[VEC], g[VEC];
    RowVec<float, VEC>::load(p + r * m.D, f);
    RowVec<float, VEC>::load(o + r * m.D, g);
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      acc[e] += f[e];
      g[e] += acc[e];
    }
    store_f32<VEC>(o + r * m.D, g);
  }
}

template <class MA, class MB>
__global__ void __launch_bounds__(kHistWaves * 64)
    hist_spread_kernel(MA a, MB b, int64_t N, int64_t nch, int64_t chunks, int causal) {
  const int lane = threadIdx.x & 63;
  const int64_t tasks = a.wave_tasks + b.wave_tasks;
  for (int64_t t = int64_t(blockIdx.x) * kHistWaves + (threadIdx.x >> 6); t < tasks;
       t += int64_t(gridDim.x) * kHistWaves) {
    if (t < a.wave_tasks)
      spread_task(a, t, lane, N, nch, chunks, causal);
    else
      spread_task(b, t - a.wave_tasks, lane, N, nch, chunks, causal);
  }
}

unsigned grid_for(int64_t wave_tasks) {
  const int64_t want = ceil_div(wave_tasks, kHistWaves);
  return unsigned(want < 1 ? 1 : (want < (int64_t(1) << 20) ? want : (int64_t(1) << 20)));
}

// The two matrices' places in the workspace and their wave counts.
template <class MA, class MB>
void place(MA& a, MB& b, int64_t S, int64_t N, char* wsb) {
  const HistWs hw = hist_ws(S, N, a.D + b.D);
  const int64_t nch = ceil_div(N, kHistRows);
  float* sums = reinterpret_cast<float*>(wsb + hw.sums_off);
  float* totals = reinterpret_cast<float*>(wsb + hw.totals_off);
  a.sums = sums;
  b.sums = sums + S * nch * a.D;
  a.totals = totals;
  b.totals = totals + S * a.D;
  a.wave_tasks = ceil_div(S * nch, 64 / (a.D / MA::kVec));
  b.wave_tasks = ceil_div(S * nch, 64 / (b.D / MB::kVec));
}

template <class MA, class MB>
hipError_t mean_t(MA a, MB b, int64_t S, int64_t N, bool causal, char* wsb, hipStream_t stream) {
  place(a, b, S, N, wsb);
  const int64_t nch = ceil_div(N, kHistRows);
  const unsigned blocks = grid_for(a.wave_tasks + b.wave_tasks);
  hipLaunchKernelGGL((hist_chunk_sums_kernel<MA, MB>), dim3(blocks), dim3(kHistWaves * 64), 0, stream, a, b, N, nch,
                     S * nch);
  hipLaunchKernelGGL(hist_chunk_offsets_kernel, dim3(grid_for(S * (a.D + b.D))), dim3(kHistWaves * 64), 0, stream,
                     a.sums, a.totals, a.D, b.sums, b.totals, b.D, S, nch, 0);
  hipLaunchKernelGGL((hist_mean_kernel<MA, MB>), dim3(blocks), dim3(kHistWaves * 64), 0, stream, a, b, N, nch,
                     S * nch, causal ? 1 : 0);
  return hipGetLastError();
}

template <class MA, class MB>
hipError_t spread_t(MA a, MB b, int64_t S, int64_t N, bool causal, char* wsb, hipStream_t stream) {
  place(a, b, S, N, wsb);
  const int64_t nch = ceil_div(N, kHistRows);
  const unsigned blocks = grid_for(a.wave_tasks + b.wave_tasks);
  hipLaunchKernelGGL((hist_chunk_sums_kernel<MA, MB>), dim3(blocks), dim3(kHistWaves * 64), 0, stream, a, b, N, nch,
                     S * nch);
  hipLaunchKernelGGL(hist_chunk_offsets_kernel, dim3(grid_for(S * (a.D + b.D))), dim3(kHistWaves * 64), 0, stream,
                     a.sums, a.totals, a.D, b.sums, b.totals, b.D, S, nch, 1);
  hipLaunchKernelGGL((hist_spread_kernel<MA, MB>), dim3(blocks), dim3(kHistWaves * 64), 0, stream, a, b, N, nch,
                     S * nch, causal ? 1 : 0);
  return hipGetLastError();
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// 16-byte lane loads when the rows and pointers allow it (and the row fits
// 64 lanes), else one element per lane (D <= 64).
template <typename T>
int vec_for(const void* x, const float* out, int D) {
  constexpr int kV = 16 / int(sizeof(T));
  if (D % kV == 0 && D / kV <= 64 && aligned16(x) && aligned16(out)) return kV;
  return D <= 64 ? 1 : 0;
}

template <typename T>
hipError_t mean_typed(const T* k, const T* v, int64_t S, int64_t N, int dk, int dv, bool causal, float* mk,
                      float* mv, char* wsb, hipStream_t stream) {
  constexpr int kV = 16 / int(sizeof(T));
  const int va = vec_for<T>(v, mv, dv), vb = vec_for<T>(k, mk, dk);
  if (va == 0 || vb == 0) return hipErrorInvalidValue;
  ScanMat<T, kV> av{v, mv, dv, 0, nullptr, nullptr};
  ScanMat<T, 1> a1{v, mv, dv, 0, nullptr, nullptr};
  ScanMat<T, kV> bv{k, mk, dk, 0, nullptr, nullptr};
  ScanMat<T, 1> b1{k, mk, dk, 0, nullptr, nullptr};
  if (va == kV) {
    if (vb == kV) return mean_t(av, bv, S, N, causal, wsb, stream);
    return mean_t(av, b1, S, N, causal, wsb, stream);
  }
  if (vb == kV) return mean_t(a1, bv, S, N, causal, wsb, stream);
  return mean_t(a1, b1, S, N, causal, wsb, stream);
}

}  // namespace

hipError_t launch_history_mean(const void* k, const void* v, bool is_bf16, int64_t S, int64_t N, int dk, int dv,
                               bool causal, float* mean_k, float* mean_v, void* workspace, hipStream_t stream) {
  char* wsb = static_cast<char*>(workspace);
  if (is_bf16)
    return mean_typed(static_cast<const uint16_t*>(k), static_cast<const uint16_t*>(v), S, N, dk, dv, causal, mean_k,
                      mean_v, wsb, stream);
  return mean_typed(static_cast<const float*>(k), static_cast<const float*>(v), S, N, dk, dv, causal, mean_k, mean_v,
                    wsb, stream);
}

hipError_t launch_history_spread(const float* xa, float* outa, int Da, const float* xb, float* outb, int Db, int64_t S,
                                 int64_t N, bool causal, void* workspace, hipStream_t stream) {
  char* wsb = static_cast<char*>(workspace);
  const int va = vec_for<float>(xa, outa, Da), vb = vec_for<float>(xb, outb, Db);
  if (va == 0 || vb == 0) return hipErrorInvalidValue;
  ScanMat<float, 4> a4{xa, outa, Da, 0, nullptr, nullptr};
  ScanMat<float, 1> a1{xa, outa, Da, 0, nullptr, nullptr};
  ScanMat<float, 4> b4{xb, outb, Db, 0, nullptr, nullptr};
  ScanMat<float, 1> b1{xb, outb, Db, 0, nullptr, nullptr};
  if (va == 4) {
    if (vb == 4) return spread_t(a4, b4, S, N, causal, wsb, stream);
    return spread_t(a4, b1, S, N, causal, wsb, stream);
  }
  if (vb == 4) return spread_t(a1, b4, S, N, causal, wsb, stream);
  return spread_t(a1, b1, S, N, causal, wsb, stream);
}

}  // namespace zeta
