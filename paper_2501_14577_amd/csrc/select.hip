// Candidate window of every query (Section 3.2.2: binary search for the
// query's insertion point among the sorted keys it may see, then a window of
// k keys centred there; Algorithm 1, Steps 3-5).
//
// Causal pools {0..i} differ per query, so the window cannot be cut from the
// full sorted list directly.  Instead of the paper's fixed chunks (which pick
// a different, coarser pool), the keys are re-filed into doubling prefix
// lists: F_t holds the keys at positions < 2^t in (code, position) order, for
// 2^t0 >= k and 2^t < N.  Query i searches F_t with t = max(t0, bitlen(i))
// (or the full list when no such level exists).  That list holds the whole
// pool, in pool order, and at least half of its entries are in the pool, so
// the wavefront that serves the query skips at most as many entries as it
// keeps.  Filtering F_t by position <= i gives exactly the pool's order, so
// the result is the definition's, not an approximation of it.
//
// Kernels:
//   list_count:   per tile of the sorted list, how many keys fall in each F_t;
//   list_scatter: stable compaction of each tile into every F_t it feeds
//                 (one ballot per level and 64 keys; earlier tiles' counts
//                 give the base);
// The windows themselves are found by the one-pass call's kernels (tile.hip):
// window_bounds gives each query's list-index bounds, and idx_rows writes the
// rows from them.
//
// query_order (the zeta_query_order entry point) regroups a processing order,
// typically the Z-order of the query codes, by the list each query searches,
// keeping the given order inside each group (one stable radix pass on the
// level).  A run of that order searches one list with non-decreasing codes, so
// the window-bounds kernel stages one stretch of the list for 64 queries and
// attend's tiles share value rows the same way.
#include <stdint.h>

#include "attend_device.h"
#include "device_common.h"
#include "kernels.h"
#include "layout.h"
#include "select_device.h"

namespace zeta {
namespace {


__global__ void __launch_bounds__(kSortThreads)
    list_count_kernel(const int32_t* __restrict__ perm, int64_t N, int64_t tiles, int t0, int levels,
                      uint32_t* __restrict__ cnt) {
  // Tiles of one segment run under one L2 (see xcd_contiguous_block).
  const int64_t blk = xcd_contiguous_block(blockIdx.x, gridDim.x);
  const int64_t seg = blk / tiles;
  const int64_t tile = blk % tiles;
  const int tid = threadIdx.x;
  __shared__ uint32_t h[kMaxLevels + 1];  // keys per bit length of their position
  if (tid <= kMaxLevels) h[tid] = 0;
  __syncthreads();
  const int64_t e0 = tile * kSortTile;
  const int64_t e1 = (e0 + kSortTile < N) ? e0 + kSortTile : N;
  const int32_t* ps = perm + seg * N;
  for (int64_t e = e0 + tid; e < e1; e += kSortThreads) atomicAdd(&h[bit_length(uint32_t(ps[e]))], 1u);
  __syncthreads();
  if (tid < levels) {
    // Keys with position < 2^t are those whose bit length is <= t.
    const int t = t0 + tid;
    uint32_t c = 0;
    for (int b = 0; b <= t; ++b) c += h[b];
    cnt[(seg * tiles + tile) * kMaxLevels + tid] = c;
  }
}

__global__ void __launch_bounds__(kSortThreads)
    list_scatter_kernel(const uint32_t* __restrict__ sorted_codes, const int32_t* __restrict__ perm,
                        int64_t N, int64_t tiles, int t0, int levels, int64_t cap,
                        const uint32_t* __restrict__ cnt, uint32_t* __restrict__ list_codes,
                        int32_t* __restrict__ list_pos, const uint16_t* __restrict__ k_rows,
                        uint2* __restrict__ keys_full, uint2* __restrict__ keys_list) {
  // Tiles of one segment run under one L2: its key rows, gathered by
  // position, and the list lines several tiles write then stay there.
  const int64_t blk = xcd_contiguous_block(blockIdx.x, gridDim.x);
  const int64_t seg = blk / tiles;
  const int64_t tile = blk % tiles;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  constexpr int kGroups = kSortThreads / kMaxLevels;
  __shared__ uint32_t s_before[kGroups][kMaxLevels];           // entries of earlier tiles, by tile group
  __shared__ uint32_t s_wave[kSortThreads / 64][kMaxLevels];  // per-wave counts, then prefixes

  {
    // Entries of the earlier tiles per level: thread (g, l) sums the tiles
    // t < tile with t % kGroups == g.
    const int l = tid % kMaxLevels, g = tid / kMaxLevels;
    uint32_t b = 0;
    if (l < levels) {
      // Independent loads in batches, so their latencies overlap.
      constexpr int kBatch = 4;
      const uint32_t* c = cnt + seg * tiles * kMaxLevels + l;
      for (int64_t t = g; t < tile; t += kBatch * kGroups) {
        uint32_t x[kBatch];
#pragma unroll
        for (int j = 0; j < kBatch; ++j) x[j] = t + j * kGroups < tile ? c[(t + j * kGroups) * kMaxLevels] : 0u;
#pragma unroll
        for (int j = 0; j < kBatch; ++j) b += x[j];
      }
    }
    s_before[g][l] = b;
  }
  const int64_t seg_off = seg * N;
  const int64_t first = tile * kSortTile + int64_t(wave) * (kSortChunks * 64);
  uint32_t code[kSortChunks];
  int32_t pos[kSortChunks];
  uint2 krow[kSortChunks];  // with k_rows: the entry's key row, written to every list it joins
#pragma unroll
  for (int c = 0; c < kSortChunks; ++c) {
    const int64_t e = first + c * 64 + lane;
    const bool valid = e < N;
    code[c] = valid ? sorted_codes[seg_off + e] : 0u;
    pos[c] = valid ? perm[seg_off + e] : 0x7FFFFFFF;  // never below any 2^t
    krow[c] = make_uint2(0u, 0u);
  }
  if (k_rows != nullptr) {
    // Each entry's key row (three bfloat16 values) gathered by position: three
    // 16-bit loads per entry, always in bounds and without a branch, so the
    // entries' gathers are in flight together; then packed as x | y << 16, z.
    uint32_t kx[kSortChunks], ky[kSortChunks], kz[kSortChunks];
#pragma unroll
    for (int c = 0; c < kSortChunks; ++c) {
      const int64_t r = (first + c * 64 + lane < N ? seg_off + pos[c] : 0) * 3;
      kx[c] = k_rows[r];
      ky[c] = k_rows[r + 1];
      kz[c] = k_rows[r + 2];
    }
#pragma unroll
    for (int c = 0; c < kSortChunks; ++c) {
      const int64_t e = first + c * 64 + lane;
      krow[c] = make_uint2(kx[c] | (ky[c] << 16), kz[c]);
      if (e < N) keys_full[seg_off + e] = krow[c];
    }
  }
  for (int l = 0; l < levels; ++l) {
    const int32_t lim = int32_t(1) << (t0 + l);
    uint32_t n = 0;
#pragma unroll
    for (int c = 0; c < kSortChunks; ++c) n += uint32_t(__popcll(wave_ballot(pos[c] < lim)));
    if (lane == 0) s_wave[wave][l] = n;
  }
  __syncthreads();
  if (tid < levels) {
    uint32_t run = 0;
#pragma unroll
    for (int g = 0; g < kGroups; ++g) run += s_before[g][tid];
#pragma unroll
    for (int w = 0; w < kSortThreads / 64; ++w) {
      const uint32_t t = s_wave[w][tid];
      s_wave[w][tid] = run;
      run += t;
    }
  }
  __syncthreads();
  uint32_t* lc = list_codes + seg * cap;
  int32_t* lp = list_pos + seg * cap;
  for (int l = 0; l < levels; ++l) {
    const int t = t0 + l;
    const int32_t lim = int32_t(1) << t;
    const int64_t list_off = (int64_t(1) << t) - (int64_t(1) << t0);
    uint32_t run = s_wave[wave][l];
#pragma unroll
    for (int c = 0; c < kSortChunks; ++c) {
      const bool in = pos[c] < lim;
      const uint64_t bal = wave_ballot(in);
      if (in) {
        const int64_t dst = list_off + run + lanes_below(bal);
        lc[dst] = code[c];
        lp[dst] = pos[c];
        if (k_rows != nullptr) keys_list[seg * cap + dst] = krow[c];
      }
      run += uint32_t(__popcll(bal));
    }
  }
}

// order_out[slot] = q_order[slot], or the slot's position when q_order is NULL.
__global__ void __launch_bounds__(256)
    copy_order_kernel(const int32_t* __restrict__ q_order, int64_t total, int64_t N, int32_t* __restrict__ order_out) {
  const int64_t slot = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (slot >= total) return;
  order_out[slot] = q_order != nullptr ? q_order[slot] : int32_t(slot % N);
}


}  // namespace

hipError_t launch_query_order(const int32_t* q_order, int64_t S, int64_t N, int topk, bool causal, int chunk,
                              int32_t* order_out, void* workspace, hipStream_t stream) {
  const ListPlan lp = list_plan(N, topk);
  const int64_t total = S * N;
  const unsigned blocks = unsigned(ceil_div(total, 256));
  if (!causal || lp.levels == 0) {
    // One list for every query: the given order (or position order) as is.
    hipLaunchKernelGGL(copy_order_kernel, dim3(blocks), dim3(256), 0, stream, q_order, total, N, order_out);
    return hipGetLastError();
  }
  const QueryOrderWs ws = query_order_ws(S, N);
  char* wsb = static_cast<char*>(workspace);
  uint32_t* phist = reinterpret_cast<uint32_t*>(wsb + ws.phist_off);
  const int32_t* given = q_order;
  if (q_order != nullptr && q_order == order_out) {
    // In place: partition from a copy.
    int32_t* copy = reinterpret_cast<int32_t*>(wsb + ws.given_off);
    hipLaunchKernelGGL(copy_order_kernel, dim3(blocks), dim3(256), 0, stream, q_order, total, N, copy);
    given = copy;
  }
  return launch_level_partition(given, S, N, lp.t0, lp.t_hi, lp.levels, chunk, order_out, phist, stream);
}

hipError_t launch_prefix_lists(const uint32_t* sorted_codes, const int32_t* perm, int64_t S, int64_t N, int topk,
                               void* workspace, hipStream_t stream, const uint32_t** list_codes,
                               const int32_t** list_pos, const uint16_t* k_rows, uint2* keys_full,
                               uint2* keys_list) {
  const ListPlan lp = list_plan(N, topk);
  *list_codes = nullptr;
  *list_pos = nullptr;
  if (lp.levels == 0) return hipSuccess;
  const SelectWs ws = select_ws(S, N, topk, 1);
  char* wsb = static_cast<char*>(workspace);
  uint32_t* cnt = reinterpret_cast<uint32_t*>(wsb + ws.cnt_off);
  uint32_t* lc = reinterpret_cast<uint32_t*>(wsb + ws.codes_off);
  int32_t* lpos = reinterpret_cast<int32_t*>(wsb + ws.pos_off);
  const int64_t tiles = ceil_div(N, kSortTile);
  const dim3 grid(unsigned(S * tiles)), block(kSortThreads);
  hipLaunchKernelGGL(list_count_kernel, grid, block, 0, stream, perm, N, tiles, lp.t0, lp.levels, cnt);
  hipLaunchKernelGGL(list_scatter_kernel, grid, block, 0, stream, sorted_codes, perm, N, tiles, lp.t0, lp.levels,
                     lp.cap, cnt, lc, lpos, k_rows, keys_full, keys_list);
  *list_codes = lc;
  *list_pos = lpos;
  return hipGetLastError();
}

hipError_t launch_select(const uint32_t* q_codes, const uint32_t* sorted_codes, const int32_t* perm,
                         int64_t S, int64_t N, int topk, bool causal, int chunk, const int32_t* q_order, int32_t* idx,
                         void* workspace, hipStream_t stream) {
  const uint32_t* list_codes = nullptr;
  const int32_t* list_pos = nullptr;
  if (causal) {
    const hipError_t e = launch_prefix_lists(sorted_codes, perm, S, N, topk, workspace, stream, &list_codes, &list_pos);
    if (e != hipSuccess) return e;
  }
  // The windows as list-index bounds, then the rows from the bounds.
  int2* bounds = reinterpret_cast<int2*>(static_cast<char*>(workspace) + select_ws(S, N, topk, causal).bounds_off);
  return launch_tile_windows(nullptr, S, N, 0, topk, causal, chunk, q_codes, sorted_codes, perm, list_codes, list_pos,
                             q_order, idx, bounds, nullptr, nullptr, true, stream);
}

}  // namespace zeta
