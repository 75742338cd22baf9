// Stable segmented LSD radix sort of (code, position) pairs (Section 3.2.2;
// Algorithm 1, Step 2; Appendix B sorts the codes with a radix sort).
//
// Every segment is cut into tiles of 1024 keys.  One pass over a digit of at
// most 9 bits runs three kernels:
//   hist:    per tile, the count of each digit value (LDS atomics);
//   scan:    per segment and digit value, the counts of earlier tiles
//            (written over the tile counts) and the segment total;
//   scatter: per tile, the digit's global base (an exclusive scan over digit
//            values of the segment totals, plus the earlier tiles' counts),
//            then a stable rank of every key inside the tile: each wavefront
//            walks its 256 keys in order, 64 at a time, finding same-digit
//            lanes with one ballot per digit bit and counting them with
//            mbcnt; per-wave running counts live in LDS.
// A pass preserves the order of equal digits, so after the last pass equal
// codes are in ascending position order.  ceil(code_bits / 9) passes split
// the bits evenly (18-bit codes: two passes of 9).
#include "device_common.h"
#include "kernels.h"
#include "layout.h"
#include "select_device.h"

namespace zeta {
namespace {

// Digit of an element: the key's bits [shift, shift+nbits) (kByLevel false), or
// the prefix-list level class of the carried position (kByLevel true; the
// level regrouping of a processing order: the level of the list that
// position's causal pool is searched in, see pool_limit and pool_level).
template <bool kByLevel>
__device__ __forceinline__ uint32_t radix_digit(uint32_t key, int32_t val, int shift, uint32_t mask, int t0,
                                                int t_hi, int chunk, int64_t N) {
  if (kByLevel) return (val >= 0 && val < N) ? uint32_t(pool_level(pool_limit(val, chunk), t0, t_hi) - t0) : 0u;
  return (key >> shift) & mask;
}

template <bool kByLevel>
__global__ void __launch_bounds__(kSortThreads)
    radix_hist_kernel(const uint32_t* __restrict__ keys, const int32_t* __restrict__ vals, int64_t N, int64_t tiles,
                      int shift, int nbits, int t0, int t_hi, int chunk, uint32_t* __restrict__ hist) {
  const int64_t seg = blockIdx.x / tiles;
  const int64_t tile = blockIdx.x % tiles;
  const int tid = threadIdx.x;
  __shared__ uint32_t h[kRadixMax];
  for (int d = tid; d < kRadixMax; d += kSortThreads) h[d] = 0;
  __syncthreads();
  const uint32_t mask = (1u << nbits) - 1u;
  const int64_t e0 = tile * kSortTile;
  const int64_t e1 = (e0 + kSortTile < N) ? e0 + kSortTile : N;
  for (int64_t e = e0 + tid; e < e1; e += kSortThreads) {
    const uint32_t key = kByLevel ? 0u : keys[seg * N + e];
    const int32_t val = kByLevel ? (vals != nullptr ? vals[seg * N + e] : int32_t(e)) : 0;
    atomicAdd(&h[radix_digit<kByLevel>(key, val, shift, mask, t0, t_hi, chunk, N)], 1u);
  }
  __syncthreads();
  for (int d = tid; d < kRadixMax; d += kSortThreads) hist[(seg * tiles + tile) * kRadixMax + d] = h[d];
}

// Tiles of one segment are split into kScanGroups contiguous groups; wave g
// of the block sums group g for 64 digit values, the groups' sums are
// combined through LDS, and each wave then rewrites its tiles' counts as
// exclusive prefixes.  Grid: S * (kRadixMax / 64) blocks.
constexpr int kScanGroups = kSortThreads / 64;
constexpr int kScanBatch = 16;

__global__ void __launch_bounds__(kSortThreads)
    radix_scan_kernel(int64_t tiles, uint32_t* __restrict__ hist, uint32_t* __restrict__ totals) {
  const int64_t seg = blockIdx.x / (kRadixMax / 64);
  const int d = int(blockIdx.x % (kRadixMax / 64)) * 64 + (threadIdx.x & 63);
  const int g = threadIdx.x >> 6;
  const int64_t per = (tiles + kScanGroups - 1) / kScanGroups;
  const int64_t t_begin = g * per < tiles ? g * per : tiles;
  const int64_t t_end = t_begin + per < tiles ? t_begin + per : tiles;
  uint32_t* h = hist + seg * tiles * kRadixMax + d;
  __shared__ uint32_t s_sum[kScanGroups][64];

  uint32_t sum = 0;
  for (int64_t t = t_begin; t < t_end; t += kScanBatch) {
    uint32_t c[kScanBatch];
#pragma unroll
    for (int j = 0; j < kScanBatch; ++j) c[j] = (t + j < t_end) ? h[(t + j) * kRadixMax] : 0u;
#pragma unroll
    for (int j = 0; j < kScanBatch; ++j) sum += c[j];
  }
  s_sum[g][threadIdx.x & 63] = sum;
  __syncthreads();
  uint32_t run = 0, total = 0;
#pragma unroll
  for (int j = 0; j < kScanGroups; ++j) {
    const uint32_t x = s_sum[j][threadIdx.x & 63];
    run += (j < g) ? x : 0u;
    total += x;
  }
  if (g == 0) totals[seg * kRadixMax + d] = total;
  for (int64_t t = t_begin; t < t_end; t += kScanBatch) {
    uint32_t c[kScanBatch];
#pragma unroll
    for (int j = 0; j < kScanBatch; ++j) c[j] = (t + j < t_end) ? h[(t + j) * kRadixMax] : 0u;
#pragma unroll
    for (int j = 0; j < kScanBatch; ++j) {
      if (t + j < t_end) h[(t + j) * kRadixMax] = run;
      run += c[j];
    }
  }
}

template <bool kHasPos, bool kByLevel>
__global__ void __launch_bounds__(kSortThreads)
    radix_scatter_kernel(const uint32_t* __restrict__ keys_in, const int32_t* __restrict__ pos_in,
                         int64_t N, int64_t tiles, int shift, int nbits, int t0, int t_hi, int chunk,
                         const uint32_t* __restrict__ hist, const uint32_t* __restrict__ totals,
                         uint32_t* __restrict__ keys_out, int32_t* __restrict__ pos_out) {
  const int64_t seg = blockIdx.x / tiles;
  const int64_t tile = blockIdx.x % tiles;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const uint32_t mask = (1u << nbits) - 1u;

  __shared__ uint32_t s_base[kRadixMax];              // first output slot of each digit in this tile
  __shared__ uint32_t s_wcnt[kSortThreads / 64][kRadixMax];  // per-wave running / prefix counts
  __shared__ uint32_t s_scan[4];

  constexpr int kPer = kRadixMax / kSortThreads;  // digit values per thread: tid*kPer ..
  {
    // Digit totals of the segment and counts of the tiles before this one.
    uint32_t tot[kPer], bef[kPer], sum = 0;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int d = tid * kPer + i;
      tot[i] = totals[seg * kRadixMax + d];
      bef[i] = hist[(seg * tiles + tile) * kRadixMax + d];
      sum += tot[i];
    }
    uint32_t excl = block256_exclusive_scan(sum, s_scan);
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      s_base[tid * kPer + i] = excl + bef[i];
      excl += tot[i];
#pragma unroll
      for (int w = 0; w < kSortThreads / 64; ++w) s_wcnt[w][tid * kPer + i] = 0;
    }
  }
  __syncthreads();

  const int64_t seg_off = seg * N;
  const int64_t first = tile * kSortTile + int64_t(wave) * (kSortChunks * 64);
  uint32_t key[kSortChunks];
  int32_t pos[kSortChunks];
  uint32_t rank[kSortChunks];
#pragma unroll
  for (int c = 0; c < kSortChunks; ++c) {
    const int64_t e = first + c * 64 + lane;
    const bool valid = e < N;
    const uint32_t kk = (valid && !kByLevel) ? keys_in[seg_off + e] : 0u;
    int32_t pp;
    if (kHasPos)
      pp = valid ? pos_in[seg_off + e] : 0;
    else
      pp = int32_t(e);
    const uint32_t d = radix_digit<kByLevel>(kk, pp, shift, mask, t0, t_hi, chunk, N);
    uint64_t peers = wave_ballot(valid);
    for (int b = 0; b < nbits; ++b) {
      const bool bit = (d >> b) & 1u;
      const uint64_t ones = wave_ballot(bit);
      peers &= bit ? ones : ~ones;
    }
    const uint32_t below = lanes_below(peers);
    const uint32_t base = s_wcnt[wave][d];
    if (valid && below == 0) s_wcnt[wave][d] = base + uint32_t(__popcll(peers));
    key[c] = kk;
    pos[c] = pp;
    rank[c] = base + below;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    uint32_t run = 0;
#pragma unroll
    for (int w = 0; w < kSortThreads / 64; ++w) {
      const uint32_t t = s_wcnt[w][tid * kPer + i];
      s_wcnt[w][tid * kPer + i] = run;
      run += t;
    }
  }
  __syncthreads();
#pragma unroll
  for (int c = 0; c < kSortChunks; ++c) {
    const int64_t e = first + c * 64 + lane;
    if (e < N) {
      const uint32_t d = radix_digit<kByLevel>(key[c], pos[c], shift, mask, t0, t_hi, chunk, N);
      const int64_t dst = int64_t(s_base[d]) + s_wcnt[wave][d] + rank[c];
      if (!kByLevel) keys_out[seg_off + dst] = key[c];
      pos_out[seg_off + dst] = pos[c];
    }
  }
}

}  // namespace

hipError_t launch_level_partition(const int32_t* vals, int64_t S, int64_t N, int t0, int t_hi, int levels, int chunk,
                                  int32_t* vals_out, uint32_t* hist, hipStream_t stream) {
  const int64_t tiles = ceil_div(N, kSortTile);
  const dim3 grid(unsigned(S * tiles)), block(kSortThreads);
  int nbits = 1;
  while ((1 << nbits) < levels + 1) ++nbits;
  uint32_t* totals = hist + S * tiles * kRadixMax;
  hipLaunchKernelGGL(radix_hist_kernel<true>, grid, block, 0, stream, nullptr, vals, N, tiles, 0, nbits, t0, t_hi,
                     chunk, hist);
  hipLaunchKernelGGL(radix_scan_kernel, dim3(unsigned(S * (kRadixMax / 64))), block, 0, stream, tiles, hist, totals);
  if (vals != nullptr)
    hipLaunchKernelGGL((radix_scatter_kernel<true, true>), grid, block, 0, stream, nullptr, vals, N, tiles, 0, nbits,
                       t0, t_hi, chunk, hist, totals, nullptr, vals_out);
  else
    hipLaunchKernelGGL((radix_scatter_kernel<false, true>), grid, block, 0, stream, nullptr, vals, N, tiles, 0, nbits,
                       t0, t_hi, chunk, hist, totals, nullptr, vals_out);
  return hipGetLastError();
}

hipError_t launch_sort(const uint32_t* k_codes, int64_t S, int64_t N, int code_bits,
                       uint32_t* sorted_codes, int32_t* perm, void* workspace, hipStream_t stream) {
  const SortPlan plan = sort_plan(N, code_bits);
  const SortWs ws = sort_ws(S, N, code_bits);
  char* wsb = static_cast<char*>(workspace);
  uint32_t* hist = reinterpret_cast<uint32_t*>(wsb + ws.hist_off);
  uint32_t* totals = hist + S * plan.tiles * kRadixMax;
  uint32_t* tmp_keys = reinterpret_cast<uint32_t*>(wsb + ws.keys_off);
  int32_t* tmp_pos = reinterpret_cast<int32_t*>(wsb + ws.pos_off);
  const dim3 grid(unsigned(S * plan.tiles)), block(kSortThreads);

  const uint32_t* src_keys = k_codes;
  const int32_t* src_pos = nullptr;
  for (int p = 0; p < plan.passes; ++p) {
    const int shift = p * plan.digit_bits;
    const int nbits = (code_bits - shift < plan.digit_bits) ? code_bits - shift : plan.digit_bits;
    // The last pass lands in the caller's outputs; earlier passes alternate.
    const bool to_out = ((plan.passes - 1 - p) % 2) == 0;
    uint32_t* dst_keys = to_out ? sorted_codes : tmp_keys;
    int32_t* dst_pos = to_out ? perm : tmp_pos;
    hipLaunchKernelGGL(radix_hist_kernel<false>, grid, block, 0, stream, src_keys, nullptr, N, plan.tiles, shift,
                       nbits, 0, 0, 0, hist);
    hipLaunchKernelGGL(radix_scan_kernel, dim3(unsigned(S * (kRadixMax / 64))), block, 0, stream, plan.tiles, hist,
                       totals);
    if (src_pos == nullptr)
      hipLaunchKernelGGL((radix_scatter_kernel<false, false>), grid, block, 0, stream, src_keys, src_pos, N,
                         plan.tiles, shift, nbits, 0, 0, 0, hist, totals, dst_keys, dst_pos);
    else
      hipLaunchKernelGGL((radix_scatter_kernel<true, false>), grid, block, 0, stream, src_keys, src_pos, N,
                         plan.tiles, shift, nbits, 0, 0, 0, hist, totals, dst_keys, dst_pos);
    src_keys = dst_keys;
    src_pos = dst_pos;
  }
  return hipGetLastError();
}

}  // namespace zeta
