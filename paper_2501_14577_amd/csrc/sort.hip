// Stable segmented LSD radix sort of (code, position) pairs (Section 3.2.2;
// Algorithm 1, Step 2; Appendix B sorts the codes with a radix sort).
//
// Every segment is cut into tiles of 4096 keys (2048 for the level
// partition of a processing order).  One pass over a digit of at
// most 9 bits runs two kernels (three when a segment has more than 32 tiles):
//   hist:    per tile, the count of each digit value (LDS atomics);
//   [scan:   per segment and digit value, the counts of earlier tiles
//            (written over the tile counts) and the segment total;]
//   scatter: per tile, the digit's first output slot (an exclusive scan over
//            digit values of the segment totals, plus the earlier tiles'
//            counts, which the scatter sums itself for up to 32 tiles), a
//            stable rank of every key inside the tile (each wavefront walks
//            its 512 keys in order, 64 at a time, finding same-digit lanes
//            with one ballot per digit bit and counting them with mbcnt), the
//            tile reordered by digit in LDS, and then the tile written out in
//            that order, so that each digit's keys leave as one run of
//            consecutive addresses.
// Tiles of one segment run on one XCD (xcd_contiguous_block): the runs
// several tiles write into the same output lines merge in that XCD's L2.
// A pass preserves the order of equal digits, so after the last pass equal
// codes are in ascending position order.  ceil(code_bits / 9) passes split
// the bits evenly (18-bit codes: two passes of 9).
#include "device_common.h"
#include "kernels.h"
#include "layout.h"
#include "select_device.h"

namespace zeta {
namespace {

constexpr int kRadixWaves = kRadixThreads / 64;
static_assert(kRadixThreads == kRadixMax, "one digit value per thread");
constexpr int kDigitBits = 9;  // the most bits one pass takes
static_assert((1 << kDigitBits) == kRadixMax, "a digit indexes the per-tile counts");

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

template <bool kByLevel, int kChunks>
__global__ void __launch_bounds__(kRadixThreads)
    radix_hist_kernel(const uint32_t* __restrict__ keys, const int32_t* __restrict__ vals, int64_t N, int64_t tiles,
                      int shift, int nbits, int t0, int t_hi, int chunk, uint32_t* __restrict__ hist) {
  // Tiles of one segment run under one L2 (see xcd_contiguous_block).
  const int64_t blk = xcd_contiguous_block(blockIdx.x, gridDim.x);
  const int64_t seg = blk / tiles;
  const int64_t tile = blk % tiles;
  const int tid = threadIdx.x;
  __shared__ uint32_t h[kRadixMax];
  h[tid] = 0;
  __syncthreads();
  const uint32_t mask = (1u << nbits) - 1u;
  constexpr int64_t kTile = int64_t(kRadixThreads) * kChunks;
  const int64_t e0 = tile * kTile;
  // Every load issued first (an element past the segment's end reads its
  // last one, then is left out), so that their latencies overlap.
  uint32_t key[kChunks];
  int32_t val[kChunks];
#pragma unroll
  for (int c = 0; c < kChunks; ++c) {
    const int64_t e = e0 + c * kRadixThreads + tid;
    const int64_t ec = e < N ? e : N - 1;
    key[c] = kByLevel ? 0u : keys[seg * N + ec];
    val[c] = kByLevel ? (vals != nullptr ? vals[seg * N + ec] : int32_t(e)) : 0;
  }
#pragma unroll
  for (int c = 0; c < kChunks; ++c) {
    if (e0 + c * kRadixThreads + tid < N)
      atomicAdd(&h[radix_digit<kByLevel>(key[c], val[c], shift, mask, t0, t_hi, chunk, N)], 1u);
  }
  __syncthreads();
  hist[(seg * tiles + tile) * kRadixMax + tid] = h[tid];
}

// Tiles of one segment are split into kScanGroups contiguous groups; wave g
// of the block sums group g for 64 digit values, the groups' sums are
// combined through LDS, and each wave then rewrites its tiles' counts as
// exclusive prefixes.  Grid: S * (kRadixMax / 64) blocks of kScanThreads.
constexpr int kScanThreads = 256;
constexpr int kScanGroups = kScanThreads / 64;
constexpr int kScanBatch = 16;

__global__ void __launch_bounds__(kScanThreads)
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

// kInline: the tile counts in `hist` are raw (no scan ran) and the segment
// has at most kRadixInlineTiles tiles; otherwise `hist` holds the earlier
// tiles' counts and `totals` the segment totals.
template <bool kHasPos, bool kByLevel, bool kInline, int kChunks>
__global__ void __launch_bounds__(kRadixThreads)
    radix_scatter_kernel(const uint32_t* __restrict__ keys_in, const int32_t* __restrict__ pos_in,
                         int64_t N, int64_t tiles, int shift, int nbits, int t0, int t_hi, int chunk,
                         const uint32_t* __restrict__ hist, const uint32_t* __restrict__ totals,
                         uint32_t* __restrict__ keys_out, int32_t* __restrict__ pos_out) {
  const int64_t blk = xcd_contiguous_block(blockIdx.x, gridDim.x);
  const int64_t seg = blk / tiles;
  const int64_t tile = blk % tiles;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const uint32_t mask = (1u << nbits) - 1u;

  __shared__ uint32_t s_base[kRadixMax];               // output slot of the tile's first key of each digit
  __shared__ uint32_t s_lstart[kRadixMax];             // tile-local slot of the first key of each digit
  __shared__ uint32_t s_wcnt[kRadixWaves][kRadixMax];  // per-wave running, then prefix, counts
  constexpr int kTile = kRadixThreads * kChunks;
  __shared__ uint32_t s_key[kByLevel ? 1 : kTile];
  __shared__ int32_t s_val[kTile];
  __shared__ uint32_t s_scan[kRadixWaves];

  // This wavefront's keys, loaded before anything else so that their
  // latency overlaps the digit offsets' loads: every load issued (an element
  // past the segment's end reads its last one, then is left out).
  const int64_t seg_off = seg * N;
  const int64_t tile0 = tile * kTile;
  const int64_t first = tile0 + int64_t(wave) * (kChunks * 64);
  uint32_t key[kChunks];
  int32_t pos[kChunks];
#pragma unroll
  for (int c = 0; c < kChunks; ++c) {
    const int64_t e = first + c * 64 + lane;
    const int64_t ec = e < N ? e : N - 1;
    key[c] = kByLevel ? 0u : keys_in[seg_off + ec];
    pos[c] = kHasPos ? pos_in[seg_off + ec] : int32_t(e);
  }

  {
    // This thread's digit value: its count in earlier tiles and in the
    // whole segment.
    const int d = tid;
    uint32_t before = 0, total = 0;
    const uint32_t* h = hist + seg * tiles * kRadixMax + d;
    if (kInline) {
      // Independent loads in batches, so their latencies overlap.
      constexpr int kBatch = 8;
      for (int64_t t0 = 0; t0 < tiles; t0 += kBatch) {
        uint32_t c[kBatch];
#pragma unroll
        for (int j = 0; j < kBatch; ++j) c[j] = t0 + j < tiles ? h[(t0 + j) * kRadixMax] : 0u;
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
          before += t0 + j < tile ? c[j] : 0u;
          total += c[j];
        }
      }
    } else {
      before = h[tile * kRadixMax];
      total = totals[seg * kRadixMax + d];
    }
    const uint32_t excl = block_exclusive_scan<kRadixWaves>(total, s_scan);
    s_base[d] = excl + before;
#pragma unroll
    for (int w = 0; w < kRadixWaves; ++w) s_wcnt[w][d] = 0;
  }
  __syncthreads();

  uint32_t rank[kChunks];
#pragma unroll
  for (int c = 0; c < kChunks; ++c) {
    const int64_t e = first + c * 64 + lane;
    const bool valid = e < N;
    const uint32_t kk = (valid && !kByLevel) ? key[c] : 0u;
    const int32_t pp = kHasPos ? (valid ? pos[c] : 0) : int32_t(e);
    const uint32_t d = radix_digit<kByLevel>(kk, pp, shift, mask, t0, t_hi, chunk, N);
    // Lanes with this lane's digit: for every digit bit, those whose bit
    // equals this lane's, i.e. peers & ~(ones ^ s) per 32-bit half with s all
    // ones where the bit is set (one three-input bit operation; its table
    // 0x90 is that function of the operand patterns 0xF0, 0xCC, 0xAA).
    const uint64_t valid_m = wave_ballot(valid);
    uint32_t plo = uint32_t(valid_m), phi = uint32_t(valid_m >> 32);
#pragma unroll
    for (int b = 0; b < kDigitBits; ++b) {
      if (b < nbits) {
        const uint32_t s = uint32_t(int32_t(d << (31 - b)) >> 31);
        const uint64_t ones = wave_ballot(s != 0u);
        plo = __builtin_amdgcn_bitop3_b32(plo, uint32_t(ones), s, 0x90);
        phi = __builtin_amdgcn_bitop3_b32(phi, uint32_t(ones >> 32), s, 0x90);
      }
    }
    const uint64_t peers = (uint64_t(phi) << 32) | plo;
    const uint32_t below = lanes_below(peers);
    const uint32_t base = s_wcnt[wave][d];
    if (valid && below == 0) s_wcnt[wave][d] = base + uint32_t(__popcll(peers));
    key[c] = kk;
    pos[c] = pp;
    rank[c] = base + below;
  }
  __syncthreads();
  {
    // Per digit: earlier waves' counts, then the digit's first slot in the
    // tile (exclusive scan of the tile's digit counts).
    const int d = tid;
    uint32_t run = 0;
#pragma unroll
    for (int w = 0; w < kRadixWaves; ++w) {
      const uint32_t t = s_wcnt[w][d];
      s_wcnt[w][d] = run;
      run += t;
    }
    s_lstart[d] = block_exclusive_scan<kRadixWaves>(run, s_scan);
  }
  __syncthreads();
  // The tile in digit order, in LDS.
#pragma unroll
  for (int c = 0; c < kChunks; ++c) {
    const int64_t e = first + c * 64 + lane;
    if (e < N) {
      const uint32_t d = radix_digit<kByLevel>(key[c], pos[c], shift, mask, t0, t_hi, chunk, N);
      const uint32_t slot = s_lstart[d] + s_wcnt[wave][d] + rank[c];
      if (!kByLevel) s_key[slot] = key[c];
      s_val[slot] = pos[c];
    }
  }
  __syncthreads();
  // Written in that order: consecutive threads of one digit write
  // consecutive slots.
  const int n = int(N - tile0 < kTile ? N - tile0 : kTile);
  for (int i = tid; i < n; i += kRadixThreads) {
    const uint32_t kk = kByLevel ? 0u : s_key[i];
    const int32_t vv = s_val[i];
    const uint32_t d = radix_digit<kByLevel>(kk, vv, shift, mask, t0, t_hi, chunk, N);
    const int64_t dst = int64_t(s_base[d]) + (uint32_t(i) - s_lstart[d]);
    if (!kByLevel) keys_out[seg_off + dst] = kk;
    pos_out[seg_off + dst] = vv;
  }
}

// One pass over tiles of kRadixThreads * kChunks keys: hist, [scan,] scatter.
template <bool kHasPos, bool kByLevel, int kChunks>
void radix_pass(const uint32_t* keys_in, const int32_t* pos_in, int64_t S, int64_t N, int64_t tiles, int shift,
                int nbits, int t0, int t_hi, int chunk, uint32_t* hist, uint32_t* keys_out, int32_t* pos_out,
                hipStream_t stream) {
  const dim3 grid(unsigned(S * tiles)), block(kRadixThreads);
  uint32_t* totals = hist + S * tiles * kRadixMax;
  hipLaunchKernelGGL((radix_hist_kernel<kByLevel, kChunks>), grid, block, 0, stream, keys_in, pos_in, N, tiles, shift, nbits, t0,
                     t_hi, chunk, hist);
  if (tiles <= kRadixInlineTiles) {
    hipLaunchKernelGGL((radix_scatter_kernel<kHasPos, kByLevel, true, kChunks>), grid, block, 0, stream, keys_in, pos_in, N,
                       tiles, shift, nbits, t0, t_hi, chunk, hist, totals, keys_out, pos_out);
  } else {
    hipLaunchKernelGGL(radix_scan_kernel, dim3(unsigned(S * (kRadixMax / 64))), dim3(kScanThreads), 0, stream, tiles,
                       hist, totals);
    hipLaunchKernelGGL((radix_scatter_kernel<kHasPos, kByLevel, false, kChunks>), grid, block, 0, stream, keys_in, pos_in, N,
                       tiles, shift, nbits, t0, t_hi, chunk, hist, totals, keys_out, pos_out);
  }
}

}  // namespace

hipError_t launch_level_partition(const int32_t* vals, int64_t S, int64_t N, int t0, int t_hi, int levels, int chunk,
                                  int32_t* vals_out, uint32_t* hist, hipStream_t stream) {
  // Smaller tiles than the sort's: few digit values, long runs, and more
  // blocks in flight.
  constexpr int kChunks = int(kLevelTile / kRadixThreads);
  const int64_t tiles = ceil_div(N, kLevelTile);
  int nbits = 1;
  while ((1 << nbits) < levels + 1) ++nbits;
  if (vals != nullptr)
    radix_pass<true, true, kChunks>(nullptr, vals, S, N, tiles, 0, nbits, t0, t_hi, chunk, hist, nullptr, vals_out,
                                    stream);
  else
    radix_pass<false, true, kChunks>(nullptr, vals, S, N, tiles, 0, nbits, t0, t_hi, chunk, hist, nullptr, vals_out,
                                     stream);
  return hipGetLastError();
}

hipError_t launch_sort(const uint32_t* k_codes, int64_t S, int64_t N, int code_bits,
                       uint32_t* sorted_codes, int32_t* perm, void* workspace, hipStream_t stream) {
  const SortPlan plan = sort_plan(N, code_bits);
  const SortWs ws = sort_ws(S, N, code_bits);
  char* wsb = static_cast<char*>(workspace);
  uint32_t* hist = reinterpret_cast<uint32_t*>(wsb + ws.hist_off);
  uint32_t* tmp_keys = reinterpret_cast<uint32_t*>(wsb + ws.keys_off);
  int32_t* tmp_pos = reinterpret_cast<int32_t*>(wsb + ws.pos_off);

  const uint32_t* src_keys = k_codes;
  const int32_t* src_pos = nullptr;
  for (int p = 0; p < plan.passes; ++p) {
    const int shift = p * plan.digit_bits;
    const int nbits = (code_bits - shift < plan.digit_bits) ? code_bits - shift : plan.digit_bits;
    // The last pass lands in the caller's outputs; earlier passes alternate.
    const bool to_out = ((plan.passes - 1 - p) % 2) == 0;
    uint32_t* dst_keys = to_out ? sorted_codes : tmp_keys;
    int32_t* dst_pos = to_out ? perm : tmp_pos;
    if (src_pos == nullptr)
      radix_pass<false, false, kRadixChunks>(src_keys, src_pos, S, N, plan.tiles, shift, nbits, 0, 0, 0, hist,
                                             dst_keys, dst_pos, stream);
    else
      radix_pass<true, false, kRadixChunks>(src_keys, src_pos, S, N, plan.tiles, shift, nbits, 0, 0, 0, hist,
                                            dst_keys, dst_pos, stream);
    src_keys = dst_keys;
    src_pos = dst_pos;
  }
  return hipGetLastError();
}

}  // namespace zeta
