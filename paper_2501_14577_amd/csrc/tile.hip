// Candidate selection and Cauchy-softmax attention for bfloat16 inputs, 16
// queries at a time on the matrix cores (Section 3.2.2 and Algorithm 1,
// Steps 3-5, for the windows; Section 3.3, equation cauchy, Section 3.4 and
// Appendix E.1 for the attention).
//
// A query's window is a run of its sorted list: every in-pool entry of the
// list range [a, b] around its insertion point (select_window's window as
// list-index bounds).  In the processing order of zeta_query_order, 16
// consecutive queries search one list at nearby insertion points, so their
// ranges overlap: together they span about twice the window length where
// gathering per query would read 16 windows.
//
// Two kernels:
//  1. window_bounds: each query's range [a, b], 8 bytes per processing-order
//     slot, one query per lane, reading a copy of the list around the run's
//     insertion points in LDS;
//  2. the tile kernel: a wavefront takes 16 consecutive slots and walks the
//     union of their ranges in chunks of 16 list entries.  The positions and
//     key rows of up to 512 entries are staged in LDS in one burst.  Then for
//     each chunk it
//       - scores the 16 x 16 (query, entry) pairs, S = 1 / (|q - k|^2 + eps)
//         when the entry lies in the query's range and pool, else 0;
//       - loads each entry's value row once for the whole tile (the next
//         chunk's rows load while the current chunk is multiplied);
//       - accumulates V^T (16 value columns x 16 entries) times S^T (16
//         entries x 16 queries), for the high and low score parts together,
//         with one v_mfma_f32_16x16x32_bf16 per 16 value columns.
// Only the weighted sum runs on the matrix cores: it is a dense contraction
// with reuse, since each staged value row is loaded once and serves all 16
// queries of the tile (about half of the 16 x chunk scores are nonzero).  The
// scores, distances over d_k = 3 coordinates, stay on the vector ALUs.
//
// Scores are float32 (hardware reciprocal, 1 ulp); each is split into a
// bfloat16 high part and a bfloat16 remainder, and both products are
// accumulated (the product's 32 K slots hold the 16 entries twice), so the
// weights carry 16 significant bits and the products are exact in the
// float32 accumulator.
// The normaliser sums the float32 scores.  The optional history-mean
// candidate (Section 3.4, last paragraph) is each query's own row, so each
// lane starts its accumulators and the normaliser from it, in float32.
//
// Operand layout of the product (lane l, kg = l / 16; lane l holds 8 of the
// 32 K slots):
//   A (value columns x slots): lane l holds entries 4kg..4kg+3 of column
//     l % 16, twice;
//   B (slots x queries): the high parts of entries 4kg..4kg+3 of query l % 16,
//     then their low parts;
//   D (columns x queries): columns 4kg..4kg+3 of query l % 16.
// Column c of block j is value element c * E + j (E = d_v / 16), so a lane
// loads E consecutive elements of each of its 4 rows with one instruction and
// ends with 4E consecutive outputs of one query.
//
// Chunks are aligned to multiples of 16 in the list and a query's scores are
// zero outside its range, so its output depends only on its own window: the
// result is the same whatever tile the query falls in, i.e. for any
// processing order.
//
// The attend call given index rows and a processing order runs the same
// chunk pipeline (kIdx): a wavefront takes 16 consecutive queries of the
// order and stages the union of their index rows as one run of chunks, each
// entry with the mask of the tile's queries whose rows hold it (a query's
// score is zero where its bit is clear).  There the high and low score parts
// are two 16 x 16 x 16 products on one read of each value fragment.  The union is found without
// barriers, per wavefront: for segments of at most 65536 rows as a bitmap of
// positions (entries in position order, each entry's index its rank), else
// in a hash table keyed by position (entries in slot order).  A union larger
// than the stage, or a row that repeats a position (each occurrence is its
// own term), splits the tile in halves, down to one query, whose row is
// staged slot by slot.  A query's sums are then grouped by the union it
// shares, so its last bits depend on its tile.
#include "attend_device.h"
#include "device_common.h"
#include "kernels.h"
#include "layout.h"
#include "select_device.h"
#include "tile_device.h"

#include <type_traits>

namespace zeta {
namespace {

constexpr int kTileQ = 16;     // queries per tile (product columns)
constexpr int kChunk = 16;     // list entries per product step
constexpr int kTileWaves = 4;  // wavefronts per block

// Index-row tiles (the attend call given a processing order): the union of a
// tile's index rows is built in a per-wavefront hash table of kIdxHash
// positions (linear probing, at most kIdxProbes slots per insertion) that
// lives in the wavefront's value-row buffers, and holds at most
// kIdxUnionCap entries.
constexpr int kIdxHashBits = 10;
constexpr int kIdxHash = 1 << kIdxHashBits;
constexpr int kIdxProbes = 8;
constexpr int kIdxUnionCap = 288;
constexpr uint32_t kIdxEmpty = 0xFFFFFFFFu;

// ---- window bounds ---------------------------------------------------------
// Each lane serves one slot of the processing order (a run of 64 consecutive
// slots per wavefront) and writes its query's window as list-index bounds
// (a, b); slots without a query get (0, -1).  The window is select_window's,
// found by the same steps one entry at a time: the lower bound of the code,
// then up to k - floor(k/2) in-pool entries from it rightwards, floor(k/2)
// plus the right side's shortfall leftwards, and more on the right when the
// left side runs out.
//
// Consecutive slots search one list at nearby insertion points.  The list
// range of kRegion entries around the run's first insertion point is copied
// to LDS (codes and positions); a lane reads the list itself only outside it
// or when its query searches another list.
constexpr int kBndWaves = 4;
constexpr int kRegion = 512;   // list entries staged per wavefront (a multiple of 32)
constexpr int kMargin = 192;    // of them before the run's first insertion point (about)

// Each wavefront's copy of a list range, in LDS.  Declared at file scope and
// indexed directly, so that every access compiles to an LDS instruction (a
// pointer kept in a struct would lose the address space and go through the
// slower flat path).
// Positions are stored in blocks of kScanStep entries at a stride of
// kPosStride: block b starts in 16-byte bank group 9b mod 16, so the scans of
// lanes in different blocks of the region read different bank groups.
constexpr int kPosStride = 36;
__shared__ uint32_t s_bnd_codes[kBndWaves][kRegion];
__shared__ __align__(16) int32_t s_bnd_pos[kBndWaves][kRegion / 32 * kPosStride];
// Segments of at most 65536 rows: positions as 16-bit values, biased by
// 2^15 (pos - 32768 as a signed 16-bit number), 40 to a block of 32 entries
// (80 bytes: the 16 blocks of a region start in 16 different bank groups),
// each entry at element pos16_slot(j) of its block.
constexpr int kPos16Stride = 40;
__shared__ __align__(16) uint16_t s_bnd_pos16[kBndWaves][kRegion / 32 * kPos16Stride];

struct LaneList {
  const uint32_t* codes;
  const int32_t* pos;
  int wave;
  int32_t n, limit, r0, r1;  // [r0, r1): the range copied to LDS (empty when not staged)
  uint32_t lim2;             // 16-bit positions: the biased limit in both halves
};

constexpr int kScanStep = 32;  // list entries examined per step of lane_scan (one bit each of a 32-bit mask)
static_assert(kScanStep == 32, "the scan masks are 32-bit words");
static_assert(kRegion % 64 == 0, "staged in whole rounds of 64 entries, two blocks each");

// Element of its block that holds entry j of the block (16-bit positions).
// The gather in pool_bits sets bit 8c + k from element 4k + c; entry j
// belongs in bit 31 - j.
__device__ __forceinline__ int pos16_slot(int j) {
  const int q = 31 - j;
  return 4 * (q & 7) + (q >> 3);
}

typedef short short2_t __attribute__((ext_vector_type(2)));

// The query's in-pool entries B .. B + kScanStep - 1 (B a multiple of
// kScanStep, B < n) as a bit mask, first entry in the highest bit: bit 31 - j
// is entry B + j.  A block inside the staged range is read from LDS, any other
// block from the list itself, with entries outside [0, n) counted out.
//
// 32-bit positions: an entry is in the pool when pos <= limit, i.e. when
// pos - limit - 1 is negative; each entry's sign bit is shifted in with one
// funnel shift (staged entries past the list's end hold INT32_MAX, in no
// pool).
// 16-bit positions (biased by 2^15): one saturating packed subtraction
// limit - pos covers two entries, negative exactly when pos > limit (the
// clamp keeps the sign); a byte permute spreads the sign bits of four entries
// into four bytes, and one masked OR per four entries packs them.  Entries
// past the list's end are cleared from the mask.
template <bool kPos16>
__device__ __forceinline__ uint32_t pool_bits(const LaneList& L, int32_t B) {
  const uint32_t nl = uint32_t(-1 - L.limit);  // pos + nl < 0 exactly when pos <= limit (no overflow)
  uint32_t mask = 0u;
  if (L.r1 > L.r0 && B >= L.r0 && B + kScanStep <= L.r0 + kRegion) {
    if constexpr (kPos16) {
      const uint4* blk = reinterpret_cast<const uint4*>(&s_bnd_pos16[L.wave][(B - L.r0) / kScanStep * kPos16Stride]);
      uint32_t w[16];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const uint4 v = blk[t];
        w[4 * t] = v.x;
        w[4 * t + 1] = v.y;
        w[4 * t + 2] = v.z;
        w[4 * t + 3] = v.w;
      }
      const short2_t lim = __builtin_bit_cast(short2_t, L.lim2);
      uint32_t out = 0u;  // bit set: entry out of the pool
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const uint32_t d0 = __builtin_bit_cast(uint32_t, __builtin_elementwise_sub_sat(lim, __builtin_bit_cast(short2_t, w[2 * k])));
        const uint32_t d1 =
            __builtin_bit_cast(uint32_t, __builtin_elementwise_sub_sat(lim, __builtin_bit_cast(short2_t, w[2 * k + 1])));
        // Selectors 8..11: the sign bits of the four 16-bit halves, each as a byte.
        out |= __builtin_amdgcn_perm(d1, d0, 0x0B0A0908u) & (0x01010101u << k);
      }
      const int32_t rem = L.n - B;  // >= 1
      const int sh = rem < kScanStep ? kScanStep - rem : 0;
      mask = ~out & (~0u << sh);
    } else {
      const int4* blk = reinterpret_cast<const int4*>(&s_bnd_pos[L.wave][(B - L.r0) / kScanStep * kPosStride]);
#pragma unroll
      for (int t = 0; t < kScanStep / 4; ++t) {
        const int4 v = blk[t];
        mask = __builtin_amdgcn_alignbit(mask, uint32_t(v.x) + nl, 31);
        mask = __builtin_amdgcn_alignbit(mask, uint32_t(v.y) + nl, 31);
        mask = __builtin_amdgcn_alignbit(mask, uint32_t(v.z) + nl, 31);
        mask = __builtin_amdgcn_alignbit(mask, uint32_t(v.w) + nl, 31);
      }
    }
  } else {
    using G = __attribute__((address_space(1))) const int32_t;
    G* gp = (G*)L.pos;
#pragma unroll
    for (int j = 0; j < kScanStep; ++j) {
      const int32_t x = B + j;
      const int32_t v = gp[x < 0 ? 0 : (x < L.n ? x : L.n - 1)];
      mask = __builtin_amdgcn_alignbit(mask, (x >= 0 && x < L.n) ? uint32_t(v) + nl : 0u, 31);
    }
  }
  return mask;
}

// Index of the n-th set bit of m (n from 1 to popcount(m)), by halving.
__device__ __forceinline__ int nth_set_bit(uint32_t m, int n) {
  int pos = 0;
#pragma unroll
  for (int w = 16; w >= 1; w >>= 1) {
    const int c = __popc(m & ((1u << w) - 1u));
    if (n > c) {
      n -= c;
      m >>= w;
      pos += w;
    }
  }
  return pos;
}

// Scan from entry e in direction dir (+1 or -1) for up to `need` in-pool
// entries beyond the `got` already taken; records the first and last entry
// taken (first only when got is 0).  Returns the new count; `e` ends just
// past the last entry taken, or past the list's end.  Entries are examined in
// aligned blocks of kScanStep as a bit mask (bit k: entry base + dir*k); only
// the block where the count is reached is searched for its bit, once, after
// the loop.  Called only with n > 0.
template <bool kPos16>
__device__ __forceinline__ int lane_scan(const LaneList& L, int32_t& e, int dir, int need, int got, int32_t& first,
                                         int32_t& last) {
  uint32_t end_mask = 0u;  // the block where the count is reached, and the bit wanted there
  int32_t end_base = 0;
  int end_n = 0;
  while (got < need && e >= 0 && e < L.n) {
    const int32_t B = e & ~(kScanStep - 1);
    uint32_t mask = pool_bits<kPos16>(L, B);  // bit 31 - j: entry B + j
    int32_t base;
    if (dir > 0) {
      base = B;
      mask = __builtin_bitreverse32(mask) & (~0u << (e - B));
    } else {
      base = B + kScanStep - 1;
      mask &= ~0u << (base - e);
    }
    const int cnt = __popc(mask);
    if (cnt == 0) {
      e = base + dir * kScanStep;
      continue;
    }
    if (got == 0) first = base + dir * (__ffs(int(mask)) - 1);
    if (got + cnt < need) {
      got += cnt;
      last = base + dir * (31 - __clz(int(mask)));
      e = base + dir * kScanStep;
    } else {
      end_mask = mask;
      end_base = base;
      end_n = need - got;
      got = need;
    }
  }
  if (end_n > 0) {
    last = end_base + dir * nth_set_bit(end_mask, end_n);
    e = last + dir;
  }
  return got;
}

template <bool kPos16>
__global__ void __launch_bounds__(kBndWaves * 64)
    window_bounds_kernel(const uint32_t* __restrict__ q_codes, const uint32_t* __restrict__ sorted_codes,
                         const int32_t* __restrict__ perm, const uint32_t* __restrict__ list_codes,
                         const int32_t* __restrict__ list_pos, const int32_t* __restrict__ order, int64_t total,
                         int64_t N, int topk, int causal, int chunk, int t0, int t_hi, int64_t cap,
                         int2* __restrict__ bounds) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int64_t runs = (total + 63) / 64;
  const int64_t nb = gridDim.x;
  for (int64_t blk = xcd_contiguous_block(blockIdx.x, nb); blk * kBndWaves < runs; blk += nb) {
    const int64_t run = blk * kBndWaves + wave;
    if (run >= runs) continue;
    const int64_t slot = run * 64 + lane;
    int32_t my_i = -1;
    uint32_t key = 0;
    int64_t seg = 0;
    if (slot < total) {
      seg = int64_t(uint32_t(slot) / uint32_t(N));  // slots < B*H*N < 2^31
      const int64_t ii = order != nullptr ? int64_t(order[slot]) : slot - seg * N;
      if (ii >= 0 && ii < N) {
        my_i = int32_t(ii);
        key = q_codes[seg * N + ii];
      }
    }
    // A query with an empty pool (the chunked rule's first chunk) gets an
    // empty window and takes no part in the search.
    const bool has_q = my_i >= 0;
    const bool valid = has_q && (causal == 0 || pool_limit(my_i, chunk) >= 0);
    const uint64_t qmask = wave_ballot(has_q);
    if (qmask == 0ull) continue;
    const uint64_t vmask = wave_ballot(valid);
    const QueryList Lq = query_list(sorted_codes, perm, list_codes, list_pos, seg, N, valid ? my_i : 0, causal, t0,
                                    t_hi, cap, valid ? chunk : 0);
    LaneList L;
    L.codes = Lq.codes;
    L.pos = Lq.pos;
    L.wave = wave;
    L.n = Lq.n;
    L.limit = Lq.limit;
    L.r0 = 0;
    L.r1 = 0;
    {
      const int32_t lc = Lq.limit < 0 ? 0 : (Lq.limit > 65535 ? 65535 : Lq.limit);
      const uint32_t b16 = uint32_t(lc) ^ 0x8000u;
      L.lim2 = b16 | (b16 << 16);
    }
    int2 res = make_int2(0, -1);
    if (vmask != 0ull) {
      // Stage the leader's list around the leader's insertion point.
      const int leader = __ffsll((unsigned long long)vmask) - 1;
      const uint32_t* g_codes = readlane_ptr(Lq.codes, leader);
      const int32_t* g_pos = readlane_ptr(Lq.pos, leader);
      const int32_t g_n = __builtin_amdgcn_readlane(Lq.n, leader);
      const uint32_t g_key = uint32_t(__builtin_amdgcn_readlane(int32_t(key), leader));
      const int32_t p0 = wave_lower_bound(g_codes, 0, g_n, g_key, lane);
      const int32_t r0 = (p0 - kMargin > 0 ? p0 - kMargin : 0) & ~(kScanStep - 1);
      const int32_t r1 = r0 + kRegion < g_n ? r0 + kRegion : g_n;
      {
        uint32_t cv[kRegion / 64];
        int32_t pv[kRegion / 64];
#pragma unroll
        for (int t = 0; t < kRegion / 64; ++t) {
          const int32_t e = r0 + t * 64 + lane;
          cv[t] = e < r1 ? g_codes[e] : 0u;
          pv[t] = e < r1 ? g_pos[e] : INT32_MAX;  // past the list's end: in no pool
        }
        const int slot16 = pos16_slot(lane % kScanStep);
#pragma unroll
        for (int t = 0; t < kRegion / 64; ++t) {
          s_bnd_codes[wave][t * 64 + lane] = cv[t];
          if constexpr (kPos16)  // positions < 65536; past the list's end: counted out by pool_bits
            s_bnd_pos16[wave][(2 * t + lane / kScanStep) * kPos16Stride + slot16] = uint16_t(uint32_t(pv[t]) ^ 0x8000u);
          else
            s_bnd_pos[wave][(2 * t + lane / kScanStep) * kPosStride + lane % kScanStep] = pv[t];
        }
      }
      wave_lds_sync();

      const bool staged = Lq.codes == g_codes;
      L.r0 = staged ? r0 : 0;
      L.r1 = staged ? r1 : 0;

      // Lower bound of the code: in the staged range when it brackets the key.
      int32_t p = 0;
      bool found = false;
      if (valid && staged && (r0 == 0 || s_bnd_codes[wave][0] < key) && (r1 == L.n || s_bnd_codes[wave][r1 - r0 - 1] >= key)) {
        int32_t lo = r0, hi = r1;
        while (lo < hi) {
          const int32_t mid = (lo + hi) >> 1;
          if (s_bnd_codes[wave][mid - r0] < key)
            lo = mid + 1;
          else
            hi = mid;
        }
        p = lo;
        found = true;
      }
      // The rest search the list itself, one query at a time, wavefront-wide.
      for (uint64_t m = wave_ballot(valid && !found); m != 0ull; m &= m - 1ull) {
        const int u = __ffsll((unsigned long long)m) - 1;
        const uint32_t* uc_p = readlane_ptr(L.codes, u);
        const int32_t un = __builtin_amdgcn_readlane(L.n, u);
        const uint32_t uk = uint32_t(__builtin_amdgcn_readlane(int32_t(key), u));
        const int32_t up = wave_lower_bound(uc_p, 0, un, uk, lane);
        if (lane == u) p = up;
      }

      // The window, entry by entry.
      if (valid) {
        const int half = topk / 2;
        const int need_r = topk - half;
        // Right side: first and last entry taken; left side: nearest and
        // farthest entry taken.
        int32_t r_first = 0, r_last = -1, l_near = -1, l_far = 0;
        int32_t cur_r = p;
        int got_r = lane_scan<kPos16>(L, cur_r, +1, need_r, 0, r_first, r_last);
        const int need_l = half + (need_r - got_r);
        int32_t cur_l = p - 1;
        const int got_l = lane_scan<kPos16>(L, cur_l, -1, need_l, 0, l_near, l_far);
        if (got_l < need_l && got_r == need_r)
          got_r = lane_scan<kPos16>(L, cur_r, +1, topk - got_l, got_r, r_first, r_last);
        if (got_l + got_r > 0) res = make_int2(got_l > 0 ? l_far : r_first, got_r > 0 ? r_last : l_near);
      }
    }  // some lane has a pool
    if (slot < total) bounds[slot] = res;

    wave_lds_sync();
  }
}

// ---- index rows from window bounds -------------------------------------------
// Writes each query's window as positions: its in-pool entries of the list
// range [a, b] in list order, then -1 (select_window's row, from the bounds
// window_bounds wrote).  A wavefront takes 16 consecutive slots of the
// processing order.  Queries searching one list (nearly always all 16) have
// overlapping ranges: their union's positions are read once into LDS (up to
// kRowsStage entries; a longer union is read from the list itself).  Each
// query's row is then written 64 entries at a time, the in-pool ones by
// ballot compaction into consecutive slots of the row.
constexpr int kRowsWaves = 4;
constexpr int kRowsStage = 1024;
__shared__ int32_t s_rows_pos[kRowsWaves][kRowsStage];

__global__ void __launch_bounds__(kRowsWaves * 64)
    idx_rows_kernel(const uint32_t* __restrict__ sorted_codes, const int32_t* __restrict__ perm,
                    const uint32_t* __restrict__ list_codes, const int32_t* __restrict__ list_pos,
                    const int32_t* __restrict__ order, const int2* __restrict__ bounds, int64_t total, int64_t N,
                    int topk, int causal, int chunk, int t0, int t_hi, int64_t cap, int32_t* __restrict__ idx) {
  constexpr int kQ = 16;  // slots per wavefront
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
  const int64_t groups = (total + kQ - 1) / kQ;
  const int64_t nb = gridDim.x;
  for (int64_t blk = xcd_contiguous_block(blockIdx.x, nb); blk * kRowsWaves < groups; blk += nb) {
    const int64_t grp = blk * kRowsWaves + wave;
    if (grp >= groups) continue;
    // Lanes 0..15: one slot each (its query, list, pool limit and window).
    int32_t my_i = -1, my_lvl = 0, my_a = 0, my_b = -1;
    int64_t my_seg = 0;
    if (lane < kQ) {
      const int64_t sl = grp * kQ + lane;
      if (sl < total) {
        const int64_t sg = int64_t(uint32_t(sl) / uint32_t(N));  // slots < B*H*N < 2^31
        const int64_t ii = order != nullptr ? int64_t(order[sl]) : sl - sg * N;
        if (ii >= 0 && ii < N) {
          my_i = int32_t(ii);
          my_seg = sg;
          const int2 bd = bounds[sl];
          my_a = bd.x;
          my_b = bd.y;
          const int32_t lim = causal ? pool_limit(my_i, chunk) : int32_t(N - 1);
          my_lvl = causal ? (lim < 0 ? -1 : query_level(lim, t0, t_hi)) : 0;
        }
      }
    }
    uint32_t pending = uint32_t(wave_ballot(my_i >= 0)) & 0xFFFFu;
    while (pending != 0u) {
      const int leader = __ffs(int(pending)) - 1;
      const int64_t g_seg = __builtin_amdgcn_readlane(int32_t(my_seg), leader);
      const int g_lvl = __builtin_amdgcn_readlane(my_lvl, leader);
      const uint32_t gmask =
          uint32_t(wave_ballot(my_i >= 0 && my_seg == g_seg && my_lvl == g_lvl)) & pending;
      pending &= ~gmask;
      const int32_t g_i = __builtin_amdgcn_readlane(my_i, leader);
      const QueryList L = query_list(sorted_codes, perm, list_codes, list_pos, g_seg, N, g_i, causal, t0, t_hi,
                                     cap, chunk);
      // The union of the group's windows (a window outside the list counts
      // as empty).
      const bool in_grp = ((gmask >> lane) & 1u) != 0u;
      const bool has = in_grp && 0 <= my_a && my_a <= my_b && my_b < L.n;
      const int32_t ua = wave_min_int(has ? my_a : INT32_MAX);
      const int32_t ub = wave_max_int(has ? my_b : INT32_MIN);
      const bool staged = ua <= ub && ub - ua < kRowsStage;
      if (staged) {
        for (int32_t e0 = ua; e0 <= ub; e0 += 4 * 64) {
          int32_t pv[4];
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const int32_t e = e0 + t * 64 + lane;
            pv[t] = e <= ub ? L.pos[e] : 0;
          }
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            const int32_t e = e0 + t * 64 + lane;
            if (e <= ub) s_rows_pos[wave][e - ua] = pv[t];
          }
        }
      }
      wave_lds_sync();
      for (uint32_t m = gmask; m != 0u; m &= m - 1u) {
        const int u = __ffs(int(m)) - 1;
        const int32_t a = __builtin_amdgcn_readlane(my_a, u), b = __builtin_amdgcn_readlane(my_b, u);
        const int32_t i = __builtin_amdgcn_readlane(my_i, u);
        const int32_t lim = causal ? pool_limit(i, chunk) : int32_t(N - 1);
        int32_t* row = idx + (g_seg * N + i) * int64_t(topk);
        int cnt = 0;
        if (0 <= a && a <= b && b < L.n) {
          if (staged) {
            // Two blocks per step, both read before either is compacted
            // (indices past the union clamped into the stage, then masked).
            for (int32_t e0 = a; e0 <= b; e0 += 128) {
              const int32_t e1 = e0 + lane, e2 = e1 + 64;
              const int32_t o1 = e1 - ua < kRowsStage ? e1 - ua : kRowsStage - 1;
              const int32_t o2 = e2 - ua < kRowsStage ? e2 - ua : kRowsStage - 1;
              int32_t p1 = s_rows_pos[wave][o1], p2 = s_rows_pos[wave][o2];
              p1 = e1 <= b ? p1 : INT32_MAX;
              p2 = e2 <= b ? p2 : INT32_MAX;
              const bool ok1 = p1 <= lim, ok2 = p2 <= lim;
              const uint64_t b1 = wave_ballot(ok1), b2 = wave_ballot(ok2);
              const int at1 = cnt + int(lanes_below(b1));
              const int at2 = cnt + __popcll(b1) + int(lanes_below(b2));
              if (ok1 && at1 < topk) row[at1] = p1;
              if (ok2 && at2 < topk) row[at2] = p2;
              cnt += __popcll(b1) + __popcll(b2);
            }
          } else {
            for (int32_t e0 = a; e0 <= b; e0 += 64) {
              const int32_t e = e0 + lane;
              const int32_t pv = e <= b ? L.pos[e] : INT32_MAX;
              const bool ok = pv <= lim;
              const uint64_t bal = wave_ballot(ok);
              const int at = cnt + int(lanes_below(bal));
              if (ok && at < topk) row[at] = pv;
              cnt += __popcll(bal);
            }
          }
        }
        if (cnt < topk)
          for (int c = cnt + lane; c < topk; c += 64) row[c] = -1;
      }
      // Every read of the staged positions is done before they are replaced.
      wave_lds_sync();
    }
  }
}

// ---- key rows in list order (d_k = 3) ----------------------------------------
// Entry e of a sorted list gets the key row of its position, as three bfloat16
// values in 8 bytes (x | y << 16, z), so that the tile kernel reads the key
// rows of a list range with coalesced loads instead of gathering them by
// position.  One thread per entry, over the full sorted lists (S*N entries)
// and then the prefix lists (S*cap entries; cap is 0 when there are none, and
// list_pos is then not read).
__global__ void __launch_bounds__(256)
    list_keys_kernel(const uint16_t* __restrict__ k, int64_t total, int64_t N, const int32_t* __restrict__ perm,
                     const int32_t* __restrict__ list_pos, int64_t cap, int64_t S, uint2* __restrict__ keys_full,
                     uint2* __restrict__ keys_list) {
  const int64_t t = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t n_full = S * N;
  int64_t seg, pv;
  uint2* dst;
  if (t < n_full) {
    seg = t / N;
    pv = perm[t];
    dst = keys_full + t;
  } else if (list_pos != nullptr && t < n_full + S * cap) {
    const int64_t u = t - n_full;
    seg = u / cap;
    pv = list_pos[u];
    dst = keys_list + u;
  } else {
    return;
  }
  *dst = packed_key_row(k, seg * N + pv, total);
}

// ---- attention over the windows ----------------------------------------------

// Value rows reach the matrix cores through LDS.  Per chunk of 16 entries the
// wavefront copies the 16 value rows straight from global memory into LDS
// (global_load_lds_dwordx4: lane L's 16 bytes land at byte 16 L of the
// instruction's 1 KiB), then reads each product's A operand with one
// transposing LDS read (ds_read_b64_tr_b16: within each group of 16 lanes,
// output lane i receives element i % 4 of the 8-byte reads of lanes
// 4j + i / 4, j = 0..3).  With lane (g, s) of a group pointing at entry row
// 4g + s / 4, columns 16 blk + 4 (s % 4) .. + 3, output lane i holds column
// 16 blk + i of entries 4g .. 4g + 3: the A operand (value columns x
// entries) of a 16 x 16 x 16 product, with no register shuffling (the kernel
// repeats it in the upper K half of a 16 x 16 x 32 product, against the low
// score parts).
//
// LDS row order.  One copy instruction fills R = 512 / d_v consecutive LDS
// rows (P = d_v / 8 pieces of 16 bytes each).  For d_v <= 128 the lanes that
// fill one LDS row share a tile-entry group kg, so each lane copies one of its
// own 4 entries (whose position it already holds): LDS row
// rho = j R + q (instruction j, q = lane / P) holds entry
// 4 kg + j (16 / P) + q % (16 / P).  For d_v = 256 row rho holds entry rho.
// Pieces are XOR-swizzled by row (sw below): physical piece p of row rho
// holds logical piece p ^ sw(rho), so that the transposing reads are free of
// bank conflicts.
// Transposing LDS reads (ds_read_b64_tr_b16) at addr[j] + kOff, kCopies of
// each (into a[kCopies j] .. a[kCopies j + kCopies - 1]), issued once the
// copies into LDS made before the last kPending copy instructions have landed
// (kPending -1: no wait here); read_tr_wait then waits for the results.
// Written as inline assembly, with the waits, because the compiler would
// otherwise wait for every copy still in flight (including the next chunk's,
// which must keep loading meanwhile) before any such read.  LDS operations of
// one wavefront complete in order, so the compiler's own waits on its later
// LDS reads stay correct with these older ones in flight.
template <int E, int kCopies, uint32_t kOff, int kPending>
__device__ __forceinline__ void read_tr_issue(const uint32_t (&addr)[E], s16x4_t (&a)[E * kCopies]) {
  static_assert(kPending >= -1 && kPending < 16, "vmcnt immediate (-1: no wait)");
  if constexpr (kPending >= 0) asm volatile("s_waitcnt vmcnt(%0)" ::"n"(kPending) : "memory");
#pragma unroll
  for (int j = 0; j < E; ++j)
#pragma unroll
    for (int c = 0; c < kCopies; ++c)
      asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2"
                   : "=v"(a[kCopies * j + c])
                   : "v"(addr[j]), "n"(kOff)
                   : "memory");
}

// Waits for every LDS read of this wavefront; the reads' results are then
// used only after the wait (each passes through an ordered empty statement).
template <int N>
__device__ __forceinline__ void read_tr_wait(s16x4_t (&a)[N]) {
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a[0])::"memory");
#pragma unroll
  for (int j = 1; j < N; ++j) asm volatile("" : "+v"(a[j]));
}

template <int DV>
struct VStage {
  static constexpr int kRowBytes = 2 * DV;
  static constexpr int kP = DV / 8;                   // 16-byte pieces per row
  static constexpr int kR = 64 / kP;                  // LDS rows per copy instruction
  static constexpr int kLoads = kChunk / kR;          // copy instructions per chunk
  static constexpr int kOwn = kP <= 16 ? 16 / kP : 0; // rows of one entry group per instruction
  static constexpr int kBlocks = DV / 16;             // products (16 value columns each) per chunk
  static constexpr int kBytes = kChunk * kRowBytes;   // one chunk's rows
  static_assert(kR >= 2 && kChunk % kR == 0, "d_v must be 32, 64, 128 or 256");
  // Piece swizzle of LDS row rho.  A transposing read is served in two
  // halves of 32 lanes (entry groups kg = 0, 1 and kg = 2, 3), each reading
  // 256 bytes: the 16 (row, piece) pairs of one half must fall in 16
  // different 16-byte bank groups.  Row rho's bank group is set by the row's
  // offset within 256 bytes and the physical piece; the swizzle puts the
  // row bits that the offset does not separate into the piece bits that the
  // block index leaves free.
  __device__ static constexpr int sw(int rho) {
    if constexpr (kP == 16) {  // rho = 4u + kg: u into piece bits 2-3, kg's low bit into bit 1
      return (rho & 12) | ((rho & 1) << 1);
    } else if constexpr (kP == 8) {  // rho = 8(u >> 1) + 2kg + (u & 1)
      return (((rho >> 1) & 1) << 1) | (((rho >> 3) & 1) << 2);
    } else if constexpr (kP == 4) {  // rho = 4kg + u
      return ((rho >> 2) & 1) << 1;
    } else {  // kP == 32, rho = 4kg + u
      return ((rho & 3) << 1) | (((rho >> 2) & 1) << 3);
    }
  }
  // Chunk entry held by LDS row rho.
  __device__ static constexpr int entry_of_row(int rho) {
    if constexpr (kP > 16) {
      return rho;
    } else {
      const int j = rho / kR, q = rho % kR;
      return 4 * (q / kOwn) + j * kOwn + q % kOwn;
    }
  }
  // LDS row holding chunk entry e.
  __device__ static constexpr int row_of_entry(int e) {
    if constexpr (kP > 16) {
      return e;
    } else {
      const int kg = e / 4, u = e % 4;
      return (u / kOwn) * kR + kg * kOwn + u % kOwn;
    }
  }
};

// kIdx: the windows are index rows (idx, topk <= kIdxTileMaxTopk, d_k = 3)
// instead of list ranges; `order` is then required and the list arguments
// are unused.
template <int DV, int DK, bool kOff32, bool kHist, int kMode, bool kIdx>
__global__ void __launch_bounds__(kTileWaves * 64)
    __attribute__((amdgpu_waves_per_eu((kOff32 && (DV == 128 || (DV < 128 && kMode != kScoreCauchy))) ? 3 : 1)))
    select_attend_tile_kernel(const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                              const uint16_t* __restrict__ v, const int32_t* __restrict__ sorted_pos,
                              const int32_t* __restrict__ list_pos, const int32_t* __restrict__ order,
                              const int2* __restrict__ bounds, const uint2* __restrict__ keys_full,
                              const uint2* __restrict__ keys_list, int64_t total, int64_t N, int dk_rt, int causal,
                              int chunk, int t0, int t_hi, int64_t cap, float eps,
                              const float* __restrict__ mk, const float* __restrict__ mv, uint16_t* __restrict__ out,
                              const int32_t* __restrict__ idx, int topk) {
  using VS = VStage<DV>;
  constexpr int E = VS::kBlocks;  // products per chunk; a lane ends with 4 columns of each block
  constexpr int KD = DK > 0 ? DK : kMaxDk;
  static_assert(!kIdx || DK == 3, "index-row tiles are compiled for d_k = 3");
  // Entries whose key rows and positions are staged at once (LDS per wave:
  // these plus two chunks of value rows).
  constexpr int kStageEntries = kIdx ? kIdxUnionCap : (DK == 3 && DV <= 128) ? 320 : 128;
  constexpr int kStage = kStageEntries / kChunk;
  // List ranges are staged in whole rounds of 64 entries (every staged
  // entry written); index-row unions in whole chunks.
  static_assert(kIdx || kStageEntries % 64 == 0, "list staging fills rounds of 64 entries");
  static_assert(kStageEntries % kChunk == 0, "the stage holds whole chunks");
  static_assert(E >= 2, "d_v must be a multiple of 32");
  // The high and low score parts of a block: index-row tiles take two
  // 16 x 16 x 16 products on one read of the A fragment; list ranges one
  // 16 x 16 x 32 product whose K halves both hold the fragment, read from LDS
  // twice where the registers allow it, else read once and copied (faster
  // there, measured: the extra products cost more than the saved reads).
  constexpr bool kSplitK = kIdx;
  constexpr int kTrCopies = kSplitK ? 1 : (DV <= 128 && kOff32) ? 2 : 1;
  using Off = typename RowOff<kOff32>::type;
  const int dk = DK > 0 ? DK : dk_rt;
  // Score (compile time): the Cauchy score, or a variant (softmax variants
  // run an online softmax per query: a running maximum shared by the
  // query's 4 lanes, the accumulators and the normaliser rescaled when it
  // grows).
  constexpr bool kVar = kMode != kScoreCauchy;
  constexpr int score = kMode;
  constexpr bool smax = kVar && score_is_softmax(kMode);
  const float rsd = 1.0f / sqrtf(float(dk));

  // One record per staged entry: its key row, then its position (as the bits
  // of a float), padded to whole 16-byte LDS reads; for d_k = 3 one read
  // (x, y, z, position).
  constexpr int KD4 = (KD + 3) / 4 * 4;
  constexpr int kPosSlot = DK == 3 ? 3 : KD4;
  constexpr int KREC = DK == 3 ? 4 : KD4 + 4;
  __shared__ __align__(16) float s_ent[kTileWaves][kStageEntries][KREC];
  // Two chunks of value rows per wave (even chunks, then odd chunks); with
  // index rows also the union's hash table (positions, then query masks)
  // while the union is built.
  constexpr int kVBufBytes = (kIdx && 2 * VS::kBytes < 8 * kIdxHash) ? 8 * kIdxHash : 2 * VS::kBytes;
  __shared__ __align__(16) unsigned char s_v[kTileWaves][kVBufBytes];
  // With index rows: the union entries' query masks (bit t: tile query t).
  __shared__ __align__(16) uint16_t s_um[kTileWaves][kIdx ? kStageEntries : 8];

  const int lane = threadIdx.x & 63;
  // Wave-uniform (the LDS destination of a copy instruction must be).
  const int wave = __builtin_amdgcn_readfirstlane(int(threadIdx.x >> 6));
  const int qn = lane & (kTileQ - 1);  // this lane's query in the tile
  const int kg = lane >> 4;            // this lane's entries in a chunk: 4kg .. 4kg+3
  const int64_t tiles = (total + kTileQ - 1) / kTileQ;
  const int64_t nb = gridDim.x;

  // Copy instruction j: this lane's LDS row, and its byte offset within the
  // value row it copies (its piece, swizzled).
  const int vq = lane / VS::kP, vp = lane % VS::kP;
  uint32_t copy_off[VS::kLoads];
#pragma unroll
  for (int j = 0; j < VS::kLoads; ++j) copy_off[j] = uint32_t(16 * (vp ^ VS::sw(j * VS::kR + vq)));
  // Transposing read of block blk: this lane points at entry 4kg + qn / 4,
  // columns 16 blk + 4 (qn % 4) .. +3 (LDS address in the wave's even-chunk
  // buffer; the odd-chunk buffer follows it).
  uint32_t tr_addr[E];
  {
    const int rho = VS::row_of_entry(4 * kg + qn / 4);
    const int x = (qn % 4) / 2, half = qn % 2;
    const uint32_t base = uint32_t(reinterpret_cast<uintptr_t>(
        (const __attribute__((address_space(3))) unsigned char*)(&s_v[wave][0])));
#pragma unroll
    for (int blk = 0; blk < E; ++blk)
      tr_addr[blk] = base + uint32_t(rho * VS::kRowBytes + 16 * ((2 * blk + x) ^ VS::sw(rho)) + 8 * half);
  }

  // The processing-order entry and window bounds of this lane's slot in a
  // tile, loaded one tile ahead: they arrive while the tile before is
  // processed.
  int32_t nx_o = 0;
  int2 nx_b = make_int2(0, -1);
  auto fetch_slot = [&](int64_t t_) {
    const int64_t sl = t_ * kTileQ + qn;
    if (sl < total) {
      if (order != nullptr) nx_o = order[sl];
      if constexpr (!kIdx) nx_b = bounds[sl];
    }
  };
  // Output rows of the last group of queries wait in this wavefront's
  // value-row buffers (s_orow[wave][r]: the output row of LDS row r, -1 for
  // none) and are stored once the next staged entries are being loaded: the
  // stores then overlap those loads instead of holding up the next tile.
  // Piece p of LDS row r sits at physical piece p ^ (r % kOutP), so that the
  // 8-byte writes and the 16-byte reads are both spread evenly over the banks.
  constexpr int kOutP = DV / 8;       // 16-byte pieces per output row
  constexpr int kOutRows = 64 / kOutP;  // rows per store instruction
  constexpr int kOutRowB = 2 * DV;    // bytes per output row
  static_assert(kTileQ * kOutRowB <= 2 * VS::kBytes, "the output rows fit in the value-row buffers");
  __shared__ int32_t s_orow[kTileWaves][kTileQ];
  bool out_pending = false;
  auto flush_out = [&]() {
    if (out_pending) {
      const unsigned char* so = s_v[wave];
#pragma unroll
      for (int t = 0; t < kTileQ / kOutRows; ++t) {
        const int r = t * kOutRows + lane / kOutP, c = lane % kOutP;
        const uint4 piece = *reinterpret_cast<const uint4*>(so + r * kOutRowB + 16 * (c ^ (r % kOutP)));
        const int32_t orow = s_orow[wave][r];
        // Streaming stores: the output is not read again here, and keeping
        // it out of L2 leaves room for value rows that later tiles reuse.
        if (orow >= 0) {
          uint32_t* dst = reinterpret_cast<uint32_t*>(out + int64_t(orow) * DV + 8 * c);
          __builtin_nontemporal_store(piece.x, dst);
          __builtin_nontemporal_store(piece.y, dst + 1);
          __builtin_nontemporal_store(piece.z, dst + 2);
          __builtin_nontemporal_store(piece.w, dst + 3);
        }
      }
      out_pending = false;
      // Every read of the rows is done before the buffers are written again.
      wave_lds_sync();
    }
  };
  const int64_t blk0 = xcd_contiguous_block(blockIdx.x, nb);
  fetch_slot(blk0 * kTileWaves + wave);
  for (int64_t blk = blk0; blk * kTileWaves < tiles; blk += nb) {
    const int64_t tile = blk * kTileWaves + wave;
    if (tile >= tiles) continue;
    const int32_t cur_o = nx_o;
    const int2 cur_b = nx_b;
    fetch_slot(tile + nb * kTileWaves);

    // The tile's queries and windows: lanes with equal qn hold the same one.
    int32_t my_i = -1;
    int64_t my_seg = 0;
    int my_lvl = 0;
    int32_t my_a = 0, my_b = -1;
    {
      const int64_t sl = tile * kTileQ + qn;
      if (sl < total) {
        const int64_t sg = int64_t(uint32_t(sl) / uint32_t(N));  // slots < B*H*N < 2^31
        const int64_t ii = order != nullptr ? int64_t(cur_o) : sl - sg * N;
        if (ii >= 0 && ii < N) {
          my_i = int32_t(ii);
          my_seg = sg;
          if constexpr (!kIdx) {
            my_lvl = causal ? pool_level(pool_limit(my_i, chunk), t0, t_hi) : 0;
            my_a = cur_b.x;
            my_b = cur_b.y;
          }
        }
      }
    }
    uint32_t pending = uint32_t(wave_ballot(my_i >= 0)) & 0xFFFFu;
    // d_k = 3 (Cauchy score, no history candidate): the query row is read
    // with the staged entries, so that one wait covers both.
    constexpr bool kLateQ = DK == 3 && !kVar && !kHist && !kIdx;

    // ---- index rows: the union of a group's rows ----
    // Slot s of tile query t's row is element 128t + s of the tile's rows;
    // round r holds elements 64r .. 64r + 63 (slots of one row), one per
    // lane.
    constexpr int kRowStride = kIdxTileMaxTopk;
    constexpr int kRounds = kTileQ * kRowStride / 64;
    // Calls body(j, t, s) for every element of the tile's rows, one round at
    // a time: j is slot s of query t's row, or -1 where t is not in `sub` or
    // s >= topk.  The index loads run kAhead rounds ahead of their use; each
    // is issued whatever its slot (one outside the rows reads a slot that
    // exists and is replaced by -1), so that the loads in flight are counted
    // exactly and a round waits only for its own.
    auto for_rows = [&](uint32_t sub, int64_t seg, auto&& body) {
      constexpr int kAhead = 8;  // divides kRounds
      const int32_t my_row = ((sub >> qn) & 1u) != 0u ? int32_t(seg * N + my_i) : -1;  // rows < 2^31
      // The raw loaded value; whether it is a slot of a row is decided where
      // it is used, so that nothing waits for a load before its round.
      auto load = [&](int r) -> int32_t {
        const int rr = r < kRounds ? r : 0;
        const int qq = rr * 64 / kRowStride, sl = rr * 64 % kRowStride + lane;
        const int32_t row = __builtin_amdgcn_readlane(my_row, qq);
        return idx[int64_t(row >= 0 ? row : 0) * topk + (sl < topk ? sl : 0)];
      };
      int32_t ring[kAhead];
#pragma unroll
      for (int u = 0; u < kAhead; ++u) ring[u] = load(u);
      // Straight-line code (all rounds unrolled): the wait before each round
      // is then exactly for its own load.
#pragma unroll
      for (int r0 = 0; r0 < kRounds; r0 += kAhead) {
#pragma unroll
        for (int u = 0; u < kAhead; ++u) {
          const int r = r0 + u;
          const int qq = r * 64 / kRowStride, sl = r * 64 % kRowStride + lane;
          const bool ok = __builtin_amdgcn_readlane(my_row, qq) >= 0 && sl < topk;
          int32_t x = ring[u];
          asm volatile("" : "+v"(x));  // used here, after this round's wait
          const int32_t j = ok ? x : -1;
          if (r + kAhead < kRounds) ring[u] = load(r + kAhead);
          body(j, qq, sl);
        }
      }
    };
    // Inserts the rows of the queries in `sub` into the hash table (keyed by
    // position, each slot also holding the mask of the queries whose rows
    // hold that position), then lists the occupied slots in slot order as
    // the union's entries: positions in s_ent, masks in s_um.  Returns the
    // number of entries, or -1 when the union does not fit (more than
    // kStageEntries entries, a probe sequence exhausted, or a position
    // repeated within one row, which needs an entry per occurrence).
    auto hash_union = [&](uint32_t sub, int64_t seg) -> int {
      uint32_t* const hpos = reinterpret_cast<uint32_t*>(&s_v[wave][0]);
      uint32_t* const hqm = hpos + kIdxHash;
#pragma unroll
      for (int t = 0; t < 2 * kIdxHash / 256; ++t) {
        const uint32_t f = t < kIdxHash / 256 ? kIdxEmpty : 0u;
        reinterpret_cast<uint4*>(hpos)[t * 64 + lane] = make_uint4(f, f, f, f);
      }
      wave_lds_sync();
      int cnt = 0;
      bool bad = false;
      uint32_t dup = 0u;
      for_rows(sub, seg, [&](int32_t j, int qq, int) {
        if (bad) return;
        bool todo = uint32_t(j) < uint32_t(N);
        const uint32_t bit = 1u << (qq & (kTileQ - 1));
        uint32_t h = (uint32_t(j) * 0x9E3779B1u) >> (32 - kIdxHashBits);
#pragma unroll 1
        for (int pr = 0; pr < kIdxProbes; ++pr) {
          uint32_t old = 0u;
          if (todo) old = atomicCAS(&hpos[h], kIdxEmpty, uint32_t(j));
          const bool won = todo && old == kIdxEmpty;
          const bool here = won || (todo && old == uint32_t(j));
          if (here) dup |= atomicOr(&hqm[h], bit) & bit;
          cnt += __popcll(wave_ballot(won));
          todo = todo && !here;
          h = (h + 1u) & uint32_t(kIdxHash - 1);
          if (wave_ballot(todo) == 0ull) break;
        }
        bad = wave_ballot(todo) != 0ull || cnt > kStageEntries;
      });
      if (bad || wave_ballot(dup != 0u) != 0ull) return -1;
      wave_lds_sync();
      int n = 0;
#pragma unroll
      for (int t = 0; t < kIdxHash / 64; ++t) {
        const uint32_t p = hpos[t * 64 + lane];
        const uint64_t m = wave_ballot(p != kIdxEmpty);
        if (p != kIdxEmpty) {
          const int id = n + int(lanes_below(m));
          s_ent[wave][id][kPosSlot] = __int_as_float(int32_t(p));
          s_um[wave][id] = uint16_t(hqm[t * 64 + lane]);
        }
        n += __popcll(m);
      }
      return n;
    };
    // The same for segments of at most 65536 rows, without hashing: the
    // union's positions as a bitmap (one bit per row, 8 KB, in the value-row
    // buffers), then per word the count of union entries before it, so that
    // an entry's index is its rank among the union's positions; a second
    // pass over the rows sets the query masks.  The entries are in position
    // order.  Lane l owns bitmap words 32l .. 32l + 31 (and their counts);
    // the 16-byte pieces of each lane's words are stored XOR-swizzled by
    // lane so that the wavefront's piece-wise reads and writes fall in
    // different bank groups.
    auto bitmap_union = [&](uint32_t sub, int64_t seg) -> int {
      uint32_t* const bm = reinterpret_cast<uint32_t*>(&s_v[wave][0]);
      uint16_t* const pre = reinterpret_cast<uint16_t*>(&s_ent[wave][0][0]);  // until the positions are written
      uint32_t* const mq = reinterpret_cast<uint32_t*>(&s_um[wave][0]);         // two masks per word
      // Physical index of bitmap word w (pieces of 4 words) and of count w
      // (pieces of 8 counts).
      // (Piece bits of w XORed with bits of its owner lane w >> 5.)
      auto bm_at = [](uint32_t w) -> uint32_t { return w ^ ((w >> 4) & 0x1Cu); };
      auto pre_at = [](uint32_t w) -> uint32_t { return w ^ ((w >> 4) & 0x18u); };
      const int bsw = (lane >> 1) & 7, psw = (lane >> 2) & 3;
      uint32_t wd[32];
      auto read_words = [&]() {
#pragma unroll
        for (int t = 0; t < 8; ++t) {
          const uint4 x = reinterpret_cast<const uint4*>(bm)[lane * 8 + (t ^ bsw)];
          wd[4 * t] = x.x;
          wd[4 * t + 1] = x.y;
          wd[4 * t + 2] = x.z;
          wd[4 * t + 3] = x.w;
        }
      };
#pragma unroll
      for (int t = 0; t < 8; ++t) reinterpret_cast<uint4*>(bm)[t * 64 + lane] = make_uint4(0u, 0u, 0u, 0u);
      wave_lds_sync();
      for_rows(sub, seg, [&](int32_t j, int, int) {
        if (uint32_t(j) < uint32_t(N)) atomicOr(&bm[bm_at(uint32_t(j) >> 5)], 1u << (j & 31));
      });
      wave_lds_sync();
      read_words();
      uint32_t tot = 0u;
#pragma unroll
      for (int i = 0; i < 32; ++i) tot += uint32_t(__popc(wd[i]));
      uint32_t incl = tot;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const uint32_t y = __shfl_up(incl, off, 64);
        if (lane >= off) incl += y;
      }
      const int total_u = __builtin_amdgcn_readlane(int(incl), 63);
      if (total_u > kStageEntries) return -1;
      const uint32_t base = incl - tot;
      {
        uint32_t run = base;
        uint32_t packed[16];
#pragma unroll
        for (int i = 0; i < 32; i += 2) {
          const uint32_t a0 = run;
          run += uint32_t(__popc(wd[i]));
          packed[i / 2] = a0 | (run << 16);
          run += uint32_t(__popc(wd[i + 1]));
        }
#pragma unroll
        for (int t = 0; t < 4; ++t)
          reinterpret_cast<uint4*>(pre)[lane * 4 + (t ^ psw)] =
              make_uint4(packed[4 * t], packed[4 * t + 1], packed[4 * t + 2], packed[4 * t + 3]);
      }
      if (lane < kStageEntries / 8) reinterpret_cast<uint4*>(mq)[lane] = make_uint4(0u, 0u, 0u, 0u);
      wave_lds_sync();
      uint32_t dup = 0u;
      for_rows(sub, seg, [&](int32_t j, int qq, int) {
        if (uint32_t(j) < uint32_t(N)) {
          const uint32_t w = uint32_t(j) >> 5;
          const int id = int(pre[pre_at(w)]) + __popc(bm[bm_at(w)] & ((1u << (j & 31)) - 1u));
          const uint32_t bit = (1u << qq) << (16 * (id & 1));
          dup |= atomicOr(&mq[id >> 1], bit) & bit;
        }
      });
      if (wave_ballot(dup != 0u) != 0ull) return -1;
      wave_lds_sync();
      // Positions, lane by lane in word order (the counts are no longer read).
      read_words();
      int id = int(base);
#pragma unroll
      for (int i = 0; i < 32; ++i) {
        uint32_t m = wd[i];
        while (m != 0u) {
          const int b = __ffs(int(m)) - 1;
          s_ent[wave][id][kPosSlot] = __int_as_float(((lane * 32 + i) << 5) + b);
          ++id;
          m &= m - 1u;
        }
      }
      return total_u;
    };
    // The union of the index rows of the queries in gm (segment seg), staged
    // as the entries of one run: positions, key rows and query masks, padded
    // to whole chunks with entries that no query takes.  When the union of
    // all of gm does not fit, the lower half of the queries is tried, and so
    // on down to one query, whose row is its own union (slot order, an entry
    // per slot).  Returns the queries covered; n receives the entry count.
    auto build_union = [&](uint32_t gm, int64_t seg, int& n) -> uint32_t {
      flush_out();  // the value-row buffers hold the bitmap or the hash table next
      uint32_t sub = gm;
      for (;;) {
        const int nq = __popc(sub);
        int cnt;
        if (nq == 1) {
          for_rows(sub, seg, [&](int32_t j, int qq, int sl) {
            if (((sub >> qq) & 1u) != 0u && sl < topk) {
              const bool ok = uint32_t(j) < uint32_t(N);
              s_ent[wave][sl][kPosSlot] = __int_as_float(ok ? j : 0);
              s_um[wave][sl] = ok ? uint16_t(1u << qq) : uint16_t(0);
            }
          });
          cnt = topk;
        } else {
          cnt = N <= 65536 ? bitmap_union(sub, seg) : hash_union(sub, seg);
        }
        if (cnt >= 0) {
          n = cnt;
          break;
        }
        uint32_t half = 0u, m = sub;
        for (int c = 0; c < nq / 2; ++c) {
          half |= m & (0u - m);
          m &= m - 1u;
        }
        sub = half;
      }
      wave_lds_sync();
      // Key rows by position (zeros for the padding).
      const int padded = (n + kChunk - 1) / kChunk * kChunk;
      constexpr int kT = (kStageEntries + 63) / 64;
      int32_t pv[kT];
      uint2 kw[kT];
#pragma unroll
      for (int t = 0; t < kT; ++t) {
        const int e = t * 64 + lane;
        pv[t] = e < n ? __float_as_int(s_ent[wave][e < kStageEntries ? e : 0][kPosSlot]) : 0;
        kw[t] = e < n ? packed_key_row(k, seg * N + pv[t], total) : make_uint2(0u, 0u);
      }
#pragma unroll
      for (int t = 0; t < kT; ++t) {
        const int e = t * 64 + lane;
        if (e < padded) {
          *reinterpret_cast<float4*>(&s_ent[wave][e][0]) =
              make_float4(__uint_as_float(kw[t].x << 16), __uint_as_float(kw[t].x & 0xFFFF0000u),
                          __uint_as_float(kw[t].y << 16), __int_as_float(pv[t]));
          if (e >= n) s_um[wave][e] = uint16_t(0);
        }
      }
      wave_lds_sync();
      return sub;
    };

    // Queries that search one list form a group (nearly always the whole tile).
    while (pending != 0u) {
      const int leader = __ffs(int(pending)) - 1;
      const int64_t g_seg = __builtin_amdgcn_readlane(int32_t(my_seg), leader);
      const int g_lvl = __builtin_amdgcn_readlane(my_lvl, leader);
      uint32_t gmask = uint32_t(wave_ballot(my_i >= 0 && my_seg == g_seg && my_lvl == g_lvl)) & pending;
      int n_union = 0;  // index rows: the entries of the group's union
      if constexpr (kIdx) gmask = build_union(gmask, g_seg, n_union);
      pending &= ~gmask;
      const int32_t* lpos = sorted_pos + g_seg * N;
      const uint2* lkey = keys_full + g_seg * N;  // key rows in list order (d_k = 3)
      int32_t ln = int32_t(N);
      if (!kIdx && causal && g_lvl <= t_hi) {
        const int64_t off = g_seg * cap + ((int64_t(1) << g_lvl) - (int64_t(1) << t0));
        lpos = list_pos + off;
        lkey = keys_list + off;
        ln = int32_t(1) << g_lvl;
      }

      // A window outside the list (not produced by the bounds kernel) counts
      // as empty.
      const bool in_grp = ((gmask >> qn) & 1u) != 0u;
      const bool mine = in_grp && (kIdx || (0 <= my_a && my_a <= my_b && my_b < ln));
      const int32_t my_lim = causal ? pool_limit(my_i, chunk) : int32_t(N - 1);
      float qv[KD];
      if constexpr (kLateQ) {
#pragma unroll
        for (int a = 0; a < KD; ++a) qv[a] = 0.0f;
      } else if (kHist ? in_grp : mine) {
        if constexpr (DK == 3) {
          Row3<uint16_t>::load(q, g_seg * N + my_i, total, qv);
        } else {
#pragma unroll
          for (int a = 0; a < KD; ++a) qv[a] = a < dk ? bf16_bits_to_float(q[(g_seg * N + my_i) * dk + a]) : 0.0f;
        }
      } else {
#pragma unroll
        for (int a = 0; a < KD; ++a) qv[a] = 0.0f;
      }

      // acc[blk]: value columns 16 blk + 4kg .. 16 blk + 4kg + 3 of query qn.
      f32x4_t acc[E];
#pragma unroll
      for (int j = 0; j < E; ++j) acc[j] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
      float zpart = 0.0f;
      float run_max = -INFINITY;  // softmax variants: the query's largest logit so far
      const float qnorm = (kVar && score == kScoreNormDot) ? row_norm<KD>(qv, dk) : 0.0f;
      // The history-mean candidate starts the sums, in float32: its score
      // (counted once, by the kg = 0 lanes) and its weighted mean value in
      // this lane's output columns.  Under a softmax variant its logit
      // starts the running maximum and its weight is 1.
      if constexpr (kHist) {
        if (in_grp) {
          const int64_t gq = g_seg * N + my_i;
          float s_mean;
          if constexpr (kVar) {
            float mkv[KD];
#pragma unroll
            for (int a = 0; a < KD; ++a) mkv[a] = a < dk ? mk[gq * dk + a] : 0.0f;
            s_mean = variant_term<KD>(score, qv, mkv, dk, eps, rsd, qnorm);
            if (smax) {
              run_max = s_mean;
              s_mean = 1.0f;
            }
          } else {
            s_mean = mean_score<KD>(mk, gq, dk, qv, eps);
          }
          if (kg == 0) zpart = s_mean;
          const float* mrow = mv + gq * DV + 4 * kg;
#pragma unroll
          for (int j = 0; j < E; ++j) {
            const float4 m = *reinterpret_cast<const float4*>(mrow + 16 * j);
            acc[j] = f32x4_t{s_mean * m.x, s_mean * m.y, s_mean * m.z, s_mean * m.w};
          }
        }
      }
      const unsigned char* vbytes = reinterpret_cast<const unsigned char*>(v + g_seg * N * DV);
      const uint16_t* kseg = k + g_seg * N * dk;

      // Window and pool tests as single unsigned compares: entry r is in the
      // window when r - a <= b - a, its position in the pool when
      // pos <= limit (an entry past the list's end holds position 0 and lies
      // outside every window).
      const uint32_t span = mine ? uint32_t(my_b - my_a) : 0u;
      const int32_t a_eff = mine ? my_a : INT32_MIN;
      const uint32_t lim_u = uint32_t(my_lim);

      // Positions of this lane's 4 entries of staged chunk ch.
      auto entry_pos = [&](int ch, int32_t(&pvs)[4]) {
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) pvs[kk] = __float_as_int(s_ent[wave][ch * kChunk + kg * 4 + kk][kPosSlot]);
      };
      // Copy the value rows of staged chunk ch into LDS buffer `buf` (every
      // lane copies one piece of one row per instruction; a missing entry
      // reads row 0, finite by contract, and has weight 0).
      auto copy_rows = [&](int ch, unsigned char* buf, const int32_t(&pvs)[4]) {
#pragma unroll
        for (int j = 0; j < VS::kLoads; ++j) {
          int32_t pv;
          if constexpr (VS::kP > 16) {
            pv = __float_as_int(s_ent[wave][ch * kChunk + VS::entry_of_row(j * VS::kR + vq)][kPosSlot]);
          } else {
            // Entry 4kg + j*kOwn + vq % kOwn: one of this lane's own four.
            // Selected by the bits of r, among values first made opaque
            // (selects among the array's elements themselves are folded into
            // an indexed private array, which lives in scratch memory).
            const int u0 = j * VS::kOwn;
            const int r = vq % VS::kOwn;
            if constexpr (VS::kOwn == 1) {
              pv = pvs[u0];
            } else if constexpr (VS::kOwn == 2) {
              int32_t p0 = pvs[u0], p1 = pvs[u0 + 1];
              asm("" : "+v"(p0), "+v"(p1));
              pv = (r & 1) ? p1 : p0;
            } else {
              static_assert(VS::kOwn == 4, "d_v >= 32");
              int32_t p0 = pvs[u0], p1 = pvs[u0 + 1], p2 = pvs[u0 + 2], p3 = pvs[u0 + 3];
              asm("" : "+v"(p0), "+v"(p1), "+v"(p2), "+v"(p3));
              pv = (r & 2) ? ((r & 1) ? p3 : p2) : ((r & 1) ? p1 : p0);
            }
          }
          const Off boff = Off(pv) * Off(VS::kRowBytes) + Off(copy_off[j]);
          __builtin_amdgcn_global_load_lds(
              (const __attribute__((address_space(1))) void*)(vbytes + boff),
              (__attribute__((address_space(3))) void*)(buf + 1024 * j), 16, 0, 0);
        }
      };
      // Scores of this lane's 4 entries of staged chunk ch for its query,
      // split into bfloat16 parts.  The reciprocal is the hardware one
      // (1 ulp).  A score s is split as hi = bf16(s) and lo = bf16(s - hi),
      // both rounded to nearest even; s - hi is exact, so hi + lo is within
      // 2^-17 of s.
      auto score4 = [&](int cb, int ch, uint32_t(&bh)[2], uint32_t(&bl)[2], float& scl) {
        const int32_t r0 = (cb + ch) * kChunk;
        float sc[4];
        const float* krow = &s_ent[wave][ch * kChunk + kg * 4][0];
        int32_t pvs[4];
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) pvs[kk] = __float_as_int(krow[kk * KREC + kPosSlot]);
        scl = 1.0f;
        // Whether entry kk of this lane's four is in its query's window:
        // index rows, bit qn of the entry's query mask; list ranges, the
        // range and pool tests.
        uint2 qm = make_uint2(0u, 0u);
        if constexpr (kIdx) qm = *reinterpret_cast<const uint2*>(&s_um[wave][r0 + kg * 4]);
        if constexpr (!kVar) {
#pragma unroll
          for (int kk = 0; kk < 4; ++kk) {
            const int32_t r = r0 + kg * 4 + kk;
            const bool in = kIdx ? (((kk < 2 ? qm.x : qm.y) >> (16 * (kk & 1) + qn)) & 1u) != 0u
                                 : uint32_t(r) - uint32_t(a_eff) <= span && uint32_t(pvs[kk]) <= lim_u;
            // eps + the squared distance, eps first (one addition fewer).
            float d2 = eps;
#pragma unroll
            for (int a = 0; a < KD; ++a) {
              if (a < dk) {
                const float diff = qv[a] - krow[kk * KREC + a];
                d2 = fmaf(diff, diff, d2);
              }
            }
            const float rc = __builtin_amdgcn_rcpf(d2);
            sc[kk] = in ? rc : 0.0f;
            zpart += sc[kk];
          }
        } else {
          // Rounded as written: this lambda is inlined at several call sites.
#pragma clang fp contract(off)
          bool ins[4];
#pragma unroll
          for (int kk = 0; kk < 4; ++kk) {
            const int32_t r = r0 + kg * 4 + kk;
            ins[kk] = kIdx ? (((kk < 2 ? qm.x : qm.y) >> (16 * (kk & 1) + qn)) & 1u) != 0u
                           : uint32_t(r) - uint32_t(a_eff) <= span && uint32_t(pvs[kk]) <= lim_u;
            sc[kk] = variant_term<KD>(score, qv, krow + kk * KREC, dk, eps, rsd, qnorm);
          }
          if (smax) {
            // Online softmax: the chunk's largest logit of the query (its 4
            // lanes), the new running maximum, the factor for the sums so far.
            float cm = -INFINITY;
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) cm = ins[kk] ? fmaxf(cm, sc[kk]) : cm;
            cm = fmaxf(cm, __shfl_xor(cm, 16, 64));
            cm = fmaxf(cm, __shfl_xor(cm, 32, 64));
            const float nm = fmaxf(run_max, cm);
            if (nm > run_max) {
              scl = run_max > -INFINITY ? __expf(run_max - nm) : 0.0f;
              run_max = nm;
            }
            zpart *= scl;
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) sc[kk] = ins[kk] ? __expf(sc[kk] - run_max) : 0.0f;
          } else {
#pragma unroll
            for (int kk = 0; kk < 4; ++kk) sc[kk] = ins[kk] ? sc[kk] : 0.0f;
          }
#pragma unroll
          for (int kk = 0; kk < 4; ++kk) zpart += sc[kk];
        }
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const bf16x2_t h = {(__bf16)sc[2 * t], (__bf16)sc[2 * t + 1]};
          uint32_t hw = __builtin_bit_cast(uint32_t, h);
          asm("" : "+v"(hw));  // the packed pair, reused as is (one conversion)
          const bf16x2_t l = {(__bf16)(sc[2 * t] - __uint_as_float(hw << 16)),
                              (__bf16)(sc[2 * t + 1] - __uint_as_float(hw & 0xFFFF0000u))};
          bh[t] = hw;
          bl[t] = __builtin_bit_cast(uint32_t, l);
        }
      };
      // acc[blk] += V^T (columns 16 blk .. +15 x the chunk's 16 entries) *
      // S^T (entries x queries), the high then the low score parts; `a`
      // holds the chunk's transposing reads, issued before its scoring.
      auto mma = [&](s16x4_t(&a)[kTrCopies * E], const uint32_t(&bh)[2], const uint32_t(&bl)[2], float scl) {
        // Softmax variants: the sums so far to the chunk's running maximum.
        if (smax && wave_ballot(scl != 1.0f) != 0ull) {
#pragma unroll
          for (int j = 0; j < E; ++j) acc[j] *= scl;
        }
        if constexpr (kSplitK) {
          // Two 16 x 16 x 16 products per block on the same A fragment (the
          // 4 entries' values): against the high score parts of every block
          // first, then against the low parts, so that consecutive products
          // into one accumulator stand E products apart.
          Frag b_hi, b_lo;
          b_hi.w[0] = bh[0];
          b_hi.w[1] = bh[1];
          b_lo.w[0] = bl[0];
          b_lo.w[1] = bl[1];
          read_tr_wait<kTrCopies * E>(a);
#pragma unroll
          for (int j = 0; j < E; ++j) acc[j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a[j], b_hi.v, acc[j], 0, 0, 0);
#pragma unroll
          for (int j = 0; j < E; ++j) acc[j] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a[j], b_lo.v, acc[j], 0, 0, 0);
        } else {
          // One 16 x 16 x 32 product per block: its 32 K slots hold the 4
          // entries' values twice against their high, then their low score
          // parts (B).
          Frag8 b;
          b.w[0] = bh[0];
          b.w[1] = bh[1];
          b.w[2] = bl[0];
          b.w[3] = bl[1];
          read_tr_wait<kTrCopies * E>(a);
#pragma unroll
          for (int j = 0; j < E; ++j) {
            const bf16x8_t a8 = __builtin_bit_cast(
                bf16x8_t, __builtin_shufflevector(a[kTrCopies * j], a[kTrCopies * j + kTrCopies - 1], 0, 1, 2, 3, 4,
                                                  5, 6, 7));
            acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a8, b.v, acc[j], 0, 0, 0);
          }
        }
      };

      // The chunks that meet some window, in list order: run by run (a run is
      // a stretch of chunks the windows cover without a gap; nearly always one
      // per tile), each run kStage chunks at a time.  Index rows: the staged
      // union is one run of at most kStage chunks.
      const int a_ch = !mine ? INT32_MAX : kIdx ? (n_union > 0 ? 0 : INT32_MAX) : my_a / kChunk;
      const int b_ch = !mine ? INT32_MIN : kIdx ? (n_union + kChunk - 1) / kChunk - 1 : my_b / kChunk;
      unsigned char* const v0 = s_v[wave];
      unsigned char* const v1 = s_v[wave] + VS::kBytes;
      for (int c = wave_min_int(a_ch); c != INT32_MAX;) {
        // Extend the run to the last chunk of every window that starts in it
        // or right after it.
        int e = c - 1;
        for (;;) {
          const int e2 = wave_max_int(a_ch <= e + 1 ? b_ch : e);
          if (e2 == e) break;
          e = e2;
        }
        for (int cb = c; cb <= e; cb += kStage) {
          const int nch = e - cb + 1 < kStage ? e - cb + 1 : kStage;
          // Stage the positions and key rows of list entries cb*kChunk ..
          // (cb + nch)*kChunk - 1 (index rows: staged with the union).
          if constexpr (!kIdx) {
            const int32_t base = cb * kChunk;
            // This lane's query row as bfloat16 bits (row 0 for a lane
            // without a window: read, not used).  The opaque row index keeps
            // the read here rather than hoisted out of the loop, where it
            // would wait alone.
            uint32_t q3[3];
            if constexpr (kLateQ) {
              int32_t qr = mine ? int32_t(g_seg * N + my_i) : 0;  // rows < 2^31
              asm volatile("" : "+v"(qr));
              const int64_t qe = int64_t(qr) * 3;
#pragma unroll
              for (int a = 0; a < 3; ++a) q3[a] = q[qe + a];
            }
            int32_t pv[kStageEntries / 64];
            uint2 kw[kStageEntries / 64];  // d_k = 3: key rows read in list order with the positions
#pragma unroll
            for (int t = 0; t < kStageEntries / 64; ++t) {
              const int e_ = t * 64 + lane;
              const int32_t r = base + e_;
              pv[t] = 0;  // an entry past the list's end: outside every window
              kw[t] = make_uint2(0u, 0u);
              if (e_ < nch * kChunk && r < ln) {
                pv[t] = lpos[r];
                if constexpr (DK == 3) kw[t] = lkey[r];
              }
            }
            flush_out();
            if constexpr (kLateQ) {
              // Converted here, before any value-row copy is issued (a wait
              // for the row after one would also wait for that copy).
#pragma unroll
              for (int a = 0; a < 3; ++a) qv[a] = mine ? __uint_as_float(q3[a] << 16) : 0.0f;
              asm volatile("" ::"v"(qv[0]), "v"(qv[1]), "v"(qv[2]));
            }
#pragma unroll
            for (int t = 0; t < kStageEntries / 64; ++t) {
              const int e_ = t * 64 + lane;
              if (e_ < nch * kChunk) {
                float kv[KD];
                if constexpr (DK == 3) {
                  kv[0] = __uint_as_float(kw[t].x << 16);
                  kv[1] = __uint_as_float(kw[t].x & 0xFFFF0000u);
                  kv[2] = __uint_as_float(kw[t].y << 16);
                } else {
#pragma unroll
                  for (int a = 0; a < KD; ++a)
                    kv[a] = a < dk ? bf16_bits_to_float(kseg[int64_t(pv[t]) * dk + a]) : 0.0f;
                }
                if constexpr (DK == 3) {
                  *reinterpret_cast<float4*>(&s_ent[wave][e_][0]) = make_float4(kv[0], kv[1], kv[2], __int_as_float(pv[t]));
                } else {
#pragma unroll
                  for (int a = 0; a < KD4; a += 4)
                    *reinterpret_cast<float4*>(&s_ent[wave][e_][a]) =
                        make_float4(kv[a], a + 1 < KD ? kv[a + 1] : 0.0f, a + 2 < KD ? kv[a + 2] : 0.0f,
                                    a + 3 < KD ? kv[a + 3] : 0.0f);
                  s_ent[wave][e_][kPosSlot] = __int_as_float(pv[t]);
                }
              }
            }
          }
          wave_lds_sync();

          // Chunk ch+1's value rows are copied while chunk ch is scored and
          // multiplied (even chunks in v0, odd chunks in v1).
          // Past the stage's last chunk the other buffer receives a copy of
          // the current chunk's rows again, so that exactly one chunk's
          // copies are always in flight behind the one being read.
          // Chunk ch's transposing reads are issued before its scoring and
          // waited for after it.
          int32_t pv4[4];
          uint32_t bh[2], bl[2];
          float scl;
          s16x4_t a[kTrCopies * E];
          entry_pos(0, pv4);
          copy_rows(0, v0, pv4);
          for (int ch = 0; ch < nch; ch += 2) {
            const int c1 = ch + 1 < nch ? ch + 1 : ch;
            entry_pos(c1, pv4);
            copy_rows(c1, v1, pv4);
            read_tr_issue<E, kTrCopies, 0, VS::kLoads>(tr_addr, a);
            score4(cb, ch, bh, bl, scl);
            mma(a, bh, bl, scl);
            if (ch + 1 >= nch) break;
            const int c2 = ch + 2 < nch ? ch + 2 : ch + 1;
            entry_pos(c2, pv4);
            copy_rows(c2, v0, pv4);
            read_tr_issue<E, kTrCopies, VS::kBytes, VS::kLoads>(tr_addr, a);
            score4(cb, ch + 1, bh, bl, scl);
            mma(a, bh, bl, scl);
          }
          // Every copy has landed before the buffers are refilled.
          asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
          wave_lds_sync();
        }
        c = wave_min_int(a_ch > e ? a_ch : INT32_MAX);
      }

      // Normalise, then leave the rows in LDS for flush_out.  Lane (qn, kg)
      // holds columns 16 blk + 4kg .. + 3 of query qn for every block; each
      // query's row will leave as whole 16-byte pieces, kOutP lanes per row
      // and full cache lines.
      float z = zpart;
      z += __shfl_xor(z, 16, 64);
      z += __shfl_xor(z, 32, 64);
      const float inv = z > 0.0f ? 1.0f / z : 0.0f;
      flush_out();  // an earlier group's rows, when this group staged nothing
      unsigned char* const so = s_v[wave];
#pragma unroll
      for (int j = 0; j < E; ++j) {
        // Rounded to bfloat16 (nearest even), two values per conversion.
        const bf16x2_t p0 = {(__bf16)(acc[j][0] * inv), (__bf16)(acc[j][1] * inv)};
        const bf16x2_t p1 = {(__bf16)(acc[j][2] * inv), (__bf16)(acc[j][3] * inv)};
        const int piece = 2 * j + (kg >> 1);
        *reinterpret_cast<uint2*>(so + qn * kOutRowB + 16 * (piece ^ (qn % kOutP)) + 8 * (kg & 1)) =
            make_uint2(__builtin_bit_cast(uint32_t, p0), __builtin_bit_cast(uint32_t, p1));
      }
      if (lane < kTileQ) s_orow[wave][lane] = in_grp ? int32_t(g_seg * N + my_i) : -1;  // rows < 2^31
      wave_lds_sync();
      out_pending = true;
    }
  }
  flush_out();
}

template <int DV, int DK>
hipError_t launch_tile_t(const uint16_t* q, const uint16_t* k, const uint16_t* v, int64_t S, int64_t N, int dk,
                         int topk, bool causal, int chunk, const int32_t* perm, const int32_t* list_pos,
                         const int32_t* q_order, const int2* bounds, const uint2* keys_full, const uint2* keys_list,
                         int score, float eps, HistMean hm, uint16_t* out, hipStream_t stream) {
  const ListPlan lp = list_plan(N, topk);
  const int64_t total = S * N;
  const int64_t tiles = ceil_div(total, kTileQ);
  const int64_t want = ceil_div(tiles, kTileWaves);
  const unsigned blocks = unsigned(want < (int64_t(1) << 20) ? want : (int64_t(1) << 20));
  const bool off32 = N * int64_t(DV) <= int64_t(0x7FFFFFFF);
#define ZETA_TILE_LAUNCH(OFF, HIST, MODE)                                                                          \
  hipLaunchKernelGGL((select_attend_tile_kernel<DV, DK, OFF, HIST, MODE, false>), dim3(blocks), dim3(kTileWaves * 64), \
                     0, stream, q, k, v, perm, list_pos, q_order, bounds, keys_full, keys_list, total, N, dk,         \
                     causal ? 1 : 0, chunk, lp.t0, lp.t_hi, lp.cap, eps, hm.k, hm.v, out, nullptr, 0)
#define ZETA_TILE_LAUNCH4(MODE)             \
  if (off32) {                              \
    if (hist)                               \
      ZETA_TILE_LAUNCH(true, true, MODE);   \
    else                                    \
      ZETA_TILE_LAUNCH(true, false, MODE);  \
  } else {                                  \
    if (hist)                               \
      ZETA_TILE_LAUNCH(false, true, MODE);  \
    else                                    \
      ZETA_TILE_LAUNCH(false, false, MODE); \
  }
  const bool hist = hm.k != nullptr;
  // The score variants are compiled for d_k = 3 only.
  if constexpr (DK == 3) {
    switch (score) {
      case kScoreDot:
        ZETA_TILE_LAUNCH4(kScoreDot)
        return hipGetLastError();
      case kScoreNegEuclid:
        ZETA_TILE_LAUNCH4(kScoreNegEuclid)
        return hipGetLastError();
      case kScoreInvEuclid:
        ZETA_TILE_LAUNCH4(kScoreInvEuclid)
        return hipGetLastError();
      case kScoreNormDot:
        ZETA_TILE_LAUNCH4(kScoreNormDot)
        return hipGetLastError();
      default:
        break;
    }
  }
  ZETA_TILE_LAUNCH4(kScoreCauchy)
#undef ZETA_TILE_LAUNCH4
#undef ZETA_TILE_LAUNCH
  return hipGetLastError();
}

template <int DV>
hipError_t launch_tile_dk(const uint16_t* q, const uint16_t* k, const uint16_t* v, int64_t S, int64_t N, int dk,
                          int topk, bool causal, int chunk, const int32_t* perm, const int32_t* list_pos,
                          const int32_t* q_order, const int2* bounds, const uint2* keys_full, const uint2* keys_list,
                          int score, float eps, HistMean hm, uint16_t* out, hipStream_t stream) {
  if (dk == 3)
    return launch_tile_t<DV, 3>(q, k, v, S, N, dk, topk, causal, chunk, perm, list_pos, q_order, bounds, keys_full,
                                keys_list, score, eps, hm, out, stream);
  return launch_tile_t<DV, 0>(q, k, v, S, N, dk, topk, causal, chunk, perm, list_pos, q_order, bounds, keys_full,
                              keys_list, score, eps, hm, out, stream);
}

// The attend call's matrix-core tiles (d_k = 3): 16 consecutive queries of
// the processing order per wavefront, over the union of their index rows.
template <int DV>
hipError_t launch_idx_tile_t(const uint16_t* q, const uint16_t* k, const uint16_t* v, int64_t S, int64_t N,
                             int topk, const int32_t* idx, const int32_t* q_order, int score, float eps, HistMean hm,
                             uint16_t* out, hipStream_t stream) {
  const int64_t total = S * N;
  const int64_t tiles = ceil_div(total, kTileQ);
  const int64_t want = ceil_div(tiles, kTileWaves);
  const unsigned blocks = unsigned(want < (int64_t(1) << 20) ? want : (int64_t(1) << 20));
  const bool off32 = N * int64_t(DV) <= int64_t(0x7FFFFFFF);
#define ZETA_IDX_LAUNCH(OFF, HIST, MODE)                                                                         \
  hipLaunchKernelGGL((select_attend_tile_kernel<DV, 3, OFF, HIST, MODE, true>), dim3(blocks), dim3(kTileWaves * 64), \
                     0, stream, q, k, v, nullptr, nullptr, q_order, nullptr, nullptr, nullptr, total, N, 3, 0, 0, 0, \
                     0, 0, eps, hm.k, hm.v, out, idx, topk)
#define ZETA_IDX_LAUNCH4(MODE)            \
  if (off32) {                            \
    if (hist)                             \
      ZETA_IDX_LAUNCH(true, true, MODE);  \
    else                                  \
      ZETA_IDX_LAUNCH(true, false, MODE); \
  } else {                                \
    if (hist)                             \
      ZETA_IDX_LAUNCH(false, true, MODE); \
    else                                  \
      ZETA_IDX_LAUNCH(false, false, MODE);\
  }
  const bool hist = hm.k != nullptr;
  switch (score) {
    case kScoreDot:
      ZETA_IDX_LAUNCH4(kScoreDot)
      break;
    case kScoreNegEuclid:
      ZETA_IDX_LAUNCH4(kScoreNegEuclid)
      break;
    case kScoreInvEuclid:
      ZETA_IDX_LAUNCH4(kScoreInvEuclid)
      break;
    case kScoreNormDot:
      ZETA_IDX_LAUNCH4(kScoreNormDot)
      break;
    default:
      ZETA_IDX_LAUNCH4(kScoreCauchy)
      break;
  }
#undef ZETA_IDX_LAUNCH4
#undef ZETA_IDX_LAUNCH
  return hipGetLastError();
}

}  // namespace

bool tile_supports(int dv) { return tile_dv(dv); }

hipError_t launch_attend_idx_tile(const void* q, const void* k, const void* v, int64_t S, int64_t N, int dv, int topk,
                                  const int32_t* idx, const int32_t* q_order, int score, float eps, HistMean hm,
                                  void* out, hipStream_t stream) {
  const uint16_t* qq = static_cast<const uint16_t*>(q);
  const uint16_t* kk = static_cast<const uint16_t*>(k);
  const uint16_t* vv = static_cast<const uint16_t*>(v);
  uint16_t* oo = static_cast<uint16_t*>(out);
  switch (dv) {
    case 32:
      return launch_idx_tile_t<32>(qq, kk, vv, S, N, topk, idx, q_order, score, eps, hm, oo, stream);
    case 64:
      return launch_idx_tile_t<64>(qq, kk, vv, S, N, topk, idx, q_order, score, eps, hm, oo, stream);
    case 128:
      return launch_idx_tile_t<128>(qq, kk, vv, S, N, topk, idx, q_order, score, eps, hm, oo, stream);
    default:
      return hipErrorInvalidValue;
  }
}

hipError_t launch_tile_windows(const void* k, int64_t S, int64_t N, int dk, int topk, bool causal, int chunk,
                               const uint32_t* q_codes, const uint32_t* sorted_codes, const int32_t* perm,
                               const uint32_t* list_codes, const int32_t* list_pos, const int32_t* q_order,
                               int32_t* idx_out, int2* bounds, uint2* keys_full, uint2* keys_list, bool keys_built,
                               hipStream_t stream) {
  const ListPlan lp = list_plan(N, topk);
  const int64_t total = S * N;
  if (dk == 3 && !keys_built) {
    // Prefix lists exist only for causal calls with levels.
    const bool have_lists = causal && lp.levels > 0 && list_pos != nullptr;
    const int64_t cap = have_lists ? lp.cap : 0;
    const unsigned blocks = unsigned(ceil_div(total + S * cap, 256));
    hipLaunchKernelGGL(list_keys_kernel, dim3(blocks), dim3(256), 0, stream, static_cast<const uint16_t*>(k), total, N,
                       perm, have_lists ? list_pos : nullptr, cap, S, keys_full, keys_list);
  }
  {
    const int64_t runs = ceil_div(total, 64);
    const int64_t want = ceil_div(runs, kBndWaves);
    const unsigned blocks = unsigned(want < (int64_t(1) << 20) ? want : (int64_t(1) << 20));
    // Positions fit 16 bits when the segment has at most 65536 rows.
    auto kern = N <= 65536 ? window_bounds_kernel<true> : window_bounds_kernel<false>;
    hipLaunchKernelGGL(kern, dim3(blocks), dim3(kBndWaves * 64), 0, stream, q_codes, sorted_codes, perm, list_codes,
                       list_pos, q_order, total, N, topk, causal ? 1 : 0, chunk, lp.t0, lp.t_hi, lp.cap, bounds);
  }
  if (idx_out != nullptr) {
    const int64_t groups = ceil_div(total, 16);
    const int64_t want = ceil_div(groups, kRowsWaves);
    const unsigned blocks = unsigned(want < (int64_t(1) << 20) ? want : (int64_t(1) << 20));
    hipLaunchKernelGGL(idx_rows_kernel, dim3(blocks), dim3(kRowsWaves * 64), 0, stream, sorted_codes, perm,
                       list_codes, list_pos, q_order, bounds, total, N, topk, causal ? 1 : 0, chunk, lp.t0, lp.t_hi,
                       lp.cap, idx_out);
  }
  return hipGetLastError();
}

hipError_t launch_select_attend_tile(const void* q, const void* k, const void* v, int64_t S, int64_t N, int dk, int dv,
                                     int topk, bool causal, int chunk, const uint32_t* q_codes,
                                     const uint32_t* sorted_codes,
                                     const int32_t* perm, const uint32_t* list_codes, const int32_t* list_pos,
                                     const int32_t* q_order, int score, float eps, HistMean hm, void* out,
                                     int32_t* idx_out, int2* bounds, uint2* keys_full, uint2* keys_list,
                                     bool keys_built, hipStream_t stream) {
  const hipError_t e = launch_tile_windows(k, S, N, dk, topk, causal, chunk, q_codes, sorted_codes, perm, list_codes,
                                           list_pos, q_order, idx_out, bounds, keys_full, keys_list, keys_built,
                                           stream);
  if (e != hipSuccess) return e;
  const uint16_t* qq = static_cast<const uint16_t*>(q);
  const uint16_t* kk = static_cast<const uint16_t*>(k);
  const uint16_t* vv = static_cast<const uint16_t*>(v);
  uint16_t* oo = static_cast<uint16_t*>(out);
#define ZETA_TILE_CASE(DVV) \
  case DVV:                 \
    return launch_tile_dk<DVV>(qq, kk, vv, S, N, dk, topk, causal, chunk, perm, list_pos, q_order, bounds, keys_full, \
                               keys_list, score, eps, hm, oo, stream);
  switch (dv) {
    ZETA_TILE_CASE(32)
    ZETA_TILE_CASE(64)
    ZETA_TILE_CASE(128)
    ZETA_TILE_CASE(256)
    default:
      return hipErrorInvalidValue;
  }
#undef ZETA_TILE_CASE
}

}  // namespace zeta
