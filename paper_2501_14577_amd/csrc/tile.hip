// Candidate selection and Cauchy-softmax attention for bfloat16 inputs, 16
// queries at a time on the matrix cores (Section 3.2.2 and Algorithm 1,
// Steps 3-5, for the windows; Section 3.3, equation cauchy, Section 3.4 and
// Appendix E.1 for the attention).
//
// A query's window is a run of its sorted list: every in-pool entry of the
// list range [a, b] around its insertion point (select_window_bounds).  In the
// processing order of zeta_query_order, 16 consecutive queries search one list
// at nearby insertion points, so their ranges overlap: together they span
// about twice the window length where gathering per query would read 16
// windows.
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
#include "attend_device.h"
#include "device_common.h"
#include "kernels.h"
#include "layout.h"
#include "select_device.h"
#include "tile_device.h"

namespace zeta {
namespace {

constexpr int kTileQ = 16;     // queries per tile (product columns)
constexpr int kChunk = 16;     // list entries per product step
constexpr int kTileWaves = 4;  // wavefronts per block

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
// or when its query searches another list.  With idx_out the run's windows
// are also written as position rows, one wavefront-wide pass per query.
constexpr int kBndWaves = 4;
constexpr int kRegion = 512;   // list entries staged per wavefront
constexpr int kMargin = 192;    // of them before the run's first insertion point

// Each wavefront's copy of a list range, in LDS.  Declared at file scope and
// indexed directly, so that every access compiles to an LDS instruction (a
// pointer kept in a struct would lose the address space and go through the
// slower flat path).
__shared__ uint32_t s_bnd_codes[kBndWaves][kRegion];
__shared__ int32_t s_bnd_pos[kBndWaves][kRegion];

struct LaneList {
  const uint32_t* codes;
  const int32_t* pos;
  int wave;
  int32_t n, limit, r0, r1;  // [r0, r1): the range copied to LDS (empty when not staged)
};

constexpr int kScanStep = 16;  // list entries examined per step of lane_scan

// Bit j set when entry lo + j is in the query's pool.  A block inside the LDS
// copy is read from there; any other block from the list itself, with entries
// outside [0, n) counted out.  Both branches are straight-line code, so a
// block's reads issue together and the lane waits once for them.
__device__ __forceinline__ uint32_t pool_bits(const LaneList& L, int32_t lo) {
  uint32_t mask = 0u;
  if (lo >= L.r0 && lo + kScanStep <= L.r1) {
    const int32_t b = lo - L.r0;
#pragma unroll
    for (int j = 0; j < kScanStep; ++j) mask |= (s_bnd_pos[L.wave][b + j] <= L.limit ? 1u : 0u) << j;
  } else {
    using G = __attribute__((address_space(1))) const int32_t;
    G* gp = (G*)L.pos;
    int32_t v[kScanStep];
#pragma unroll
    for (int j = 0; j < kScanStep; ++j) {
      const int32_t x = lo + j;
      v[j] = gp[x < 0 ? 0 : (x < L.n ? x : L.n - 1)];
    }
#pragma unroll
    for (int j = 0; j < kScanStep; ++j) {
      const int32_t x = lo + j;
      mask |= (x >= 0 && x < L.n && v[j] <= L.limit ? 1u : 0u) << j;
    }
  }
  return mask;
}

// Scan from entry e in direction dir (+1 or -1) for up to `need` in-pool
// entries beyond the `got` already taken; records the first and last entry
// taken (first only when got is 0).  Returns the new count; `e` ends just
// past the last entry taken, or past the list's end.  Entries are examined
// kScanStep at a time as a bit mask (bit j: entry e + dir*j is in the pool);
// only the block where the count is reached is searched bit by bit.  Called
// only with n > 0.
__device__ __forceinline__ int lane_scan(const LaneList& L, int32_t& e, int dir, int need, int got, int32_t& first,
                                         int32_t& last) {
  while (got < need && e >= 0 && e < L.n) {
    // Lowest index of the block, in ascending list order.
    const int32_t lo = dir > 0 ? e : e - (kScanStep - 1);
    uint32_t mask = pool_bits(L, lo);
    // Bit j of `mask` is entry lo + j; reorder so bit j is entry e + dir*j.
    if (dir < 0) mask = __builtin_bitreverse32(mask) >> (32 - kScanStep);
    const int cnt = __popc(mask);
    if (cnt == 0) {
      e += dir * kScanStep;
      continue;
    }
    if (got == 0) first = e + dir * (__ffs(int(mask)) - 1);
    if (got + cnt < need) {
      got += cnt;
      last = e + dir * (31 - __clz(int(mask)));
      e += dir * kScanStep;
    } else {
      // The (need - got)-th set bit ends the scan.
      uint32_t m = mask;
      for (int t = 1; t < need - got; ++t) m &= m - 1u;
      const int j = __ffs(int(m)) - 1;
      last = e + dir * j;
      e = last + dir;
      got = need;
    }
  }
  return got;
}

__global__ void __launch_bounds__(kBndWaves * 64)
    window_bounds_kernel(const uint32_t* __restrict__ q_codes, const uint32_t* __restrict__ sorted_codes,
                         const int32_t* __restrict__ perm, const uint32_t* __restrict__ list_codes,
                         const int32_t* __restrict__ list_pos, const int32_t* __restrict__ order, int64_t total,
                         int64_t N, int topk, int causal, int chunk, int t0, int t_hi, int64_t cap,
                         int2* __restrict__ bounds, int32_t* __restrict__ idx_out) {
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
      seg = slot / N;
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
    int2 res = make_int2(0, -1);
    if (vmask != 0ull) {
      // Stage the leader's list around the leader's insertion point.
      const int leader = __ffsll((unsigned long long)vmask) - 1;
      const uint32_t* g_codes = readlane_ptr(Lq.codes, leader);
      const int32_t* g_pos = readlane_ptr(Lq.pos, leader);
      const int32_t g_n = __builtin_amdgcn_readlane(Lq.n, leader);
      const uint32_t g_key = uint32_t(__builtin_amdgcn_readlane(int32_t(key), leader));
      const int32_t p0 = wave_lower_bound(g_codes, 0, g_n, g_key, lane);
      const int32_t r0 = p0 - kMargin > 0 ? p0 - kMargin : 0;
      const int32_t r1 = r0 + kRegion < g_n ? r0 + kRegion : g_n;
      {
        uint32_t cv[kRegion / 64];
        int32_t pv[kRegion / 64];
#pragma unroll
        for (int t = 0; t < kRegion / 64; ++t) {
          const int32_t e = r0 + t * 64 + lane;
          cv[t] = e < r1 ? g_codes[e] : 0u;
          pv[t] = e < r1 ? g_pos[e] : 0;
        }
#pragma unroll
        for (int t = 0; t < kRegion / 64; ++t) {
          s_bnd_codes[wave][t * 64 + lane] = cv[t];
          s_bnd_pos[wave][t * 64 + lane] = pv[t];
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
        int got_r = lane_scan(L, cur_r, +1, need_r, 0, r_first, r_last);
        const int need_l = half + (need_r - got_r);
        int32_t cur_l = p - 1;
        const int got_l = lane_scan(L, cur_l, -1, need_l, 0, l_near, l_far);
        if (got_l < need_l && got_r == need_r) got_r = lane_scan(L, cur_r, +1, topk - got_l, got_r, r_first, r_last);
        if (got_l + got_r > 0) res = make_int2(got_l > 0 ? l_far : r_first, got_r > 0 ? r_last : l_near);
      }
    }  // some lane has a pool
    if (slot < total) bounds[slot] = res;

    if (idx_out != nullptr) {
      // The windows' positions in list order, then -1: one query at a time.
      for (uint64_t m = qmask; m != 0ull; m &= m - 1ull) {
        const int u = __ffsll((unsigned long long)m) - 1;
        const int32_t* upos = readlane_ptr(L.pos, u);
        const int32_t ua = __builtin_amdgcn_readlane(res.x, u), ub = __builtin_amdgcn_readlane(res.y, u);
        const int32_t ulim = __builtin_amdgcn_readlane(L.limit, u);
        const int32_t ui = __builtin_amdgcn_readlane(my_i, u);
        const int64_t useg = (run * 64 + u) / N;
        int32_t* row = idx_out + (useg * N + ui) * int64_t(topk);
        int cnt = 0;
        for (int32_t e0 = ua; e0 <= ub; e0 += 64) {
          const int32_t e = e0 + lane;
          const int32_t pv = e <= ub ? upos[e] : INT32_MAX;
          const bool ok = pv <= ulim;
          const uint64_t bal = wave_ballot(ok);
          if (ok) row[cnt + int(lanes_below(bal))] = pv;
          cnt += __popcll(bal);
        }
        for (int c = cnt + lane; c < topk; c += 64) row[c] = -1;
      }
    }
    wave_lds_sync();
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

template <int DV, int DK, bool kOff32, bool kHist, int kMode>
__global__ void __launch_bounds__(kTileWaves * 64)
    __attribute__((amdgpu_waves_per_eu((DV <= 128 && kMode != kScoreCauchy) ? 3 : 1)))
    select_attend_tile_kernel(const uint16_t* __restrict__ q, const uint16_t* __restrict__ k,
                              const uint16_t* __restrict__ v, const int32_t* __restrict__ sorted_pos,
                              const int32_t* __restrict__ list_pos, const int32_t* __restrict__ order,
                              const int2* __restrict__ bounds, const uint2* __restrict__ keys_full,
                              const uint2* __restrict__ keys_list, int64_t total, int64_t N, int dk_rt, int causal,
                              int chunk, int t0, int t_hi, int64_t cap, float eps,
                              const float* __restrict__ mk, const float* __restrict__ mv, uint16_t* __restrict__ out) {
  constexpr int E = DV / 16;  // value elements per lane and row; also product blocks per chunk
  constexpr int W = E / 2;    // 32-bit words per lane and row
  constexpr int KD = DK > 0 ? DK : kMaxDk;
  constexpr int kStageEntries = DK == 3 ? 512 : 128;  // entries whose positions and key rows are staged at once
  constexpr int kStage = kStageEntries / kChunk;
  static_assert(E >= 2 && E % 2 == 0, "d_v must be a multiple of 32");
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

  // Key rows padded to a multiple of 4 floats, so 4 consecutive entries'
  // positions and each key row are whole 16-byte LDS reads.
  constexpr int KD4 = (KD + 3) / 4 * 4;
  __shared__ __align__(16) int32_t s_pos[kTileWaves][kStageEntries];
  __shared__ __align__(16) float s_k[kTileWaves][kStageEntries][KD4];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int qn = lane & (kTileQ - 1);  // this lane's query in the tile; also its value column in a block
  const int kg = lane >> 4;            // this lane's entries in a chunk: 4kg .. 4kg+3
  const int64_t tiles = (total + kTileQ - 1) / kTileQ;
  const int64_t nb = gridDim.x;

  for (int64_t blk = xcd_contiguous_block(blockIdx.x, nb); blk * kTileWaves < tiles; blk += nb) {
    const int64_t tile = blk * kTileWaves + wave;
    if (tile >= tiles) continue;

    // The tile's queries and windows: lanes with equal qn hold the same one.
    int32_t my_i = -1;
    int64_t my_seg = 0;
    int my_lvl = 0;
    int32_t my_a = 0, my_b = -1;
    {
      const int64_t sl = tile * kTileQ + qn;
      if (sl < total) {
        const int64_t sg = sl / N;
        const int64_t ii = order != nullptr ? int64_t(order[sl]) : sl - sg * N;
        if (ii >= 0 && ii < N) {
          my_i = int32_t(ii);
          my_seg = sg;
          my_lvl = causal ? pool_level(pool_limit(my_i, chunk), t0, t_hi) : 0;
          const int2 bb = bounds[sl];
          my_a = bb.x;
          my_b = bb.y;
        }
      }
    }
    uint32_t pending = uint32_t(wave_ballot(my_i >= 0)) & 0xFFFFu;

    // Queries that search one list form a group (nearly always the whole tile).
    while (pending != 0u) {
      const int leader = __ffs(int(pending)) - 1;
      const int64_t g_seg = __builtin_amdgcn_readlane(int32_t(my_seg), leader);
      const int g_lvl = __builtin_amdgcn_readlane(my_lvl, leader);
      const uint32_t gmask =
          uint32_t(wave_ballot(my_i >= 0 && my_seg == g_seg && my_lvl == g_lvl)) & pending;
      pending &= ~gmask;
      const int32_t* lpos = sorted_pos + g_seg * N;
      const uint2* lkey = keys_full + g_seg * N;  // key rows in list order (d_k = 3)
      int32_t ln = int32_t(N);
      if (causal && g_lvl <= t_hi) {
        const int64_t off = g_seg * cap + ((int64_t(1) << g_lvl) - (int64_t(1) << t0));
        lpos = list_pos + off;
        lkey = keys_list + off;
        ln = int32_t(1) << g_lvl;
      }

      // A window outside the list (not produced by the bounds kernel) counts
      // as empty.
      const bool in_grp = ((gmask >> qn) & 1u) != 0u;
      const bool mine = in_grp && 0 <= my_a && my_a <= my_b && my_b < ln;
      const int32_t my_lim = causal ? pool_limit(my_i, chunk) : int32_t(N - 1);
      float qv[KD];
      if (kHist ? in_grp : mine) {
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

      f32x4_t acc[E];
#pragma unroll
      for (int j = 0; j < E; ++j) acc[j] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
      float zpart = 0.0f;
      float run_max = -INFINITY;  // softmax variants: the query's largest logit so far
      const float qnorm = (kVar && score == kScoreNormDot) ? row_norm<KD>(qv, dk) : 0.0f;
      // The history-mean candidate starts the sums, in float32: its score
      // (counted once, by the kg = 0 lanes) and its weighted mean value in
      // this lane's output elements kg*4E .. kg*4E + 4E - 1.  Under a softmax
      // variant its logit starts the running maximum and its weight is 1.
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
          const float* mrow = mv + gq * DV + kg * 4 * E;
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < E; j += 4) {
              const float4 m = *reinterpret_cast<const float4*>(mrow + i * E + j);
              acc[j][i] = s_mean * m.x;
              acc[j + 1][i] = s_mean * m.y;
              acc[j + 2][i] = s_mean * m.z;
              acc[j + 3][i] = s_mean * m.w;
            }
        }
      }
      const uint16_t* vseg = v + g_seg * N * DV;
      const unsigned char* vbytes = reinterpret_cast<const unsigned char*>(vseg);
      const uint16_t* kseg = k + g_seg * N * dk;
      const Off col = Off(qn * E);

      // Window and pool tests as single unsigned compares: entry r is in the
      // window when r - a <= b - a, its position in the pool when
      // pos <= limit (an entry past the list's end holds position 0 and lies
      // outside every window).
      const uint32_t span = mine ? uint32_t(my_b - my_a) : 0u;
      const int32_t a_eff = mine ? my_a : INT32_MIN;
      const uint32_t lim_u = uint32_t(my_lim);

      // Scores of this lane's 4 entries of staged chunk `ch` for its query,
      // split into bfloat16 parts, and the loads of the entries' value rows.
      // Branch-free, so that loads in flight can be counted across chunks: a
      // chunk index at or past nch scores nothing, and every lane loads a
      // row (a missing entry reads row 0, finite by contract; a row no query
      // takes has weight 0).  The reciprocal is the hardware one (1 ulp).  A
      // score s is split as hi = bf16(s) and lo = bf16(s - hi), both rounded
      // to nearest even; s - hi is exact, so hi + lo is within 2^-17 of s.
      auto prep = [&](int cb, int ch, int nch_, uint32_t(&raw)[4][W], uint32_t(&bh)[2], uint32_t(&bl)[2],
                      float& scl) {
        const bool live = ch < nch_;
        const int chc = live ? ch : 0;
        const int32_t r0 = (cb + chc) * kChunk;
        float sc[4];
        int32_t pvs[4];
        {
          const int4 p4 = *reinterpret_cast<const int4*>(&s_pos[wave][chc * kChunk + kg * 4]);
          pvs[0] = p4.x;
          pvs[1] = p4.y;
          pvs[2] = p4.z;
          pvs[3] = p4.w;
        }
        // The entries' value rows first (a wave-uniform base and a 32-bit byte
        // offset per lane when the segment's values span under 4 GiB, so no
        // 64-bit address arithmetic), kept ahead of the scoring and of the
        // previous chunk's products so that they load while those run.
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const Off boff = (Off(pvs[kk]) * Off(DV) + col) * Off(2);
          load_words<W>(reinterpret_cast<const uint16_t*>(vbytes + boff), raw[kk]);
        }
        __builtin_amdgcn_sched_barrier(0);
        const float* krow = &s_k[wave][chc * kChunk + kg * 4][0];
        scl = 1.0f;
        if constexpr (!kVar) {
#pragma unroll
          for (int kk = 0; kk < 4; ++kk) {
            const int32_t r = r0 + kg * 4 + kk;
            const int32_t pv = pvs[kk];
            const bool in = live && uint32_t(r) - uint32_t(a_eff) <= span && uint32_t(pv) <= lim_u;
            float d2 = 0.0f;
#pragma unroll
            for (int a = 0; a < KD; ++a) {
              if (a < dk) {
                const float diff = qv[a] - krow[kk * KD4 + a];
                d2 = fmaf(diff, diff, d2);
              }
            }
            const float rc = __builtin_amdgcn_rcpf(d2 + eps);
            sc[kk] = in ? rc : 0.0f;
            zpart += sc[kk];
          }
        } else {
          // Rounded as written: this lambda is inlined at several call sites,
          // and a chunk's site depends on where its run starts.
#pragma clang fp contract(off)
          bool ins[4];
#pragma unroll
          for (int kk = 0; kk < 4; ++kk) {
            const int32_t r = r0 + kg * 4 + kk;
            ins[kk] = live && uint32_t(r) - uint32_t(a_eff) <= span && uint32_t(pvs[kk]) <= lim_u;
            sc[kk] = variant_term<KD>(score, qv, krow + kk * KD4, dk, eps, rsd, qnorm);
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
          const uint32_t hw = __builtin_bit_cast(uint32_t, h);
          const bf16x2_t l = {(__bf16)(sc[2 * t] - __uint_as_float(hw << 16)),
                              (__bf16)(sc[2 * t + 1] - __uint_as_float(hw & 0xFFFF0000u))};
          bh[t] = hw;
          bl[t] = __builtin_bit_cast(uint32_t, l);
        }
      };
      // acc[j] += V^T (block j) * S^T for one chunk, high and low score parts
      // in one 16x16x32 product: a lane's eight K slots hold its 4 entries'
      // values twice, against their high and then their low score parts (A
      // and B slots correspond lane by lane, so the sum pairs each value with
      // both parts of its own score).
      auto mma = [&](const uint32_t(&raw)[4][W], const uint32_t(&bh)[2], const uint32_t(&bl)[2], float scl) {
        // Softmax variants: the sums so far to the chunk's running maximum.
        if (smax && wave_ballot(scl != 1.0f) != 0ull) {
#pragma unroll
          for (int j = 0; j < E; ++j) acc[j] *= scl;
        }
        Frag8 b;
        b.w[0] = bh[0];
        b.w[1] = bh[1];
        b.w[2] = bl[0];
        b.w[3] = bl[1];
#pragma unroll
        for (int j = 0; j < E; ++j) {
          Frag8 a;
#pragma unroll
          for (int t = 0; t < 2; ++t) {
            // One byte permute: element j of two consecutive rows, x below y
            // (the low halves for even j, the high halves for odd j).
            const uint32_t x = raw[2 * t][j >> 1], y = raw[2 * t + 1][j >> 1];
            a.w[t] = __builtin_amdgcn_perm(y, x, (j & 1) ? 0x07060302u : 0x05040100u);
            a.w[t + 2] = a.w[t];
          }
          acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v, b.v, acc[j], 0, 0, 0);
        }
      };

      // The chunks that meet some window, in list order: run by run (a run is
      // a stretch of chunks the windows cover without a gap; nearly always one
      // per tile), each run kStage chunks at a time.
      const int a_ch = mine ? my_a / kChunk : INT32_MAX;
      const int b_ch = mine ? my_b / kChunk : INT32_MIN;
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
          // (cb + nch)*kChunk - 1.
          {
            const int32_t base = cb * kChunk;
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
                s_pos[wave][e_] = pv[t];
#pragma unroll
                for (int a = 0; a < KD4; a += 4)
                  *reinterpret_cast<float4*>(&s_k[wave][e_][a]) =
                      make_float4(kv[a], a + 1 < KD ? kv[a + 1] : 0.0f, a + 2 < KD ? kv[a + 2] : 0.0f,
                                  a + 3 < KD ? kv[a + 3] : 0.0f);
              }
            }
          }
          wave_lds_sync();

          // Value rows of chunk ch+1 load while chunk ch is multiplied.
          uint32_t rA[4][W], rB[4][W], hA[2], lA[2], hB[2], lB[2];
          float sA, sB;
          prep(cb, 0, nch, rA, hA, lA, sA);
          for (int ch = 0; ch < nch; ch += 2) {
            prep(cb, ch + 1, nch, rB, hB, lB, sB);
            mma(rA, hA, lA, sA);
            if (ch + 1 >= nch) break;
            prep(cb, ch + 2, nch, rA, hA, lA, sA);
            mma(rB, hB, lB, sB);
          }
          wave_lds_sync();
        }
        c = wave_min_int(a_ch > e ? a_ch : INT32_MAX);
      }

      // Normalise and store: lane holds columns 4kg..4kg+3 of every block,
      // i.e. value elements 4kg*E .. 4kg*E + 4E - 1 of query qn.
      float z = zpart;
      z += __shfl_xor(z, 16, 64);
      z += __shfl_xor(z, 32, 64);
      if (in_grp) {
        const float inv = z > 0.0f ? 1.0f / z : 0.0f;
        float o[4 * E];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < E; ++j) o[i * E + j] = acc[j][i] * inv;
        // Rounded to bfloat16 (nearest even), two values per conversion.
        uint32_t w[2 * E];
#pragma unroll
        for (int t = 0; t < 2 * E; ++t) {
          const bf16x2_t pr = {(__bf16)o[2 * t], (__bf16)o[2 * t + 1]};
          w[t] = __builtin_bit_cast(uint32_t, pr);
        }
        uint4* dst = reinterpret_cast<uint4*>(out + (g_seg * N + my_i) * int64_t(DV) + kg * 4 * E);
#pragma unroll
        for (int t = 0; t < 2 * E; t += 4) dst[t / 4] = make_uint4(w[t], w[t + 1], w[t + 2], w[t + 3]);
      }
    }
  }
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
#define ZETA_TILE_LAUNCH(OFF, HIST, MODE)                                                                         \
  hipLaunchKernelGGL((select_attend_tile_kernel<DV, DK, OFF, HIST, MODE>), dim3(blocks), dim3(kTileWaves * 64), 0,    \
                     stream, q, k, v, perm, list_pos, q_order, bounds, keys_full, keys_list, total, N, dk,           \
                     causal ? 1 : 0, chunk, lp.t0, lp.t_hi, lp.cap, eps, hm.k, hm.v, out)
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

}  // namespace

bool tile_supports(int dv) { return tile_dv(dv); }

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
    hipLaunchKernelGGL(window_bounds_kernel, dim3(blocks), dim3(kBndWaves * 64), 0, stream, q_codes, sorted_codes,
                       perm, list_codes, list_pos, q_order, total, N, topk, causal ? 1 : 0, chunk, lp.t0, lp.t_hi,
                       lp.cap, bounds, idx_out);
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
