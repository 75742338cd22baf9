// Device-side pieces of candidate selection shared by the select kernel and
// the fused select-and-attend kernel: list search, window scans and the
// doubling-prefix-list addressing (Section 3.2.2; Algorithm 1, Steps 3-5).
#pragma once

#include <stdint.h>

#include "device_common.h"

namespace zeta {
namespace {

__device__ __forceinline__ int bit_length(uint32_t x) { return x ? 32 - __clz(int(x)) : 0; }

// First index in codes[lo..n) whose code is >= key, given that every entry
// before lo is below key, found by a wavefront: each round 64 lanes probe
// evenly spaced entries and the ballot of "probe < key" (a prefix of the
// lanes, the list being sorted) narrows the range 64x.
__device__ __forceinline__ int32_t wave_lower_bound(const uint32_t* __restrict__ codes, int32_t lo, int32_t n,
                                                    uint32_t key, int lane) {
  int32_t hi = n;
  while (hi > lo) {
    const int32_t len = hi - lo;
    const int32_t stride = (len + 63) >> 6;
    const int32_t x = lo + lane * stride;
    const bool probe = x < hi;
    const bool less = probe && codes[x] < key;
    const int cnt = __popcll(wave_ballot(less));
    if (cnt == 0) {
      hi = lo;
    } else {
      const int32_t next_hi = lo + cnt * stride;
      lo = lo + (cnt - 1) * stride + 1;
      hi = next_hi < hi ? next_hi : hi;
    }
  }
  return lo;
}

// The same search when the answer is expected just after `lo` (the previous
// query's insertion point in the same list, for a code no smaller): probe the
// 64 entries from lo first, and fall back to the 64-way search beyond them.
__device__ __forceinline__ int32_t wave_lower_bound_near(const uint32_t* __restrict__ codes, int32_t lo,
                                                         int32_t n, uint32_t key, int lane) {
  const int32_t x = lo + lane;
  const bool less = x < n && codes[x] < key;
  const int cnt = __popcll(wave_ballot(less));
  if (cnt < 64) return lo + cnt;
  return wave_lower_bound(codes, lo + 64, n, key, lane);
}

// Chunks of 64 list entries fetched on each side of the insertion point
// before the scans start, so that the common case needs one round trip.
constexpr int kPre = 2;

// Append up to `need` in-pool entries (position <= limit), in list order,
// from the 64 entries whose positions this wavefront holds in `pv` (entry
// cur + lane; out-of-list lanes hold INT_MAX) to buf[got..].  Returns the new
// count; `cur` ends just past the last entry taken, or 64 further on.
__device__ __forceinline__ int take_right(int32_t pv, int32_t limit, int32_t n, int32_t& cur, int need, int got,
                                          int32_t* buf) {
  const bool ok = pv <= limit;
  const uint64_t bal = wave_ballot(ok);
  const int avail = __popcll(bal);
  const int want = need - got;
  const int take = avail < want ? avail : want;
  const int slot = int(lanes_below(bal));
  if (ok && slot < take) buf[got + slot] = pv;
  if (take < avail) {
    // Stop just past the take-th in-pool entry of this chunk.
    const uint64_t last = wave_ballot(ok && slot == take - 1);
    cur = cur + (__ffsll((unsigned long long)last) - 1) + 1;
  } else {
    cur = cur + 64 < n ? cur + 64 : n;
  }
  return got + take;
}

// Collect up to `need` in-pool entries, nearest first, from the 64 entries
// cur-64 .. cur-1 held in `pv` (out-of-list lanes hold INT_MAX), into
// buf[cap_end-1-got], buf[cap_end-2-got], ... so that the collected run ends at
// buf[cap_end-1] in ascending list order.  Returns the new count.
__device__ __forceinline__ int take_left(int32_t pv, int32_t limit, int need, int got, int32_t* buf, int cap_end) {
  const bool ok = pv <= limit;
  const uint64_t bal = wave_ballot(ok);
  const int avail = __popcll(bal);
  const int want = need - got;
  const int take = avail < want ? avail : want;
  const int from_top = avail - 1 - int(lanes_below(bal));
  if (ok && from_top < take) buf[cap_end - 1 - (got + from_top)] = pv;
  return got + take;
}

// Scan entries cur, cur+1, ... of pos[0..n) and append up to `need` in-pool
// ones to buf[got..].  Returns the new count; `cur` is left just past the
// last entry taken (or at n).
__device__ __forceinline__ int scan_right(const int32_t* __restrict__ pos, int32_t n, int32_t limit,
                                          int32_t& cur, int need, int got, int32_t* buf, int lane) {
  while (got < need && cur < n) {
    const int32_t e = cur + lane;
    const int32_t pv = e < n ? pos[e] : INT32_MAX;
    got = take_right(pv, limit, n, cur, need, got, buf);
  }
  return got;
}

// Scan entries cur-1, cur-2, ... and collect up to `need` in-pool entries,
// nearest first, after the `got` already collected (see take_left).
__device__ __forceinline__ int scan_left(const int32_t* __restrict__ pos, int32_t limit, int32_t cur, int need,
                                         int got, int32_t* buf, int cap_end, int lane) {
  while (got < need && cur > 0) {
    const int32_t e = cur - 64 + lane;
    const int32_t pv = e >= 0 ? pos[e] : INT32_MAX;
    got = take_left(pv, limit, need, got, buf, cap_end);
    cur -= 64;
  }
  return got;
}

// Level of the list a causal query at position i searches: t0..t_hi for the
// prefix lists, t_hi + 1 for the full sorted list.
__device__ __forceinline__ int query_level(int32_t i, int t0, int t_hi) {
  const int bl = bit_length(uint32_t(i));
  const int t = bl > t0 ? bl : t0;
  return t <= t_hi ? t : t_hi + 1;
}

// Largest key position in the causal pool of query i: i for the exact
// prefix (chunk 0), floor(i / M) * M - 1 for the paper's chunked rule with
// chunk size M = chunk (Section 3.2.2; Algorithm 1, Step 4); -1 when the
// pool is empty (the first chunk).
__device__ __forceinline__ int32_t pool_limit(int32_t i, int chunk) {
  return chunk > 0 ? (i / chunk) * chunk - 1 : i;
}

// Level of the list searched for a causal pool ending at `limit` (t0 for an
// empty pool, which reads no entry).
__device__ __forceinline__ int pool_level(int32_t limit, int t0, int t_hi) {
  return limit < 0 ? t0 : query_level(limit, t0, t_hi);
}

// Where a query's candidates live: the sorted list it searches (codes and
// positions, n entries) and the largest position in its pool.  An empty
// causal pool gives n = 0.
struct QueryList {
  const uint32_t* codes;
  const int32_t* pos;
  int32_t n;
  int32_t limit;
};

__device__ __forceinline__ QueryList query_list(const uint32_t* __restrict__ sorted_codes,
                                                const int32_t* __restrict__ perm,
                                                const uint32_t* __restrict__ list_codes,
                                                const int32_t* __restrict__ list_pos, int64_t seg, int64_t N,
                                                int32_t i, int causal, int t0, int t_hi, int64_t cap,
                                                int chunk = 0) {
  QueryList L;
  L.codes = sorted_codes + seg * N;
  L.pos = perm + seg * N;
  L.n = int32_t(N);
  L.limit = int32_t(N - 1);  // every position is in the non-causal pool
  if (causal) {
    L.limit = pool_limit(i, chunk);
    if (L.limit < 0) {
      L.n = 0;
      return L;
    }
    const int t = query_level(L.limit, t0, t_hi);
    if (t <= t_hi) {
      const int64_t off = seg * cap + ((int64_t(1) << t) - (int64_t(1) << t0));
      L.codes = list_codes + off;
      L.pos = list_pos + off;
      L.n = int32_t(1) << t;
    }
  }
  return L;
}

// The window of a query whose insertion point in L is p: floor(k/2) pool keys
// before p and the rest from p on, shifted inward when one side of the pool
// runs out.  The left part ends at lbuf[topk-1] (got_l entries, ascending list
// order), the right part starts at rbuf[0] (got_r entries).  The first kPre
// chunks on each side are fetched together; further chunks as needed.
__device__ __forceinline__ void select_window(const QueryList& L, int32_t p, int topk, int32_t* lbuf,
                                              int32_t* rbuf, int lane, int& got_l_out, int& got_r_out) {
  const int half = topk / 2;
  int32_t pre_r[kPre], pre_l[kPre];
#pragma unroll
  for (int c = 0; c < kPre; ++c) {
    const int32_t er = p + c * 64 + lane;
    const int32_t el = p - (c + 1) * 64 + lane;
    pre_r[c] = er < L.n ? L.pos[er] : INT32_MAX;
    pre_l[c] = el >= 0 ? L.pos[el] : INT32_MAX;
  }
  const int need_r = topk - half;
  int32_t cur_r = p;
  int got_r = 0;
#pragma unroll
  for (int c = 0; c < kPre; ++c)
    if (got_r < need_r && cur_r < L.n) got_r = take_right(pre_r[c], L.limit, L.n, cur_r, need_r, got_r, rbuf);
  got_r = scan_right(L.pos, L.n, L.limit, cur_r, need_r, got_r, rbuf, lane);
  const int need_l = half + (need_r - got_r);
  int got_l = 0;
  int32_t cur_l = p;
#pragma unroll
  for (int c = 0; c < kPre; ++c) {
    if (got_l < need_l && cur_l > 0) {
      got_l = take_left(pre_l[c], L.limit, need_l, got_l, lbuf, topk);
      cur_l -= 64;
    }
  }
  got_l = scan_left(L.pos, L.limit, cur_l, need_l, got_l, lbuf, topk, lane);
  if (got_l < need_l && got_r == need_r)
    got_r = scan_right(L.pos, L.n, L.limit, cur_r, topk - got_l, got_r, rbuf, lane);
  got_l_out = got_l;
  got_r_out = got_r;
}

}  // namespace
}  // namespace zeta
