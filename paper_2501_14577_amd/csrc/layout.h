// Host-side shape arithmetic shared by argument validation, workspace sizing
// and the kernel launchers.  Pure C++: no HIP types, no device code.
#pragma once

#include <stddef.h>
#include <stdint.h>

namespace zeta {

constexpr int kWave = 64;
constexpr int kMaxDk = 8;       // largest d_k compiled
constexpr int kMaxTopk = 1024;  // largest k compiled
constexpr int kMaxBits = 24;    // grid cells per axis stay exact in float32

// ---- encode ---------------------------------------------------------------
// Rows of q (and of k) reduced by one block of the range kernel.
constexpr int64_t kEncRowsPerChunk = 512;
// Rows of q (and of k) encoded by one block of the encode kernel.
constexpr int64_t kEncRowsPerBlock = 256;
// Bytes of the per-GPU array that holds the range partials of the
// allocation-free encode call.
constexpr size_t kEncStaticScratchBytes = size_t(1) << 20;

// ---- sort -----------------------------------------------------------------
// Keys per tile of the prefix-list kernels: 4 waves x 4 chunks of 64 keys.
constexpr int kSortThreads = 256;
constexpr int kSortChunks = 4;
constexpr int64_t kSortTile = int64_t(kSortThreads) * kSortChunks;
// Keys per tile of the radix passes: 8 waves x 8 chunks of 64 keys, so that a
// tile holds about 8 keys of each of the 512 digit values and its reordered
// output is written in runs.
constexpr int kRadixThreads = 512;
constexpr int kRadixChunks = 8;
constexpr int64_t kRadixTile = int64_t(kRadixThreads) * kRadixChunks;
constexpr int kRadixMax = 512;  // digits of at most 9 bits
// Keys per tile of the level partition (zeta_query_order).
constexpr int64_t kLevelTile = 2048;
// Up to this many tiles per segment the scatter sums the earlier tiles' counts
// itself; beyond it a scan kernel writes them first.
constexpr int64_t kRadixInlineTiles = 32;

// ---- select ---------------------------------------------------------------
constexpr int kMaxLevels = 32;

// ---- attend ---------------------------------------------------------------
constexpr int kAttWavesPerBlock = 8;

inline size_t align_up(size_t x, size_t a = 256) { return (x + a - 1) / a * a; }

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Smallest t with 2^t >= x (x >= 1).
inline int ceil_log2(int64_t x) {
  int t = 0;
  while ((int64_t(1) << t) < x) ++t;
  return t;
}

struct SortPlan {
  int passes;      // radix passes
  int digit_bits;  // bits per pass (the last pass may use fewer)
  int64_t tiles;   // tiles per segment
};

inline SortPlan sort_plan(int64_t N, int code_bits) {
  SortPlan p;
  p.passes = (code_bits + 8) / 9;
  p.digit_bits = (code_bits + p.passes - 1) / p.passes;
  p.tiles = ceil_div(N, kRadixTile);
  return p;
}

// Doubling prefix lists used by causal selection.  List F_t holds the keys at
// positions below 2^t in (code, position) order, for t0 <= t <= t_hi, where
// 2^t0 >= topk and 2^t_hi < N.  F_t starts at entry 2^t - 2^t0 of its
// segment's region of `cap` entries.  A query at position i reads
// F_{max(t0, bitlen(i))} when that level exists and the full sorted list
// otherwise; either list contains its whole causal pool and at least half of
// the list's entries belong to the pool (or the list has under 2*topk entries).
struct ListPlan {
  int t0;
  int t_hi;
  int levels;   // t_hi - t0 + 1, or 0 when no list is needed
  int64_t cap;  // entries per segment
};

inline ListPlan list_plan(int64_t N, int topk) {
  ListPlan p;
  p.t0 = ceil_log2(topk);
  p.t_hi = ceil_log2(N) - 1;
  if (p.t0 <= p.t_hi) {
    p.levels = p.t_hi - p.t0 + 1;
    p.cap = (int64_t(1) << (p.t_hi + 1)) - (int64_t(1) << p.t0);
  } else {
    p.levels = 0;
    p.cap = 0;
  }
  return p;
}

// ---- workspace layouts (byte offsets into the caller's buffer) ------------

struct EncodeWs {
  int64_t chunks;
  size_t partial_off, bytes;
};
inline EncodeWs encode_ws(int64_t S, int64_t N, int dk) {
  EncodeWs w;
  w.chunks = ceil_div(N, kEncRowsPerChunk);
  w.partial_off = 0;
  w.bytes = align_up(size_t(S) * size_t(w.chunks) * 2 * size_t(dk) * sizeof(float));
  return w;
}

struct SortWs {
  size_t hist_off, keys_off, pos_off, bytes;
};
inline SortWs sort_ws(int64_t S, int64_t N, int code_bits) {
  SortPlan p = sort_plan(N, code_bits);
  SortWs w;
  w.hist_off = 0;
  // Per-tile counts, then per-segment digit totals.
  w.keys_off = align_up(size_t(S) * size_t(p.tiles + 1) * kRadixMax * sizeof(uint32_t));
  size_t buf = p.passes > 1 ? align_up(size_t(S) * size_t(N) * sizeof(uint32_t)) : 0;
  w.pos_off = w.keys_off + buf;
  w.bytes = w.pos_off + buf;
  return w;
}

// bytes: the prefix lists (none for non-causal calls or short segments);
// call_bytes: zeta_select_topk's need, the lists and then the window bounds
// (8 bytes per query) at bounds_off.
struct SelectWs {
  size_t cnt_off, codes_off, pos_off, bytes, bounds_off, call_bytes;
};
inline SelectWs select_ws(int64_t S, int64_t N, int topk, int causal) {
  SelectWs w;
  w.cnt_off = w.codes_off = w.pos_off = w.bytes = 0;
  ListPlan lp = list_plan(N, topk);
  if (causal && lp.levels > 0) {
    const int64_t tiles = ceil_div(N, kSortTile);
    const size_t list = align_up(size_t(S) * size_t(lp.cap) * sizeof(uint32_t));
    w.codes_off = align_up(size_t(S) * size_t(tiles) * kMaxLevels * sizeof(uint32_t));
    w.pos_off = w.codes_off + list;
    w.bytes = w.pos_off + list;
  }
  w.bounds_off = align_up(w.bytes);
  w.call_bytes = w.bounds_off + align_up(size_t(S) * size_t(N) * 2 * sizeof(int32_t));
  return w;
}

// Value widths compiled for the matrix-core tiles.
inline bool tile_dv(int dv) { return dv == 32 || dv == 64 || dv == 128 || dv == 256; }

// Largest k of the attend call's matrix-core tiles (index rows shared by 16
// neighbouring queries of a processing order).
constexpr int kIdxTileMaxTopk = 128;

// Whether the attend call runs on those tiles: a processing order given,
// bfloat16 inputs, d_k = 3, d_v up to 128 and k up to kIdxTileMaxTopk.
inline bool idx_tile_path(bool is_bf16, int dk, int dv, int topk, bool have_order) {
  return have_order && is_bf16 && dk == 3 && (dv == 32 || dv == 64 || dv == 128) && topk <= kIdxTileMaxTopk;
}

// Whether the one-pass call runs on the matrix-core tiles (and so needs the
// fused_ws layout, 16-byte aligned): bfloat16 inputs, a compiled d_v, and the
// Cauchy score, or any score when d_k = 3.  Validation and the launcher both
// decide with this one test.
inline bool tile_path(bool is_bf16, int dv, bool cauchy, int dk) {
  return is_bf16 && tile_dv(dv) && (cauchy || dk == 3);
}

// One-pass select and attend on the matrix cores: the prefix lists (as for
// select), then each processing-order slot's window bounds (two int32).
// For d_k = 3 it also keeps the key rows of the full sorted lists and of the
// prefix lists in list order (8 bytes per entry).
struct FusedWs {
  size_t bounds_off, keys_full_off, keys_list_off, bytes;
};
inline FusedWs fused_ws(int64_t S, int64_t N, int topk, int causal) {
  FusedWs w;
  const SelectWs sel = select_ws(S, N, topk, causal);
  w.bounds_off = sel.bounds_off;
  w.keys_full_off = sel.call_bytes;
  w.keys_list_off = w.keys_full_off + align_up(size_t(S) * size_t(N) * 8);
  const ListPlan lp = list_plan(N, topk);
  const size_t lists = (causal && lp.levels > 0) ? size_t(S) * size_t(lp.cap) : 0;
  w.bytes = w.keys_list_off + align_up(lists * 8);
  return w;
}

// ---- locality experiment -------------------------------------------------------
// Keys per query sorted in LDS by the exact nearest-key search, and segment
// length covered by the overlap count's LDS bit set.
constexpr int kKnnMaxN = 4096;
constexpr int64_t kOverlapMaxN = 65536;

// ---- history mean ---------------------------------------------------------
// Segmented scans over [S][N][D] matrices (values and keys together): rows
// per chunk, and the most columns scanned at once (d_k + d_v).
constexpr int64_t kHistRows = 32;
constexpr int kHistMaxCols = kMaxDk + 256;

// Per (segment, chunk, column) sums, turned in place into exclusive prefix
// (or suffix) sums, and per (segment, column) totals.
struct HistWs {
  size_t sums_off, totals_off, bytes;
};
inline HistWs hist_ws(int64_t S, int64_t N, int D) {
  HistWs w;
  w.sums_off = 0;
  w.totals_off = align_up(size_t(S) * size_t(ceil_div(N, kHistRows)) * size_t(D) * sizeof(float));
  w.bytes = w.totals_off + align_up(size_t(S) * size_t(D) * sizeof(float));
  return w;
}

// Attention gradients: per-query partial sums of the eps gradient and the
// per-block sums of their fixed-order reduction; per query (Z_i, c_i); the
// key of every window slot, the slots sorted by key (keys and the sort's
// permutation); each key's run of sorted slots; the sort's own workspace.
// With the history-mean candidate also the gradients reaching each query's
// mean key and mean value (divided by the history's length) and the scan
// that passes them back to the history's rows.
struct BwdWs {
  size_t part_off, block_off, zc_off, keys_off, sorted_off, slot_off, runs_off, sort_off;
  size_t hist_k_off, hist_v_off, hist_scan_off, bytes;
  int key_bits;  // bits of a slot key (keys run to N inclusive)
};
inline BwdWs bwd_ws(int64_t S, int64_t N, int topk, int dk = 0, int dv = 0, bool history = false) {
  BwdWs w;
  const size_t rows = size_t(S) * size_t(N);
  const size_t slots = rows * size_t(topk);
  w.key_bits = 1;
  while ((int64_t(1) << w.key_bits) <= N) ++w.key_bits;
  w.part_off = 0;
  w.block_off = w.part_off + align_up(rows * sizeof(float));
  w.zc_off = w.block_off + align_up(256 * sizeof(float));
  w.keys_off = w.zc_off + align_up(rows * 2 * sizeof(float));
  w.sorted_off = w.keys_off + align_up(slots * sizeof(uint32_t));
  w.slot_off = w.sorted_off + align_up(slots * sizeof(uint32_t));
  w.runs_off = w.slot_off + align_up(slots * sizeof(int32_t));
  w.sort_off = w.runs_off + align_up(rows * 2 * sizeof(int32_t));
  w.hist_k_off = w.sort_off + align_up(sort_ws(S, N * topk, w.key_bits).bytes);
  w.hist_v_off = w.hist_k_off;
  w.hist_scan_off = w.hist_k_off;
  w.bytes = w.hist_k_off;
  if (history) {
    w.hist_v_off = w.hist_k_off + align_up(rows * size_t(dk) * sizeof(float));
    w.hist_scan_off = w.hist_v_off + align_up(rows * size_t(dv) * sizeof(float));
    w.bytes = w.hist_scan_off + hist_ws(S, N, dk + dv).bytes;
  }
  return w;
}

// Regrouping a processing order by list level: a copy of the given order
// (when it is regrouped in place) and the radix pass's histograms.
struct QueryOrderWs {
  size_t given_off, phist_off, bytes;
};
inline QueryOrderWs query_order_ws(int64_t S, int64_t N) {
  QueryOrderWs w;
  w.given_off = 0;
  w.phist_off = align_up(size_t(S) * size_t(N) * sizeof(int32_t));
  w.bytes = w.phist_off + align_up(size_t(S) * size_t(ceil_div(N, kLevelTile) + 1) * kRadixMax * sizeof(uint32_t));
  return w;
}

// Gradients of the bfloat16 one-pass attention: the one-pass call's lists,
// bounds and key rows, then per slot a 32-byte record, a copy of the dout row
// and the deps part, each tile's window range per list and their envelopes,
// each chunk's candidate tiles (in the envelopes' layout), the block sums of
// deps and, with the history-mean candidate, the gradients reaching the means
// and their scan's sums.
constexpr int64_t kTileBwdRedPer = 4096;  // deps parts per block sum (at least)
constexpr int64_t kTileBwdRedMax = 1024;  // block sums at most
inline int tile_bwd_levels(int64_t N, int topk, bool causal) {
  const ListPlan lp = list_plan(N, topk);
  return causal ? lp.levels + 1 : 1;  // the prefix lists, then the full list
}
struct TileBwdWs {
  FusedWs fused;
  size_t rec_off, dslot_off, part_off, env_off, env2_off, ranges_off, sums_off;
  size_t hist_k_off, hist_v_off, hist_scan_off, bytes;
};
inline TileBwdWs tile_bwd_ws(int64_t S, int64_t N, int dv, int topk, int causal, bool history = false) {
  TileBwdWs w;
  w.fused = fused_ws(S, N, topk, causal);
  const size_t rows = size_t(S) * size_t(N);
  const size_t tiles = size_t(S) * size_t((N + 15) / 16);
  const size_t env = size_t(tile_bwd_levels(N, topk, causal != 0)) * tiles * 2 * sizeof(int32_t);
  w.rec_off = align_up(w.fused.bytes);
  w.dslot_off = w.rec_off + align_up(rows * 32);
  w.part_off = w.dslot_off + align_up(rows * size_t(dv) * 2);
  w.env_off = w.part_off + align_up(rows * sizeof(float));
  w.env2_off = w.env_off + align_up(env);
  w.ranges_off = w.env2_off + align_up(env);
  w.sums_off = w.ranges_off + align_up(env);
  w.hist_k_off = w.sums_off + align_up(size_t(kTileBwdRedMax) * sizeof(float));
  w.hist_v_off = w.hist_k_off;
  w.hist_scan_off = w.hist_k_off;
  w.bytes = w.hist_k_off;
  if (history) {  // the gradients reaching the means (d_k = 3) and their scan
    w.hist_v_off = w.hist_k_off + align_up(rows * 3 * sizeof(float));
    w.hist_scan_off = w.hist_v_off + align_up(rows * size_t(dv) * sizeof(float));
    w.bytes = w.hist_scan_off + hist_ws(S, N, 3 + dv).bytes;
  }
  return w;
}

}  // namespace zeta
