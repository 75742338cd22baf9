// Gradients of the bfloat16 one-pass attention over the windows of
// zeta_select_attend_fwd (Appendix E.2, summary of gradient computations), on
// the matrix cores.  With S_ij = 1 / delta_ij, delta_ij = |q_i - k_j|^2 + eps,
// Z_i = sum_j S_ij, A_ij = S_ij / Z_i, p_ij = dout_i . v_j,
// c_i = dout_i . o_i = sum_j A_ij p_ij and w_ij = (p_ij - c_i) S_ij^2 / Z_i:
//   dv_j = sum_i A_ij dout_i,        dk_j = 2 sum_i w_ij (q_i - k_j),
//   dq_i = -2 sum_j w_ij (q_i - k_j), deps = -sum_ij w_ij.
//
// A tile is 16 consecutive slots of one segment's processing order.
//  1. Query pass, one wavefront per tile, walking the union of its windows in
//     16-entry chunks as the forward tile kernel does.  Per chunk the 16 x 16
//     dot products p_ij are one matrix-core product per 32 value columns (V
//     rows times dout^T).  Each lane sums over its 4 entries
//       Z = sum S, P = sum S p, X = sum S^2 p, Y = sum S^2,
//       U = sum S^2 p (q - k), R = sum S^2 (q - k),
//     so one walk gives c = P / Z, dq = -(2 / Z)(U - c R) and the query's
//     part of deps, -(X - c Y) / Z.  Per slot it stores a 32-byte record (q,
//     list, 1/Z, c, window bounds, pool limit) and the query's dout row, so
//     that a tile's data is contiguous for the key pass; per list it stores
//     the first and last list index of the tile's windows.
//  2. Envelopes, per segment and level: the running maximum (from the first
//     tile) of the tiles' last indices and the running minimum (from the last
//     tile) of their first indices.  Both are non-decreasing, so the tiles
//     whose windows meet a chunk lie between two positions, found by binary
//     search per chunk.
//  3. Key pass, one launch per list (the full sorted list first, then each
//     prefix list), one wavefront per 16-entry chunk.  Over the candidate
//     tiles (64 tiles' ranges tested at once) a lane takes one entry and 4 of
//     the tile's queries: S_ij, the dot
//     products (dout x V^T, one product per 32 columns), w_ij and A_ij.  dv^T
//     accumulates as dout^T (columns x queries) times A (queries x entries),
//     with the high and low bfloat16 parts of A in one 16x16x32 product per 16
//     columns; dk accumulates in float32 on the vector ALUs.  The full list's
//     launch writes the rows of every key (each key is in it once); a prefix
//     list's launch adds to the rows of its keys.
// Launches run in a fixed order and a chunk visits its tiles in processing
// order: no atomics, and the outputs are the same from run to run for a given
// processing order.  Any processing order is correct; the one from
// zeta_query_order keeps each chunk's candidate tiles few.
//
// With the history-mean candidate (Section 3.4, last paragraph) the query pass
// adds the pair (mean_k[i], mean_v[i]) to its sums once per query (float32,
// its dot product dout_i . mean_v[i] from the lanes' dout slices) and writes
// the gradients reaching the means, divided by the history's length; after
// the key passes a reverse scan adds them to the rows of every history.
#include "attend_device.h"
#include "device_common.h"
#include "kernels.h"
#include "layout.h"
#include "select_device.h"
#include "tile_device.h"

namespace zeta {
namespace {

constexpr int kBtWaves = 4;          // wavefronts per block
constexpr int kBtStage = 512;        // list entries staged at once by the query pass
constexpr int kBtChunk = 16;         // list entries per product step
constexpr int kBtStageChunks = kBtStage / kBtChunk;
constexpr int kRedThreads = 256;
constexpr uint32_t kNoList = 0xFFFFu;  // record of a slot whose query has no window

// What the key pass needs of a slot's query, in 32 bytes: q as bfloat16 bits,
// the list index (kNoList: no window), 1/Z, c, the window's list-index bounds
// and the pool limit.
struct alignas(16) SlotRec {
  uint32_t q01;     // q[0] | q[1] << 16
  uint32_t q2_list;  // q[2] | list index << 16
  float zinv, c;
  int32_t a, b;
  uint32_t lim, pad;
};

// The list of a level: the full sorted list, or prefix list `lvl`.
struct LevelList {
  const int32_t* pos;
  const uint2* key;
  int32_t n;
};

__device__ __forceinline__ LevelList level_list(const int32_t* sorted_pos, const int32_t* list_pos,
                                                const uint2* keys_full, const uint2* keys_list, int64_t seg,
                                                int64_t N, int causal, int lvl, int t0, int t_hi, int64_t cap) {
  LevelList L;
  L.pos = sorted_pos + seg * N;
  L.key = keys_full + seg * N;
  L.n = int32_t(N);
  if (causal && lvl <= t_hi) {
    const int64_t off = seg * cap + ((int64_t(1) << lvl) - (int64_t(1) << t0));
    L.pos = list_pos + off;
    L.key = keys_list + off;
    L.n = int32_t(1) << lvl;
  }
  return L;
}

// Key row (d_k = 3) from its list-order copy: x | y << 16, z.
__device__ __forceinline__ void key_row(uint2 w, float (&kv)[3]) {
  kv[0] = __uint_as_float(w.x << 16);
  kv[1] = __uint_as_float(w.x & 0xFFFF0000u);
  kv[2] = __uint_as_float(w.y << 16);
}

// Eight bfloat16 values (16 bytes) at a 16-byte aligned address.
__device__ __forceinline__ void load8(const uint16_t* p, uint32_t (&o)[4]) {
  const uint4 x = *reinterpret_cast<const uint4*>(p);
  o[0] = x.x;
  o[1] = x.y;
  o[2] = x.z;
  o[3] = x.w;
}

__device__ __forceinline__ Frag8 frag8(const uint32_t (&w)[4]) {
  Frag8 f;
  f.w[0] = w[0];
  f.w[1] = w[1];
  f.w[2] = w[2];
  f.w[3] = w[3];
  return f;
}

// Sum over the 4 lanes of a column of the product layout (lanes l, l^16,
// l^32, l^48).
__device__ __forceinline__ float kg_sum(float x) {
  x += __shfl_xor(x, 16, 64);
  x += __shfl_xor(x, 32, 64);
  return x;
}

// The index of a list among a call's lists: prefix list lvl is lvl - t0, the
// full sorted list (lvl > t_hi) comes after the `levels` prefix lists; 0 when
// not causal (the full list only).
__device__ __forceinline__ int level_index(int lvl, int causal, int t0, int t_hi, int levels) {
  return causal ? (lvl > t_hi ? levels : lvl - t0) : 0;
}

// ---- 1. query pass ----------------------------------------------------------
template <int DV, bool kHist>
__global__ void __launch_bounds__(kBtWaves * 64) __attribute__((amdgpu_waves_per_eu(DV <= 128 ? 3 : 1)))
    bwd_tile_query_kernel(const uint16_t* __restrict__ q, const uint16_t* __restrict__ v,
                          const uint16_t* __restrict__ dout, const int32_t* __restrict__ sorted_pos,
                          const int32_t* __restrict__ list_pos, const int32_t* __restrict__ order,
                          const int2* __restrict__ bounds, const uint2* __restrict__ keys_full,
                          const uint2* __restrict__ keys_list, int64_t S, int64_t N, int64_t ct, int causal,
                          int chunk, int t0, int t_hi, int levels, int64_t cap, float eps, float* __restrict__ dq,
                          SlotRec* __restrict__ rec, uint16_t* __restrict__ dslot, float* __restrict__ deps_part,
                          int2* __restrict__ env, const float* __restrict__ mk, const float* __restrict__ mv,
                          float* __restrict__ hk, float* __restrict__ hv) {
  constexpr int NS = DV / 32;  // 32-column slices of a row: one product each
  static_assert(DV % 32 == 0, "d_v must be a multiple of 32");
  __shared__ __align__(16) int32_t s_pos[kBtWaves][kBtStage];
  __shared__ __align__(16) float s_k[kBtWaves][kBtStage][4];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int qn = lane & 15;  // this lane's query (B column) and entry (A row)
  const int kg = lane >> 4;  // this lane's entries 4kg..4kg+3 and column slice 8kg..8kg+7
  const int64_t tiles = S * ct;
  const int64_t nb = gridDim.x;

  for (int64_t blk = xcd_contiguous_block(blockIdx.x, nb); blk * kBtWaves < tiles; blk += nb) {
    const int64_t tile = blk * kBtWaves + wave;
    if (tile >= tiles) continue;
    const int64_t seg = tile / ct;
    const int64_t tau = tile - seg * ct;
    const int64_t xs = tau * 16 + qn;  // slot within the segment
    const int64_t slot = seg * N + xs;
    int32_t my_i = -1, my_a = 0, my_b = -1;
    int my_lvl = 0;
    if (xs < N) {
      const int64_t ii = order != nullptr ? int64_t(order[slot]) : xs;
      if (ii >= 0 && ii < N) {
        my_i = int32_t(ii);
        my_lvl = causal ? pool_level(pool_limit(my_i, chunk), t0, t_hi) : 0;
        const int2 bb = bounds[slot];
        my_a = bb.x;
        my_b = bb.y;
      }
    }
    // Slots without a query still hold a defined record, deps part and (zero)
    // dout row.
    if (xs < N && my_i < 0) {
      if (kg == 0) {
        SlotRec r = {};
        r.q2_list = kNoList << 16;
        rec[slot] = r;
        deps_part[slot] = 0.0f;
      }
#pragma unroll
      for (int s2 = 0; s2 < NS; ++s2)
        *reinterpret_cast<uint4*>(dslot + slot * DV + 32 * s2 + 8 * kg) = make_uint4(0u, 0u, 0u, 0u);
    }
    uint32_t pending = uint32_t(wave_ballot(my_i >= 0)) & 0xFFFFu;

    // Queries that search one list form a group (nearly always the whole tile).
    while (pending != 0u) {
      const int leader = __ffs(int(pending)) - 1;
      const int g_lvl = __builtin_amdgcn_readlane(my_lvl, leader);
      const uint32_t gmask = uint32_t(wave_ballot(my_i >= 0 && my_lvl == g_lvl)) & pending;
      pending &= ~gmask;
      const LevelList L = level_list(sorted_pos, list_pos, keys_full, keys_list, seg, N, causal, g_lvl, t0, t_hi, cap);
      const bool in_grp = ((gmask >> qn) & 1u) != 0u;
      const bool mine = in_grp && 0 <= my_a && my_a <= my_b && my_b < L.n;
      const int32_t my_lim = causal ? pool_limit(my_i, chunk) : int32_t(N - 1);

      // The group's window range in this list, for the key pass.
      {
        const int lo = wave_min_int(mine ? my_a : INT32_MAX);
        const int hi = wave_max_int(mine ? my_b : INT32_MIN);
        if (lane == 0) env[(int64_t(level_index(g_lvl, causal, t0, t_hi, levels)) * S + seg) * ct + tau] = make_int2(lo, hi);
      }

      float qv[3] = {0.0f, 0.0f, 0.0f};
      uint32_t dfr[NS][4];  // dout of query qn, columns 32s + 8kg .. 32s + 8kg + 7
#pragma unroll
      for (int s = 0; s < NS; ++s) dfr[s][0] = dfr[s][1] = dfr[s][2] = dfr[s][3] = 0u;
      // With the history-mean candidate every query has a candidate.
      if (kHist ? in_grp : mine) {
        const int64_t gq = seg * N + my_i;
        Row3<uint16_t>::load(q, gq, S * N, qv);
#pragma unroll
        for (int s = 0; s < NS; ++s) load8(dout + gq * DV + 32 * s + 8 * kg, dfr[s]);
      }
      // The slot's copy of its dout row (zeros without a window).
      if (in_grp) {
#pragma unroll
        for (int s = 0; s < NS; ++s)
          *reinterpret_cast<uint4*>(dslot + slot * DV + 32 * s + 8 * kg) =
              make_uint4(dfr[s][0], dfr[s][1], dfr[s][2], dfr[s][3]);
      }
      float z = 0.0f, pz = 0.0f, xz = 0.0f, yz = 0.0f;
      float u[3] = {0.0f, 0.0f, 0.0f}, rr[3] = {0.0f, 0.0f, 0.0f};

      // Window and pool tests as single unsigned compares (as in the forward).
      const uint32_t span = mine ? uint32_t(my_b - my_a) : 0u;
      const int32_t a_eff = mine ? my_a : INT32_MIN;
      const uint32_t lim_u = uint32_t(my_lim);
      const uint16_t* vseg = v + seg * N * DV;

      // Value slices of entry qn of staged chunk ch (row 0 for a chunk past
      // the burst: loaded, never used).
      auto load_v = [&](int ch, int nch_, uint32_t(&vf)[NS][4]) {
        const int chc = ch < nch_ ? ch : 0;
        const int32_t pv = s_pos[wave][chc * kBtChunk + qn];
#pragma unroll
        for (int s = 0; s < NS; ++s) load8(vseg + int64_t(pv) * DV + 32 * s + 8 * kg, vf[s]);
      };
      // Sums over this lane's 4 entries of chunk ch.
      auto accumulate = [&](int cb, int ch, const uint32_t(&vf)[NS][4]) {
        f32x4_t d = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int s = 0; s < NS; ++s) d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(frag8(vf[s]).v, frag8(dfr[s]).v, d, 0, 0, 0);
        const int4 p4 = *reinterpret_cast<const int4*>(&s_pos[wave][ch * kBtChunk + kg * 4]);
        const int32_t pvs[4] = {p4.x, p4.y, p4.z, p4.w};
        const int32_t r0 = (cb + ch) * kBtChunk + kg * 4;
#pragma unroll
        for (int kk = 0; kk < 4; ++kk) {
          const float4 kr = *reinterpret_cast<const float4*>(&s_k[wave][ch * kBtChunk + kg * 4 + kk][0]);
          const float df[3] = {qv[0] - kr.x, qv[1] - kr.y, qv[2] - kr.z};
          const float d2 = fmaf(df[2], df[2], fmaf(df[1], df[1], df[0] * df[0]));
          const bool in = uint32_t(r0 + kk) - uint32_t(a_eff) <= span && uint32_t(pvs[kk]) <= lim_u;
          const float sc = in ? __builtin_amdgcn_rcpf(d2 + eps) : 0.0f;
          const float p = d[kk];
          const float s2 = sc * sc;
          z += sc;
          pz = fmaf(sc, p, pz);
          yz += s2;
          const float s2p = s2 * p;
          xz += s2p;
#pragma unroll
          for (int a = 0; a < 3; ++a) {
            u[a] = fmaf(s2p, df[a], u[a]);
            rr[a] = fmaf(s2, df[a], rr[a]);
          }
        }
      };

      // The chunks that meet some window, run by run, kBtStageChunks at a time.
      const int a_ch = mine ? my_a / kBtChunk : INT32_MAX;
      const int b_ch = mine ? my_b / kBtChunk : INT32_MIN;
      for (int c = wave_min_int(a_ch); c != INT32_MAX;) {
        int e = c - 1;
        for (;;) {
          const int e2 = wave_max_int(a_ch <= e + 1 ? b_ch : e);
          if (e2 == e) break;
          e = e2;
        }
        for (int cb = c; cb <= e; cb += kBtStageChunks) {
          const int nch = e - cb + 1 < kBtStageChunks ? e - cb + 1 : kBtStageChunks;
          {
            const int32_t base = cb * kBtChunk;
            int32_t pv[kBtStage / 64];
            uint2 kw[kBtStage / 64];
#pragma unroll
            for (int t = 0; t < kBtStage / 64; ++t) {
              const int e_ = t * 64 + lane;
              const int32_t r = base + e_;
              pv[t] = 0;  // an entry past the list's end: outside every window
              kw[t] = make_uint2(0u, 0u);
              if (e_ < nch * kBtChunk && r < L.n) {
                pv[t] = L.pos[r];
                kw[t] = L.key[r];
              }
            }
#pragma unroll
            for (int t = 0; t < kBtStage / 64; ++t) {
              const int e_ = t * 64 + lane;
              if (e_ < nch * kBtChunk) {
                float kv[3];
                key_row(kw[t], kv);
                s_pos[wave][e_] = pv[t];
                *reinterpret_cast<float4*>(&s_k[wave][e_][0]) = make_float4(kv[0], kv[1], kv[2], 0.0f);
              }
            }
          }
          wave_lds_sync();
          // Value slices of chunk ch+1 load while chunk ch is summed.
          uint32_t vA[NS][4], vB[NS][4];
          load_v(0, nch, vA);
          for (int ch = 0; ch < nch; ch += 2) {
            load_v(ch + 1, nch, vB);
            accumulate(cb, ch, vA);
            if (ch + 1 >= nch) break;
            load_v(ch + 2, nch, vA);
            accumulate(cb, ch + 1, vB);
          }
          wave_lds_sync();
        }
        c = wave_min_int(a_ch > e ? a_ch : INT32_MAX);
      }

      z = kg_sum(z);
      pz = kg_sum(pz);
      xz = kg_sum(xz);
      yz = kg_sum(yz);
#pragma unroll
      for (int a = 0; a < 3; ++a) {
        u[a] = kg_sum(u[a]);
        rr[a] = kg_sum(rr[a]);
      }
      // The history-mean candidate's terms, once per query (every lane of the
      // query adds them to its totals).
      float s_m = 0.0f, p_m = 0.0f, dm[3] = {0.0f, 0.0f, 0.0f};
      if constexpr (kHist) {
        if (in_grp) {
          const int64_t gq = seg * N + my_i;
          const float4* mrow = reinterpret_cast<const float4*>(mv + gq * DV);
          float part = 0.0f;
#pragma unroll
          for (int s = 0; s < NS; ++s) {
            const float4 m0 = mrow[(32 * s + 8 * kg) / 4], m1 = mrow[(32 * s + 8 * kg) / 4 + 1];
            const float mvv[8] = {m0.x, m0.y, m0.z, m0.w, m1.x, m1.y, m1.z, m1.w};
#pragma unroll
            for (int t = 0; t < 4; ++t) {
              part = fmaf(__uint_as_float(dfr[s][t] << 16), mvv[2 * t], part);
              part = fmaf(__uint_as_float(dfr[s][t] & 0xFFFF0000u), mvv[2 * t + 1], part);
            }
          }
          p_m = kg_sum(part);
#pragma unroll
          for (int a = 0; a < 3; ++a) dm[a] = qv[a] - mk[gq * 3 + a];
          s_m = __builtin_amdgcn_rcpf(fmaf(dm[2], dm[2], fmaf(dm[1], dm[1], dm[0] * dm[0])) + eps);
          const float s2 = s_m * s_m;
          z += s_m;
          pz = fmaf(s_m, p_m, pz);
          yz += s2;
          xz = fmaf(s2, p_m, xz);
#pragma unroll
          for (int a = 0; a < 3; ++a) {
            u[a] = fmaf(s2 * p_m, dm[a], u[a]);
            rr[a] = fmaf(s2, dm[a], rr[a]);
          }
        }
      }
      if constexpr (kHist) {
        if (in_grp) {
          // The gradients reaching mean_k[i] and mean_v[i], divided by the
          // history's length.
          const float inv = z > 0.0f ? 1.0f / z : 0.0f;
          const float cc = pz * inv;
          const float inv_cnt = 1.0f / float(causal ? my_i + 1 : N);
          const int64_t gq = seg * N + my_i;
          const float w_m = (p_m - cc) * s_m * s_m * inv;
          if (kg == 0) {
#pragma unroll
            for (int a = 0; a < 3; ++a) hk[gq * 3 + a] = 2.0f * w_m * dm[a] * inv_cnt;
          }
          const float am = s_m * inv * inv_cnt;
#pragma unroll
          for (int s = 0; s < NS; ++s) {
            float4* dst = reinterpret_cast<float4*>(hv + gq * DV + 32 * s + 8 * kg);
            dst[0] = make_float4(am * __uint_as_float(dfr[s][0] << 16), am * __uint_as_float(dfr[s][0] & 0xFFFF0000u),
                                 am * __uint_as_float(dfr[s][1] << 16), am * __uint_as_float(dfr[s][1] & 0xFFFF0000u));
            dst[1] = make_float4(am * __uint_as_float(dfr[s][2] << 16), am * __uint_as_float(dfr[s][2] & 0xFFFF0000u),
                                 am * __uint_as_float(dfr[s][3] << 16), am * __uint_as_float(dfr[s][3] & 0xFFFF0000u));
          }
        }
      }
      if (in_grp && kg == 0) {
        const float inv = z > 0.0f ? 1.0f / z : 0.0f;
        const float cc = pz * inv;
        const int64_t gq = seg * N + my_i;
#pragma unroll
        for (int a = 0; a < 3; ++a) dq[gq * 3 + a] = -2.0f * inv * (u[a] - cc * rr[a]);
        deps_part[slot] = -inv * (xz - cc * yz);
        SlotRec r;
        r.q01 = (__float_as_uint(qv[0]) >> 16) | (__float_as_uint(qv[1]) & 0xFFFF0000u);
        const uint32_t list = mine ? uint32_t(level_index(g_lvl, causal, t0, t_hi, levels)) : kNoList;
        r.q2_list = (__float_as_uint(qv[2]) >> 16) | (list << 16);
        r.zinv = inv;
        r.c = cc;
        r.a = my_a;
        r.b = my_b;
        r.lim = uint32_t(my_lim);
        r.pad = 0u;
        rec[slot] = r;
      }
    }
  }
}

// ---- 2. envelopes ---------------------------------------------------------------
// One block per (list, segment): out[t] = (min over t' >= t of the first
// index, max over t' <= t of the last index).  Each thread scans a stretch of
// consecutive tiles; the stretches' totals are scanned in LDS.
constexpr int kEnvThreads = 256;

__global__ void __launch_bounds__(kEnvThreads)
    bwd_envelope_kernel(const int2* __restrict__ env, int64_t ct, int2* __restrict__ env2) {
  __shared__ int s_mx[kEnvThreads];
  __shared__ int s_mn[kEnvThreads];
  const int tid = threadIdx.x;
  const int2* in = env + int64_t(blockIdx.x) * ct;
  int2* out = env2 + int64_t(blockIdx.x) * ct;
  const int64_t per = (ct + kEnvThreads - 1) / kEnvThreads;
  const int64_t b0 = int64_t(tid) * per < ct ? int64_t(tid) * per : ct;
  const int64_t b1 = b0 + per < ct ? b0 + per : ct;
  int mx = INT32_MIN, mn = INT32_MAX;
  for (int64_t t = b0; t < b1; ++t) {
    const int2 r = in[t];
    mx = r.y > mx ? r.y : mx;
    mn = r.x < mn ? r.x : mn;
  }
  s_mx[tid] = mx;
  s_mn[tid] = mn;
  __syncthreads();
  // Inclusive scans: maximum from the first stretch, minimum from the last.
  for (int off = 1; off < kEnvThreads; off <<= 1) {
    const int a = tid >= off ? s_mx[tid - off] : INT32_MIN;
    const int b = tid + off < kEnvThreads ? s_mn[tid + off] : INT32_MAX;
    __syncthreads();
    s_mx[tid] = a > s_mx[tid] ? a : s_mx[tid];
    s_mn[tid] = b < s_mn[tid] ? b : s_mn[tid];
    __syncthreads();
  }
  int carry = tid > 0 ? s_mx[tid - 1] : INT32_MIN;
  for (int64_t t = b0; t < b1; ++t) {
    const int y = in[t].y;
    carry = y > carry ? y : carry;
    out[t].y = carry;
  }
  carry = tid + 1 < kEnvThreads ? s_mn[tid + 1] : INT32_MAX;
  for (int64_t t = b1 - 1; t >= b0; --t) {
    const int x = in[t].x;
    carry = x < carry ? x : carry;
    out[t].x = carry;
  }
}

// First tile t in [0, ct) with key(t) >= want for a non-decreasing key
// (ct when none): the running maximum of last indices (kHi) or the running
// minimum of first indices.
template <bool kHi>
__device__ __forceinline__ int64_t first_at_least(const int2* p, int64_t ct, int want) {
  int64_t lo = 0, hi = ct;
  while (lo < hi) {
    const int64_t mid = (lo + hi) >> 1;
    const int2 r = p[mid];
    if ((kHi ? r.y : r.x) >= want)
      hi = mid;
    else
      lo = mid + 1;
  }
  return lo;
}

// Per list, segment and chunk: the candidate tiles [ta, tb).  Tiles before ta
// end before the chunk; tiles from tb on start after it.  One thread per
// (list, segment, chunk), in the envelopes' layout.
__global__ void __launch_bounds__(256)
    bwd_ranges_kernel(const int2* __restrict__ env2, int64_t S, int64_t N, int64_t ct, int causal, int t0, int t_hi,
                      int levels, int nl, int2* __restrict__ ranges) {
  const int64_t t = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t >= int64_t(nl) * S * ct) return;
  const int64_t row = t / ct;
  const int64_t c = t - row * ct;
  const int li = int(row / S);
  const int lvl = !causal ? 0 : (li == levels ? t_hi + 1 : t0 + li);
  const int64_t ln = (causal && lvl <= t_hi) ? (int64_t(1) << lvl) : N;
  if (c * 16 >= ln) return;
  const int lo_c = int(c * 16);
  const int hi_c = int(c * 16 + 15 < ln - 1 ? c * 16 + 15 : ln - 1);
  const int2* ev2 = env2 + row * ct;
  ranges[t] = make_int2(int(first_at_least<true>(ev2, ct, lo_c)), int(first_at_least<false>(ev2, ct, hi_c + 1)));
}

// ---- 3. key pass ------------------------------------------------------------------
// A block's wavefronts take consecutive chunks of one list and segment and
// walk the union of their candidate tiles together.  Each tile's 16 records
// and 16 dout rows are staged once in LDS for all of them (two buffers: the next
// tile's bytes load while the current tile is summed, one barrier per tile);
// a wavefront skips the tiles its own chunk does not meet.  Dout rows are
// padded by 16 bytes, so that lanes reading 16 different rows use different
// banks.
constexpr int kKeyWaves = 4;  // chunks per block (one per wavefront)
constexpr int kKeyThreads = kKeyWaves * 64;

template <int DV, bool kOff32>
__global__ void __launch_bounds__(kKeyThreads) __attribute__((amdgpu_waves_per_eu(DV <= 128 ? 3 : 2)))
    bwd_tile_key_kernel(const uint16_t* __restrict__ v, const int32_t* __restrict__ sorted_pos,
                        const int32_t* __restrict__ list_pos, const uint2* __restrict__ keys_full,
                        const uint2* __restrict__ keys_list, const SlotRec* __restrict__ rec,
                        const uint16_t* __restrict__ dslot, const int2* __restrict__ env,
                        const int2* __restrict__ ranges, int64_t S, int64_t N, int64_t ct, int causal, int t0,
                        int t_hi, int levels, int64_t cap, int lvl, int first, float eps, float* __restrict__ dk,
                        float* __restrict__ dv) {
  constexpr int NS = DV / 32;
  constexpr int E = DV / 16;  // value elements per lane and row in the dv product
  constexpr int W = E / 2;
  constexpr int kRowU = DV / 8;                                   // 16-byte units per dout row
  constexpr int kDoutU = 16 * kRowU;                              // units of a tile's dout rows
  constexpr int kStU = (kDoutU + kKeyThreads - 1) / kKeyThreads;  // dout units staged per thread
  // Byte offsets into a segment's records and dout rows: 32-bit when the
  // segment's dout rows span under 4 GiB.
  using Off = typename RowOff<kOff32>::type;
  __shared__ __align__(16) uint32_t s_rec[2][16][8];
  __shared__ __align__(16) uint16_t s_dout[2][16][DV + 8];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int ent = lane & 15;  // this lane's entry (B column, and A row of the dot products)
  const int kg = lane >> 4;   // this lane's queries 4kg..4kg+3 of a tile
  const uint32_t li = uint32_t(level_index(lvl, causal, t0, t_hi, levels));
  const int64_t ln = (causal && lvl <= t_hi) ? (int64_t(1) << lvl) : N;
  const int64_t cl = (ln + kBtChunk - 1) / kBtChunk;
  const int64_t gps = (cl + kKeyWaves - 1) / kKeyWaves;  // groups of 4 chunks per segment
  const int64_t groups = S * gps;
  const int64_t nb = gridDim.x;
  const int32_t n32 = int32_t(N);

  for (int64_t blk = xcd_contiguous_block(blockIdx.x, nb); blk < groups; blk += nb) {
    const int64_t seg = blk / gps;
    const int64_t c0 = (blk - seg * gps) * kKeyWaves;
    const int64_t c_last = (c0 + kKeyWaves < cl ? c0 + kKeyWaves : cl) - 1;
    const int64_t c = c0 + wave;
    const bool live = c < cl;
    const LevelList L = level_list(sorted_pos, list_pos, keys_full, keys_list, seg, N, causal, lvl, t0, t_hi, cap);
    const int32_t e = int32_t(c * kBtChunk + ent);
    const bool valid_e = live && e < L.n;
    const int32_t pos_e = valid_e ? L.pos[e] : 0;
    float kv[3] = {0.0f, 0.0f, 0.0f};
    if (valid_e) key_row(L.key[e], kv);
    const uint16_t* vseg = v + seg * N * DV;
    uint32_t vfr[NS][4];  // value slices of this lane's entry: columns 32s + 8kg .. + 7
#pragma unroll
    for (int s = 0; s < NS; ++s) load8(vseg + int64_t(pos_e) * DV + 32 * s + 8 * kg, vfr[s]);

    f32x4_t acc[E];
#pragma unroll
    for (int j = 0; j < E; ++j) acc[j] = f32x4_t{0.0f, 0.0f, 0.0f, 0.0f};
    float gk[3] = {0.0f, 0.0f, 0.0f};
    bool touched = false;

    // This wave's chunk (empty when past the list) and the group's entries.
    const int lo_c = live ? int(c * kBtChunk) : 1;
    const int hi_c = live ? int(c * kBtChunk + kBtChunk - 1 < ln - 1 ? c * kBtChunk + kBtChunk - 1 : ln - 1) : 0;
    const int lo_g = int(c0 * kBtChunk);
    const int hi_g = int(c_last * kBtChunk + kBtChunk - 1 < ln - 1 ? c_last * kBtChunk + kBtChunk - 1 : ln - 1);
    const int2* ev = env + (int64_t(li) * S + seg) * ct;
    const int2* rgs = ranges + (int64_t(li) * S + seg) * ct;
    // The candidate ranges grow with the chunk: the group's is from its first
    // chunk's start to its last chunk's end.
    const int64_t ta = rgs[c0].x, tb = rgs[c_last].y;
    const unsigned char* rbase = reinterpret_cast<const unsigned char*>(rec + seg * N);
    const unsigned char* dbase = reinterpret_cast<const unsigned char*>(dslot + seg * N * DV);

    // The tiles whose windows meet the group, 64 candidates tested at once
    // (the same in every wavefront); with each, whether it meets this wave's
    // chunk.
    int64_t blk_base = ta, cur_base = ta;
    uint64_t pend = 0ull, mine = 0ull;
    auto next_tile = [&](bool& hit_w) -> int64_t {
      while (pend == 0ull && blk_base < tb) {
        const int64_t tl = blk_base + lane;
        bool hg = false, hw = false;
        if (tl < tb) {
          const int2 rg = ev[tl];
          hg = (rg.x <= hi_g) & (rg.y >= lo_g);
          hw = (rg.x <= hi_c) & (rg.y >= lo_c);
        }
        pend = wave_ballot(hg);
        mine = wave_ballot(hw);
        cur_base = blk_base;
        blk_base += 64;
      }
      if (pend == 0ull) return -1;
      const int b = __ffsll((unsigned long long)pend) - 1;
      pend &= pend - 1ull;
      hit_w = ((mine >> b) & 1ull) != 0ull;
      return cur_base + b;
    };
    uint4 st_rec = make_uint4(0u, 0u, 0u, 0u);  // 16 bytes of the records (threads 0..31)
    uint4 st_dout[kStU];
    auto stage = [&](int64_t tau) {
      const int32_t t16 = int32_t(tau) * 16;
      if (tid < 32) {
        const int32_t xs = t16 + (tid >> 1);
        const Off xq = Off(xs < n32 ? xs : n32 - 1);
        st_rec = *reinterpret_cast<const uint4*>(rbase + xq * Off(sizeof(SlotRec)) + Off((tid & 1) * 16));
      }
#pragma unroll
      for (int u = 0; u < kStU; ++u) {
        const int unit = u * kKeyThreads + tid;
        if (unit < kDoutU) {
          const int32_t xs = t16 + unit / kRowU;
          const Off xq = Off(xs < n32 ? xs : n32 - 1);
          st_dout[u] = *reinterpret_cast<const uint4*>(dbase + (xq * Off(DV) + Off((unit % kRowU) * 8)) * Off(2));
        }
      }
    };
    auto store = [&](int buf) {
      if (tid < 32) *reinterpret_cast<uint4*>(&s_rec[buf][tid >> 1][(tid & 1) * 4]) = st_rec;
#pragma unroll
      for (int u = 0; u < kStU; ++u) {
        const int unit = u * kKeyThreads + tid;
        if (unit < kDoutU) *reinterpret_cast<uint4*>(&s_dout[buf][unit / kRowU][(unit % kRowU) * 8]) = st_dout[u];
      }
    };
    auto sum_tile = [&](int64_t tau, int buf) {
      SlotRec rq[4];  // records of the tile's queries 4kg..4kg+3
#pragma unroll
      for (int r = 0; r < 4; ++r) rq[r] = *reinterpret_cast<const SlotRec*>(&s_rec[buf][kg * 4 + r][0]);
      // Dot products: lane holds p for queries 4kg..4kg+3 and entry ent (A
      // rows: dout of the tile's query ent).
      f32x4_t d = {0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        const uint4 x = *reinterpret_cast<const uint4*>(&s_dout[buf][ent][32 * s + 8 * kg]);
        const uint32_t dw[4] = {x.x, x.y, x.z, x.w};
        d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(frag8(dw).v, frag8(vfr[s]).v, d, 0, 0, 0);
      }
      float aw[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const SlotRec& rr = rq[r];
        const float qx = __uint_as_float(rr.q01 << 16);
        const float qy = __uint_as_float(rr.q01 & 0xFFFF0000u);
        const float qz = __uint_as_float(rr.q2_list << 16);
        const float df[3] = {qx - kv[0], qy - kv[1], qz - kv[2]};
        const float d2 = fmaf(df[2], df[2], fmaf(df[1], df[1], df[0] * df[0]));
        const bool in = ((rr.q2_list >> 16) == li) & (int32_t(tau) * 16 + kg * 4 + r < n32) & valid_e &
                        (uint32_t(e - rr.a) <= uint32_t(rr.b - rr.a)) & (uint32_t(pos_e) <= rr.lim);
        const float sc = in ? __builtin_amdgcn_rcpf(d2 + eps) : 0.0f;
        aw[r] = sc * rr.zinv;
        const float w = (d[r] - rr.c) * sc * aw[r];
#pragma unroll
        for (int a = 0; a < 3; ++a) gk[a] = fmaf(w, df[a], gk[a]);
      }
      // dv^T += dout^T (columns x queries) * A (queries x entries), high and
      // low parts of A in one product per 16 columns; A rows from the dout
      // rows of queries 4kg..4kg+3, elements ent*E .. ent*E + E - 1.
      Frag8 b;
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const bf16x2_t h = {(__bf16)aw[2 * t], (__bf16)aw[2 * t + 1]};
        const uint32_t hw = __builtin_bit_cast(uint32_t, h);
        const bf16x2_t l = {(__bf16)(aw[2 * t] - __uint_as_float(hw << 16)),
                            (__bf16)(aw[2 * t + 1] - __uint_as_float(hw & 0xFFFF0000u))};
        b.w[t] = hw;
        b.w[t + 2] = __builtin_bit_cast(uint32_t, l);
      }
      uint32_t raw[4][W];
#pragma unroll
      for (int r = 0; r < 4; ++r) load_words<W>(&s_dout[buf][kg * 4 + r][ent * E], raw[r]);
#pragma unroll
      for (int j = 0; j < E; ++j) {
        Frag8 a;
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const uint32_t x = raw[2 * t][j >> 1], y = raw[2 * t + 1][j >> 1];
          a.w[t] = __builtin_amdgcn_perm(y, x, (j & 1) ? 0x07060302u : 0x05040100u);
          a.w[t + 2] = a.w[t];
        }
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v, b.v, acc[j], 0, 0, 0);
      }
    };
    {
      bool cur_hit = false;
      int64_t cur = next_tile(cur_hit);
      int buf = 0;
      if (cur >= 0) {
        stage(cur);
        store(0);
      }
      __syncthreads();
      while (cur >= 0) {
        bool nxt_hit = false;
        const int64_t nxt = next_tile(nxt_hit);
        if (nxt >= 0) stage(nxt);
        if (cur_hit) {
          touched = true;
          sum_tile(cur, buf);
        }
        if (nxt >= 0) store(buf ^ 1);
        __syncthreads();
        cur = nxt;
        cur_hit = nxt_hit;
        buf ^= 1;
      }
    }

    // Write (full list) or add (prefix lists) this chunk's rows: lane holds
    // elements 4kg*E .. 4kg*E + 4E - 1 of entry ent's dv row.
#pragma unroll
    for (int a = 0; a < 3; ++a) gk[a] = 2.0f * kg_sum(gk[a]);
    if (valid_e && (first || touched)) {
      float* drow = dv + (seg * N + pos_e) * int64_t(DV) + kg * 4 * E;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        if constexpr (E % 4 == 0) {
#pragma unroll
          for (int j0 = 0; j0 < E; j0 += 4) {
            float4 o = make_float4(acc[j0][r], acc[j0 + 1][r], acc[j0 + 2][r], acc[j0 + 3][r]);
            float4* dst = reinterpret_cast<float4*>(drow + r * E + j0);
            if (!first) {
              const float4 old = *dst;
              o.x += old.x;
              o.y += old.y;
              o.z += old.z;
              o.w += old.w;
            }
            *dst = o;
          }
        } else {
          static_assert(E == 2, "d_v of 32 gives two elements per row and lane");
          float2 o = make_float2(acc[0][r], acc[1][r]);
          float2* dst = reinterpret_cast<float2*>(drow + r * E);
          if (!first) {
            const float2 old = *dst;
            o.x += old.x;
            o.y += old.y;
          }
          *dst = o;
        }
      }
      if (kg == 0) {
        float* krow = dk + (seg * N + pos_e) * 3;
#pragma unroll
        for (int a = 0; a < 3; ++a) krow[a] = first ? gk[a] : krow[a] + gk[a];
      }
    }
    // The next group reuses the LDS buffers.
    __syncthreads();
  }
}

// ---- deps -----------------------------------------------------------------------
// Fixed-order sum of the per-slot parts: block sums, then one block over them.
__global__ void __launch_bounds__(kRedThreads)
    bwd_tile_reduce_kernel(const float* __restrict__ part, int64_t n, int64_t per_block, float* __restrict__ sums) {
  __shared__ float s_red[kRedThreads];
  const int64_t b0 = int64_t(blockIdx.x) * per_block;
  const int64_t b1 = b0 + per_block < n ? b0 + per_block : n;
  float acc = 0.0f;
  for (int64_t t = b0 + threadIdx.x; t < b1; t += kRedThreads) acc += part[t];
  s_red[threadIdx.x] = acc;
  __syncthreads();
  for (int w = kRedThreads / 2; w > 0; w >>= 1) {
    if (int(threadIdx.x) < w) s_red[threadIdx.x] += s_red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) sums[blockIdx.x] = s_red[0];
}

__global__ void __launch_bounds__(256) bwd_tile_fill_int2_kernel(int2* __restrict__ p, int64_t n, int2 val) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t t = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; t < n; t += stride) p[t] = val;
}

template <int DV>
hipError_t launch_tile_bwd_t(const uint16_t* q, const uint16_t* v, const uint16_t* dout, int64_t S, int64_t N,
                             int topk, bool causal, int chunk, const int32_t* perm, const int32_t* list_pos,
                             const int32_t* q_order, const int2* bounds, const uint2* keys_full,
                             const uint2* keys_list, float eps, HistMean hm, float* dq, float* dk, float* dv,
                             float* deps, const TileBwdWs& ws, char* wsb, hipStream_t stream) {
  const ListPlan lp = list_plan(N, topk);
  const int64_t ct = ceil_div(N, int64_t(16));
  const int nl = tile_bwd_levels(N, topk, causal);
  const bool off32 = N * int64_t(DV) * 2 <= int64_t(0xFFFFFFFF);
  SlotRec* rec = reinterpret_cast<SlotRec*>(wsb + ws.rec_off);
  uint16_t* dslot = reinterpret_cast<uint16_t*>(wsb + ws.dslot_off);
  float* part = reinterpret_cast<float*>(wsb + ws.part_off);
  int2* env = reinterpret_cast<int2*>(wsb + ws.env_off);
  int2* env2 = reinterpret_cast<int2*>(wsb + ws.env2_off);
  int2* ranges = reinterpret_cast<int2*>(wsb + ws.ranges_off);
  float* hk = reinterpret_cast<float*>(wsb + ws.hist_k_off);
  float* hv = reinterpret_cast<float*>(wsb + ws.hist_v_off);
  float* sums = reinterpret_cast<float*>(wsb + ws.sums_off);
  const int64_t nenv = int64_t(nl) * S * ct;
  {
    const int64_t want = ceil_div(nenv, int64_t(256));
    hipLaunchKernelGGL(bwd_tile_fill_int2_kernel, dim3(unsigned(want < 65536 ? want : 65536)), dim3(256), 0, stream,
                       env, nenv, make_int2(INT32_MAX, INT32_MIN));
  }
  const int cz = causal ? 1 : 0;
  {
    const int64_t tiles = S * ct;
    const int64_t want = ceil_div(tiles, int64_t(kBtWaves));
    const unsigned blocks = unsigned(want < (int64_t(1) << 20) ? want : (int64_t(1) << 20));
#define ZETA_BT_QUERY(HIST)                                                                                     \
  hipLaunchKernelGGL((bwd_tile_query_kernel<DV, HIST>), dim3(blocks), dim3(kBtWaves * 64), 0, stream, q, v, dout, perm, \
                     list_pos, q_order, bounds, keys_full, keys_list, S, N, ct, cz, chunk, lp.t0, lp.t_hi, lp.levels,   \
                     lp.cap, eps, dq, rec, dslot, part, env, hm.k, hm.v, hk, hv)
    if (hm.k != nullptr)
      ZETA_BT_QUERY(true);
    else
      ZETA_BT_QUERY(false);
#undef ZETA_BT_QUERY
  }
  hipLaunchKernelGGL(bwd_envelope_kernel, dim3(unsigned(int64_t(nl) * S)), dim3(kEnvThreads), 0, stream, env, ct,
                     env2);
  hipLaunchKernelGGL(bwd_ranges_kernel, dim3(unsigned(ceil_div(nenv, int64_t(256)))), dim3(256), 0, stream, env2, S, N,
                     ct, cz, lp.t0, lp.t_hi, lp.levels, nl, ranges);
  // The full list first (its launch writes every key's rows), then the prefix
  // lists from the longest down.
  for (int li = nl - 1; li >= 0; --li) {
    const int lvl = !causal ? 0 : (li == lp.levels ? lp.t_hi + 1 : lp.t0 + li);
    const int64_t ln = (causal && lvl <= lp.t_hi) ? (int64_t(1) << lvl) : N;
    const int64_t want = S * ceil_div(ceil_div(ln, int64_t(16)), int64_t(kKeyWaves));  // groups of chunks
    const unsigned blocks = unsigned(want < (int64_t(1) << 20) ? want : (int64_t(1) << 20));
#define ZETA_BT_KEY(OFF)                                                                                       \
  hipLaunchKernelGGL((bwd_tile_key_kernel<DV, OFF>), dim3(blocks), dim3(kKeyThreads), 0, stream, v, perm, list_pos,    \
                     keys_full, keys_list, rec, dslot, env, ranges, S, N, ct, cz, lp.t0, lp.t_hi, lp.levels, lp.cap,  \
                     lvl, li == nl - 1 ? 1 : 0, eps, dk, dv)
    if (off32)
      ZETA_BT_KEY(true);
    else
      ZETA_BT_KEY(false);
#undef ZETA_BT_KEY
  }
  if (hm.k != nullptr) {
    // The gradients reaching the means pass to the rows of every history.
    const hipError_t e = launch_history_spread(hv, dv, DV, hk, dk, 3, S, N, causal, wsb + ws.hist_scan_off, stream);
    if (e != hipSuccess) return e;
  }
  const int64_t total = S * N;
  const int64_t nred = ceil_div(total, kTileBwdRedPer) < kTileBwdRedMax ? ceil_div(total, kTileBwdRedPer)
                                                                        : kTileBwdRedMax;
  const int64_t per = ceil_div(total, nred);
  hipLaunchKernelGGL(bwd_tile_reduce_kernel, dim3(unsigned(nred)), dim3(kRedThreads), 0, stream, part, total, per,
                     sums);
  hipLaunchKernelGGL(bwd_tile_reduce_kernel, dim3(1), dim3(kRedThreads), 0, stream, sums, nred, nred, deps);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_select_attend_bwd(const void* q, const void* k, const void* v, const void* dout, int64_t S,
                                    int64_t N, int dk_, int dv_, int topk, bool causal, int chunk,
                                    const uint32_t* q_codes, const uint32_t* sorted_codes, const int32_t* perm,
                                    const int32_t* q_order, float eps, HistMean hm, float* dq, float* dk,
                                    float* dv, float* deps, void* workspace, hipStream_t stream) {
  const uint32_t* list_codes = nullptr;
  const int32_t* list_pos = nullptr;
  const TileBwdWs ws = tile_bwd_ws(S, N, dv_, topk, causal ? 1 : 0, hm.k != nullptr);
  char* wsb = static_cast<char*>(workspace);
  int2* bounds = reinterpret_cast<int2*>(wsb + ws.fused.bounds_off);
  uint2* keys_full = reinterpret_cast<uint2*>(wsb + ws.fused.keys_full_off);
  uint2* keys_list = reinterpret_cast<uint2*>(wsb + ws.fused.keys_list_off);
  if (causal) {
    // The key rows in list order come with the prefix lists.
    const hipError_t e = launch_prefix_lists(sorted_codes, perm, S, N, topk, workspace, stream, &list_codes,
                                             &list_pos, static_cast<const uint16_t*>(k), keys_full, keys_list);
    if (e != hipSuccess) return e;
  }
  hipError_t e = launch_tile_windows(k, S, N, dk_, topk, causal, chunk, q_codes, sorted_codes, perm, list_codes,
                                     list_pos, q_order, nullptr, bounds, keys_full, keys_list, list_codes != nullptr,
                                     stream);
  if (e != hipSuccess) return e;
  const uint16_t* qq = static_cast<const uint16_t*>(q);
  const uint16_t* vv = static_cast<const uint16_t*>(v);
  const uint16_t* dd = static_cast<const uint16_t*>(dout);
#define ZETA_TILE_BWD_CASE(DVV)                                                                                      \
  case DVV:                                                                                                          \
    return launch_tile_bwd_t<DVV>(qq, vv, dd, S, N, topk, causal, chunk, perm, list_pos, q_order, bounds, keys_full, \
                                  keys_list, eps, hm, dq, dk, dv, deps, ws, wsb, stream);
  switch (dv_) {
    ZETA_TILE_BWD_CASE(32)
    ZETA_TILE_BWD_CASE(64)
    ZETA_TILE_BWD_CASE(128)
    ZETA_TILE_BWD_CASE(256)
    default:
      return hipErrorInvalidValue;
  }
#undef ZETA_TILE_BWD_CASE
}

}  // namespace zeta
