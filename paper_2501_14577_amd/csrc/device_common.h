// Wavefront primitives and element conversions shared by the gfx950 kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace zeta {

// Number of set bits of `mask` held by lanes below the calling lane.
__device__ __forceinline__ uint32_t lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi(uint32_t(mask >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(mask), 0u));
}

__device__ __forceinline__ uint32_t lane_id() { return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u)); }

__device__ __forceinline__ uint64_t wave_ballot(bool p) { return __ballot(p); }

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off, 64);
  return x;
}

__device__ __forceinline__ int wave_max(int x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    int y = __shfl_xor(x, off, 64);
    x = y > x ? y : x;
  }
  return x;
}

__device__ __forceinline__ float wave_max_f(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x = fmaxf(x, __shfl_xor(x, off, 64));
  return x;
}

// Orders this wave's earlier LDS writes before its later LDS reads (lanes of
// one wavefront exchanging data through LDS without a block barrier).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Workgroups are dispatched to the 8 XCDs round-robin (block b runs on XCD
// b % 8).  This maps a hardware block index to a logical one so that each XCD
// receives one contiguous range of logical blocks, keeping neighbouring work
// (which shares data) under one L2.  A bijection on [0, nb).
__device__ __forceinline__ int64_t xcd_contiguous_block(int64_t b, int64_t nb) {
  constexpr int64_t kXcds = 8;
  const int64_t per = nb / kXcds, extra = nb % kXcds;
  const int64_t x = b % kXcds, l = b / kXcds;
  return (x < extra) ? x * (per + 1) + l : extra * (per + 1) + (x - extra) * per + l;
}

// Exclusive prefix sum over a block of exactly 64 * kWaves threads (one value
// each).  `scratch` must hold kWaves words.  Contains block barriers: every
// thread calls it.
template <int kWaves>
__device__ __forceinline__ uint32_t block_exclusive_scan(uint32_t x, uint32_t* scratch) {
  const uint32_t lane = threadIdx.x & 63u, wave = threadIdx.x >> 6;
  uint32_t incl = x;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    uint32_t y = __shfl_up(incl, off, 64);
    if (lane >= uint32_t(off)) incl += y;
  }
  if (lane == 63) scratch[wave] = incl;
  __syncthreads();
  uint32_t base = 0;
  for (uint32_t w = 0; w < wave; ++w) base += scratch[w];
  __syncthreads();
  return base + incl - x;
}

// ---- element conversions -------------------------------------------------

__device__ __forceinline__ float bf16_bits_to_float(uint16_t b) { return __uint_as_float(uint32_t(b) << 16); }

// Round to nearest, ties to even (inputs are finite).
__device__ __forceinline__ uint16_t float_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return uint16_t(u >> 16);
}

template <typename T>
struct Elem;

template <>
struct Elem<float> {
  __device__ __forceinline__ static float load(const float* p) { return *p; }
};

template <>
struct Elem<uint16_t> {
  __device__ __forceinline__ static float load(const uint16_t* p) { return bf16_bits_to_float(*p); }
};

}  // namespace zeta
