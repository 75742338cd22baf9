// Matrix-core operand types and wavefront helpers shared by the bfloat16
// tile kernels (the one-pass attention and its gradients).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace zeta {

typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));

union Frag {  // four bfloat16 values
  uint32_t w[2];
  s16x4_t v;
};

union Frag8 {  // eight bfloat16 values
  uint32_t w[4];
  bf16x8_t v;
};

// Minimum / maximum over the wavefront, read by every lane: within each row
// of 16 lanes by four DPP exchanges (swap neighbours, swap pairs, mirror the
// half row, mirror the row), then rows 1 and 3 take row 0's and row 2's
// result (row_bcast:15) and rows 2 and 3 take lane 31's (row_bcast:31), so
// lane 63 holds the wavefront's result.  No LDS round trip (unlike a
// shuffle through ds_bpermute).
template <bool kMax>
__device__ __forceinline__ int wave_reduce_minmax(int x) {
  auto op = [](int a, int b) { return kMax ? (a > b ? a : b) : (a < b ? a : b); };
  x = op(x, __builtin_amdgcn_update_dpp(x, x, 0xB1, 0xF, 0xF, false));   // quad_perm [1,0,3,2]
  x = op(x, __builtin_amdgcn_update_dpp(x, x, 0x4E, 0xF, 0xF, false));   // quad_perm [2,3,0,1]
  x = op(x, __builtin_amdgcn_update_dpp(x, x, 0x141, 0xF, 0xF, false));  // row_half_mirror
  x = op(x, __builtin_amdgcn_update_dpp(x, x, 0x140, 0xF, 0xF, false));  // row_mirror
  x = op(x, __builtin_amdgcn_update_dpp(x, x, 0x142, 0xA, 0xF, false));  // row_bcast:15 into rows 1, 3
  x = op(x, __builtin_amdgcn_update_dpp(x, x, 0x143, 0xC, 0xF, false));  // row_bcast:31 into rows 2, 3
  return __builtin_amdgcn_readlane(x, 63);
}

__device__ __forceinline__ int wave_min_int(int x) { return wave_reduce_minmax<false>(x); }

__device__ __forceinline__ int wave_max_int(int x) { return wave_reduce_minmax<true>(x); }

// Lane `src`'s value of a pointer, read by every lane.  Each 32-bit half goes
// through uint32_t: widening a negative int32 would sign-extend into the
// high half.
template <typename T>
__device__ __forceinline__ T* readlane_ptr(T* p, int src) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = uint32_t(__builtin_amdgcn_readlane(int32_t(uint32_t(v)), src));
  const uint32_t hi = uint32_t(__builtin_amdgcn_readlane(int32_t(uint32_t(v >> 32)), src));
  // Rebuilt as a global-memory pointer, so that loads through it are global
  // loads rather than flat ones.
  using G = __attribute__((address_space(1))) T;
  G* g = (G*)((uint64_t(hi) << 32) | uint64_t(lo));
  return (T*)g;
}

// E consecutive bfloat16 elements (E / 2 words) from a 2E-byte aligned address.
template <int W>
__device__ __forceinline__ void load_words(const uint16_t* p, uint32_t (&o)[W]) {
  if constexpr (W % 4 == 0) {
#pragma unroll
    for (int t = 0; t < W / 4; ++t) {
      const uint4 x = reinterpret_cast<const uint4*>(p)[t];
      o[4 * t] = x.x;
      o[4 * t + 1] = x.y;
      o[4 * t + 2] = x.z;
      o[4 * t + 3] = x.w;
    }
  } else if constexpr (W == 2) {
    const uint2 x = *reinterpret_cast<const uint2*>(p);
    o[0] = x.x;
    o[1] = x.y;
  } else {
    static_assert(W == 1, "unsupported row slice");
    o[0] = *reinterpret_cast<const uint32_t*>(p);
  }
}

}  // namespace zeta
