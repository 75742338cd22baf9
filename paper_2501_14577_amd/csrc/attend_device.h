// Device-side row access shared by the attend and fused select-and-attend
// kernels: 16-byte lane loads of value rows widened to float32, one-load key
// and query rows for d_k = 3, and row offsets.
#pragma once

#include <stdint.h>

#include "device_common.h"

namespace zeta {
namespace {

template <typename T>
struct Vec16;  // one 16-byte lane load of a value row, widened to float32

template <>
struct Vec16<float> {
  static constexpr int kElems = 4;
  __device__ __forceinline__ static void widen(const uint4& x, float* f) {
    f[0] = __uint_as_float(x.x);
    f[1] = __uint_as_float(x.y);
    f[2] = __uint_as_float(x.z);
    f[3] = __uint_as_float(x.w);
  }
  __device__ __forceinline__ static void store(float* p, const float* f) {
    *reinterpret_cast<float4*>(p) = make_float4(f[0], f[1], f[2], f[3]);
  }
};

template <>
struct Vec16<uint16_t> {
  static constexpr int kElems = 8;
  __device__ __forceinline__ static void widen(const uint4& x, float* f) {
    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = __uint_as_float(w[i] << 16);
      f[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  }
  __device__ __forceinline__ static void store(uint16_t* p, const float* f) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = uint32_t(float_to_bf16_bits(f[2 * i])) | (uint32_t(float_to_bf16_bits(f[2 * i + 1])) << 16);
    *reinterpret_cast<uint4*>(p) = make_uint4(w[0], w[1], w[2], w[3]);
  }
};

// The three coordinates of row `row` of a [rows][3] array, widened to
// float32, with one memory instruction: a float32 row is one 12-byte load; a
// bfloat16 row (6 bytes, 2-byte aligned) lies inside the 8 bytes starting at
// the 4-byte boundary at or below it, except that the array's very last row
// may end 2 bytes before that window does, so it is read element by element.
struct alignas(4) Words2 {
  uint32_t a, b;
};
struct alignas(4) Floats3 {
  float x, y, z;
};

template <typename T>
struct Row3;

template <>
struct Row3<float> {
  __device__ __forceinline__ static void load(const float* base, int64_t row, int64_t /*rows*/, float* f) {
    const Floats3 r = *reinterpret_cast<const Floats3*>(base + row * 3);
    f[0] = r.x;
    f[1] = r.y;
    f[2] = r.z;
  }
};

template <>
struct Row3<uint16_t> {
  __device__ __forceinline__ static void load(const uint16_t* base, int64_t row, int64_t rows, float* f) {
    const int64_t e = row * 3;
    const int64_t a = e & ~int64_t(1);
    if (a + 4 <= rows * 3) {
      const Words2 w = *reinterpret_cast<const Words2*>(base + a);
      if (e == a) {
        f[0] = __uint_as_float(w.a << 16);
        f[1] = __uint_as_float(w.a & 0xFFFF0000u);
        f[2] = __uint_as_float(w.b << 16);
      } else {
        f[0] = __uint_as_float(w.a & 0xFFFF0000u);
        f[1] = __uint_as_float(w.b << 16);
        f[2] = __uint_as_float(w.b & 0xFFFF0000u);
      }
    } else {
      f[0] = bf16_bits_to_float(base[e]);
      f[1] = bf16_bits_to_float(base[e + 1]);
      f[2] = bf16_bits_to_float(base[e + 2]);
    }
  }
};

// Row `row` of a bfloat16 [rows][3] array as three bfloat16 bit patterns in
// 8 bytes (x | y << 16, z), read the way Row3 reads it.
__device__ __forceinline__ uint2 packed_key_row(const uint16_t* base, int64_t row, int64_t rows) {
  const int64_t e = row * 3;
  const int64_t a = e & ~int64_t(1);
  uint32_t x, y, z;
  if (a + 4 <= rows * 3) {
    const Words2 w = *reinterpret_cast<const Words2*>(base + a);
    if (e == a) {
      x = w.a & 0xFFFFu;
      y = w.a >> 16;
      z = w.b & 0xFFFFu;
    } else {
      x = w.a >> 16;
      y = w.b & 0xFFFFu;
      z = w.b >> 16;
    }
  } else {
    x = base[e];
    y = base[e + 1];
    z = base[e + 2];
  }
  return make_uint2(x | (y << 16), z);
}

// Byte offset of a value row inside its segment: 32-bit when the segment's
// values span less than 4 GiB, else 64-bit.
template <bool kOff32>
struct RowOff {
  using type = int64_t;
};
template <>
struct RowOff<true> {
  using type = uint32_t;
};

// Score of the history-mean candidate of query row g (Section 3.4): the
// Cauchy score against the float32 mean key row mk[g].
template <int KD>
__device__ __forceinline__ float mean_score(const float* __restrict__ mk, int64_t g, int dk, const float* qv,
                                            float eps) {
  float d2 = 0.0f;
#pragma unroll
  for (int a = 0; a < KD; ++a) {
    if (a < dk) {
      const float diff = qv[a] - mk[g * dk + a];
      d2 = fmaf(diff, diff, d2);
    }
  }
  return 1.0f / (d2 + eps);
}

// Score variants (Section 4.3; Appendix G.2; equation 3) over the same
// candidates.  mode: 1 dot-product softmax, 2 negative-Euclidean softmax,
// 3 inverse Euclidean, 4 normalised dot-product softmax (the Cauchy score,
// mode 0, is computed inline by the kernels).  Returns the weight itself
// (inverse Euclidean: 1 / (|q - k| + eps)) or the logit of a softmax
// (q.k / sqrt(d), -|q - k|^2 / sqrt(d), (q/|q|).(k/|k|) / sqrt(d); a zero
// vector gives 0).  rsd = 1 / sqrt(d); qn = |q|.  The result is rounded as
// written (no multiply fused into the caller's next add), so every inlined
// copy of a kernel's scoring gives the same bits.
template <int KD>
__device__ __forceinline__ float variant_term(int mode, const float* qv, const float* kv, int dk, float eps, float rsd,
                                              float qn) {
#pragma clang fp contract(off)
  float d2 = 0.0f, dot = 0.0f, kk = 0.0f;
#pragma unroll
  for (int a = 0; a < KD; ++a) {
    if (a < dk) {
      const float diff = qv[a] - kv[a];
      d2 = fmaf(diff, diff, d2);
      dot = fmaf(qv[a], kv[a], dot);
      kk = fmaf(kv[a], kv[a], kk);
    }
  }
  switch (mode) {
    case 1:
      return dot * rsd;
    case 2:
      return -d2 * rsd;
    case 3:
      return 1.0f / (sqrtf(d2) + eps);
    default: {
      const float kn = sqrtf(kk);
      return (qn > 0.0f && kn > 0.0f) ? dot / (qn * kn) * rsd : 0.0f;
    }
  }
}

// |q| of a query row (for the normalised dot product).
template <int KD>
__device__ __forceinline__ float row_norm(const float* qv, int dk) {
  float s = 0.0f;
#pragma unroll
  for (int a = 0; a < KD; ++a)
    if (a < dk) s = fmaf(qv[a], qv[a], s);
  return sqrtf(s);
}

// Softmax variants: turns this lane's logits s_w[c] into exp(z - zmax) over
// the slots it scored (slot pairs 2*lane, 2*lane + 1 of every 128; bit b of
// okmask marks its b-th slot valid; zloc is its largest valid logit), and the
// history-mean candidate's logit into its weight; returns the wavefront's
// sum of the weights.  zmax is the largest logit of the window and the
// candidate (0 when there is none).
__device__ __forceinline__ float softmax_weights(float* s_w, int topk, int lane, uint32_t okmask, float zloc,
                                                 bool has_mean, float& s_mean) {
  float zmax = wave_max_f(zloc);
  if (has_mean) zmax = fmaxf(zmax, s_mean);
  if (!(zmax > -INFINITY)) zmax = 0.0f;
  float zs = 0.0f;
  int b = 0;
  for (int c0 = 2 * lane; c0 < topk; c0 += 128) {
#pragma unroll
    for (int h = 0; h < 2; ++h, ++b) {
      if ((okmask >> b) & 1u) {
        const float e = expf(s_w[c0 + h] - zmax);
        s_w[c0 + h] = e;
        zs += e;
      }
    }
  }
  float z = wave_sum(zs);
  if (has_mean) {
    s_mean = expf(s_mean - zmax);
    z += s_mean;
  }
  return z;
}

// acc[e] += s * mean value row elements [0, n) at p (16-byte aligned float32).
template <int n>
__device__ __forceinline__ void add_mean_value(const float* __restrict__ p, float s, float* acc) {
#pragma unroll
  for (int e = 0; e < n; e += 4) {
    const float4 m = *reinterpret_cast<const float4*>(p + e);
    acc[e] = fmaf(s, m.x, acc[e]);
    acc[e + 1] = fmaf(s, m.y, acc[e + 1]);
    acc[e + 2] = fmaf(s, m.z, acc[e + 2]);
    acc[e + 3] = fmaf(s, m.w, acc[e + 3]);
  }
}

}  // namespace
}  // namespace zeta
