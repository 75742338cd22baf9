// Z-order encoding of queries and keys (Section 3.1, equation Z).
//
// Two kernels:
//  1. range_partial: per (segment, chunk of rows) min/max of every axis over
//     the chunk's query and key rows.  Consecutive threads read consecutive
//     elements; the block is 64*d_k threads so each thread stays on one axis.
//  2. encode: every block first folds its segment's partial ranges (all
//     threads load partials at once, then combine per axis in LDS), then
//     quantises and interleaves 256 query rows and 256 key rows, each row read
//     with one load.  Quantisation is float32 with one rounding per operation,
//     matching the definition bit for bit.
#include "attend_device.h"
#include "device_common.h"
#include "kernels.h"
#include "layout.h"

#include <mutex>

namespace zeta {
namespace {

template <typename T>
__global__ void range_partial_kernel(const T* __restrict__ q, const T* __restrict__ k, int64_t N,
                                     int dk, int64_t chunks, float* __restrict__ partial) {
  const int64_t seg = blockIdx.x / chunks;
  const int64_t chunk = blockIdx.x % chunks;
  const int64_t r0 = chunk * kEncRowsPerChunk;
  const int64_t r1 = (r0 + kEncRowsPerChunk < N) ? r0 + kEncRowsPerChunk : N;
  const int tid = threadIdx.x;  // blockDim.x == 64 * dk
  const int64_t e_end = r1 * dk;
  const int64_t stride = int64_t(blockDim.x);
  const T* qs = q + seg * N * dk;
  const T* ks = k + seg * N * dk;
  float lo = __builtin_huge_valf(), hi = -__builtin_huge_valf();
  for (int64_t e = r0 * dk + tid; e < e_end; e += stride) {
    float a = Elem<T>::load(qs + e);
    float b = Elem<T>::load(ks + e);
    lo = fminf(lo, fminf(a, b));
    hi = fmaxf(hi, fmaxf(a, b));
  }
  __shared__ float s_lo[64 * kMaxDk];
  __shared__ float s_hi[64 * kMaxDk];
  s_lo[tid] = lo;
  s_hi[tid] = hi;
  __syncthreads();
  if (tid < dk) {
    float l = s_lo[tid], h = s_hi[tid];
    for (int t = tid + dk; t < int(blockDim.x); t += dk) {
      l = fminf(l, s_lo[t]);
      h = fmaxf(h, s_hi[t]);
    }
    float* out = partial + (seg * chunks + chunk) * 2 * dk;
    out[tid] = l;
    out[dk + tid] = h;
  }
}

// Grid coordinate of one value: floor((x - lo) * (2^bits - 1) / (hi - lo)),
// clamped, in float32 with one rounding per operation.
__device__ __forceinline__ uint32_t quantise(float x, float lo, float hi, int bits) {
#pragma clang fp contract(off)
  const uint32_t top = (1u << bits) - 1u;
  const float den = hi - lo;
  if (!(den > 0.0f)) return 0u;
  const float t = x - lo;
  const float u = t * float(top);
  const float w = __fdiv_rn(u, den);
  const float f = floorf(w);
  if (!(f > 0.0f)) return 0u;
  if (f >= float(top)) return top;
  return uint32_t(f);
}

// Spread the low 10 bits of x to every third bit position.
__device__ __forceinline__ uint32_t spread3(uint32_t x) {
  x &= 0x3FFu;
  x = (x | (x << 16)) & 0x030000FFu;
  x = (x | (x << 8)) & 0x0300F00Fu;
  x = (x | (x << 4)) & 0x030C30C3u;
  x = (x | (x << 2)) & 0x09249249u;
  return x;
}

// Code of row `r` of a [rows][dk] array.
template <typename T>
__device__ __forceinline__ uint32_t encode_row(const T* base, int64_t r, int64_t rows, const float* lo,
                                               const float* hi, int dk, int bits) {
  if (dk == 3) {
    float x[3];
    Row3<T>::load(base, r, rows, x);
    const uint32_t c0 = quantise(x[0], lo[0], hi[0], bits);
    const uint32_t c1 = quantise(x[1], lo[1], hi[1], bits);
    const uint32_t c2 = quantise(x[2], lo[2], hi[2], bits);
    return (spread3(c0) << 2) | (spread3(c1) << 1) | spread3(c2);
  }
  const T* row = base + r * dk;
  uint32_t z = 0;
  for (int a = 0; a < dk; ++a) {
    const uint32_t c = quantise(Elem<T>::load(row + a), lo[a], hi[a], bits);
    for (int s = 0; s < bits; ++s) z |= ((c >> s) & 1u) << (dk * s + (dk - 1 - a));
  }
  return z;
}

template <typename T>
__global__ void __launch_bounds__(256) encode_kernel(const T* __restrict__ q, const T* __restrict__ k,
                                                     int64_t N, int dk, int bits,
                                                     const float* __restrict__ partial, int64_t chunks,
                                                     const float* __restrict__ range_lohi,
                                                     float* __restrict__ range_out,
                                                     uint32_t* __restrict__ q_codes,
                                                     uint32_t* __restrict__ k_codes,
                                                     int64_t blocks_per_seg, int64_t S) {
  const int64_t seg = blockIdx.x / blocks_per_seg;
  const int64_t blk = blockIdx.x % blocks_per_seg;
  __shared__ float s_lo[kMaxDk], s_hi[kMaxDk];
  __shared__ float s_plo[kEncRowsPerBlock], s_phi[kEncRowsPerBlock];
  const int tid = threadIdx.x;
  if (range_lohi != nullptr) {
    if (tid < dk) {
      s_lo[tid] = range_lohi[seg * 2 * dk + tid];
      s_hi[tid] = range_lohi[seg * 2 * dk + dk + tid];
    }
  } else {
    // Fold the segment's partial ranges: every thread takes the partials of
    // one axis (tid % dk) from chunks tid / dk, tid / dk + 256 / dk, ...
    // (all loads independent), then threads of one axis combine in LDS.
    const int per = kEncRowsPerBlock / dk;  // partials of one axis per round
    const int a = tid % dk;
    float lo = __builtin_huge_valf(), hi = -__builtin_huge_valf();
    if (tid < per * dk) {
      const float* p = partial + seg * chunks * 2 * dk;
      for (int64_t c = tid / dk; c < chunks; c += per) {
        lo = fminf(lo, p[c * 2 * dk + a]);
        hi = fmaxf(hi, p[c * 2 * dk + dk + a]);
      }
    }
    s_plo[tid] = lo;
    s_phi[tid] = hi;
    __syncthreads();
    if (tid < dk) {
      for (int t = tid + dk; t < per * dk; t += dk) {
        lo = fminf(lo, s_plo[t]);
        hi = fmaxf(hi, s_phi[t]);
      }
      s_lo[tid] = lo;
      s_hi[tid] = hi;
    }
  }
  __syncthreads();
  if (range_out != nullptr && blk == 0 && tid < dk) {
    range_out[seg * 2 * dk + tid] = s_lo[tid];
    range_out[seg * 2 * dk + dk + tid] = s_hi[tid];
  }
  const int64_t r = blk * kEncRowsPerBlock + tid;
  if (r < N) {
    const int64_t off = seg * N + r;
    q_codes[off] = encode_row(q, off, S * N, s_lo, s_hi, dk, bits);
    k_codes[off] = encode_row(k, off, S * N, s_lo, s_hi, dk, bits);
  }
}

template <typename T>
hipError_t launch_encode_t(const T* q, const T* k, int64_t S, int64_t N, int dk, int bits,
                           const float* range_lohi, float* range_out, uint32_t* q_codes,
                           uint32_t* k_codes, void* workspace, hipStream_t stream) {
  const EncodeWs ws = encode_ws(S, N, dk);
  float* partial = nullptr;
  if (range_lohi == nullptr) {
    partial = reinterpret_cast<float*>(static_cast<char*>(workspace) + ws.partial_off);
    hipLaunchKernelGGL(range_partial_kernel<T>, dim3(unsigned(S * ws.chunks)), dim3(64 * dk), 0,
                       stream, q, k, N, dk, ws.chunks, partial);
  }
  const int64_t bps = ceil_div(N, kEncRowsPerBlock);
  hipLaunchKernelGGL(encode_kernel<T>, dim3(unsigned(S * bps)), dim3(unsigned(kEncRowsPerBlock)), 0,
                     stream, q, k, N, dk, bits, partial, ws.chunks, range_lohi, range_out, q_codes,
                     k_codes, bps, S);
  return hipGetLastError();
}

// Range partials of the allocation-free entry point: one copy per GPU, held
// until the process ends.  Host code never passes `scratch` itself (its name
// is a host-side stand-in, not a device address); it passes the address that
// hipGetSymbolAddress returns for the device, taken once per device.
static __device__ __align__(256) unsigned char scratch[kEncStaticScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the stream's device (the current device for
// the null stream), looked up with that device current on its first use.
hipError_t static_scratch(hipStream_t stream, void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (stream != nullptr) {
    hipDevice_t sd = 0;
    e = hipStreamGetDevice(stream, &sd);
    if (e != hipSuccess) return e;
    dev = int(sd);
  }
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    int cur = 0;
    e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (cur != dev) {
      const hipError_t e2 = hipSetDevice(cur);
      if (e == hipSuccess) e = e2;
    }
    if (e != hipSuccess) return e;
    if (ptr == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

hipError_t launch_encode_static(const void* q, const void* k, bool is_bf16, int64_t S, int64_t N, int dk, int bits,
                                const float* range_lohi, float* range_out, uint32_t* q_codes, uint32_t* k_codes,
                                hipStream_t stream) {
  void* ws = nullptr;
  if (range_lohi == nullptr) {
    const hipError_t e = static_scratch(stream, &ws);
    if (e != hipSuccess) return e;
  }
  return launch_encode(q, k, is_bf16, S, N, dk, bits, range_lohi, range_out, q_codes, k_codes, ws, stream);
}

hipError_t launch_encode(const void* q, const void* k, bool is_bf16, int64_t S, int64_t N, int dk,
                         int bits, const float* range_lohi, float* range_out, uint32_t* q_codes,
                         uint32_t* k_codes, void* workspace, hipStream_t stream) {
  if (is_bf16)
    return launch_encode_t(static_cast<const uint16_t*>(q), static_cast<const uint16_t*>(k), S, N, dk,
                           bits, range_lohi, range_out, q_codes, k_codes, workspace, stream);
  return launch_encode_t(static_cast<const float*>(q), static_cast<const float*>(k), S, N, dk, bits,
                         range_lohi, range_out, q_codes, k_codes, workspace, stream);
}

}  // namespace zeta
