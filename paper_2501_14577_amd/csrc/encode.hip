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
// For d_k = 3 with 16-byte aligned tensors and N a multiple of 8 (every
// workload here) both kernels take a vector form instead: a thread owns 8
// consecutive rows, read as whole 16-byte vectors (24 values: three loads of
// bfloat16, six of float32) and written as two 16-byte code stores; a block
// covers 1024 rows of one segment (grid: chunks x segments, no index
// division; up to 65535 segments).  The quotient of the quantiser comes from the hardware
// reciprocal unless it lies close enough to an integer that the correctly
// rounded division could floor differently; then the IEEE division decides
// (the codes are those of the definition either way).
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

// ---- d_k = 3, vector form ---------------------------------------------------

constexpr int kEnc3Threads = 128;
constexpr int kEnc3Rows = 8;                                  // rows per thread
constexpr int64_t kEnc3Chunk = int64_t(kEnc3Threads) * kEnc3Rows;  // rows per block

// Rows r .. r+7 of a [rows][3] array whose row r starts on a 16-byte
// boundary: 24 values.
template <typename T>
__device__ __forceinline__ void load_rows8(const T* base, int64_t r, float (&x)[24]) {
  const uint4* p = reinterpret_cast<const uint4*>(base + r * 3);
  if constexpr (sizeof(T) == 2) {
    const uint4 a = p[0], b = p[1], c = p[2];
    const uint32_t w[12] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w, c.x, c.y, c.z, c.w};
#pragma unroll
    for (int i = 0; i < 12; ++i) {
      x[2 * i] = __uint_as_float(w[i] << 16);
      x[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
  } else {
#pragma unroll
    for (int i = 0; i < 6; ++i) {
      const uint4 v = p[i];
      x[4 * i] = __uint_as_float(v.x);
      x[4 * i + 1] = __uint_as_float(v.y);
      x[4 * i + 2] = __uint_as_float(v.z);
      x[4 * i + 3] = __uint_as_float(v.w);
    }
  }
}

// Per-axis min and max of (lo[a], hi[a]) over the block (128 threads), result
// in s_lo / s_hi.
__device__ __forceinline__ void block128_range3(float (&lo)[3], float (&hi)[3], float* s_lo, float* s_hi) {
  __shared__ float s_part[2][6];
#pragma unroll
  for (int a = 0; a < 3; ++a) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      lo[a] = fminf(lo[a], __shfl_xor(lo[a], off, 64));
      hi[a] = fmaxf(hi[a], __shfl_xor(hi[a], off, 64));
    }
  }
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
#pragma unroll
    for (int a = 0; a < 3; ++a) {
      s_part[wave][a] = lo[a];
      s_part[wave][3 + a] = hi[a];
    }
  }
  __syncthreads();
  if (threadIdx.x < 3) {
    s_lo[threadIdx.x] = fminf(s_part[0][threadIdx.x], s_part[1][threadIdx.x]);
    s_hi[threadIdx.x] = fmaxf(s_part[0][3 + threadIdx.x], s_part[1][3 + threadIdx.x]);
  }
  __syncthreads();
}

// Range partials: per (segment, 1024-row chunk), lo then hi of each axis.
template <typename T>
__global__ void __launch_bounds__(kEnc3Threads)
    range3_kernel(const T* __restrict__ q, const T* __restrict__ k, int64_t N, float* __restrict__ partial) {
  const int64_t chunk = blockIdx.x, seg = blockIdx.y;
  const int64_t r = chunk * kEnc3Chunk + int64_t(threadIdx.x) * kEnc3Rows;
  float lo[3], hi[3];
#pragma unroll
  for (int a = 0; a < 3; ++a) {
    lo[a] = __builtin_huge_valf();
    hi[a] = -__builtin_huge_valf();
  }
  if (r < N) {  // N is a multiple of 8: all 8 rows exist
    float x[24], y[24];
    load_rows8(q, seg * N + r, x);
    load_rows8(k, seg * N + r, y);
#pragma unroll
    for (int i = 0; i < 24; ++i) {
      lo[i % 3] = fminf(lo[i % 3], fminf(x[i], y[i]));
      hi[i % 3] = fmaxf(hi[i % 3], fmaxf(x[i], y[i]));
    }
  }
  __shared__ float s_lo[3], s_hi[3];
  block128_range3(lo, hi, s_lo, s_hi);
  if (threadIdx.x < 3) {
    float* out = partial + (seg * int64_t(gridDim.x) + chunk) * 6;
    out[threadIdx.x] = s_lo[threadIdx.x];
    out[3 + threadIdx.x] = s_hi[threadIdx.x];
  }
}

// quantise() with the division done by the hardware reciprocal where that
// provably floors the same: w' = u * rcp(den) is within 2^-21.5 * w' of the
// correctly rounded quotient, so when w' is farther than 2^-20 * w' from the
// nearest integer both lie strictly on the same side of it, inside the same
// unit interval, and floor alike.  Otherwise (or for w' >= 2^19, where that
// margin reaches half a unit) the IEEE division is taken.
__device__ __forceinline__ uint32_t quantise_fast(float x, float lo, float den, float rden, float topf, uint32_t top) {
#pragma clang fp contract(off)
  if (!(den > 0.0f)) return 0u;
  const float t = x - lo;
  const float u = t * topf;
  float w = u * rden;
  const float n = rintf(w);
  const float margin = w * 0x1p-20f;
  if (!(fabsf(w - n) > margin) || !(w < 0x1p19f)) w = __fdiv_rn(u, den);
  const float f = floorf(w);
  if (!(f > 0.0f)) return 0u;
  if (f >= topf) return top;
  return uint32_t(f);
}

template <typename T>
__global__ void __launch_bounds__(kEnc3Threads)
    encode3_kernel(const T* __restrict__ q, const T* __restrict__ k, int64_t N, int bits,
                   const float* __restrict__ partial, const float* __restrict__ range_lohi,
                   float* __restrict__ range_out, uint32_t* __restrict__ q_codes, uint32_t* __restrict__ k_codes) {
  const int64_t chunk = blockIdx.x, seg = blockIdx.y;
  const int64_t chunks = gridDim.x;
  // This thread's rows are loaded first, so that their latency overlaps the
  // range fold (a thread past the segment's end reads its first rows, and
  // writes nothing).
  const int64_t r = chunk * kEnc3Chunk + int64_t(threadIdx.x) * kEnc3Rows;
  const int64_t rr = r < N ? r : 0;
  float xq[24], xk[24];
  load_rows8(q, seg * N + rr, xq);
  load_rows8(k, seg * N + rr, xk);
  __shared__ float s_lo[3], s_hi[3];
  if (range_lohi != nullptr) {
    if (threadIdx.x < 3) {
      s_lo[threadIdx.x] = range_lohi[seg * 6 + threadIdx.x];
      s_hi[threadIdx.x] = range_lohi[seg * 6 + 3 + threadIdx.x];
    }
    __syncthreads();
  } else {
    // Fold the segment's partial ranges.
    float lo[3], hi[3];
#pragma unroll
    for (int a = 0; a < 3; ++a) {
      lo[a] = __builtin_huge_valf();
      hi[a] = -__builtin_huge_valf();
    }
    const float* p = partial + seg * chunks * 6;
    for (int64_t c = threadIdx.x; c < chunks; c += kEnc3Threads) {
#pragma unroll
      for (int a = 0; a < 3; ++a) {
        lo[a] = fminf(lo[a], p[c * 6 + a]);
        hi[a] = fmaxf(hi[a], p[c * 6 + 3 + a]);
      }
    }
    block128_range3(lo, hi, s_lo, s_hi);
  }
  if (range_out != nullptr && chunk == 0 && threadIdx.x < 3) {
    range_out[seg * 6 + threadIdx.x] = s_lo[threadIdx.x];
    range_out[seg * 6 + 3 + threadIdx.x] = s_hi[threadIdx.x];
  }
  if (r >= N) return;
  const uint32_t top = (1u << bits) - 1u;
  const float topf = float(top);
  float lo[3], den[3], rden[3];
#pragma unroll
  for (int a = 0; a < 3; ++a) {
    lo[a] = s_lo[a];
    {
#pragma clang fp contract(off)
      den[a] = s_hi[a] - s_lo[a];
    }
    rden[a] = __builtin_amdgcn_rcpf(den[a]);
  }
#pragma unroll
  for (int which = 0; which < 2; ++which) {
    const float(&x)[24] = which == 0 ? xq : xk;
    uint32_t c[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const uint32_t c0 = quantise_fast(x[3 * i], lo[0], den[0], rden[0], topf, top);
      const uint32_t c1 = quantise_fast(x[3 * i + 1], lo[1], den[1], rden[1], topf, top);
      const uint32_t c2 = quantise_fast(x[3 * i + 2], lo[2], den[2], rden[2], topf, top);
      c[i] = (spread3(c0) << 2) | (spread3(c1) << 1) | spread3(c2);
    }
    uint4* dst = reinterpret_cast<uint4*>((which == 0 ? q_codes : k_codes) + seg * N + r);
    dst[0] = make_uint4(c[0], c[1], c[2], c[3]);
    dst[1] = make_uint4(c[4], c[5], c[6], c[7]);
  }
}

bool aligned16_ptr(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

template <typename T>
hipError_t launch_encode_t(const T* q, const T* k, int64_t S, int64_t N, int dk, int bits,
                           const float* range_lohi, float* range_out, uint32_t* q_codes,
                           uint32_t* k_codes, void* workspace, hipStream_t stream) {
  const EncodeWs ws = encode_ws(S, N, dk);
  if (dk == 3 && N % kEnc3Rows == 0 && S <= 65535 && aligned16_ptr(q) && aligned16_ptr(k) && aligned16_ptr(q_codes) &&
      aligned16_ptr(k_codes)) {
    // Vector form; its partials (one per 1024-row chunk) fit in the space
    // sized for 512-row chunks.
    const dim3 grid(unsigned(ceil_div(N, kEnc3Chunk)), unsigned(S));
    float* partial = nullptr;
    if (range_lohi == nullptr) {
      partial = reinterpret_cast<float*>(static_cast<char*>(workspace) + ws.partial_off);
      hipLaunchKernelGGL(range3_kernel<T>, grid, dim3(kEnc3Threads), 0, stream, q, k, N, partial);
    }
    hipLaunchKernelGGL(encode3_kernel<T>, grid, dim3(kEnc3Threads), 0, stream, q, k, N, bits, partial, range_lohi,
                       range_out, q_codes, k_codes);
    return hipGetLastError();
  }
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
