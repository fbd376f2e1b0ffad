// Achievable-peak microbenchmarks (measurement only; declared in include/asv_microbench.h).
#include <hip/hip_runtime.h>

#include "asv_microbench.h"

namespace {

constexpr int kThreads = 256;
constexpr int kUnroll = 8;

// Workgroup g reads the 16-byte words [g * per, min((g + 1) * per, n16)).
__global__ __launch_bounds__(kThreads) void k_stream_read(const uint4* __restrict__ p,
                                                           size_t n16, size_t per,
                                                           uint32_t* __restrict__ sink) {
  const size_t base = blockIdx.x * per;
  const size_t end = base + per < n16 ? base + per : n16;
  uint32_t acc = 0;
  for (size_t i = base + threadIdx.x; i < end; i += (size_t)kThreads * kUnroll) {
    uint4 v[kUnroll];
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) {
      const size_t j = i + (size_t)u * kThreads;
      v[u] = j < end ? p[j] : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < kUnroll; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  if (acc == 0x9e3779b9u) sink[blockIdx.x] = acc;
}

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
constexpr int kUnrollNt = 4;

// Interleaved read with the non-temporal hint: round k of workgroup g reads the 16-byte words
// (k grid + g) 1024 + u 256 + t, u < 4 (t = thread).
__global__ __launch_bounds__(kThreads) void k_stream_read_nt(const u32x4* __restrict__ p,
                                                              size_t n16,
                                                              uint32_t* __restrict__ sink) {
  uint32_t acc = 0;
  const size_t step = (size_t)gridDim.x * kThreads * kUnrollNt;
  for (size_t i = blockIdx.x * (size_t)kThreads * kUnrollNt + threadIdx.x; i < n16; i += step) {
    u32x4 v[kUnrollNt];
#pragma unroll
    for (int u = 0; u < kUnrollNt; ++u) {
      const size_t j = i + (size_t)u * kThreads;
      v[u] = j < n16 ? __builtin_nontemporal_load(p + j) : u32x4{0u, 0u, 0u, 0u};
    }
#pragma unroll
    for (int u = 0; u < kUnrollNt; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  if (acc == 0x9e3779b9u) sink[blockIdx.x] = acc;
}

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x16 __attribute__((__vector_size__(16 * sizeof(float))));

__global__ __launch_bounds__(kThreads) void k_mfma_loop(float* __restrict__ sink, int iters) {
  const int t = threadIdx.x;
  bf16x8 a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.001f * (float)((t + i) & 15));
    b[i] = (__bf16)(0.002f * (float)((t * 3 + i) & 7));
  }
  f32x16 acc[8];
#pragma unroll
  for (int k = 0; k < 8; ++k)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[k][e] = 0.f;
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[k], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < 8; ++k)
#pragma unroll
    for (int e = 0; e < 16; ++e) s += acc[k][e];
  sink[blockIdx.x * kThreads + t] = s;
}

constexpr int kLdsUnits = 1024;   // 16 KB of 16-byte units

// Each wave reads one 16-byte unit per lane, the same every iteration; `mask` is zero at run
// time, so the address is fixed, but the compiler cannot hoist the read out of the loop.
__global__ __launch_bounds__(kThreads) void k_lds_read(const int32_t* __restrict__ unit_of_lane,
                                                        int iters, int mask,
                                                        uint32_t* __restrict__ sink) {
  __shared__ uint4 buf[kLdsUnits];
  for (int i = threadIdx.x; i < kLdsUnits; i += kThreads)
    buf[i] = make_uint4(i, i + 1, i + 2, i + 3);
  __syncthreads();
  const int u = unit_of_lane[threadIdx.x & 63] & (kLdsUnits - 1);
  uint32_t acc = 0;
  for (int it = 0; it < iters; ++it) {
    const uint4 v = buf[u ^ (it & mask)];
    acc += v.x ^ v.y ^ v.z ^ v.w;
  }
  sink[blockIdx.x * kThreads + threadIdx.x] = acc;
}

}  // namespace

extern "C" int asvb_stream_read(const void* buf, uint64_t bytes, uint32_t* sink, int32_t grid,
                                void* stream) {
  if (!buf || !sink || grid < 1 || bytes == 0 || bytes % 16 != 0 ||
      (reinterpret_cast<uintptr_t>(buf) & 15u) != 0)
    return -1;
  const size_t n16 = bytes / 16, per = (n16 + grid - 1) / grid;
  (void)hipGetLastError();
  k_stream_read<<<grid, kThreads, 0, reinterpret_cast<hipStream_t>(stream)>>>(
      static_cast<const uint4*>(buf), n16, per, sink);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

extern "C" int asvb_stream_read_nt(const void* buf, uint64_t bytes, uint32_t* sink,
                                   int32_t grid, void* stream) {
  if (!buf || !sink || grid < 1 || bytes == 0 || bytes % 16 != 0 ||
      (reinterpret_cast<uintptr_t>(buf) & 15u) != 0)
    return -1;
  (void)hipGetLastError();
  k_stream_read_nt<<<grid, kThreads, 0, reinterpret_cast<hipStream_t>(stream)>>>(
      static_cast<const u32x4*>(buf), bytes / 16, sink);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

extern "C" int asvb_mfma_loop(float* sink, int32_t iters, int32_t grid, void* stream) {
  if (!sink || iters < 1 || grid < 1) return -1;
  (void)hipGetLastError();
  k_mfma_loop<<<grid, kThreads, 0, reinterpret_cast<hipStream_t>(stream)>>>(sink, iters);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

extern "C" int asvb_lds_read(const int32_t* unit_of_lane, int32_t iters, uint32_t* sink,
                             int32_t grid, void* stream) {
  if (!unit_of_lane || !sink || iters < 1 || grid < 1) return -1;
  (void)hipGetLastError();
  k_lds_read<<<grid, kThreads, 0, reinterpret_cast<hipStream_t>(stream)>>>(unit_of_lane, iters,
                                                                          0, sink);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}
