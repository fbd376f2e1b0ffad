// Shared device helpers of libasv (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace asv {

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_inff();
constexpr int kNoIndex = 0x7fffffff;

// Online (max, sum of exp relative to max, lowest argmax) record of a set of logits.
struct Rec {
  float m;   // max, -inf for an empty set
  float s;   // sum_v exp(z_v - m), 0 for an empty set
  int a;     // lowest index attaining m, kNoIndex for an empty set
};

__device__ __forceinline__ Rec rec_empty() { return Rec{kNegInf, 0.f, kNoIndex}; }

// Base-2 exponential of the hardware (v_exp_f32). Every use here exponentiates a value taken
// relative to a maximum (argument <= 0); results below 2^-126 flush to zero, which changes a
// sum of such terms (at least one of which is 1) by less than 2^-126 relative.
__device__ __forceinline__ float exp2_rel(float x) { return __builtin_amdgcn_exp2f(x); }

// Merge two records; the argmax keeps the lowest index among equal maxima.
__device__ __forceinline__ Rec rec_merge(Rec x, Rec y) {
  Rec r;
  r.m = fmaxf(x.m, y.m);
  float sx = (x.m == kNegInf) ? 0.f : x.s * exp2_rel((x.m - r.m) * kLog2e);
  float sy = (y.m == kNegInf) ? 0.f : y.s * exp2_rel((y.m - r.m) * kLog2e);
  r.s = sx + sy;
  r.a = (x.m > y.m) ? x.a : (y.m > x.m) ? y.a : min(x.a, y.a);
  return r;
}

__device__ __forceinline__ Rec rec_shfl_xor(Rec x, int mask) {
  Rec y;
  y.m = __shfl_xor(x.m, mask, kWave);
  y.s = __shfl_xor(x.s, mask, kWave);
  y.a = __shfl_xor(x.a, mask, kWave);
  return y;
}

// Full-wave reduction; every lane ends with the merged record.
__device__ __forceinline__ Rec rec_wave_reduce(Rec x) {
#pragma unroll
  for (int mask = 32; mask >= 1; mask >>= 1) x = rec_merge(x, rec_shfl_xor(x, mask));
  return x;
}

// ---- wave-wide reductions without LDS round trips: rotations within each 16-lane row (DPP
// row_ror), then the four row results read as scalars. Every lane returns the same value; the
// combination order is fixed, so results are deterministic.
template <int N>
__device__ __forceinline__ int row_ror(int x) {
  return __builtin_amdgcn_update_dpp(0, x, 0x120 + N, 0xf, 0xf, false);
}
template <int N>
__device__ __forceinline__ float row_ror(float x) {
  return __int_as_float(row_ror<N>(__float_as_int(x)));
}
__device__ __forceinline__ float lane_value(float x, int l) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), l));
}
__device__ __forceinline__ int lane_value(int x, int l) { return __builtin_amdgcn_readlane(x, l); }

__device__ __forceinline__ float wave_max(float x) {
  x = fmaxf(x, row_ror<8>(x));
  x = fmaxf(x, row_ror<4>(x));
  x = fmaxf(x, row_ror<2>(x));
  x = fmaxf(x, row_ror<1>(x));
  return fmaxf(fmaxf(lane_value(x, 0), lane_value(x, 16)),
               fmaxf(lane_value(x, 32), lane_value(x, 48)));
}
__device__ __forceinline__ float wave_sum(float x) {
  x += row_ror<8>(x);
  x += row_ror<4>(x);
  x += row_ror<2>(x);
  x += row_ror<1>(x);
  return (lane_value(x, 0) + lane_value(x, 16)) + (lane_value(x, 32) + lane_value(x, 48));
}
__device__ __forceinline__ int wave_min(int x) {
  x = min(x, row_ror<8>(x));
  x = min(x, row_ror<4>(x));
  x = min(x, row_ror<2>(x));
  x = min(x, row_ror<1>(x));
  return min(min(lane_value(x, 0), lane_value(x, 16)), min(lane_value(x, 32), lane_value(x, 48)));
}

// Wave-wide merge of lane records: M = max m, s = sum s_l exp(m_l - M), a = lowest a_l with
// m_l = M. Lanes with an empty record (m = -inf, s = 0) contribute nothing; at least one lane
// must hold a finite m.
__device__ __forceinline__ Rec rec_wave_reduce_dpp(Rec x) {
  const float M = wave_max(x.m);
  const float part = x.m == kNegInf ? 0.f : x.s * exp2_rel((x.m - M) * kLog2e);
  return Rec{M, wave_sum(part), wave_min(x.m == M ? x.a : kNoIndex)};
}

// Device-coherent access without cache maintenance, for data one workgroup writes and another
// workgroup of the same launch reads: device-scope relaxed atomic stores write through the
// XCD's L2 and device-scope relaxed atomic loads miss it, so neither needs the whole-L2
// write-back / invalidate that a device-scope fence costs.
__device__ __forceinline__ void st_device(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_device(int32_t* p, int32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_device(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int32_t ld_device(const int32_t* p) {
  return __hip_atomic_load(const_cast<int32_t*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// LDS writes of every lane of this wave are visible to its later LDS reads: the LDS executes a
// wave's instructions in order, so a compiler fence plus the drain of this wave's LDS queue
// suffice (no workgroup barrier, which would need every wave of the workgroup).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0)
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// f(std::integral_constant<int, i>{}) for i = 0 .. M-1, each i a compile-time constant (a
// fully unrolled loop whose body may select code with if constexpr).
template <int M, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (M > 0) {
    static_for<M - 1>(f);
    f(std::integral_constant<int, M - 1>{});
  }
}

// Wait until every global store this wave issued has completed (vmcnt(0)).
__device__ __forceinline__ void wait_stores() { __builtin_amdgcn_s_waitcnt(0x0f70); }

}  // namespace asv
