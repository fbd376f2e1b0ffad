// Shared device helpers of libasv (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

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

// Merge two records; the argmax keeps the lowest index among equal maxima.
__device__ __forceinline__ Rec rec_merge(Rec x, Rec y) {
  Rec r;
  r.m = fmaxf(x.m, y.m);
  float sx = (x.m == kNegInf) ? 0.f : x.s * exp2f((x.m - r.m) * kLog2e);
  float sy = (y.m == kNegInf) ? 0.f : y.s * exp2f((y.m - r.m) * kLog2e);
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

}  // namespace asv
