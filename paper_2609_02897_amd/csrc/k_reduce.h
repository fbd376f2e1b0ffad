// K4: partial (max, sum-exp) records over the draft logits of each request's root row, the
//     input of the draft top-1 confidence p_draft(top1) of Sec. 3.3, Eq. (2).
#pragma once

#include "k_common.h"

namespace asv {

constexpr int kConfPerThread = 8;
constexpr int kConfThreads = 256;
constexpr int kConfChunk = kConfPerThread * kConfThreads;   // draft logits per K4 workgroup

// Grid (chunks, B). Workgroup (ch, b) reduces draft_logits[root_b][ch*kConfChunk ...] to one
// (max, sum of exp(q - max)) record in one pass: each thread issues its eight loads (entry
// lo + 256 i + t, coalesced per wave) before using any, then reduces them in registers.
// Entries past V read as -inf and add nothing. An out-of-range root (malformed offsets,
// reported by K3) yields an empty record and reads nothing.
__global__ __launch_bounds__(kConfThreads)
void k_draft_conf_partial(int N, int V, const int32_t* __restrict__ req_offsets,
                          const float* __restrict__ q, float* __restrict__ part_m,
                          float* __restrict__ part_s) {
  __shared__ float sm[kConfThreads / kWave], ss[kConfThreads / kWave];
  const int ch = blockIdx.x, b = blockIdx.y, nch = gridDim.x;
  const int root = req_offsets[b];
  const int lo = ch * kConfChunk, hi = min(lo + kConfChunk, V);
  Rec r = rec_empty();
  if (root >= 0 && root < N) {
    const float* row = q + (size_t)root * V;
    float x[kConfPerThread];
#pragma unroll
    for (int i = 0; i < kConfPerThread; ++i) {
      const int v = lo + i * kConfThreads + (int)threadIdx.x;
      x[i] = v < hi ? row[v] : kNegInf;
    }
    float m = x[0];
#pragma unroll
    for (int i = 1; i < kConfPerThread; ++i) m = fmaxf(m, x[i]);
    float s = 0.f;
    if (m != kNegInf) {
      const float mb = m * kLog2e;
#pragma unroll
      for (int i = 0; i < kConfPerThread; ++i) s += exp2_rel(fmaf(x[i], kLog2e, -mb));
    }
    r = Rec{m, s, 0};
  }
  r = rec_wave_reduce(r);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sm[w] = r.m;
    ss[w] = r.s;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    Rec t{sm[0], ss[0], 0};
    for (int i = 1; i < kConfThreads / kWave; ++i) t = rec_merge(t, Rec{sm[i], ss[i], 0});
    part_m[(size_t)b * nch + ch] = t.m;
    part_s[(size_t)b * nch + ch] = t.s;
  }
}

}  // namespace asv
