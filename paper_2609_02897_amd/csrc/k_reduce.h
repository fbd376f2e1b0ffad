// K4: partial (max, sum-exp) records over the draft logits of each request's root row, the
//     input of the draft top-1 confidence p_draft(top1) of Sec. 3.3, Eq. (2).
#pragma once

#include "k_common.h"

namespace asv {

constexpr int kConfChunk = 8192;        // draft logits per K4 workgroup
constexpr int kConfThreads = 256;

// Grid (chunks, B). Workgroup (ch, b) reduces draft_logits[root_b][ch*kConfChunk ...] to one
// (max, sum of exp(q - max)) record. An out-of-range root (malformed offsets, reported by K3)
// yields an empty record and reads nothing.
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
    float m = kNegInf;
    for (int v = lo + threadIdx.x; v < hi; v += kConfThreads) m = fmaxf(m, row[v]);
    float s = 0.f;
    const float mb = m * kLog2e;
    for (int v = lo + threadIdx.x; v < hi; v += kConfThreads)
      s += exp2_rel(fmaf(row[v], kLog2e, -mb));
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
