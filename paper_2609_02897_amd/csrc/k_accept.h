// K3: margin rule, tree walk, bonus token and policy-state update; one wave per request.
//
// Margin rule (Sec. 3.2, Eq. (1)): a node c with parent p and drafted token d is accepted when
// p_target(d) / p_target(top1) = exp(z_p[d] - max z_p) >= kappa, i.e. z_p[d] - max >= ln kappa;
// an exact match d == argmax z_p is accepted outright, kappa == 0 accepts everything.
// Walk: from the root, repeatedly take the child with the highest drafted logit (lowest row id
// on ties) while it is accepted; a child that is not the current row's argmax is a promotion
// and counts against params.max_promotions (-1 = unlimited). The bonus token is the argmax of
// the last accepted node's row (greedy decoding).
// State (Sec. 3.3): EMA of the accept fraction len / (n - 1), a 16-slot history ring, the
// zero-accept streak and the circuit breaker.
#pragma once

#include "k_common.h"
#include "asv.h"

namespace asv {

__device__ __forceinline__ int wave_or(int x) {
#pragma unroll
  for (int mask = 32; mask >= 1; mask >>= 1) x |= __shfl_xor(x, mask, kWave);
  return x;
}

// (g, c) with the larger g, the smaller c on equal g.
__device__ __forceinline__ void best_child_reduce(float& g, int& c) {
#pragma unroll
  for (int mask = 32; mask >= 1; mask >>= 1) {
    const float g2 = __shfl_xor(g, mask, kWave);
    const int c2 = __shfl_xor(c, mask, kWave);
    if (g2 > g || (g2 == g && c2 < c)) {
      g = g2;
      c = c2;
    }
  }
}

__global__ __launch_bounds__(kWave)
void k_tree_accept(int B, int N, int V, const int32_t* __restrict__ off,
                   const int32_t* __restrict__ parent, const int32_t* __restrict__ tok,
                   const float* __restrict__ tau, const float* __restrict__ row_max,
                   const int32_t* __restrict__ row_arg, const float* __restrict__ g,
                   uint8_t* __restrict__ accept, int32_t* __restrict__ acc_len,
                   int32_t* __restrict__ bonus, int32_t* __restrict__ path,
                   const float* __restrict__ conf_m, const float* __restrict__ conf_s,
                   int n_conf, float* __restrict__ draft_conf, asv_req_state* __restrict__ state,
                   int32_t* __restrict__ status, asv_params prm) {
  const int b = blockIdx.x, lane = threadIdx.x;
  const int lo = off[b], hi = off[b + 1];
  if (lo < 0 || lo >= hi || hi > N || (b == 0 && lo != 0) || (b == B - 1 && hi != N)) {
    if (lane == 0) {
      status[b] = ASV_RS_BAD_OFFSETS;
      acc_len[b] = 0;
      bonus[b] = -1;
      if (draft_conf) draft_conf[b] = __builtin_nanf("");
    }
    return;
  }

  // ---- validate the tree
  const float kappa = tau[b];
  int st = 0;
  if (!(kappa >= 0.f && kappa <= 1.f)) st |= ASV_RS_BAD_TAU;
  if (lane == 0 && parent[lo] != -1) st |= ASV_RS_BAD_ROOT;
  for (int c = lo + 1 + lane; c < hi; c += kWave) {
    const int p = parent[c], d = tok[c];
    if (p < lo || p >= c) st |= ASV_RS_BAD_PARENT;
    if (d < 0 || d >= V) st |= ASV_RS_BAD_TOKEN;
  }
  st = wave_or(st);
  if (st) {
    for (int c = lo + lane; c < hi; c += kWave) {
      accept[c] = 0;
      path[c] = -1;
    }
    if (lane == 0) {
      status[b] = st;
      acc_len[b] = 0;
      bonus[b] = -1;
      if (draft_conf) draft_conf[b] = __builtin_nanf("");
    }
    return;
  }

  // ---- Eq. (1) for every node of the request
  const float ln_kappa = kappa > 0.f ? logf(kappa) : kNegInf;
  for (int c = lo + lane; c < hi; c += kWave) {
    uint8_t ok = 1;
    if (c != lo) {
      const int p = parent[c];
      ok = (tok[c] == row_arg[p]) || kappa == 0.f || (g[c] - row_max[p] >= ln_kappa);
    }
    accept[c] = ok;
  }

  // ---- walk
  int cur = lo, len = 0, promos = 0;
  for (;;) {
    float bg = kNegInf;
    int bc = kNoIndex;
    for (int c = lo + 1 + lane; c < hi; c += kWave) {
      if (parent[c] == cur) {
        const float gc = g[c];
        if (bc == kNoIndex || gc > bg || (gc == bg && c < bc)) {
          bg = gc;
          bc = c;
        }
      }
    }
    best_child_reduce(bg, bc);
    if (bc == kNoIndex) break;
    const int arg = row_arg[cur];
    const int d = tok[bc];
    const bool ok = (d == arg) || kappa == 0.f || (bg - row_max[cur] >= ln_kappa);
    if (!ok) break;
    if (d != arg) {
      if (prm.max_promotions >= 0 && promos >= prm.max_promotions) break;
      ++promos;
    }
    if (lane == 0) path[lo + len] = bc;
    ++len;
    cur = bc;
  }
  for (int c = lo + len + lane; c < hi; c += kWave) path[c] = -1;

  // ---- draft top-1 confidence of the root row: 1 / sum_v exp(q_v - max q)
  float conf = 0.f;
  if (n_conf > 0) {
    Rec r = rec_empty();
    for (int i = lane; i < n_conf; i += kWave)
      r = rec_merge(r, Rec{conf_m[(size_t)b * n_conf + i], conf_s[(size_t)b * n_conf + i], 0});
    r = rec_wave_reduce(r);
    conf = 1.f / r.s;
  }

  if (lane != 0) return;
  acc_len[b] = len;
  bonus[b] = row_arg[cur];
  status[b] = 0;
  if (n_conf > 0 && draft_conf) draft_conf[b] = conf;
  if (!state) return;

  // ---- policy state (one lane)
  asv_req_state* s = state + b;
  const int n = hi - lo;
  if (n > 1) {
    const float x = (float)len / (float)(n - 1);
    s->rar = s->rar + prm.alpha * (x - s->rar);
    const int head = ((s->hist_head % ASV_HIST_WINDOW) + ASV_HIST_WINDOW) % ASV_HIST_WINDOW;
    s->hist[head] = x;
    const int new_head = (head + 1) % ASV_HIST_WINDOW;
    const int count = min(max(s->hist_count, 0) + 1, ASV_HIST_WINDOW);
    float sum = 0.f;
    for (int i = 0; i < count; ++i)
      sum += s->hist[(new_head - 1 - i + 2 * ASV_HIST_WINDOW) % ASV_HIST_WINDOW];
    s->hist_head = new_head;
    s->hist_count = count;
    s->hist_mean = sum / (float)count;
    const int streak = (len == 0) ? s->zero_streak + 1 : 0;
    const int trip = streak >= prm.breaker_n ? 1 : 0;
    s->breaker = trip;
    s->zero_streak = streak;
    if (trip) {
      s->rar = prm.rar0;
      for (int i = 0; i < ASV_HIST_WINDOW; ++i) s->hist[i] = 0.f;
      s->hist_head = 0;
      s->hist_count = 0;
      s->hist_mean = prm.rar0;
      s->zero_streak = 0;
    }
  } else {
    s->breaker = 0;
  }
  s->steps = s->steps + 1;
  if (n_conf > 0) s->draft_conf = conf;
}

__global__ void k_state_init(asv_req_state* state, int B, asv_params prm) {
  const int b = blockIdx.x * blockDim.x + threadIdx.x;
  if (b >= B) return;
  asv_req_state* s = state + b;
  s->rar = prm.rar0;
  for (int i = 0; i < ASV_HIST_WINDOW; ++i) s->hist[i] = 0.f;
  s->hist_head = 0;
  s->hist_count = 0;
  s->zero_streak = 0;
  s->breaker = 0;
  s->steps = 0;
  s->hist_mean = prm.rar0;
  s->draft_conf = 0.f;
}

}  // namespace asv
