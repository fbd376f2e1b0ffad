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

// Requests with at most this many nodes are staged in LDS with one round of loads and walked
// there; larger ones are walked from global memory (same arithmetic).
constexpr int kStageNodes = 1024;

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
  __shared__ int32_t s_par[kStageNodes], s_tok[kStageNodes], s_arg[kStageNodes];
  __shared__ float s_g[kStageNodes], s_max[kStageNodes];
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
  const int n = hi - lo;
  const float kappa = tau[b];

  // draft-confidence partials: issued now, merged after the walk
  Rec conf_r = rec_empty();
  for (int i = lane; i < n_conf; i += kWave)
    conf_r = rec_merge(conf_r, Rec{conf_m[(size_t)b * n_conf + i],
                                   conf_s[(size_t)b * n_conf + i], 0});

  // ---- stage the request: parent, token, drafted logit and the row max / argmax of every node,
  // plus the 24-word policy state (one word per lane), all in one round of loads
  static_assert(sizeof(asv_req_state) == 24 * 4, "state layout");
  __shared__ asv_req_state s_st;
  uint32_t* const sh_words = reinterpret_cast<uint32_t*>(&s_st);
  uint32_t* const st_words = state ? reinterpret_cast<uint32_t*>(state + b) : nullptr;
  if (state && lane < 24) sh_words[lane] = st_words[lane];
  const bool staged = n <= kStageNodes;
  if (staged) {
    for (int i0 = 0; i0 < n; i0 += 4 * kWave) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int i = i0 + u * kWave + lane;
        if (i < n) {
          s_par[i] = parent[lo + i];
          s_tok[i] = tok[lo + i];
          s_g[i] = g[lo + i];
          s_max[i] = row_max[lo + i];
          s_arg[i] = row_arg[lo + i];
        }
      }
    }
  }
  __syncthreads();
  auto P = [&](int c) { return staged ? s_par[c - lo] : parent[c]; };
  auto D = [&](int c) { return staged ? s_tok[c - lo] : tok[c]; };
  auto Gc = [&](int c) { return staged ? s_g[c - lo] : g[c]; };
  auto Mr = [&](int r) { return staged ? s_max[r - lo] : row_max[r]; };
  auto Ar = [&](int r) { return staged ? s_arg[r - lo] : row_arg[r]; };

  // ---- validate the tree
  int st = 0;
  if (!(kappa >= 0.f && kappa <= 1.f)) st |= ASV_RS_BAD_TAU;
  if (lane == 0 && P(lo) != -1) st |= ASV_RS_BAD_ROOT;
  for (int c = lo + 1 + lane; c < hi; c += kWave) {
    const int p = P(c), d = D(c);
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
      const int p = P(c);
      ok = (D(c) == Ar(p)) || kappa == 0.f || (Gc(c) - Mr(p) >= ln_kappa);
    }
    accept[c] = ok;
  }

  // ---- walk
  int cur = lo, len = 0, promos = 0;
  for (;;) {
    float bg = kNegInf;
    int bc = kNoIndex;
    for (int c = lo + 1 + lane; c < hi; c += kWave) {
      if (P(c) == cur) {
        const float gc = Gc(c);
        if (bc == kNoIndex || gc > bg || (gc == bg && c < bc)) {
          bg = gc;
          bc = c;
        }
      }
    }
    best_child_reduce(bg, bc);
    if (bc == kNoIndex) break;
    const int arg = Ar(cur);
    const int d = D(bc);
    const bool ok = (d == arg) || kappa == 0.f || (bg - Mr(cur) >= ln_kappa);
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
    conf_r = rec_wave_reduce(conf_r);
    conf = 1.f / conf_r.s;
  }

  if (lane == 0) {
    acc_len[b] = len;
    bonus[b] = Ar(cur);
    status[b] = 0;
    if (n_conf > 0 && draft_conf) draft_conf[b] = conf;
  }
  if (!state) return;

  // ---- policy state (staged above): updated by lane 0 in LDS, written back one word per lane
  if (lane == 0) {
    asv_req_state& q = s_st;
    if (n > 1) {
      const float x = (float)len / (float)(n - 1);
      q.rar = q.rar + prm.alpha * (x - q.rar);
      const int head = ((q.hist_head % ASV_HIST_WINDOW) + ASV_HIST_WINDOW) % ASV_HIST_WINDOW;
      q.hist[head] = x;
      const int new_head = (head + 1) % ASV_HIST_WINDOW;
      const int count = min(max(q.hist_count, 0) + 1, ASV_HIST_WINDOW);
      float sum = 0.f;
      for (int i = 0; i < count; ++i)
        sum += q.hist[(new_head - 1 - i + 2 * ASV_HIST_WINDOW) % ASV_HIST_WINDOW];
      q.hist_head = new_head;
      q.hist_count = count;
      q.hist_mean = sum / (float)count;
      const int streak = (len == 0) ? q.zero_streak + 1 : 0;
      const int trip = streak >= prm.breaker_n ? 1 : 0;
      q.breaker = trip;
      q.zero_streak = streak;
      if (trip) {
        q.rar = prm.rar0;
        for (int i = 0; i < ASV_HIST_WINDOW; ++i) q.hist[i] = 0.f;
        q.hist_head = 0;
        q.hist_count = 0;
        q.hist_mean = prm.rar0;
        q.zero_streak = 0;
      }
    } else {
      q.breaker = 0;
    }
    q.steps = q.steps + 1;
    if (n_conf > 0) q.draft_conf = conf;
  }
  __syncthreads();
  if (lane < 24) st_words[lane] = sh_words[lane];
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
