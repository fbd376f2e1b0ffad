// Margin rule, tree walk, bonus token and policy-state update of one request, run by one wave,
// and the two kernels that run it after the LM-head pass:
//   k_merge_accept (K2+K3 fused, batches of up to kFusedMaxB requests): merges each row's slab
//     records and, in the workgroup that completes a request's last row, walks that request;
//   k_slab_merge + k_tree_accept (larger batches): the same two steps as separate launches.
//
// Margin rule (Sec. 3.2, Eq. (1)): a node c with parent p and drafted token d is accepted when
// p_target(d) / p_target(top1) = exp(z_p[d] - max z_p) >= kappa, i.e. z_p[d] - max >= ln kappa;
// an exact match d == argmax z_p is accepted outright, kappa == 0 accepts everything. With a
// temperature T (params.temperature) the target distribution is softmax(z / T) and the test
// becomes z_p[d] - max >= T ln kappa.
// Walk: from the root, repeatedly take the child with the highest drafted logit (lowest row id
// on ties) while it is accepted; a child that is not the current row's argmax is a promotion
// and counts against params.max_promotions (-1 = unlimited). The bonus token is the argmax of
// the last accepted node's row (greedy decoding).
// State (Sec. 3.3): EMA of the accept fraction len / (n - 1), a 16-slot history ring, the
// zero-accept streak and the circuit breaker, then the Draft Confidence Score and the tree
// shape it selects for the next draft (Eq. (2)).
#pragma once

#include "k_common.h"
#include "asv.h"

namespace asv {

static_assert(ASV_HIST_WINDOW == 16, "the ring arithmetic below assumes 16 slots");

__device__ __forceinline__ bool wave_any(bool x) { return __ballot(x) != 0; }

// ---- per-row merge of the slab records (the first half of the finishing step)

// One wave per tree row: lane l holds records s = l, l + 64, ... of the row's S slab records.
// row_lse = M + log(sum_s l_s * exp(m_s - M)); the argmax is the lowest index among the slabs
// attaining M (each slab's own argmax is its lowest). Each lane issues the loads of
// kMergeBatch records before using any, so a row of up to 64 * kMergeBatch slabs
// (V <= 163840 with 256-entry slabs) costs one memory round trip, and reduces them with
// independent operations (one max, then the scaled sum and the tie minimum), not a chain of
// pairwise merges.
constexpr int kMergeBatch = 10;
struct RecBatch {
  float m[kMergeBatch], s[kMergeBatch];
  int32_t a[kMergeBatch];
};

__device__ __forceinline__ void load_rec_batch(RecBatch& bt, size_t base, int s0, int S, int lane,
                                               const float* __restrict__ rec_m,
                                               const float* __restrict__ rec_s,
                                               const int32_t* __restrict__ rec_a) {
  // Every lane loads (clamped to the row's last record, S >= 1); entries past S duplicate a
  // real record, which leaves the max and the argmax unchanged, and their sums are masked out.
#pragma unroll
  for (int u = 0; u < kMergeBatch; ++u) {
    const int s = s0 + u * kWave + lane;
    const size_t at = base + (size_t)min(s, S - 1);
    bt.m[u] = rec_m[at];
    bt.s[u] = rec_s[at] * (float)(s < S);
    bt.a[u] = rec_a[at];
  }
}

// Lane-local record of one batch.
__device__ __forceinline__ Rec batch_record(const RecBatch& bt) {
  float m = bt.m[0];
#pragma unroll
  for (int u = 1; u < kMergeBatch; ++u) m = fmaxf(m, bt.m[u]);
  float sum = 0.f;
  int a = kNoIndex;
#pragma unroll
  for (int u = 0; u < kMergeBatch; ++u) {
    sum += bt.s[u] * exp2_rel((bt.m[u] - m) * kLog2e);
    a = min(a, bt.m[u] == m ? bt.a[u] : kNoIndex);
  }
  return m == kNegInf ? rec_empty() : Rec{m, sum, a};
}

// Merges the batch already loaded for s0 = 0 with the remaining batches of the row at base.
__device__ __forceinline__ Rec merge_row_rest(const RecBatch& first, size_t base, int S, int lane,
                                              const float* __restrict__ rec_m,
                                              const float* __restrict__ rec_s,
                                              const int32_t* __restrict__ rec_a) {
  Rec r = batch_record(first);
  for (int s0 = kWave * kMergeBatch; s0 < S; s0 += kWave * kMergeBatch) {
    RecBatch bt;
    load_rec_batch(bt, base, s0, S, lane, rec_m, rec_s, rec_a);
    r = rec_merge(r, batch_record(bt));
  }
  return rec_wave_reduce_dpp(r);
}

// The offsets array as a whole is well formed: req_offsets[0] = 0, strictly increasing,
// req_offsets[B] = N. When it is not, every request of the batch reports ASV_RS_BAD_OFFSETS
// (a malformed offsets array leaves the ownership of every row in doubt).
__device__ __forceinline__ bool offset_pair_bad(int b, int B, int N, int lo, int hi) {
  return lo >= hi || (b == 0 && lo != 0) || (b == B - 1 && hi != N);
}

// ---- one request's walk, run by one wave

// Everything the walk reads and writes. row_max / row_arg may be written by other workgroups
// of the same launch (the fused kernel); they are read with device-coherent loads and are
// deliberately not restrict-qualified.
struct AcceptArgs {
  int B, N, V;
  const int32_t* off;
  const int32_t* parent;
  const int32_t* tok;
  const float* tau;
  const float* row_max;
  const int32_t* row_arg;
  const float* g;
  uint8_t* accept;
  int32_t* acc_len;
  int32_t* bonus;
  int32_t* path;
  const float* conf_m;
  const float* conf_s;
  int n_conf;
  float* draft_conf;
  asv_req_state* state;
  int32_t* status;
  asv_params prm;
};

// Requests with at most this many nodes are staged in the wave's LDS slice and walked there;
// larger ones are walked from global memory (same arithmetic, slower walk).
constexpr int kWaveStage = 256;
constexpr int kStagePerLane = kWaveStage / kWave;
struct WalkSmem {
  uint64_t best[kWaveStage];  // packed key of each node's best child, 0 = none
  int32_t par[kWaveStage], tok[kWaveStage], arg[kWaveStage], pathl[kWaveStage];
  float g[kWaveStage], mx[kWaveStage];
  uint8_t ok[kWaveStage];     // Eq. (1) verdict of each node
  asv_req_state st;
};
constexpr int kStateWords = 28;
static_assert(sizeof(asv_req_state) == kStateWords * 4, "state layout");
static_assert(kStateWords <= kWave, "one state word per lane");

// Draft Confidence Score and the tree shape it selects (Sec. 3.3, Eq. (2)):
// dcs = min(1, draft_conf * rar / d); each member of (nsteps, topk, ndt) moves linearly from
// shape_lo at score 0 to shape_hi at score 1 and is rounded to the nearest integer, halves
// down; a request whose breaker tripped takes the starting configuration. The score decides
// integers, so every operation is rounded on its own (no contraction into fused operations).
__device__ __forceinline__ void tree_shape(asv_req_state& q, const asv_params& prm) {
  const float dcs = fminf(1.f, __fdiv_rn(__fmul_rn(q.draft_conf, q.rar), prm.dcs_divisor));
  q.dcs = dcs;
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    const float x = __fadd_rn((float)prm.shape_lo[k],
                              __fmul_rn((float)(prm.shape_hi[k] - prm.shape_lo[k]), dcs));
    q.shape[k] = q.breaker ? prm.shape_start[k] : (int)ceilf(x - 0.5f);
  }
}

// Per-lane registers of a request's staged inputs (parent, token, drafted logit), loaded ahead
// of the walk and written to LDS later.
struct StageRegs {
  int32_t par[kStagePerLane], tok[kStagePerLane];
  float g[kStagePerLane];
};

// Straight-line loads of nodes [lo, lo + min(n, kWaveStage)), clamped into [0, N) so that any lo
// is safe (entries past n are loaded but unused).
__device__ __forceinline__ void stage_load(const AcceptArgs& a, int lo, int lane, StageRegs& r) {
  const int base = min(max(lo, 0), a.N - 1);
#pragma unroll
  for (int u = 0; u < kStagePerLane; ++u) {
    const int c = min(base + u * kWave + lane, a.N - 1);
    r.par[u] = a.parent[c];
    r.tok[u] = a.tok[c];
    r.g[u] = a.g[c];
  }
}

// Tree checks on the staged registers: root parent -1, every other parent inside [lo, c),
// tokens inside [0, V). Returns the ASV_RS_* bits (wave-uniform).
__device__ __forceinline__ int stage_check(const AcceptArgs& a, int lo, int n, int lane,
                                           const StageRegs& r) {
  bool bad_root = false, bad_parent = false, bad_token = false;
#pragma unroll
  for (int u = 0; u < kStagePerLane; ++u) {
    const int i = u * kWave + lane;
    if (i == 0) bad_root = r.par[u] != -1;
    if (i >= 1 && i < n) {
      bad_parent |= r.par[u] < lo || r.par[u] >= lo + i;
      bad_token |= r.tok[u] < 0 || r.tok[u] >= a.V;
    }
  }
  return (wave_any(bad_root) ? ASV_RS_BAD_ROOT : 0) |
         (wave_any(bad_parent) ? ASV_RS_BAD_PARENT : 0) |
         (wave_any(bad_token) ? ASV_RS_BAD_TOKEN : 0);
}

__device__ __forceinline__ void stage_store(int n, int lane, const StageRegs& r, WalkSmem& sm) {
#pragma unroll
  for (int u = 0; u < kStagePerLane; ++u) {
    const int i = u * kWave + lane;
    if (i < n) {
      sm.par[i] = r.par[u];
      sm.tok[i] = r.tok[u];
      sm.g[i] = r.g[u];
    }
  }
}

__device__ __forceinline__ void fail_request(const AcceptArgs& a, int b, int code) {
  a.status[b] = code;
  a.acc_len[b] = 0;
  a.bonus[b] = -1;
  if (a.draft_conf) a.draft_conf[b] = __builtin_nanf("");
}

// Draft-confidence partial records of request b, lane-local (reduced in finish_request).
__device__ __forceinline__ Rec conf_partials(const AcceptArgs& a, int b, int lane) {
  Rec r = rec_empty();
  for (int i = lane; i < a.n_conf; i += kWave)
    r = rec_merge(r, Rec{a.conf_m[(size_t)b * a.n_conf + i], a.conf_s[(size_t)b * a.n_conf + i],
                         0});
  return r;
}

// Outputs and policy-state update of a walked request: draft top-1 confidence of the root row
// 1 / sum_v exp(q_v - max q) (Eq. (2)); lane 0 updates the staged state words in LDS, then they
// are written back one word per lane.
__device__ __forceinline__ void finish_request(const AcceptArgs& a, int b, int n, int len, int bonus, Rec conf_r,
                               int lane, asv_req_state& q) {
  float conf = 0.f;
  if (a.n_conf > 0) {
    conf_r = rec_wave_reduce(conf_r);
    conf = 1.f / conf_r.s;
  }
  if (lane == 0) {
    a.acc_len[b] = len;
    a.bonus[b] = bonus;
    a.status[b] = 0;
    if (a.n_conf > 0 && a.draft_conf) a.draft_conf[b] = conf;
  }
  if (!a.state) return;
  if (lane == 0) {
    if (n > 1) {
      const float x = (float)len / (float)(n - 1);
      q.rar = q.rar + a.prm.alpha * (x - q.rar);
      const int head = q.hist_head & (ASV_HIST_WINDOW - 1);
      q.hist[head] = x;
      const int new_head = (head + 1) & (ASV_HIST_WINDOW - 1);
      const int count = min(max(q.hist_count, 0) + 1, ASV_HIST_WINDOW);
      // newest first, as many slots as are filled
      float sum = 0.f;
#pragma unroll
      for (int i = 0; i < ASV_HIST_WINDOW; ++i)
        sum += i < count ? q.hist[(new_head - 1 - i) & (ASV_HIST_WINDOW - 1)] : 0.f;
      q.hist_head = new_head;
      q.hist_count = count;
      q.hist_mean = sum / (float)count;
      const int streak = (len == 0) ? q.zero_streak + 1 : 0;
      const int trip = streak >= a.prm.breaker_n ? 1 : 0;
      q.breaker = trip;
      q.zero_streak = streak;
      if (trip) {
        q.rar = a.prm.rar0;
#pragma unroll
        for (int i = 0; i < ASV_HIST_WINDOW; ++i) q.hist[i] = 0.f;
        q.hist_head = 0;
        q.hist_count = 0;
        q.hist_mean = a.prm.rar0;
        q.zero_streak = 0;
      }
    } else {
      q.breaker = 0;
    }
    q.steps = q.steps + 1;
    if (a.n_conf > 0) q.draft_conf = conf;
    tree_shape(q, a.prm);
  }
  wave_lds_sync();
  if (lane < kStateWords)
    reinterpret_cast<uint32_t*>(a.state + b)[lane] = reinterpret_cast<const uint32_t*>(&q)[lane];
}

// Ordered key of a child: larger drafted logit first, then the lower node index. -0 is folded
// into +0 so that equal logits compare equal.
__device__ __forceinline__ uint64_t child_key(float g, int i) {
  const uint32_t u = __float_as_uint(g + 0.f);
  const uint32_t ord = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)ord << 32) | (uint32_t)(0xffffffffu - (uint32_t)i);
}

// Inputs of one request's walk that exist before the finishing step starts (parent, token,
// drafted logit, tau, state words, draft-confidence partials): loaded by stage_inputs into
// registers, lane-local, in one round.
struct WalkInputs {
  StageRegs r;
  float kappa;
  uint32_t st_word;
  Rec conf;
};

__device__ __forceinline__ void stage_inputs(const AcceptArgs& a, int b, int lo, int lane,
                                             WalkInputs& in) {
  stage_load(a, lo, lane, in.r);
  in.kappa = a.tau[b];
  in.st_word = (a.state && lane < kStateWords) ? reinterpret_cast<const uint32_t*>(a.state + b)[lane] : 0u;
  in.conf = conf_partials(a, b, lane);
}

// Request b with rows [lo, hi), 0 <= lo < hi <= N and n = hi - lo <= kWaveStage, with its
// inputs in `in` (stage_inputs). Loads the row max / argmax of the request's rows, then walks
// in LDS. Every lane of the wave calls this with the same arguments.
__device__ __forceinline__ void accept_staged(const AcceptArgs& a, int b, int lo, int hi, int lane,
                                              WalkSmem& sm, const WalkInputs& in) {
  const int n = hi - lo;
  float mx[kStagePerLane];
  int32_t arg[kStagePerLane];
#pragma unroll
  for (int u = 0; u < kStagePerLane; ++u) {
    const int c = min(lo + u * kWave + lane, a.N - 1);
    mx[u] = ld_device(a.row_max + c);
    arg[u] = ld_device(a.row_arg + c);
  }
  const float kappa = in.kappa;
  const Rec conf_r = in.conf;
  const int tree_bits = stage_check(a, lo, n, lane, in.r);
  stage_store(n, lane, in.r, sm);
#pragma unroll
  for (int u = 0; u < kStagePerLane; ++u) {
    const int i = u * kWave + lane;
    if (i < n) {
      sm.mx[i] = mx[u];
      sm.arg[i] = arg[u];
      sm.best[i] = 0;
    }
  }
  if (a.state && lane < kStateWords) reinterpret_cast<uint32_t*>(&sm.st)[lane] = in.st_word;
  wave_lds_sync();

  const int st = (!(kappa >= 0.f && kappa <= 1.f) ? ASV_RS_BAD_TAU : 0) | tree_bits;
  if (st) {
    for (int c = lo + lane; c < hi; c += kWave) {
      a.accept[c] = 0;
      a.path[c] = -1;
    }
    if (lane == 0) fail_request(a, b, st);
    return;
  }

  // ---- Eq. (1) for every node, and each node's best child (one LDS max per child)
  const float ln_kappa = kappa > 0.f ? a.prm.temperature * logf(kappa) : kNegInf;
  if (lane == 0) a.accept[lo] = 1;
  for (int i = 1 + lane; i < n; i += kWave) {
    const int p = sm.par[i] - lo;
    const float gi = sm.g[i];
    const bool ok = (sm.tok[i] == sm.arg[p]) || kappa == 0.f || (gi - sm.mx[p] >= ln_kappa);
    sm.ok[i] = ok;
    a.accept[lo + i] = ok;
    atomicMax(reinterpret_cast<unsigned long long*>(&sm.best[p]),
              (unsigned long long)child_key(gi, i));
  }
  wave_lds_sync();

  // ---- walk: follow the best-child chain while the child is accepted (wave-uniform)
  int cur = 0, len = 0, promos = 0;
  for (;;) {
    const uint64_t k = sm.best[cur];
    const uint32_t k_lo = __builtin_amdgcn_readfirstlane((uint32_t)k);
    const uint32_t k_hi = __builtin_amdgcn_readfirstlane((uint32_t)(k >> 32));
    if ((k_lo | k_hi) == 0) break;
    const int c = (int)(0xffffffffu - k_lo);
    if (!__builtin_amdgcn_readfirstlane(sm.ok[c])) break;
    if (__builtin_amdgcn_readfirstlane(sm.tok[c] != sm.arg[cur])) {
      if (a.prm.max_promotions >= 0 && promos >= a.prm.max_promotions) break;
      ++promos;
    }
    if (lane == 0) sm.pathl[len] = c;
    ++len;
    cur = c;
  }
  wave_lds_sync();
  for (int i = lane; i < n; i += kWave) a.path[lo + i] = i < len ? lo + sm.pathl[i] : -1;
  finish_request(a, b, n, len, sm.arg[cur], conf_r, lane, sm.st);
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

// Request b with more than kWaveStage nodes: the same steps, reading global memory, with one
// wave-wide best-child reduction per walk step. Only the state words are staged (sm.st).
__device__ __forceinline__ void accept_global(const AcceptArgs& a, int b, int lo, int hi, int lane,
                              WalkSmem& sm) {
  const int n = hi - lo;
  const float kappa = a.tau[b];
  const Rec conf_r = conf_partials(a, b, lane);
  if (a.state && lane < kStateWords)
    reinterpret_cast<uint32_t*>(&sm.st)[lane] =
        reinterpret_cast<const uint32_t*>(a.state + b)[lane];
  auto Mr = [&](int r) { return ld_device(a.row_max + r); };
  auto Ar = [&](int r) { return ld_device(a.row_arg + r); };

  bool bad_parent = false, bad_token = false;
  for (int c = lo + 1 + lane; c < hi; c += kWave) {
    const int p = a.parent[c], d = a.tok[c];
    bad_parent |= p < lo || p >= c;
    bad_token |= d < 0 || d >= a.V;
  }
  const int st = (!(kappa >= 0.f && kappa <= 1.f) ? ASV_RS_BAD_TAU : 0) |
                 (a.parent[lo] != -1 ? ASV_RS_BAD_ROOT : 0) |
                 (wave_any(bad_parent) ? ASV_RS_BAD_PARENT : 0) |
                 (wave_any(bad_token) ? ASV_RS_BAD_TOKEN : 0);
  if (st) {
    for (int c = lo + lane; c < hi; c += kWave) {
      a.accept[c] = 0;
      a.path[c] = -1;
    }
    if (lane == 0) fail_request(a, b, st);
    return;
  }

  const float ln_kappa = kappa > 0.f ? a.prm.temperature * logf(kappa) : kNegInf;
  for (int c = lo + lane; c < hi; c += kWave) {
    uint8_t ok = 1;
    if (c != lo) {
      const int p = a.parent[c];
      ok = (a.tok[c] == Ar(p)) || kappa == 0.f || (a.g[c] - Mr(p) >= ln_kappa);
    }
    a.accept[c] = ok;
  }

  int cur = lo, len = 0, promos = 0;
  for (;;) {
    float bg = kNegInf;
    int bc = kNoIndex;
    for (int c = lo + 1 + lane; c < hi; c += kWave) {
      if (a.parent[c] == cur) {
        const float gc = a.g[c];
        if (bc == kNoIndex || gc > bg || (gc == bg && c < bc)) {
          bg = gc;
          bc = c;
        }
      }
    }
    best_child_reduce(bg, bc);
    if (bc == kNoIndex) break;
    const int arg = Ar(cur);
    const int d = a.tok[bc];
    const bool ok = (d == arg) || kappa == 0.f || (bg - Mr(cur) >= ln_kappa);
    if (!ok) break;
    if (d != arg) {
      if (a.prm.max_promotions >= 0 && promos >= a.prm.max_promotions) break;
      ++promos;
    }
    if (lane == 0) a.path[lo + len] = bc;
    ++len;
    cur = bc;
  }
  for (int c = lo + len + lane; c < hi; c += kWave) a.path[c] = -1;
  wave_lds_sync();
  finish_request(a, b, n, len, Ar(cur), conf_r, lane, sm.st);
}

// ---- fused finishing step

constexpr int kFusedMaxB = 1024;   // largest batch of the fused finishing kernel
constexpr int kFinishWaves = 4;    // rows per workgroup, one wave per row

// Grid ceil(N / kFinishWaves); wave w of workgroup i owns row n = 4i + w. Each wave
//   1. loads the first 64 offset pairs and row n's slab records in one round, merges the
//      records and writes row n's statistics;
//   2. checks all offsets and finds the request b of row n by ballots; the wave is b's leader
//      here when row n is b's first row in this workgroup;
//   3. after a workgroup barrier, a leader adds the number of b's rows in this workgroup to
//      done_cnt[b] (one device-scope atomic per request and workgroup); the leader whose
//      addition completes b walks it.
// done_cnt[0..B) must be zero at launch (the LM-head kernel clears it). Requires B <= kFusedMaxB.
// Ordering without device-scope fences: row_max / row_argmax are written with device-coherent
// stores, and every wave waits for its stores to complete before the workgroup barrier that
// precedes the counter update; the completing wave reads them with device-coherent loads
// issued after the counter's returned value is known.
__global__ __launch_bounds__(kFinishWaves * kWave)
void k_merge_accept(int S, const float* __restrict__ rec_m, const float* __restrict__ rec_s,
                    const int32_t* __restrict__ rec_a, float* row_max, float* __restrict__ row_lse,
                    int32_t* row_argmax, int32_t* done_cnt, AcceptArgs a) {
  __shared__ WalkSmem s_walk[kFinishWaves];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r0 = blockIdx.x * kFinishWaves, n = r0 + w;
  const int r_end = min(r0 + kFinishWaves, a.N);
  const bool has_row = n < a.N;
  const size_t rbase = (size_t)(has_row ? n : 0) * S;

  // 1. first 64 offset pairs and the records in one round of loads; merge; row statistics
  const int i0 = min(lane, a.B - 1);
  const int ov0 = a.off[i0], onx0 = a.off[i0 + 1];
  RecBatch first;
  load_rec_batch(first, rbase, 0, S, lane, rec_m, rec_s, rec_a);
  if (has_row) {
    const Rec r = merge_row_rest(first, rbase, S, lane, rec_m, rec_s, rec_a);
    if (lane == 0) {
      st_device(row_max + n, r.m);
      row_lse[n] = r.m + __builtin_amdgcn_logf(r.s) * 0.69314718055994531f;
      st_device(row_argmax + n, r.a);
    }
  }

  // 2. offsets: validity (the same in every wave of the launch) and the request b of row n,
  // while the row statistics drain
  bool bad_lane = lane < a.B && offset_pair_bad(lane, a.B, a.N, ov0, onx0);
  int before_n = __popcll(__ballot(lane >= 1 && lane < a.B && ov0 <= n));
  for (int c0 = kWave; c0 < a.B; c0 += kWave) {  // batches beyond 64 requests
    const int i = c0 + lane, ic = min(i, a.B - 1);
    const int lo_i = a.off[ic], hi_i = a.off[ic + 1];
    bad_lane |= i < a.B && offset_pair_bad(i, a.B, a.N, lo_i, hi_i);
    before_n += __popcll(__ballot(i < a.B && lo_i <= n));
  }
  if (wave_any(bad_lane)) {  // every wave of every workgroup takes this branch
    for (int q = blockIdx.x * blockDim.x + threadIdx.x; q < a.B; q += gridDim.x * blockDim.x)
      fail_request(a, q, ASV_RS_BAD_OFFSETS);
    return;
  }
  const int b = before_n;
  int lo, hi;
  if (b < kWave) {
    lo = __builtin_amdgcn_readlane(ov0, b);
    hi = __builtin_amdgcn_readlane(onx0, b);
  } else {
    lo = a.off[b];
    hi = a.off[b + 1];
  }
  const bool leader = has_row && n == max(lo, r0);
  wait_stores();
  __syncthreads();

  // 3. count, and walk what this wave completed. A leader issues the loads of its request's
  // walk inputs together with the counter update, so their round trips overlap.
  if (!leader) return;
  const bool staged = hi - lo <= kWaveStage;
  WalkInputs in;
  if (staged) stage_inputs(a, b, lo, lane, in);
  int done = 0;
  if (lane == 0) {
    const int k = min(hi, r_end) - n;
    const int before = __hip_atomic_fetch_add(done_cnt + b, k, __ATOMIC_RELAXED,
                                              __HIP_MEMORY_SCOPE_AGENT);
    done = before + k == hi - lo;
  }
  if (!__builtin_amdgcn_readfirstlane(done)) return;
  if (staged)
    accept_staged(a, b, lo, hi, lane, s_walk[w], in);
  else
    accept_global(a, b, lo, hi, lane, s_walk[w]);
}

// ---- unfused finishing step, for batches beyond kFusedMaxB requests

constexpr int kMergeRowsPerBlock = 4;  // one wave per row

// Grid ceil(N / 4): merges one row per wave, and checks a slice of the offsets, raising
// *bad_flag (cleared by the LM-head kernel) when any pair is malformed.
__global__ __launch_bounds__(kMergeRowsPerBlock * kWave)
void k_slab_merge(int N, int S, const float* __restrict__ rec_m, const float* __restrict__ rec_s,
                  const int32_t* __restrict__ rec_a, float* __restrict__ row_max,
                  float* __restrict__ row_lse, int32_t* __restrict__ row_argmax, int B,
                  const int32_t* __restrict__ off, int32_t* __restrict__ bad_flag) {
  const int lane = threadIdx.x & 63;
  const int n = blockIdx.x * kMergeRowsPerBlock + (threadIdx.x >> 6);
  for (int b = blockIdx.x * blockDim.x + threadIdx.x; b < B; b += gridDim.x * blockDim.x)
    if (offset_pair_bad(b, B, N, off[b], off[b + 1])) atomicOr(bad_flag, 1);
  if (n >= N) return;
  const size_t base = (size_t)n * S;
  RecBatch first;
  load_rec_batch(first, base, 0, S, lane, rec_m, rec_s, rec_a);
  const Rec r = merge_row_rest(first, base, S, lane, rec_m, rec_s, rec_a);
  if (lane == 0) {
    row_max[n] = r.m;
    row_lse[n] = r.m + __builtin_amdgcn_logf(r.s) * 0.69314718055994531f;
    row_argmax[n] = r.a;
  }
}

// Grid B, one wave per request.
__global__ __launch_bounds__(kWave)
void k_tree_accept(const int32_t* __restrict__ bad_flag, AcceptArgs a) {
  __shared__ WalkSmem s_walk;
  const int b = blockIdx.x, lane = threadIdx.x;
  if (*bad_flag) {
    if (lane == 0) fail_request(a, b, ASV_RS_BAD_OFFSETS);
    return;
  }
  const int lo = a.off[b], hi = a.off[b + 1];
  if (hi - lo <= kWaveStage) {
    WalkInputs in;
    stage_inputs(a, b, lo, lane, in);
    accept_staged(a, b, lo, hi, lane, s_walk, in);
  } else
    accept_global(a, b, lo, hi, lane, s_walk);
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
  s->dcs = 0.f;
  for (int k = 0; k < 3; ++k) s->shape[k] = prm.shape_start[k];
}

// Grid-stride over requests: optional fresh draft confidence, then the tree shape.
__global__ void k_tree_policy(const float* __restrict__ conf, asv_req_state* state, int B,
                              asv_params prm) {
  for (int b = blockIdx.x * blockDim.x + threadIdx.x; b < B; b += gridDim.x * blockDim.x) {
    asv_req_state q = state[b];
    if (conf) q.draft_conf = conf[b];
    tree_shape(q, prm);
    state[b] = q;
  }
}

}  // namespace asv
