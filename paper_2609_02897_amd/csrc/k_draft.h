// Draft side of a decoding step (Sec. 2, "Draft"): the draft LM head reduced to each row's top-4
// and log-sum-exp, one growth step of every request's draft tree, and the final pruning to the
// verification budget.
//
// K5 k_draft_partial: the LM-head tile of K1 (same staging, MFMA and accumulator layout) with a
//   top-4 epilogue: per (draft row, vocabulary slab) it writes the slab's four best (logit, id)
//   pairs, best first, as 64-bit order keys, and the sum of exp(z - best). The logits never
//   reach memory.
// K6 k_draft_grow: one workgroup per request, one wave per draft row (4 rows per request):
//   merge the slab records of the row, then wave 0 applies the growth step to the request's tree.
// K7 k_draft_prune: one workgroup per request: rank the pool, keep the best ndt - 1 nodes in
//   pool order and write the verification layout.
//
// Order of (logit, id) pairs everywhere: higher logit first, lower id on equal logits; a logit
// that is not a number is taken as -inf before any comparison.
#pragma once

#include "asv.h"
#include "k_common.h"
#include "k_lmhead.h"

namespace asv {

constexpr int kTopK = ASV_TOPK_MAX;   // 4
constexpr int kPoolMax = ASV_POOL_MAX;
constexpr int kDraftThreads = kTopK * kWave;
constexpr int kGrowBatch = 8;         // slab records a lane loads before merging them

__device__ __forceinline__ bool pair_better(float va, int ia, float vb, int ib) {
  return va > vb || (va == vb && ia < ib);
}

// Slot a keeps the better pair.
__device__ __forceinline__ void pair_order(float& va, int& ia, float& vb, int& ib) {
  const bool sw = pair_better(vb, ib, va, ia);
  const float tv = sw ? vb : va;
  const int ti = sw ? ib : ia;
  vb = sw ? va : vb;
  ib = sw ? ia : ib;
  va = tv;
  ia = ti;
}

// A (logit, id) pair as one 64-bit key whose unsigned order is the pair order: the high word is
// the logit's bits mapped to an order-preserving unsigned integer, the low word the complement
// of the id (a lower id gives a larger key). Logits are never a non-number here; -0 is folded
// into +0 first, so that equal logits compare equal as floats do. Key 0 lies below every pair.
__host__ __device__ __forceinline__ uint64_t pair_key(float v, int id) {
  const uint32_t u = __builtin_bit_cast(uint32_t, v + 0.f);
  const uint32_t o = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  return ((uint64_t)o << 32) | (uint32_t)~id;
}
__host__ __device__ __forceinline__ float key_value(uint64_t k) {
  const uint32_t o = (uint32_t)(k >> 32);
  return __builtin_bit_cast(float, (o & 0x80000000u) ? (o & 0x7fffffffu) : ~o);
}
__host__ __device__ __forceinline__ int key_id(uint64_t k) { return (int)~(uint32_t)k; }

// Four pairs as keys in descending order, the best logit m (the value of k[0]) and the sum of
// exp(z - m) over the set they were taken from (an empty set: keys 0, m = -inf, s = 0).
struct Top4 {
  uint64_t k[kTopK];
  float m;
  float s;
};

__device__ __forceinline__ Top4 top4_empty() {
  Top4 t;
#pragma unroll
  for (int q = 0; q < kTopK; ++q) t.k[q] = 0;
  t.m = kNegInf;
  t.s = 0.f;
  return t;
}

__device__ __forceinline__ void key_order(uint64_t& a, uint64_t& b) {
  const uint64_t hi = a > b ? a : b, lo = a > b ? b : a;
  a = hi;
  b = lo;
}

// The four best pairs of two sorted lists with disjoint ids: the larger of a[q] and b[3-q] for
// every q is a bitonic sequence holding them, which two compare-exchange stages sort. The sums
// merge like online-softmax records.
__device__ __forceinline__ Top4 top4_merge(const Top4& a, const Top4& b) {
  Top4 c;
#pragma unroll
  for (int q = 0; q < kTopK; ++q) c.k[q] = a.k[q] > b.k[3 - q] ? a.k[q] : b.k[3 - q];
  key_order(c.k[0], c.k[2]);
  key_order(c.k[1], c.k[3]);
  key_order(c.k[0], c.k[1]);
  key_order(c.k[2], c.k[3]);
  const Rec r = rec_merge(Rec{a.m, a.s, 0}, Rec{b.m, b.s, 0});
  c.m = r.m;
  c.s = r.s;
  // Opaque to the optimiser: chains of these merges (a slab loop followed by a wave
  // reduction) are otherwise folded into select trees that grow exponentially with the chain
  // length and stall the compiler. The empty asm costs no instruction.
#pragma unroll
  for (int q = 0; q < kTopK; ++q) asm volatile("" : "+v"(c.k[q]));
  return c;
}

__device__ __forceinline__ uint64_t shfl_xor64(uint64_t x, int mask) {
  const uint32_t lo = __shfl_xor((uint32_t)x, mask, kWave);
  const uint32_t hi = __shfl_xor((uint32_t)(x >> 32), mask, kWave);
  return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ Top4 top4_shfl_xor(const Top4& x, int mask) {
  Top4 y;
#pragma unroll
  for (int q = 0; q < kTopK; ++q) y.k[q] = shfl_xor64(x.k[q], mask);
  y.m = __shfl_xor(x.m, mask, kWave);
  y.s = __shfl_xor(x.s, mask, kWave);
  return y;
}

template <int N>
__device__ __forceinline__ uint64_t row_ror64(uint64_t x) {
  const uint32_t lo = (uint32_t)row_ror<N>((int)(uint32_t)x);
  const uint32_t hi = (uint32_t)row_ror<N>((int)(uint32_t)(x >> 32));
  return ((uint64_t)hi << 32) | lo;
}

template <int N>
__device__ __forceinline__ Top4 top4_row_ror(const Top4& x) {
  Top4 y;
#pragma unroll
  for (int q = 0; q < kTopK; ++q) y.k[q] = row_ror64<N>(x.k[q]);
  y.m = row_ror<N>(x.m);
  y.s = row_ror<N>(x.s);
  return y;
}

__device__ __forceinline__ Top4 top4_lane(const Top4& x, int l) {
  Top4 y;
#pragma unroll
  for (int q = 0; q < kTopK; ++q) {
    const uint32_t lo = (uint32_t)lane_value((int)(uint32_t)x.k[q], l);
    const uint32_t hi = (uint32_t)lane_value((int)(uint32_t)(x.k[q] >> 32), l);
    y.k[q] = ((uint64_t)hi << 32) | lo;
  }
  y.m = lane_value(x.m, l);
  y.s = lane_value(x.s, l);
  return y;
}

// Wave-wide merge without LDS round trips: rotations within each 16-lane row (every lane ends
// with its row's merge; the merged sets are disjoint at each step), then the four rows read as
// scalars and merged in a fixed order. Every lane returns the same record.
__device__ __forceinline__ Top4 top4_wave_reduce(Top4 t) {
  t = top4_merge(t, top4_row_ror<8>(t));
  t = top4_merge(t, top4_row_ror<4>(t));
  t = top4_merge(t, top4_row_ror<2>(t));
  t = top4_merge(t, top4_row_ror<1>(t));
  return top4_merge(top4_merge(top4_lane(t, 0), top4_lane(t, 16)),
                    top4_merge(top4_lane(t, 32), top4_lane(t, 48)));
}

// ------------------------------------------------------------------------------------------ K5

template <int TV, int TR, int WV, int WR, int BK, int NST>
__global__ __launch_bounds__(WV * WR * kWave, 1)
void k_draft_partial(const uint16_t* __restrict__ X, const uint16_t* __restrict__ W, int R,
                     int H, int V, int S, int RT, uint64_t* __restrict__ rec_k,
                     float* __restrict__ rec_s, int w_packed) {
  using C = LmheadCfg<TV, TR, WV, WR, BK, NST>;
  constexpr int T = C::kThreads;
  __shared__ uint4 smem[C::kLds / 16];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wv = wave % WV, wr = wave / WV;
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  const int slab = tile / RT, rt = tile % RT;
  const int v0 = slab * TV, r0 = rt * TR;

  f32x16 acc[C::MV][C::MR];
  // The non-temporal hint on the W copies pays for tiles of up to 64 rows (4 rows: 5% less
  // time after a cache flush); the 128-row tile is faster without it, because the draft
  // weight (262 MB at 32000 ids) largely fits the last-level cache.
  lmhead_tile<TV, TR, WV, WR, BK, NST, (TR <= 64)>(X, W, R, H, V, v0, r0, smem, w_packed, acc);

  // Output block (i, j), register e of a lane holds vocabulary row
  //   v0 + wv * kWaveV + 32 i + 8 (e / 4) + 4 (lane / 32) + e % 4   and
  // tree row wr * kWaveR + 32 j + lane % 32. For a fixed lane the entry ordinal k = 16 i + e
  // visits the lane's vocabulary ids in increasing order.
  const bool full_slab = v0 + TV <= V;
  const int vlane = v0 + wv * C::kWaveV + 4 * (lane >> 5);
  auto entry_v = [&](int k) { return vlane + 32 * (k >> 4) + 8 * ((k & 15) >> 2) + (k & 3); };
  // Lane-local top-4 of row block j: the first four entries sorted, then every later entry
  // inserted where it beats a kept one strictly (it has the highest id so far, so it loses
  // ties). MASK drops entries past V (last slab).
  auto lane_top4 = [&](int j, auto mask_tag) -> Top4 {
    constexpr bool MASK = decltype(mask_tag)::value;
    auto entry = [&](int k) {
      float z = fmaxf(acc[k >> 4][j][k & 15], kNegInf);    // a non-number becomes -inf
      if constexpr (MASK) z = entry_v(k) < V ? z : kNegInf;
      return z;
    };
    float v[kTopK];
    int id[kTopK];
#pragma unroll
    for (int k = 0; k < kTopK; ++k) {
      v[k] = entry(k);
      id[k] = entry_v(k);
    }
    pair_order(v[0], id[0], v[1], id[1]);
    pair_order(v[2], id[2], v[3], id[3]);
    pair_order(v[0], id[0], v[2], id[2]);
    pair_order(v[1], id[1], v[3], id[3]);
    pair_order(v[1], id[1], v[2], id[2]);
#pragma unroll
    for (int k = kTopK; k < C::MV * 16; ++k) {
      const float z = entry(k);
      const int e = entry_v(k);
      const bool b0 = z > v[0], b1 = z > v[1], b2 = z > v[2], b3 = z > v[3];
      v[3] = b2 ? v[2] : (b3 ? z : v[3]);
      id[3] = b2 ? id[2] : (b3 ? e : id[3]);
      v[2] = b1 ? v[1] : (b2 ? z : v[2]);
      id[2] = b1 ? id[1] : (b2 ? e : id[2]);
      v[1] = b0 ? v[0] : (b1 ? z : v[1]);
      id[1] = b0 ? id[0] : (b1 ? e : id[1]);
      v[0] = b0 ? z : v[0];
      id[0] = b0 ? e : id[0];
    }
    const float mb = v[0] * kLog2e;
    float sum = 0.f;
#pragma unroll
    for (int k = 0; k < C::MV * 16; ++k) sum += exp2_rel(fmaf(entry(k), kLog2e, -mb));
    Top4 t;
#pragma unroll
    for (int k = 0; k < kTopK; ++k) t.k[k] = pair_key(v[k], id[k]);
    t.m = v[0];
    t.s = v[0] == kNegInf ? 0.f : sum;
    return t;
  };

  // Per-row exchange area in the (now idle) LDS ring: WV records of four keys and a sum per
  // tree row.
  uint64_t* const x_k = reinterpret_cast<uint64_t*>(smem);
  float* const x_s = reinterpret_cast<float*>(x_k + WV * TR * kTopK);
  static_assert(WV * TR * (8 * kTopK + 4) <= C::kLds, "exchange area exceeds the ring");
#pragma unroll
  for (int j = 0; j < C::MR; ++j) {
    if (r0 + wr * C::kWaveR + 32 * j >= R) continue;        // row block past the last row
    Top4 t = full_slab ? lane_top4(j, std::false_type{}) : lane_top4(j, std::true_type{});
    t = top4_merge(t, top4_shfl_xor(t, 32));
    if (lane < 32) {
      const int at = wv * TR + wr * C::kWaveR + 32 * j + lane;
#pragma unroll
      for (int k = 0; k < kTopK; ++k) x_k[at * kTopK + k] = t.k[k];
      x_s[at] = t.s;
    }
    __builtin_amdgcn_sched_barrier(0);
  }
  __syncthreads();
  for (int row = tid; row < TR; row += T) {
    const int n = r0 + row;
    if (n >= R) break;
    auto load = [&](int w) {
      Top4 t;
      const int at = w * TR + row;
#pragma unroll
      for (int k = 0; k < kTopK; ++k) t.k[k] = x_k[at * kTopK + k];
      t.m = key_value(t.k[0]);
      t.s = x_s[at];
      return t;
    };
    Top4 t = load(0);
#pragma unroll
    for (int w = 1; w < WV; ++w) t = top4_merge(t, load(w));
    const size_t at = (size_t)n * S + slab;
    uint4* const dst = reinterpret_cast<uint4*>(rec_k + at * kTopK);
    dst[0] = make_uint4((uint32_t)t.k[0], (uint32_t)(t.k[0] >> 32), (uint32_t)t.k[1],
                        (uint32_t)(t.k[1] >> 32));
    dst[1] = make_uint4((uint32_t)t.k[2], (uint32_t)(t.k[2] >> 32), (uint32_t)t.k[3],
                        (uint32_t)(t.k[3] >> 32));
    rec_s[at] = t.s;
  }
}

// ------------------------------------------------------------------------------------------ K6

struct DraftGrowArgs {
  int B, S, step;
  const uint64_t* rec_k;
  const float* rec_s;
  const int32_t* vocab_map;
  const asv_req_state* state;
  int shape[3];
  asv_draft_tree* tree;
  int32_t* topk_id;
  float* topk_logp;
  float* row_lse;
  int32_t* front_tok;
  float* draft_conf;
};

__device__ __forceinline__ bool draft_shape_ok(int nsteps, int topk, int ndt) {
  return nsteps >= 1 && topk >= 1 && topk <= kTopK && ndt >= 1 &&
         nsteps <= kPoolMax && topk + (nsteps - 1) * topk * topk <= kPoolMax;
}

__global__ __launch_bounds__(kDraftThreads)
void k_draft_grow(DraftGrowArgs a) {
  __shared__ int s_id[kTopK][kTopK];
  __shared__ float s_lp[kTopK][kTopK];
  __shared__ float s_sc[kTopK * kTopK];
  __shared__ int s_ft[kTopK];
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63;
  const int slot = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int row = b * kTopK + slot;

  // ---- the tree's header, read first so that its latency overlaps the merge below
  asv_draft_tree* tr = a.tree + b;
  int nsteps, topk, ndt, steps, n_pool, n_front, status;
  int front[kTopK];
  float fscore[kTopK];
  if (a.step == 0) {
    if (a.state) {
      nsteps = a.state[b].shape[0];
      topk = a.state[b].shape[1];
      ndt = a.state[b].shape[2];
    } else {
      nsteps = a.shape[0];
      topk = a.shape[1];
      ndt = a.shape[2];
    }
    steps = 0;
    n_pool = 0;
    n_front = 1;
    status = draft_shape_ok(nsteps, topk, ndt) ? 0 : ASV_DS_BAD_SHAPE;
#pragma unroll
    for (int k = 0; k < kTopK; ++k) {
      front[k] = -1;
      fscore[k] = 0.f;
    }
  } else {
    nsteps = tr->nsteps;
    topk = tr->topk;
    ndt = tr->ndt;
    steps = tr->steps;
    n_pool = tr->n_pool;
    n_front = tr->n_front;
    status = tr->status;
    if (status == 0 && !draft_shape_ok(nsteps, topk, ndt)) status = ASV_DS_BAD_SHAPE;
#pragma unroll
    for (int k = 0; k < kTopK; ++k) {
      front[k] = tr->front[k];
      fscore[k] = tr->front_score[k];
    }
  }

  // ---- merge the S slab records of this wave's row: lane l takes slabs l, l + 64, ...,
  // kGrowBatch at a time, all loads of a batch issued before any merge (addresses clamped into
  // the row, slots past S masked afterwards), merged as a pairwise tree
  Top4 t = top4_empty();
  for (int base = 0; base < a.S; base += kWave * kGrowBatch) {
    Top4 r[kGrowBatch];
#pragma unroll
    for (int q = 0; q < kGrowBatch; ++q) {
      const int sl = base + q * kWave + lane;
      const size_t at = (size_t)row * a.S + min(sl, a.S - 1);
      const uint4* const src = reinterpret_cast<const uint4*>(a.rec_k + at * kTopK);
      const uint4 k01 = src[0], k23 = src[1];
      r[q].k[0] = ((uint64_t)k01.y << 32) | k01.x;
      r[q].k[1] = ((uint64_t)k01.w << 32) | k01.z;
      r[q].k[2] = ((uint64_t)k23.y << 32) | k23.x;
      r[q].k[3] = ((uint64_t)k23.w << 32) | k23.z;
      r[q].m = key_value(r[q].k[0]);
      r[q].s = a.rec_s[at];
    }
#pragma unroll
    for (int q = 0; q < kGrowBatch; ++q)
      if (base + q * kWave + lane >= a.S) r[q] = top4_empty();
#pragma unroll
    for (int w = 1; w < kGrowBatch; w *= 2)
#pragma unroll
      for (int q = 0; q + w < kGrowBatch; q += 2 * w) r[q] = top4_merge(r[q], r[q + w]);
    t = top4_merge(t, r[0]);
  }
  t = top4_wave_reduce(t);
  const float lse = t.m == kNegInf ? kNegInf : t.m + logf(t.s);
  if (lane < kTopK) {
    uint64_t key = t.k[0];
#pragma unroll
    for (int k = 1; k < kTopK; ++k)
      if (lane == k) key = t.k[k];
    const float v = key_value(key);
    const int id = key_id(key);
    float lp = v - lse;
    lp = lp != lp ? kNegInf : lp;
    const int tok = a.vocab_map ? a.vocab_map[id] : id;
    a.topk_id[row * kTopK + lane] = tok;
    a.topk_logp[row * kTopK + lane] = lp;
    s_id[slot][lane] = tok;
    s_lp[slot][lane] = lp;
  }
  if (lane == 0) a.row_lse[row] = lse;
  __syncthreads();
  if (slot != 0) return;

  // ---- wave 0: one growth step of request b's tree
  if (a.step == 0 && a.draft_conf && lane == 0) a.draft_conf[b] = expf(s_lp[0][0]);
  // the header bounds are checked again so that a tree that was never initialised (step > 0
  // first) cannot send a write outside its pool
  const bool grow = status == 0 && steps >= 0 && steps < nsteps && n_front >= 1 &&
                    n_front <= kTopK && n_pool >= 0 && n_pool + n_front * topk <= kPoolMax;
  int new_front_tok = -1;
  if (grow) {
    // candidate q = j * topk + c: child c of frontier slot j
    const int ncand = n_front * topk;
    float sc = kNegInf;
    int tok = -1, par = -1;
    if (lane < ncand) {
      const int j = lane / topk, c = lane % topk;
      float fs = fscore[0];
      int fp = front[0];
#pragma unroll
      for (int k = 1; k < kTopK; ++k)
        if (j == k) {
          fs = fscore[k];
          fp = front[k];
        }
      sc = __fadd_rn(fs, s_lp[j][c]);
      tok = s_id[j][c];
      par = fp;
    }
    // rank of each candidate: the candidates with a higher score, or an equal score and an
    // earlier position, read back from LDS by every lane
    if (lane < ncand) s_sc[lane] = sc;
    wave_lds_sync();
    int rank = 0;
#pragma unroll
    for (int q = 0; q < kTopK * kTopK; ++q) {
      const float sq = s_sc[q];
      rank += (q < ncand && (sq > sc || (sq == sc && q < lane))) ? 1 : 0;
    }
    if (lane < ncand) {
      tr->tok[n_pool + lane] = tok;
      tr->par[n_pool + lane] = par;
      tr->score[n_pool + lane] = sc;
    }
    if (lane < ncand && rank < topk) {
      tr->front[rank] = n_pool + lane;
      tr->front_score[rank] = sc;
      s_ft[rank] = tok;
    }
    // the token of frontier slot r goes to lane r (the next forward's input order)
    wave_lds_sync();
    if (lane < topk) new_front_tok = s_ft[lane];
    if (lane == 0) {
      tr->n_pool = n_pool + ncand;
      tr->n_front = topk;
      tr->steps = steps + 1;
    }
  }
  if (a.step == 0 && lane == 0) {
    tr->nsteps = nsteps;
    tr->topk = topk;
    tr->ndt = ndt;
    tr->status = status;
    tr->reserved = 0;
    if (!grow) {
      tr->steps = 0;
      tr->n_pool = 0;
      tr->n_front = 1;
      tr->front[0] = -1;
      tr->front_score[0] = 0.f;
    }
  }
  if (lane < kTopK) a.front_tok[b * kTopK + lane] = new_front_tok;
}

// ------------------------------------------------------------------------------------------ K7

constexpr int kPruneThreads = kPoolMax;

__device__ __forceinline__ int draft_tree_rows(const asv_draft_tree* t) {
  const int n_pool = t->n_pool, ndt = t->ndt;
  if (t->status != 0 || n_pool < 0 || n_pool > kPoolMax || ndt < 1) return 1;
  return 1 + min(ndt - 1, n_pool);
}

__global__ __launch_bounds__(kPruneThreads)
void k_draft_prune(const asv_draft_tree* __restrict__ trees,
                   const int32_t* __restrict__ root_tok, int n_cap, int32_t* __restrict__ parent,
                   int32_t* __restrict__ draft_tok, int32_t* __restrict__ req_offsets,
                   int32_t* __restrict__ req_status) {
  __shared__ float s_score[kPoolMax];
  __shared__ int s_map[kPoolMax];
  __shared__ int s_part[kPruneThreads / kWave];
  const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const asv_draft_tree* t = trees + b;

  // ---- offset of this request: rows of all earlier trees
  __shared__ int s_lo;
  if (tid == 0) s_lo = 0;
  __syncthreads();
  int part = 0;
  for (int q = tid; q < b; q += kPruneThreads) part += draft_tree_rows(trees + q);
  if (part) atomicAdd(&s_lo, part);
  __syncthreads();
  const int lo = s_lo;
  const int n = draft_tree_rows(t);
  const int hi = lo + n;
  if (tid == 0) {
    req_offsets[b + 1] = hi;
    if (b == 0) req_offsets[0] = 0;
    req_status[b] = t->status | (hi > n_cap ? ASV_DS_OVERFLOW : 0);
  }
  if (hi > n_cap) return;
  if (tid == 0) {
    parent[lo] = -1;
    draft_tok[lo] = root_tok ? root_tok[b] : -1;
  }
  if (n == 1) return;

  // ---- rank the pool: the n - 1 best (higher score, earlier entry on ties) are kept
  const int P = t->n_pool, m = n - 1;
  const float sq = tid < P ? t->score[tid] : kNegInf;
  if (tid < P) s_score[tid] = sq;
  __syncthreads();
  int rank = 0;
  for (int q = 0; q < P; ++q) {
    const float s = s_score[q];
    rank += (s > sq || (s == sq && q < tid)) ? 1 : 0;
  }
  const bool keep = tid < P && rank < m;
  // ---- position of each kept entry in pool order: exclusive prefix count of `keep`
  const uint64_t bal = __ballot(keep);
  const int before = __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                               __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0));
  if (lane == 0) s_part[wave] = __popcll(bal);
  __syncthreads();
  int base = 0;
  for (int w = 0; w < wave; ++w) base += s_part[w];
  if (tid < P) s_map[tid] = keep ? 1 + base + before : -1;
  __syncthreads();
  if (keep) {
    const int node = lo + 1 + base + before;
    const int p = t->par[tid];
    // parents score at least as high and come earlier, so a kept node's parent is kept
    const int pl = p < 0 ? 0 : (p < P && s_map[p] > 0 ? s_map[p] : 0);
    parent[node] = lo + pl;
    draft_tok[node] = t->tok[tid];
  }
}

}  // namespace asv
