// The steps on either side of the target forward: tree-attention metadata before it (Sec. 1,
// Sec. 2: the whole draft tree is scored in one forward, each node attending to itself and its
// ancestors) and the commit of the accepted path after verification (Sec. 2, "Verify").
//
// K8 k_tree_meta: one workgroup per request. The request's parent links are staged in LDS;
//   each thread walks one node's chain to the root, which gives its depth and its row of the
//   ancestor bit mask (words written from the highest down, each exactly once).
// K9 k_commit: workgroups per request: its offset among the committed rows (a block sum of the
//   validated counts of the earlier requests), its tokens and rows, and a copy of the kept
//   rows' data.
#pragma once

#include "asv.h"
#include "k_common.h"

namespace asv {

constexpr int kMetaThreads = 256;
constexpr int kMetaLdsNodes = 8192;   // requests up to this size walk their links in LDS

// True when req_offsets is strictly increasing from 0 to N (every block checks all of it, so a
// malformed array flags every request, as in verification).
__device__ __forceinline__ bool offsets_ok_block(const int32_t* __restrict__ off, int B, int N,
                                                 int tid, int nthreads) {
  int bad = (tid == 0) && (off[0] != 0 || off[B] != N);
  for (int q = tid; q < B; q += nthreads) bad |= off[q] >= off[q + 1];
  return !__syncthreads_or(bad);
}

__global__ __launch_bounds__(kMetaThreads)
void k_tree_meta(const int32_t* __restrict__ parent, const int32_t* __restrict__ off, int B,
                 int N, const int32_t* __restrict__ pos_base, int mask_words,
                 int32_t* __restrict__ pos, uint32_t* __restrict__ mask,
                 int32_t* __restrict__ req_status) {
  __shared__ int s_par[kMetaLdsNodes];
  const int b = blockIdx.x, tid = threadIdx.x;
  if (!offsets_ok_block(off, B, N, tid, kMetaThreads)) {
    if (tid == 0) req_status[b] = ASV_RS_BAD_OFFSETS;
    return;
  }
  const int lo = off[b], n = off[b + 1] - lo;
  // local parent links; a root must have -1 and every other node an earlier node of its request
  int bad = 0;
  for (int c = tid; c < n; c += kMetaThreads) {
    const int p = parent[lo + c];
    if (c == 0) bad |= p != -1 ? ASV_RS_BAD_ROOT : 0;
    else bad |= (p < lo || p >= lo + c) ? ASV_RS_BAD_PARENT : 0;
    if (n <= kMetaLdsNodes) s_par[c] = c == 0 ? -1 : p - lo;
  }
  __shared__ int s_bad;
  if (tid == 0) s_bad = 0;
  __syncthreads();
  if (bad) atomicOr(&s_bad, bad);
  __syncthreads();
  const int status = s_bad | (mask && n > 32 * mask_words ? ASV_RS_MASK_SMALL : 0);
  if (tid == 0) req_status[b] = status;
  if (s_bad) return;
  const bool with_mask = mask && !(status & ASV_RS_MASK_SMALL);
  const int base = pos_base ? pos_base[b] : 0;
  for (int c = tid; c < n; c += kMetaThreads) {
    // walk c -> root; local ids strictly decrease, so mask words are completed in descending
    // order: word w is stored once the walk moves below 32 w
    uint32_t* row = with_mask ? mask + (size_t)(lo + c) * mask_words : nullptr;
    int w = mask_words - 1, depth = 0;
    uint32_t bits = 0;
    for (int j = c;; ) {
      if (row)
        for (; w > (j >> 5); --w) {
          row[w] = bits;
          bits = 0;
        }
      bits |= 1u << (j & 31);
      if (j == 0) break;
      j = n <= kMetaLdsNodes ? s_par[j] : parent[lo + j] - lo;
      ++depth;
    }
    if (row)
      for (; w >= 0; --w) {
        row[w] = bits;
        bits = 0;
      }
    if (pos) pos[lo + c] = base + depth;
  }
}

// ------------------------------------------------------------------------------------------ K9

constexpr int kCommitThreads = 256;
constexpr int kCommitSplit = 4;       // workgroups per request when rows are copied

struct CommitArgs {
  int B, N;
  const int32_t* off;
  const int32_t* tok;
  const int32_t* acc_len;
  const int32_t* path;
  const int32_t* bonus;
  int32_t* c_off;
  int32_t* c_tok;
  int32_t* c_row;
  const char* src;
  char* dst;
  long long row_bytes;
  int32_t* status;
};

// Committed length of request q (well-formed offsets), taken cooperatively by one wave:
// accepted_len + 1 when accepted_len lies in [0, n - 1] (n = its node count) and every accepted
// path entry is a non-root node of request q; else 1 (the root row and the bonus), with
// ASV_RS_BAD_PATH. Every workgroup derives each earlier request's count from the same checks,
// so the offset one request starts at is where the previous one ends.
__device__ __forceinline__ int commit_count_wave(const CommitArgs& a, int q, int lane,
                                                 int* bad) {
  const int lo = a.off[q], hi = a.off[q + 1];
  const int L = a.acc_len[q];
  if (L < 0 || L > hi - lo - 1) {
    *bad = ASV_RS_BAD_PATH;
    return 1;
  }
  bool out = false;
  for (int j = lane; j < L; j += kWave) {
    const int p = a.path[lo + j];
    out |= p <= lo || p >= hi;
  }
  if (__any(out)) {
    *bad = ASV_RS_BAD_PATH;
    return 1;
  }
  *bad = 0;
  return L + 1;
}

__global__ __launch_bounds__(kCommitThreads)
void k_commit(CommitArgs a) {
  __shared__ int s_base, s_cnt, s_bad;
  // Grid (B, G): workgroup (b, g) copies kept rows g, g + G, ... of request b; all G
  // workgroups of a request compute the same offset and checks, and only g = 0 writes the
  // status, the tokens and the row ids.
  const int b = blockIdx.x, g = blockIdx.y, G = gridDim.y, tid = threadIdx.x;
  const int lane = tid % kWave, wave = tid / kWave;
  constexpr int kWaves = kCommitThreads / kWave;
  if (!offsets_ok_block(a.off, a.B, a.N, tid, kCommitThreads)) {
    // nothing is committed: empty segments for every request
    if (tid == 0 && g == 0) {
      a.status[b] = ASV_RS_BAD_OFFSETS;
      a.c_off[b + 1] = 0;
      if (b == 0) a.c_off[0] = 0;
    }
    return;
  }
  if (tid == 0) s_base = 0;
  __syncthreads();
  // the earlier requests' validated counts, one wave per request; then this request's own
  int part = 0, bad = 0;
  for (int q = wave; q < b; q += kWaves) part += commit_count_wave(a, q, lane, &bad);
  if (lane == 0 && part) atomicAdd(&s_base, part);
  if (wave == 0) {
    const int cnt = commit_count_wave(a, b, lane, &bad);
    if (lane == 0) {
      s_cnt = cnt;
      s_bad = bad;
    }
  }
  __syncthreads();
  const int lo = a.off[b];
  const int base = s_base;
  const int sbad = s_bad;
  const int cnt = s_cnt;               // 1 (root row and bonus only) under ASV_RS_BAD_PATH
  const int len = cnt - 1;
  if (tid == 0 && g == 0) {
    a.status[b] = sbad;
    a.c_off[b + 1] = base + cnt;
    if (b == 0) a.c_off[0] = 0;
  }
  for (int j = tid; j < cnt && g == 0; j += kCommitThreads) {
    const int at = base + j;
    if (at >= a.N) break;
    const int row = j == 0 ? lo : a.path[lo + j - 1];
    a.c_row[at] = row;
    a.c_tok[at] = j < len ? a.tok[a.path[lo + j]] : a.bonus[b];
  }
  if (!a.src) return;
  // copy the kept rows: 16-byte chunks when rows allow it, else 4-byte words
  const long long rb = a.row_bytes;
  const bool wide = (rb & 15) == 0 && ((reinterpret_cast<uintptr_t>(a.src) |
                                        reinterpret_cast<uintptr_t>(a.dst)) & 15) == 0;
  const long long unit = wide ? 16 : 4;
  const long long per_row = rb / unit;
  const int mine = cnt > g ? (cnt - g + G - 1) / G : 0;     // kept rows g, g + G, ...
  const long long total = (long long)mine * per_row;
  for (long long e = tid; e < total; e += kCommitThreads) {
    const int k = (int)(e / per_row);
    const long long u = e - (long long)k * per_row;
    const int j = g + k * G;
    const int at = base + j;
    if (at >= a.N) break;
    const int row = j == 0 ? lo : a.path[lo + j - 1];
    const char* s = a.src + (long long)row * rb + u * unit;
    char* d = a.dst + (long long)at * rb + u * unit;
    if (wide) *reinterpret_cast<uint4*>(d) = *reinterpret_cast<const uint4*>(s);
    else *reinterpret_cast<uint32_t*>(d) = *reinterpret_cast<const uint32_t*>(s);
  }
}

}  // namespace asv
