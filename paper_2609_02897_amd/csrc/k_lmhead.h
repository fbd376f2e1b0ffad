// K1: fused target LM-head over every draft-tree row, reduced per vocabulary slab.
//
// For a tile of TV vocabulary rows x TR tree rows, the workgroup computes the logits
// z[n][v] = sum_h W[v][h] * X[n][h] (bf16 inputs, fp32 accumulation on the MFMA units) and,
// instead of storing them, writes one online-softmax record per (tree row, slab): the slab's
// max logit, the sum of exp(z - max) and the lowest argmax. It also writes the drafted logit
// z[parent(c)][draft_tok[c]] of every node c whose parent row and drafted token fall in the
// tile, read from the very accumulator the max saw. These are the target probabilities the
// margin rule of Sec. 3.2, Eq. (1) needs; the [N][V] logits never reach memory.
//
// Data flow: W and X tiles are staged HBM -> registers -> LDS (double buffered, 64 K-elements
// per stage, XOR-swizzled 16-byte chunks), read back in the MFMA operand layout and fed to
// v_mfma_f32_32x32x16_bf16. Both operands are K-contiguous (W is [V][H], X is [N][H]), so every
// lane moves 16 contiguous bytes per load. The MFMA's A operand is W (32 vocab rows) and B is X
// (32 tree rows): each lane then owns one tree row and 16 vocabulary entries of every 32x32
// output block, so the per-row reduction is mostly lane-local.
#pragma once

#include "k_common.h"

namespace asv {

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x16 __attribute__((__vector_size__(16 * sizeof(float))));

constexpr int kBK = 64;     // K elements per stage (one 128-byte segment of a row)
constexpr int kSlab = 256;  // vocabulary rows per workgroup = width of one record slab

// Staged tiles hold 8 chunks of 16 bytes per row; logical chunk c of row r sits at
// c ^ (r & 7), so 8 consecutive rows reading the same chunk use 8 distinct bank groups.
__device__ __forceinline__ int swz(int row, int chunk) { return row * 8 + (chunk ^ (row & 7)); }

// Word 3 of a raw buffer resource on gfx9-family GPUs (32-bit data format, no swizzle).
constexpr int kRsrcWord3 = 0x00020000;

__device__ __forceinline__ uint4 ld16(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
  return make_uint4(v.x, v.y, v.z, v.w);
}

template <int TV, int TR, int WV, int WR>
struct LmheadCfg {
  static constexpr int kThreads = WV * WR * kWave;
  static constexpr int kWaveV = TV / WV;        // vocabulary rows per wave
  static constexpr int kWaveR = TR / WR;        // tree rows per wave
  static constexpr int MV = kWaveV / 32;        // 32x32 blocks per wave, vocab direction
  static constexpr int MR = kWaveR / 32;        // 32x32 blocks per wave, tree-row direction
  static constexpr int CW = TV * 8 / kThreads;  // 16-byte W chunks each thread stages
  static constexpr int CX = TR * 8 / kThreads;  // 16-byte X chunks each thread stages
  static constexpr int kCand = 2;               // gather candidates prefetched per thread
  static_assert(TV == kSlab, "one record slab per workgroup");
  static_assert(MV >= 1 && MR >= 1 && CW >= 1 && CX >= 1, "tile too small for the wave grid");
  static_assert((TV * 8) % kThreads == 0 && (TR * 8) % kThreads == 0, "uneven staging");
  static_assert((kThreads / 8) % 8 == 0, "staged row groups must keep the swizzle phase");
};

// Map a launch-order block id to a tile so that each XCD (blocks are dealt to the 8 XCDs
// round-robin) works through a contiguous range of tiles: the row tiles of one vocabulary
// slab then run on one XCD and share that slab through its L2.
__device__ __forceinline__ int xcd_tile(int bid, int G) {
  const int q = G >> 3, rem = G & 7, xcd = bid & 7, loc = bid >> 3;
  return xcd * q + min(xcd, rem) + loc;
}

template <int TV, int TR, int WV, int WR>
__global__ __launch_bounds__(WV * WR * kWave)
void k_lmhead_partial(const uint16_t* __restrict__ X, const uint16_t* __restrict__ W,
                      const int32_t* __restrict__ parent, const int32_t* __restrict__ draft_tok,
                      const int32_t* __restrict__ req_offsets, int B, int N, int H, int V,
                      int S, int RT, float* __restrict__ rec_m, float* __restrict__ rec_s,
                      int32_t* __restrict__ rec_a, float* __restrict__ drafted_logit) {
  using C = LmheadCfg<TV, TR, WV, WR>;
  constexpr int T = C::kThreads;
  // One LDS block: two W stages, two X stages. The epilogue reuses it (gather list in the W
  // stages, reduction scratch at the start of X stage 0, two counters at X stage 1).
  __shared__ uint4 smem[2 * TV * 8 + 2 * TR * 8];
  auto sW = [&](int stage) { return smem + stage * (TV * 8); };
  auto sX = [&](int stage) { return smem + 2 * TV * 8 + stage * (TR * 8); };
  int* const s_seg_end = reinterpret_cast<int*>(sX(1));
  int* const s_cnt = s_seg_end + 1;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wv = wave % WV, wr = wave / WV;
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  const int slab = tile / RT, rt = tile % RT;
  const int v0 = slab * TV, r0 = rt * TR;
  const int v_end = min(v0 + TV, V);
  const int r_last = min(r0 + TR, N) - 1;

  // ---- staging through buffer loads: one resource per operand covering only this tile's
  // valid rows, so rows past V (last slab) or past N (last row tile) read as zeros and never
  // touch memory outside the arrays; their results are discarded below.
  const __amdgpu_buffer_rsrc_t w_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(W + (size_t)v0 * H), (short)0, (v_end - v0) * H * 2, kRsrcWord3);
  const __amdgpu_buffer_rsrc_t x_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(X + (size_t)r0 * H), (short)0, (r_last + 1 - r0) * H * 2,
      kRsrcWord3);
  // Thread t stages 16-byte chunk (t & 7) of rows (t >> 3) + i * T/8; consecutive threads read
  // consecutive 16 bytes of a row (8 threads cover one 128-byte segment).
  const int st_row = tid >> 3, st_ch = tid & 7;
  const int st_voff = st_row * H * 2 + st_ch * 16;
  const int st_dst = swz(st_row, st_ch);   // + i * T for chunk i (T/8 is a multiple of 8)
  uint4 rw[C::CW], rx[C::CX];
  auto load_stage = [&](int k0) {
#pragma unroll
    for (int i = 0; i < C::CW; ++i)
      rw[i] = ld16(w_rsrc, st_voff + i * (T / 8) * H * 2, k0 * 2);
#pragma unroll
    for (int i = 0; i < C::CX; ++i)
      rx[i] = ld16(x_rsrc, st_voff + i * (T / 8) * H * 2, k0 * 2);
  };
  auto store_stage = [&](int stage) {
#pragma unroll
    for (int i = 0; i < C::CW; ++i) sW(stage)[st_dst + i * T] = rw[i];
#pragma unroll
    for (int i = 0; i < C::CX; ++i) sX(stage)[st_dst + i * T] = rx[i];
  };
  load_stage(0);

  // ---- prefetch what the drafted-logit gather needs: the request offsets (to find the end
  // of the segment holding the tile's last row; children of the tile's rows lie before it)
  // and the parent / token of the first candidate nodes after r0.
  int off_lo = 0, off_hi = 0;
  if (tid < B) {
    off_lo = req_offsets[tid];
    off_hi = req_offsets[tid + 1];
  }
  int cc[C::kCand], cp[C::kCand], cd[C::kCand];
#pragma unroll
  for (int k = 0; k < C::kCand; ++k) {
    cc[k] = r0 + 1 + k * T + tid;
    cp[k] = -1;
    cd[k] = -1;
    if (cc[k] < N) {
      cp[k] = parent[cc[k]];
      cd[k] = draft_tok[cc[k]];
    }
  }

  store_stage(0);
  __syncthreads();

  // ---- main loop over K: prefetch stage kt+1 into registers while stage kt feeds the MFMAs
  f32x16 acc[C::MV][C::MR];
#pragma unroll
  for (int i = 0; i < C::MV; ++i)
#pragma unroll
    for (int j = 0; j < C::MR; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  const int KT = H / kBK;
  const int frag_row = lane & 31, frag_half = lane >> 5;
  for (int kt = 0; kt < KT; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < KT;
    if (more) load_stage((kt + 1) * kBK);
#pragma unroll
    for (int s = 0; s < kBK / 16; ++s) {
      bf16x8 a[C::MV], b[C::MR];
#pragma unroll
      for (int i = 0; i < C::MV; ++i) {
        const int row = wv * C::kWaveV + 32 * i + frag_row;
        a[i] = __builtin_bit_cast(bf16x8, sW(cur)[swz(row, 2 * s + frag_half)]);
      }
#pragma unroll
      for (int j = 0; j < C::MR; ++j) {
        const int row = wr * C::kWaveR + 32 * j + frag_row;
        b[j] = __builtin_bit_cast(bf16x8, sX(cur)[swz(row, 2 * s + frag_half)]);
      }
#pragma unroll
      for (int i = 0; i < C::MV; ++i)
#pragma unroll
        for (int j = 0; j < C::MR; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
    if (more) store_stage(cur ^ 1);
    __syncthreads();
  }

  // Output block (i, j), register e of a lane holds vocab row
  //   32*i + 8*(e/4) + 4*(lane/32) + e%4   (of the wave's vocab range) and
  // tree row 32*j + lane%32 (of the wave's row range).

  // ---- drafted logits: nodes whose parent row and drafted token fall inside this tile.
  // Matches are collected in LDS (the stage buffers are free now) and extracted by the lane
  // that owns the accumulator. Candidates beyond the prefetched ones are read in rounds.
  if (tid == 0) *s_seg_end = N;
  __syncthreads();
  if (tid < B && off_lo <= r_last && r_last < off_hi) atomicMin(s_seg_end, off_hi);
  for (int t = tid + T; t < B; t += T) {
    const int lo = req_offsets[t], hi = req_offsets[t + 1];
    if (lo <= r_last && r_last < hi) atomicMin(s_seg_end, hi);
  }
  __syncthreads();
  // Malformed offsets only widen or empty the candidate range; every access stays < N.
  const int cand_hi = max(r0 + 1, min(*s_seg_end, N));
  // Gather list in W stage 0, per-wave extraction scratch (64 lanes x 16 floats) in stage 1.
  int4* const s_list = reinterpret_cast<int4*>(sW(0));
  constexpr int kCap = TV * 8;
  float* const wscr = reinterpret_cast<float*>(sW(1)) + wave * (kWave * 16);
  static_assert(WV * WR * kWave * 16 * 4 <= TV * 8 * 16, "extraction scratch exceeds a stage");
  for (int base = r0 + 1; base < cand_hi; base += kCap) {
    if (tid == 0) *s_cnt = 0;
    __syncthreads();
    const int top = min(base + kCap, cand_hi);
    if (base == r0 + 1) {
#pragma unroll
      for (int k = 0; k < C::kCand; ++k) {
        const int c = cc[k], p = cp[k], d = cd[k];
        if (c < top && p >= r0 && p < r0 + TR && d >= v0 && d < v_end) {
          const int at = atomicAdd(s_cnt, 1);
          s_list[at] = make_int4(c, p - r0, d - v0, 0);
        }
      }
    }
    for (int c = max(base, r0 + 1 + C::kCand * T) + tid; c < top; c += T) {
      const int p = parent[c], d = draft_tok[c];
      if (p >= r0 && p < r0 + TR && d >= v0 && d < v_end) {
        const int at = atomicAdd(s_cnt, 1);
        s_list[at] = make_int4(c, p - r0, d - v0, 0);
      }
    }
    __syncthreads();
    const int cnt = *s_cnt;
    for (int e = 0; e < cnt; ++e) {
      const int4 m = s_list[e];
      const int pr = m.y - wr * C::kWaveR, dv = m.z - wv * C::kWaveV;
      if (pr < 0 || pr >= C::kWaveR || dv < 0 || dv >= C::kWaveV) continue;
      const int jj = pr >> 5, ii = dv >> 5, mm = dv & 31;
      const int ee = ((mm >> 3) << 2) | (mm & 3);
      const int owner = (pr & 31) + 32 * ((mm >> 2) & 1);
      // The block index is wave-uniform: branch to it, park its 16 registers in this wave's
      // LDS scratch and let the owner lane read its element back (LDS operations of one wave
      // complete in order).
#pragma unroll
      for (int i = 0; i < C::MV; ++i)
#pragma unroll
        for (int j = 0; j < C::MR; ++j)
          if (i == ii && j == jj) {
#pragma unroll
            for (int e2 = 0; e2 < 16; ++e2) wscr[e2 * kWave + lane] = acc[i][j][e2];
          }
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      if (lane == owner) drafted_logit[m.x] = wscr[ee * kWave + owner];
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    }
    __syncthreads();
  }

  // ---- per-row slab record: lane-local pass, then the two lane halves, then the waves
  // that share the same tree rows (through LDS).
  float* const red_m = reinterpret_cast<float*>(sX(0));
  float* const red_s = red_m + WV * TR;
  int* const red_a = reinterpret_cast<int*>(red_s + WV * TR);
#pragma unroll
  for (int j = 0; j < C::MR; ++j) {
    Rec r = rec_empty();
#pragma unroll
    for (int i = 0; i < C::MV; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int v = v0 + wv * C::kWaveV + 32 * i + 8 * (e >> 2) + 4 * frag_half + (e & 3);
        const float z = acc[i][j][e];
        if (v < V && z > r.m) {
          r.m = z;
          r.a = v;
        }
      }
    float s = 0.f;
    const float mb = r.m * kLog2e;
#pragma unroll
    for (int i = 0; i < C::MV; ++i)
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int v = v0 + wv * C::kWaveV + 32 * i + 8 * (e >> 2) + 4 * frag_half + (e & 3);
        if (v < V) s += exp2f(fmaf(acc[i][j][e], kLog2e, -mb));
      }
    r.s = s;
    r = rec_merge(r, rec_shfl_xor(r, 32));
    if (lane < 32) {
      const int row = wr * C::kWaveR + 32 * j + lane;
      red_m[wv * TR + row] = r.m;
      red_s[wv * TR + row] = r.s;
      red_a[wv * TR + row] = r.a;
    }
  }
  __syncthreads();
  for (int row = tid; row < TR; row += T) {
    Rec r{red_m[row], red_s[row], red_a[row]};
#pragma unroll
    for (int w = 1; w < WV; ++w) r = rec_merge(r, Rec{red_m[w * TR + row], red_s[w * TR + row],
                                                    red_a[w * TR + row]});
    const int n = r0 + row;
    if (n < N) {
      const size_t at = (size_t)n * S + slab;
      rec_m[at] = r.m;
      rec_s[at] = r.s;
      rec_a[at] = r.a;
    }
  }
}

}  // namespace asv
