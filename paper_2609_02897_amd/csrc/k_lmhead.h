// K1: fused target LM-head over every draft-tree row, reduced per vocabulary slab.
//
// For a tile of TV vocabulary rows (one record slab) x TR tree rows, the workgroup computes the logits
// z[n][v] = sum_h W[v][h] * X[n][h] (bf16 inputs, fp32 accumulation on the MFMA units) and,
// instead of storing them, writes one online-softmax record per (tree row, slab): the slab's
// max logit, the sum of exp(z - max) and the lowest argmax. It also writes the drafted logit
// z[parent(c)][draft_tok[c]] of every node c whose parent row and drafted token fall in the
// tile, read from the very accumulator the max saw. These are the target probabilities the
// margin rule of Sec. 3.2, Eq. (1) needs; the [N][V] logits never reach memory.
//
// Data flow: a ring of NST LDS stages, each holding BK K-elements of every W and X row of the
// tile. Stages are filled by direct global->LDS buffer loads (no staging registers) and their
// completion is awaited by hand (s_waitcnt vmcnt) before a workgroup barrier. Two K loops
// share this layout: lmhead_tile issues each stage's copies in one burst, NST-1 stages ahead,
// with one barrier per stage; lmhead_tile_spread / lmhead_tile_spread3 place every copy
// between two MFMAs on a fixed schedule, so the copies never stall a wave's MFMAs (the 128-
// and 256-row tiles, which are MFMA-bound). 16-byte chunks are XOR-swizzled so that
// ds_read_b128 in the MFMA operand layout is free of bank conflicts. K1 runs
// v_mfma_f32_16x16x32_bf16 with A = W (16 vocabulary rows) and B = X (16 tree rows): each lane
// then owns one tree row and 4 vocabulary entries of every 16x16 output block, so the per-row
// reduction is mostly lane-local, with two cross-lane steps. (The draft LM head, which shares
// the burst ring, runs v_mfma_f32_32x32x16_bf16: 16 entries of a 32x32 block per lane.) In
// every comparison made the two shapes gave bit-identical logits; the 16x16x32 form lets the
// chip hold a higher clock under K1's sustained MFMA load. Fragments of a later K step are read while the current MFMAs run.
// Every loop accumulates K in increasing order, so all tiles give the same logits bit for bit.
#pragma once

#include <type_traits>

#include "k_common.h"

namespace asv {

typedef __bf16 bf16x8 __attribute__((__vector_size__(8 * sizeof(__bf16))));
typedef float f32x16 __attribute__((__vector_size__(16 * sizeof(float))));
typedef float f32x4 __attribute__((__vector_size__(4 * sizeof(float))));

// The two bf16 MFMA shapes a tile can run on. Both take 8 bf16 of A and of B per lane: lane l
// holds row (of A) or column (of B) l % kBlock and the 8 consecutive K elements
// 8 (l / kBlock) .. + 7 of the instruction's K step, so a fragment is one 16-byte LDS read.
// row_of(lane, e) is the A row (vocabulary entry) of accumulator register e of a lane; its
// B column (tree row) is lane % kBlock. Within a lane, row_of increases with e.
// The 16x16x32 form does the same work per K element with a quarter of the accumulator
// registers per instruction; under sustained load the chip holds a higher shader clock with it.
struct Mfma32 {   // v_mfma_f32_32x32x16_bf16
  using Acc = f32x16;
  static constexpr int kBlock = 32, kK = 16, kRegs = 16;
  static __device__ __forceinline__ Acc mma(bf16x8 a, bf16x8 b, Acc c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ Acc mma_chained(bf16x8 a, bf16x8 b, Acc c) {
    return mma(a, b, c);
  }
  static __device__ __forceinline__ int row_of(int lane, int e) {
    return 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
  }
  // register and lane holding row m (of the block) of tree row p (of the block)
  static __device__ __forceinline__ int reg_of(int m) { return ((m >> 3) << 2) | (m & 3); }
  static __device__ __forceinline__ int lane_of(int p, int m) { return p + 32 * ((m >> 2) & 1); }
};
struct Mfma16 {   // v_mfma_f32_16x16x32_bf16
  using Acc = f32x4;
  static constexpr int kBlock = 16, kK = 32, kRegs = 4;
  // The empty asm keeps each result in accumulator registers; without it the register
  // allocator moves the 4-register accumulators between AGPRs and VGPRs on every pass of the
  // smaller tiles' K loops. It emits no instruction.
  static __device__ __forceinline__ Acc mma(bf16x8 a, bf16x8 b, Acc c) {
    Acc d = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    asm volatile("" : "+a"(d));
    return d;
  }
  // Without the pin, for a result whose only use is a later MFMA of the same loop pass. The
  // two-slot spread loop pins only each pass's last K step: pinning every step there made the
  // allocator rotate 12 accumulator registers of the 192-row tile through copies on every pass.
  static __device__ __forceinline__ Acc mma_chained(bf16x8 a, bf16x8 b, Acc c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ int row_of(int lane, int e) { return 4 * (lane >> 4) + e; }
  static __device__ __forceinline__ int reg_of(int m) { return m & 3; }
  static __device__ __forceinline__ int lane_of(int p, int m) { return p + 16 * (m >> 2); }
};

constexpr int kKAlign = 64;   // H must be a multiple of this (host check)

// Word 3 of a raw buffer resource on gfx9-family GPUs (32-bit data format, no swizzle).
constexpr int kRsrcWord3 = 0x00020000;

// A staged row of BK bf16 is CPR = BK / 8 chunks of 16 bytes. Logical chunk c of row r is
// stored at position c ^ f(r) (16-byte units from the region start). The LDS serves a wave's
// ds_read_b128 in four passes of 16 lanes over 64 four-byte banks, 16 bank groups of 16 bytes;
// a pass takes the lanes with equal lane bit 5 and equal parity of lane bits 2, 3 and 4
// (measured: this grouping reproduces the bank-conflict counts of every probe pattern), and a
// pass takes as many cycles as it has lanes on its busiest bank group. With 128-byte rows a read
// lands in group 8 (r & 1) + (c ^ f(r)) mod 8, and f(r) = (r >> 1) & 7 gives every pass 16
// distinct groups in both fragment layouts: 32x32x16 (lane l reads row l % 32, chunk
// 2 s + l / 32) and 16x16x32 (row l % 16, chunk 4 s + l / 16). 64-byte rows (32x32x16 only)
// take f(r) = ((r >> 2) ^ (r >> 1)) & 3.
template <int CPR>
__host__ __device__ __forceinline__ int swz_phase(int row) {
  static_assert(CPR == 4 || CPR == 8, "64- or 128-byte staged rows");
  return CPR == 8 ? ((row >> 1) & 7) : (((row >> 2) ^ (row >> 1)) & 3);
}
template <int CPR>
__host__ __device__ __forceinline__ int swz(int row, int chunk) {
  return row * CPR + (chunk ^ swz_phase<CPR>(row));
}

// Direct global->LDS copy of 16 bytes per lane from byte voff + soff of the buffer: lane t's
// 16 bytes land at LDS byte address lds + 16 t. A lane whose offset lies past the buffer
// resource's range writes zeros. The K loops keep each lane's offset within its row in voff
// (fixed for the whole loop) and put the K stage's offset, the same for every lane, in the
// scalar soff: the per-copy address needs no vector instruction, and the range check still
// turns every row past the valid ones into zeros (their voff alone is out of range) whether or
// not soff takes part in it.
// M0 is reserved: the compiler sets it right before each instruction that reads it and never
// keeps a value in it across other code on gfx9-family GPUs, so overwriting it here is safe;
// the clobber is declared anyway.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(int lds, int voff, int soff, __amdgpu_buffer_rsrc_t r) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               :
               : "s"(lds), "v"(voff), "s"(r), "s"(soff)
               : "memory", "m0");
}
// The same copy with the non-temporal hint (nt): for data read once and streamed, which the
// caches should not try to keep.
__device__ __forceinline__ void dma16_stream(int lds, int voff, int soff,
                                             __amdgpu_buffer_rsrc_t r) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen nt lds"
               :
               : "s"(lds), "v"(voff), "s"(r), "s"(soff)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// Wait until at most N vector-memory operations of this wave are outstanding and its LDS
// reads are done, then join the workgroup barrier. Loads complete in order, so this retires
// every older stage copy.
template <int N>
__device__ __forceinline__ void wait_vm_barrier() {
  asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" : : "n"(N) : "memory");
}

// wait_vm_barrier<newer * L>() for a run-time newer in [0, 3]: each stage issues L operations,
// and the newer stages' operations may stay in flight.
template <int L>
__device__ __forceinline__ void wait_stage_barrier(int newer) {
  if (newer >= 3) wait_vm_barrier<3 * L>();
  else if (newer == 2) wait_vm_barrier<2 * L>();
  else if (newer == 1) wait_vm_barrier<L>();
  else wait_vm_barrier<0>();
}

template <int TV, int TR, int WV, int WR, int BK, int NST, class MF = Mfma32>
struct LmheadCfg {
  static constexpr int kWaves = WV * WR;
  static constexpr int kThreads = kWaves * kWave;
  static constexpr int kWaveV = TV / WV;        // vocabulary rows per wave
  static constexpr int kWaveR = TR / WR;        // tree rows per wave
  static constexpr int MV = kWaveV / MF::kBlock;  // MFMA blocks per wave, vocab direction
  static constexpr int MR = kWaveR / MF::kBlock;  // MFMA blocks per wave, tree-row direction
  static constexpr int NS = BK / MF::kK;        // MFMA K steps per stage
  static constexpr int CPR = BK / 8;            // 16-byte chunks per staged row
  static constexpr int kRowsPerCopy = 64 / CPR; // rows one 1 KB wave copy fills
  static constexpr int kStageW = TV * BK * 2;   // bytes of W per stage
  static constexpr int kStageX = TR * BK * 2;   // bytes of X per stage
  static constexpr int kStage = kStageW + kStageX;
  static constexpr int DW = kStageW / 1024 / kWaves;  // 1 KB copies per wave per stage, W
  static constexpr int DX = kStageX / 1024 / kWaves;  // 1 KB copies per wave per stage, X
  static constexpr int kLoads = DW + DX;        // vector-memory ops per lane per stage
  static constexpr int kLds = NST * kStage;
  static constexpr int kCand = 2;               // gather candidates prefetched per thread
  static_assert(TV % 32 == 0 && TR % 32 == 0 && kWaveV % MF::kBlock == 0 &&
                kWaveR % MF::kBlock == 0, "whole MFMA blocks");
  static_assert(MV >= 1 && MR >= 1, "tile too small for the wave grid");
  static_assert(BK == 32 || BK == 64, "stage depth");
  static_assert(NST >= 1 && NST <= 5, "ring depth");
  static_assert(DW >= 1 && DX >= 1 && DW * kWaves * 1024 == kStageW &&
                DX * kWaves * 1024 == kStageX, "each wave copies whole 1 KB groups");
  static_assert(NST < 2 || (NST - 2) * kLoads <= 63, "vmcnt range");
  static_assert(kLds <= 160 * 1024, "LDS per workgroup");
};

// Map a launch-order block id to a tile so that each XCD (blocks are dealt to the 8 XCDs
// round-robin) works through a contiguous range of tiles: the row tiles of one vocabulary
// slab then run on one XCD and share that slab through its L2.
__host__ __device__ __forceinline__ int xcd_tile(int bid, int G) {
  const int q = G >> 3, rem = G & 7, xcd = bid & 7, loc = bid >> 3;
  return xcd * q + min(xcd, rem) + loc;
}

// Tile t of a launch over n_slabs vocabulary slabs x RT row tiles -> (slab within the launch,
// row tile). With blk_rows = 0 the order is slab-major (the row tiles of one slab are
// consecutive). Otherwise the slabs go in blocks of blk_slabs, each block's tiles in groups of
// blk_rows row tiles (the last group takes the rest), slab-major within a group: a run of
// blk_slabs * blk_rows consecutive tiles, which xcd_tile keeps on one XCD, then reads
// blk_slabs W slabs and blk_rows X row tiles through that XCD's L2 instead of about
// blk_slabs * blk_rows / RT slabs and all RT row tiles. Every (slab, row tile) pair is taken
// once; the order changes no result.
__host__ __device__ __forceinline__ void tile_coords(int t, int n_slabs, int RT, int blk_slabs,
                                            int blk_rows, int& slab, int& rt) {
  if (blk_rows <= 0 || blk_rows >= RT) {
    slab = t / RT;
    rt = t % RT;
    return;
  }
  const int blk = t / (blk_slabs * RT), rem = t % (blk_slabs * RT);
  const int sb = min(blk_slabs, n_slabs - blk * blk_slabs);  // slabs in this block
  const int group = sb * blk_rows, full_groups = RT / blk_rows;
  if (rem < full_groups * group) {
    const int g = rem / group, in = rem % group;
    slab = blk * blk_slabs + in / blk_rows;
    rt = g * blk_rows + in % blk_rows;
  } else {
    const int rest = RT - full_groups * blk_rows, in = rem - full_groups * group;
    slab = blk * blk_slabs + in / rest;
    rt = full_groups * blk_rows + in % rest;
  }
}

// What every K loop of a tile shares: this wave's place in the tile; one buffer resource per
// operand covering only the tile's valid rows (rows past V in the last slab or past N in the
// last row tile read as zeros and never touch memory outside the arrays; their results are
// discarded by the caller); the source offsets of this wave's stage copies; the LDS addresses
// of the MFMA fragments. Copy j of a stage region fills rows R j .. R j + R - 1
// (R = kRowsPerCopy): lane t supplies 16 bytes of row R j + t / CPR at swizzled position
// t % CPR, i.e. the logical chunk (t % CPR) ^ f(R j + t / CPR).
// W is row-major [V][H], or packed (w_packed != 0, written by k_pack_tiles with BK = 64):
// K block k holds rows 0 .. Vp - 1 (V rounded up to max(TV, 128) rows, zero past V) as
// consecutive [BK]-wide row segments, so the TV rows of slab s at K block k are one contiguous
// run starting at element k Vp BK + v0 BK. Offsets within the packed buffer are 32-bit
// unsigned (the host keeps it under 4 GiB).
// STREAM_W: copy W with the non-temporal hint. K1 takes it for launches of one or two row
// tiles, which read each W slab about once (60 rows: 13% less time), and the default policy
// for more row tiles, which share each W slab through an XCD's L2 (with the hint: 378 rows'
// three 128-row tiles a slab about 2% slower, 2048 and 3048 rows 1.5% and 4.5%).
template <int TV, int TR, int WV, int WR, int BK, int NST, bool STREAM_W = (TR <= 128),
          class MF = Mfma32>
struct TileIo {
  using C = LmheadCfg<TV, TR, WV, WR, BK, NST, MF>;
  static constexpr int CPR = C::CPR;
  static constexpr bool kStreamW = STREAM_W;
  static constexpr int NS = C::NS;
  const uint4* lds;
  int lane, wave, wv, wr, lds0, frag_row, frag_grp;
  // 16-byte units, within a ring slot, of this lane's fragment of W block 0 / X block 0 at
  // K step s. Block i sits kBlock i rows further on, at the same swizzled chunk (the swizzle
  // repeats every 16 rows), so a fragment address is one of these plus a constant, which the
  // LDS read takes as its immediate offset.
  int w_frag0[NS], x_frag0[NS];
  unsigned w_kstep;             // bytes between the W data of consecutive K stages
  __amdgpu_buffer_rsrc_t w_rsrc, x_rsrc;
  int w_voff[C::DW], x_voff[C::DX];

  __device__ __forceinline__ TileIo(const uint16_t* X, const uint16_t* W, int N, int H, int V,
                                    int v0, int r0, const uint4* smem, int w_packed)
      : lds(smem) {
    lane = threadIdx.x & 63;
    wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    wv = wave % WV;
    wr = wave / WV;
    frag_row = lane % MF::kBlock;
    frag_grp = lane / MF::kBlock;
    static_assert(MF::kBlock % 16 == 0 && C::kWaveV % 16 == 0 && C::kWaveR % 16 == 0,
                  "fragment blocks start at whole periods of the swizzle");
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      w_frag0[s] = swz<CPR>(wv * C::kWaveV + frag_row, (MF::kK / 8) * s + frag_grp);
      x_frag0[s] =
          C::kStageW / 16 + swz<CPR>(wr * C::kWaveR + frag_row, (MF::kK / 8) * s + frag_grp);
    }
    lds0 = __builtin_amdgcn_readfirstlane((int)(size_t)smem);
    const int v_end = min(v0 + TV, V);
    const int r_last = min(r0 + TR, N) - 1;
    if (w_packed) {
      constexpr unsigned kAlign = TV > 128 ? TV : 128;
      const unsigned Vp = (V + kAlign - 1) / kAlign * kAlign, tile = TV * BK * 2;
      w_kstep = Vp * BK * 2;
      w_rsrc = __builtin_amdgcn_make_buffer_rsrc(
          const_cast<uint16_t*>(W + (size_t)v0 * BK), (short)0,
          (int)((unsigned)(H / BK - 1) * w_kstep + tile), kRsrcWord3);
    } else {
      w_kstep = BK * 2;
      w_rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(W + (size_t)v0 * H),
                                                 (short)0, (v_end - v0) * H * 2, kRsrcWord3);
    }
    x_rsrc = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(X + (size_t)r0 * H),
                                               (short)0, (r_last + 1 - r0) * H * 2, kRsrcWord3);
#pragma unroll
    for (int i = 0; i < C::DW; ++i)
      w_voff[i] = copy_voff(i * C::kWaves + wave, w_packed ? BK : H);
#pragma unroll
    for (int i = 0; i < C::DX; ++i) x_voff[i] = copy_voff(i * C::kWaves + wave, H);
  }
  // byte offset of this lane's 16 bytes of copy j at K stage 0; `pitch` elements per row
  __device__ __forceinline__ int copy_voff(int j, int pitch) const {
    const int row = j * C::kRowsPerCopy + lane / CPR;
    return row * pitch * 2 + ((lane % CPR) ^ swz_phase<CPR>(row)) * 16;
  }
  // copy c of this wave (the W copies first, then the X copies) of K stage ks into ring slot
  // `slot`
  template <int c>
  __device__ __forceinline__ void copy(int slot, int ks) const {
    const int base = lds0 + slot * C::kStage;
    if constexpr (c < C::DW) {
      const int lds_at = base + (c * C::kWaves + wave) * 1024;
      const int so = __builtin_amdgcn_readfirstlane((int)((unsigned)ks * w_kstep));
      if constexpr (kStreamW)
        dma16_stream(lds_at, w_voff[c], so, w_rsrc);
      else
        dma16(lds_at, w_voff[c], so, w_rsrc);
    } else
      dma16(base + C::kStageW + ((c - C::DW) * C::kWaves + wave) * 1024, x_voff[c - C::DW],
            __builtin_amdgcn_readfirstlane(ks * BK * 2), x_rsrc);
  }
  // the fragment of W block i (of this wave's vocabulary rows), or of X block j (of its tree
  // rows), for MFMA K step s of ring slot `slot`
  __device__ __forceinline__ bf16x8 w_frag(int slot, int s, int i) const {
    const uint4* w = lds + slot * (C::kStage / 16) + w_frag0[s];
    return __builtin_bit_cast(bf16x8, w[MF::kBlock * CPR * i]);
  }
  __device__ __forceinline__ bf16x8 x_frag(int slot, int s, int j) const {
    const uint4* x = lds + slot * (C::kStage / 16) + x_frag0[s];
    return __builtin_bit_cast(bf16x8, x[MF::kBlock * CPR * j]);
  }
};

template <class Acc, int MV, int MR>
__device__ __forceinline__ void zero_acc(Acc (&acc)[MV][MR]) {
  constexpr int kRegs = sizeof(Acc) / sizeof(float);
#pragma unroll
  for (int i = 0; i < MV; ++i)
#pragma unroll
    for (int j = 0; j < MR; ++j)
#pragma unroll
      for (int e = 0; e < kRegs; ++e) acc[i][j][e] = 0.f;
}

// The logits of one tile, left in the MFMA accumulators: acc[i][j] holds the block of
// vocabulary rows v0 + wv * kWaveV + kBlock i .. and tree rows r0 + wr * kWaveR + kBlock j ..
// of this wave, summed over all of H. Rows past V or past N read as zeros. On return every
// stage copy has landed and the workgroup has passed a barrier, so the caller may reuse the
// LDS ring.
template <int TV, int TR, int WV, int WR, int BK, int NST, bool STREAM_W = (TR <= 128),
          class MF = Mfma32>
__device__ __forceinline__ void lmhead_tile(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W, int N, int H, int V,
    int v0, int r0, uint4* smem, int w_packed,
    typename MF::Acc (&acc)[LmheadCfg<TV, TR, WV, WR, BK, NST, MF>::MV]
                           [LmheadCfg<TV, TR, WV, WR, BK, NST, MF>::MR]) {
  using C = LmheadCfg<TV, TR, WV, WR, BK, NST, MF>;
  const TileIo<TV, TR, WV, WR, BK, NST, STREAM_W, MF> io(X, W, N, H, V, v0, r0, smem, w_packed);
  const int KT = H / BK;
  auto issue_stage = [&](int ks) {
    static_for<C::kLoads>([&](auto cc) { io.template copy<decltype(cc)::value>(ks % NST, ks); });
  };
  zero_acc(acc);

  bf16x8 a0[C::MV], b0[C::MR], a1[C::MV], b1[C::MR];
  // Fragments of MFMA K step `step` of the stage in ring slot `slot`.
  auto load_frags = [&](int slot, int step, bf16x8* a, bf16x8* b) {
#pragma unroll
    for (int i = 0; i < C::MV; ++i) a[i] = io.w_frag(slot, step, i);
#pragma unroll
    for (int j = 0; j < C::MR; ++j) b[j] = io.x_frag(slot, step, j);
  };
  auto mfmas = [&](const bf16x8* a, const bf16x8* b) {
#pragma unroll
    for (int i = 0; i < C::MV; ++i)
#pragma unroll
      for (int j = 0; j < C::MR; ++j) acc[i][j] = MF::mma(a[i], b[j], acc[i][j]);
  };

  // Prologue: fill the whole ring, then wait for stage 0.
  const int pro = min(NST, KT);
  for (int ks = 0; ks < pro; ++ks) issue_stage(ks);
  wait_stage_barrier<C::kLoads>(pro - 1);
  load_frags(0, 0, a0, b0);

  // Per stage k with MFMA K steps s = 0 .. NS - 1: read the fragments of step s + 1 while the
  // MFMAs of step s run. Before the last step's MFMAs (all reads of slot k done), wait for
  // stage k+1 and pass the barrier while the previous MFMAs drain, refill slot k with stage
  // k + NST, and read the first fragments of k+1 under the last step's MFMAs.
  constexpr int NS = C::NS;
  for (int k = 0; k < KT; ++k) {
    const int slot = k % NST;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      bf16x8* ca = (s & 1) ? a1 : a0;
      bf16x8* cb = (s & 1) ? b1 : b0;
      bf16x8* na = (s & 1) ? a0 : a1;
      bf16x8* nb = (s & 1) ? b0 : b1;
      if (s + 1 < NS) {
        load_frags(slot, s + 1, na, nb);
      } else if (k + 1 < KT) {
        // stage k+1 must have landed; the copies of the newer stages may stay in flight
        wait_stage_barrier<C::kLoads>(min(NST - 2, KT - 2 - k));
        if (k + NST < KT) issue_stage(k + NST);
        load_frags((k + 1) % NST, 0, na, nb);
      }
      mfmas(ca, cb);
    }
  }
  static_assert(NS % 2 == 0, "fragment double buffer alternates within a stage");
  // every copy was waited for by the last stage's predecessor
  __syncthreads();
}

// LDS reads complete, then the workgroup barrier.
__device__ __forceinline__ void wait_lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" : : : "memory");
}

// The same logits as lmhead_tile with a one-slot ring, for weight-streaming tiles that run
// three workgroups per CU: each wave reads a whole stage's fragments into registers, the
// workgroup frees the slot and refills it with the next stage while this stage's MFMAs run.
// A stage's copy latency is exposed per workgroup and hidden by the other workgroups of the
// CU. MFMAs accumulate in lmhead_tile's K order, so the logits are bit-identical.
template <int TV, int TR, int WV, int WR, int BK, bool STREAM_W, class MF>
__device__ __forceinline__ void lmhead_tile_1slot(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W, int N, int H, int V,
    int v0, int r0, uint4* smem, int w_packed,
    typename MF::Acc (&acc)[LmheadCfg<TV, TR, WV, WR, BK, 1, MF>::MV]
                           [LmheadCfg<TV, TR, WV, WR, BK, 1, MF>::MR]) {
  using C = LmheadCfg<TV, TR, WV, WR, BK, 1, MF>;
  const TileIo<TV, TR, WV, WR, BK, 1, STREAM_W, MF> io(X, W, N, H, V, v0, r0, smem, w_packed);
  const int KT = H / BK;
  auto issue_stage = [&](int ks) {
    static_for<C::kLoads>([&](auto cc) { io.template copy<decltype(cc)::value>(0, ks); });
  };
  zero_acc(acc);
  constexpr int NS = C::NS;
  bf16x8 fa[NS][C::MV], fb[NS][C::MR];
  issue_stage(0);
  for (int k = 0; k < KT; ++k) {
    wait_vm_barrier<0>();                 // stage k has landed in the slot
#pragma unroll
    for (int s = 0; s < NS; ++s) {
#pragma unroll
      for (int i = 0; i < C::MV; ++i) fa[s][i] = io.w_frag(0, s, i);
#pragma unroll
      for (int j = 0; j < C::MR; ++j) fb[s][j] = io.x_frag(0, s, j);
    }
    wait_lds_barrier();                   // every wave holds its fragments: the slot is free
    if (k + 1 < KT) issue_stage(k + 1);
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int i = 0; i < C::MV; ++i)
#pragma unroll
        for (int j = 0; j < C::MR; ++j) acc[i][j] = MF::mma(fa[s][i], fb[s][j], acc[i][j]);
  }
  __syncthreads();
}

// The same logits as lmhead_tile for 64-deep stages in a two-slot ring, with a fixed
// instruction schedule that spreads each stage's copies over the MFMAs. A stage has NS MFMA K
// steps (four K16 steps of 32x32x16, or two K32 steps of 16x16x32) of NF = MV + MR fragments
// and MV * MR MFMAs each (NM MFMAs in all); its first half is steps 0 .. NS/2 - 1, its second
// half the rest. Per stage k, in issue order (one MFMA per position m, the other work
// attached after it):
//   m < NS/2 NF     read the second half's fragments of slot k, one per MFMA;
//   m = Q1 - 1      LDS reads done + barrier: no wave reads slot k any more;
//   Q1 <= m < NM    the copies of stage k + 2 into slot k, evenly spaced;
//   m = Q2 - 1      wait until stage k + 1 has landed (only copies of stage k + 2 may be
//                   outstanding) + barrier;
//   m >= Q2         read the first half's fragments of stage k + 1, one per MFMA.
// Each wave's vector-memory queue thus never holds a whole stage of copies (issued in one
// burst, they block the wave's in-order instruction stream, and with it its MFMAs, until the
// CU's address unit has taken them); the stage copy has about 1.5 stages to land. MFMAs
// accumulate in the same K order as lmhead_tile, so the logits are bit-identical. The
// schedule is branch-free: past the last stage the copies repeat the last stage into the slot
// just freed (never read again) and the reads of the stage after the last are discarded.
template <int TV, int TR, int WV, int WR, bool STREAM_W, class MF = Mfma32>
__device__ __forceinline__ void lmhead_tile_spread(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W, int N, int H, int V,
    int v0, int r0, uint4* smem, int w_packed,
    typename MF::Acc (&acc)[LmheadCfg<TV, TR, WV, WR, 64, 2, MF>::MV]
                           [LmheadCfg<TV, TR, WV, WR, 64, 2, MF>::MR]) {
  constexpr int BK = 64, NST = 2;
  using C = LmheadCfg<TV, TR, WV, WR, BK, NST, MF>;
  constexpr int MV = C::MV, MR = C::MR, NS = C::NS, HS = NS / 2;
  constexpr int NF = MV + MR;                 // fragments per K step
  constexpr int NM = NS * MV * MR;            // MFMAs per stage
  constexpr int kCopies = C::kLoads;          // copies per wave per stage
  constexpr int RS = MF::kK / 16;             // MFMAs per fragment read (one per 32 cycles)
  constexpr int NR = RS * HS * NF;            // MFMA positions the reads of a half span
  constexpr int Q1 = NR + 2;                  // slot-free barrier after MFMA Q1 - 1
  constexpr int Q2 = NM - NR - 4;             // next-stage barrier after MFMA Q2 - 1
  static_assert(NS % 2 == 0, "two halves of K steps");
  static_assert(NR <= HS * MV * MR, "the second half is read within the first half");
  static_assert(Q1 < Q2 && Q2 + NR <= NM, "schedule points inside the stage");
  static_assert(Q2 >= HS * MV * MR, "the first half of the next stage overwrites registers "
                "this stage's first half has finished with");
  // position of copy c, and how many copies precede the next-stage barrier
  constexpr auto copy_pos = [](int c) { return Q1 + c * (NM - Q1) / kCopies; };
  constexpr int kBeforeQ2 = [&] {
    int n = 0;
    for (int c = 0; c < kCopies; ++c) n += copy_pos(c) <= Q2 - 1 ? 1 : 0;
    return n;
  }();

  const TileIo<TV, TR, WV, WR, BK, NST, STREAM_W, MF> io(X, W, N, H, V, v0, r0, smem,
                                                        w_packed);
  const int KT = H / BK;
  auto issue_copy = [&](int slot, int ks, auto cc) {
    io.template copy<decltype(cc)::value>(slot, ks);
  };
  zero_acc(acc);

  bf16x8 fa[NS][MV], fb[NS][MR];
  // fragment f of MFMA K step s of ring slot `slot`. The 32x32x16 loop reads W before X;
  // the 16x16x32 loop reads in the order the step's MFMAs first use them (W 0, every X, then
  // the other W), since its reads come closer to their use.
  auto read_frag = [&](int slot, int s, int f) {
    if constexpr (RS == 1) {
      if (f < MV) fa[s][f] = io.w_frag(slot, s, f);
      else fb[s][f - MV] = io.x_frag(slot, s, f - MV);
    } else {
      if (f == 0) fa[s][0] = io.w_frag(slot, s, 0);
      else if (f <= MR) fb[s][f - 1] = io.x_frag(slot, s, f - 1);
      else fa[s][f - MR] = io.w_frag(slot, s, f - MR);
    }
  };

  // Prologue: stages 0 and 1, wait for stage 0, read its first half.
  static_for<kCopies>([&](auto cc) { issue_copy(0, 0, cc); });
  if (KT > 1) {
    static_for<kCopies>([&](auto cc) { issue_copy(1, 1, cc); });
    wait_vm_barrier<kCopies>();
  } else {
    wait_vm_barrier<0>();
  }
#pragma unroll
  for (int s = 0; s < HS; ++s)
#pragma unroll
    for (int f = 0; f < NF; ++f) read_frag(0, s, f);

  for (int k = 0; k < KT; ++k) {
    const int slot = k & 1;
    const int ks_copy = min(k + 2, KT - 1);
    static_for<NM>([&](auto mc) {
      constexpr int m = decltype(mc)::value;
      constexpr int s = m / (MV * MR), q = m % (MV * MR), i = q / MR, j = q % MR;
      if constexpr (s == NS - 1)
        acc[i][j] = MF::mma(fa[s][i], fb[s][j], acc[i][j]);
      else
        acc[i][j] = MF::mma_chained(fa[s][i], fb[s][j], acc[i][j]);
      if constexpr (m < NR && m % RS == 0) read_frag(slot, HS + m / RS / NF, m / RS % NF);
      if constexpr (m == Q1 - 1) wait_lds_barrier();
      static_for<kCopies>([&](auto cc) {
        if constexpr (copy_pos(decltype(cc)::value) == m) issue_copy(slot, ks_copy, cc);
      });
      if constexpr (m == Q2 - 1) wait_vm_barrier<kBeforeQ2>();
      if constexpr (m >= Q2 && m < Q2 + NR && (m - Q2) % RS == 0)
        read_frag(slot ^ 1, (m - Q2) / RS / NF, (m - Q2) / RS % NF);
      __builtin_amdgcn_sched_barrier(0);
    });
  }
  // every copy lands before the caller reuses the ring and before the workgroup can exit
  asm volatile("s_waitcnt vmcnt(0)" : : : "memory");
  __syncthreads();
}

// The spread K loop for a three-slot ring: one barrier per stage. Stage j's copies go to slot
// j % 3 and are spread evenly over the window from the barrier of stage j - 3 (after which no
// wave reads that slot) to the barrier of stage j - 2 (which waits for stage j - 1); each copy
// thus has at least one stage to land. Per stage k (halves of K steps as in
// lmhead_tile_spread), one MFMA per position m:
//   m < NS/2 NF     read the second half's fragments of slot k, one per MFMA;
//   m < Q2          the remaining copies of stage k + 2;
//   m = Q2 - 1      wait until stage k + 1 has landed (only copies of stage k + 2 may be
//                   outstanding) + barrier;
//   m >= Q2         read the first half's fragments of stage k + 1; the first copies of
//                   stage k + 3.
// Past the last stage the copies repeat the last stage into slots no later stage reads.
template <int TV, int TR, int WV, int WR, bool STREAM_W, class MF = Mfma32>
__device__ __forceinline__ void lmhead_tile_spread3(
    const uint16_t* __restrict__ X, const uint16_t* __restrict__ W, int N, int H, int V,
    int v0, int r0, uint4* smem, int w_packed,
    typename MF::Acc (&acc)[LmheadCfg<TV, TR, WV, WR, 64, 3, MF>::MV]
                           [LmheadCfg<TV, TR, WV, WR, 64, 3, MF>::MR]) {
  constexpr int BK = 64, NST = 3;
  using C = LmheadCfg<TV, TR, WV, WR, BK, NST, MF>;
  constexpr int MV = C::MV, MR = C::MR, NS = C::NS, HS = NS / 2;
  constexpr int NF = MV + MR;                 // fragments per K step
  constexpr int NM = NS * MV * MR;            // MFMAs per stage
  constexpr int G = C::kLoads;                // copies per wave per stage
  constexpr int Q2 = NM - HS * NF;            // the barrier after MFMA Q2 - 1
  static_assert(NS % 2 == 0, "two halves of K steps");
  static_assert(Q2 >= HS * NF + 2, "the second half's reads land before the barrier");
  static_assert(Q2 >= HS * MV * MR, "the first half of the next stage overwrites registers "
                "this stage's first half has finished with");
  static_assert(2 * G <= 63, "vmcnt range");
  // copy c of a group sits c * NM / G MFMAs after the barrier that opens its window; the
  // first n1 of them fall in the same stage as that barrier
  constexpr auto rel = [](int c) { return c * NM / G; };
  constexpr int n1 = [&] {
    int n = 0;
    for (int c = 0; c < G; ++c) n += Q2 + rel(c) < NM ? 1 : 0;
    return n;
  }();

  const TileIo<TV, TR, WV, WR, BK, NST, STREAM_W, MF> io(X, W, N, H, V, v0, r0, smem,
                                                        w_packed);
  const int KT = H / BK;
  // copy c of stage j into slot j % 3, from K stage min(j, KT - 1)
  auto issue_copy = [&](int j, auto cc) {
    io.template copy<decltype(cc)::value>(j % NST, min(j, KT - 1));
  };
  zero_acc(acc);

  bf16x8 fa[NS][MV], fb[NS][MR];
  auto read_frag = [&](int slot, int s, int f) {
    if (f < MV) fa[s][f] = io.w_frag(slot, s, f);
    else fb[s][f - MV] = io.x_frag(slot, s, f - MV);
  };

  // Prologue: stages 0 and 1 and the first n1 copies of stage 2 (what the window of a stage
  // -1 would have issued); wait for stage 0; read its first half.
  static_for<G>([&](auto cc) { issue_copy(0, cc); });
  static_for<G>([&](auto cc) { issue_copy(1, cc); });
  static_for<G>([&](auto cc) {
    if constexpr (decltype(cc)::value < n1) issue_copy(2, cc);
  });
  wait_vm_barrier<G + n1>();
#pragma unroll
  for (int s = 0; s < HS; ++s)
#pragma unroll
    for (int f = 0; f < NF; ++f) read_frag(0, s, f);

  int slot = 0;
  for (int k = 0; k < KT; ++k) {
    const int nslot = slot == NST - 1 ? 0 : slot + 1;
    static_for<NM>([&](auto mc) {
      constexpr int m = decltype(mc)::value;
      constexpr int s = m / (MV * MR), q = m % (MV * MR), i = q / MR, j = q % MR;
      acc[i][j] = MF::mma(fa[s][i], fb[s][j], acc[i][j]);
      if constexpr (m < HS * NF) read_frag(slot, HS + m / NF, m % NF);
      static_for<G>([&](auto cc) {
        constexpr int c = decltype(cc)::value;
        if constexpr (c >= n1 && Q2 + rel(c) - NM == m) issue_copy(k + 2, cc);
        if constexpr (c < n1 && Q2 + rel(c) == m) issue_copy(k + 3, cc);
      });
      if constexpr (m == Q2 - 1) wait_vm_barrier<G>();
      if constexpr (m >= Q2 && m < Q2 + HS * NF)
        read_frag(nslot, (m - Q2) / NF, (m - Q2) % NF);
      __builtin_amdgcn_sched_barrier(0);
    });
    slot = nslot;
  }
  // every copy lands before the caller reuses the ring and before the workgroup can exit
  asm volatile("s_waitcnt vmcnt(0)" : : : "memory");
  __syncthreads();
}

// LOOP selects the K loop: 0 = the burst ring of lmhead_tile; 1 = the one-slot ring of
// lmhead_tile_1slot (three workgroups per CU); 2 and 3 = the spread loop of that ring depth
// (lmhead_tile_spread, lmhead_tile_spread3). STREAM_W: the W copies' cache
// policy (see TileIo); it changes no result. MF is the MFMA shape; every tile
// family of K1 runs the same one, so that all of them sum each logit's products in the same
// order and give the same logits bit for bit. One launch covers a contiguous range of
// vocabulary slabs (all of them, or one of two ranges whose tiles differ in height).
template <int TV, int TR, int WV, int WR, int BK, int NST, int LOOP, bool STREAM_W,
          class MF = Mfma16>
__global__ __launch_bounds__(WV * WR * kWave, LOOP == 1 ? 3 : 1)
void k_lmhead_partial(const uint16_t* __restrict__ X, const uint16_t* __restrict__ W,
                      const int32_t* __restrict__ parent, const int32_t* __restrict__ draft_tok,
                      const int32_t* __restrict__ req_offsets, int B, int N, int H, int V,
                      int S, int slab0, int RT, float* __restrict__ rec_m,
                      float* __restrict__ rec_s, int32_t* __restrict__ rec_a,
                      float* __restrict__ drafted_logit, int32_t* __restrict__ done_cnt,
                      int n_cnt, int w_packed, int blk_slabs, int blk_rows) {
  using C = LmheadCfg<TV, TR, WV, WR, BK, NST, MF>;
  constexpr int T = C::kThreads;
  constexpr int kBlock = MF::kBlock, kRegs = MF::kRegs;
  __shared__ uint4 smem[C::kLds / 16];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wv = wave % WV, wr = wave / WV;
  // clear the per-request completion counters of the finishing kernel that follows
  for (int i = blockIdx.x * T + tid; i < n_cnt; i += gridDim.x * T) done_cnt[i] = 0;
  // consecutive tiles share W slabs and X row tiles through one XCD's L2; this launch covers
  // slabs slab0 .. slab0 + gridDim.x / RT - 1 of the S slabs
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  int slab, rt;
  tile_coords(tile, gridDim.x / RT, RT, blk_slabs, blk_rows, slab, rt);
  slab += slab0;
  const int v0 = slab * TV, r0 = rt * TR;
  const int v_end = min(v0 + TV, V);
  const int r_last = min(r0 + TR, N) - 1;

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

  // ---- the tile's logits
  typename MF::Acc acc[C::MV][C::MR];
  if constexpr (LOOP == 1) {
    static_assert(NST == 1, "one-slot ring");
    lmhead_tile_1slot<TV, TR, WV, WR, BK, STREAM_W, MF>(X, W, N, H, V, v0, r0, smem, w_packed,
                                                        acc);
  } else if constexpr (LOOP == 2) {
    static_assert(BK == 64 && NST == 2, "two-slot spread loop: 64-deep stages");
    lmhead_tile_spread<TV, TR, WV, WR, STREAM_W, MF>(X, W, N, H, V, v0, r0, smem, w_packed,
                                                     acc);
  } else if constexpr (LOOP == 3) {
    static_assert(BK == 64 && NST == 3, "three-slot spread loop: 64-deep stages");
    lmhead_tile_spread3<TV, TR, WV, WR, STREAM_W, MF>(X, W, N, H, V, v0, r0, smem, w_packed,
                                                      acc);
  } else {
    static_assert(LOOP == 0, "K loop");
    lmhead_tile<TV, TR, WV, WR, BK, NST, STREAM_W, MF>(X, W, N, H, V, v0, r0, smem,
                                                       w_packed, acc);
  }

  // Output block (i, j), register e of a lane holds vocab row kBlock i + MF::row_of(lane, e)
  // (of the wave's vocab range) and tree row kBlock j + lane % kBlock (of the wave's rows).

  // Epilogue scratch reuses the ring: the gather list (kCap entries of 16 bytes), one
  // 64 x 16-float extraction area per wave, the row-reduction exchange and two counters.
  constexpr int kCap = 1024;
  constexpr int kScrOff = kCap * 16;
  constexpr int kRedOff = kScrOff + C::kWaves * kWave * 16 * 4;
  constexpr int kCntOff = kRedOff + 3 * WV * TR * 4;
  static_assert(kCntOff + 8 <= C::kLds, "epilogue scratch exceeds the LDS ring");
  char* const lds_bytes = reinterpret_cast<char*>(smem);
  int4* const s_list = reinterpret_cast<int4*>(lds_bytes);
  float* const wscr = reinterpret_cast<float*>(lds_bytes + kScrOff) + wave * (kWave * 16);
  float* const red_m = reinterpret_cast<float*>(lds_bytes + kRedOff);
  float* const red_s = red_m + WV * TR;
  int* const red_a = reinterpret_cast<int*>(red_s + WV * TR);
  int* const s_seg_end = reinterpret_cast<int*>(lds_bytes + kCntOff);
  int* const s_cnt = s_seg_end + 1;

  // ---- drafted logits: nodes whose parent row and drafted token fall inside this tile.
  // Matches are collected in LDS and extracted by the lane that owns the accumulator.
  // Candidates beyond the prefetched ones are read in rounds of kCap.
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
      // Keep the accumulator reads below inside this (rarely taken) loop body: without this
      // the compiler hoists all of them out of the loop into VGPRs and spills.
#pragma unroll
      for (int i = 0; i < C::MV; ++i)
#pragma unroll
        for (int j = 0; j < C::MR; ++j) asm volatile("" : "+a"(acc[i][j]));
      const int jj = pr / kBlock, ii = dv / kBlock, mm = dv % kBlock;
      const int ee = MF::reg_of(mm);
      const int owner = MF::lane_of(pr % kBlock, mm);
      // The block index is wave-uniform: branch to it, park its registers in this wave's
      // LDS scratch and let the owner lane read its element back (LDS operations of one wave
      // complete in order).
#pragma unroll
      for (int i = 0; i < C::MV; ++i)
#pragma unroll
        for (int j = 0; j < C::MR; ++j)
          if (i == ii && j == jj) {
#pragma unroll
            for (int e2 = 0; e2 < kRegs; ++e2) wscr[e2 * kWave + lane] = acc[i][j][e2];
          }
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      if (lane == owner) drafted_logit[m.x] = wscr[ee * kWave + owner];
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    }
    __syncthreads();
  }

  // ---- per-row slab record: lane-local pass, then the lane groups that hold the same tree
  // rows (64 / kBlock of them), then the waves that share the same tree rows (through LDS).
  // Within a lane the entries of a tree row are visited in increasing vocabulary order, so
  // "strictly greater" keeps the lowest argmax; the argmax is tracked as the entry ordinal
  // k = kRegs i + e and turned into a vocabulary id afterwards, and merges keep the lowest id
  // among equal maxima. Only the last slab needs the v < V mask. One row block at a time keeps
  // the accumulator reads short-lived (sched_barrier stops the scheduler from hoisting them).
  const bool full_slab = v0 + TV <= V;
  const int vwave = v0 + wv * C::kWaveV;
  auto entry_v = [&](int k) {
    return vwave + kBlock * (k / kRegs) + MF::row_of(lane, k % kRegs);
  };
  // Branch-free lane-local record of row block j; MASK drops entries past V (last slab).
  auto row_record = [&](int j, auto mask_tag) -> Rec {
    constexpr bool MASK = decltype(mask_tag)::value;
    float m = kNegInf;
    int kbest = 0;
#pragma unroll
    for (int i = 0; i < C::MV; ++i)
#pragma unroll
      for (int e = 0; e < kRegs; ++e) {
        const int k = kRegs * i + e;
        float z = acc[i][j][e];
        if constexpr (MASK) z = entry_v(k) < V ? z : kNegInf;
        kbest = z > m ? k : kbest;
        m = fmaxf(m, z);
      }
    const float mb = m * kLog2e;
    float sum = 0.f;
#pragma unroll
    for (int i = 0; i < C::MV; ++i)
#pragma unroll
      for (int e = 0; e < kRegs; ++e) {
        const float t = exp2_rel(fmaf(acc[i][j][e], kLog2e, -mb));
        if constexpr (MASK) sum += entry_v(kRegs * i + e) < V ? t : 0.f;
        else sum += t;
      }
    return Rec{m, m == kNegInf ? 0.f : sum, m == kNegInf ? kNoIndex : entry_v(kbest)};
  };
#pragma unroll
  for (int j = 0; j < C::MR; ++j) {
    Rec r = full_slab ? row_record(j, std::false_type{}) : row_record(j, std::true_type{});
#pragma unroll
    for (int mask = kBlock; mask < kWave; mask <<= 1) r = rec_merge(r, rec_shfl_xor(r, mask));
    if (lane < kBlock) {
      const int row = wr * C::kWaveR + kBlock * j + lane;
      red_m[wv * TR + row] = r.m;
      red_s[wv * TR + row] = r.s;
      red_a[wv * TR + row] = r.a;
    }
    __builtin_amdgcn_sched_barrier(0);
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

// ---- packed weights
// packed[((k T + s) PR + r) 64 + c] = W[PR s + r][64 k + c], zero where PR s + r >= V, with T
// tiles of PR rows per 64-column block (T PR = V rounded up to max(PR, 128) rows). Workgroup b
// writes tile b = k T + s, PR x 128 bytes: thread t stores the 16-byte units t + 256 i, i.e.
// row t / 8 + 32 i, columns 64 k + 8 (t % 8) .. + 7. Stores are contiguous; each group of 8
// lanes reads 128 contiguous bytes of one row.
constexpr int kPackDepth = 64, kPackThreads = 256;

template <int PR>
__global__ __launch_bounds__(kPackThreads)
void k_pack_tiles(const uint4* __restrict__ W, uint4* __restrict__ P, int V, int H, int T) {
  static_assert(PR % 32 == 0, "whole rows per pass");
  const int b = blockIdx.x, s = b % T, k = b / T, t = threadIdx.x;
  const int row_units = H / 8;                        // 16-byte units per row of W
  uint4* out = P + (size_t)b * (PR * kPackDepth / 8);
#pragma unroll
  for (int i = 0; i < PR / 32; ++i) {
    const int r = t / 8 + 32 * i;
    const int v = s * PR + r;
    uint4 val = make_uint4(0u, 0u, 0u, 0u);
    if (v < V) val = W[(size_t)v * row_units + k * (kPackDepth / 8) + (t & 7)];
    out[t + kPackThreads * i] = val;
  }
}

}  // namespace asv
