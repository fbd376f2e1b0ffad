/* Achievable-peak microbenchmarks for MI355X (gfx950), measurement only: they give the
 * measured ceilings that the verification kernels' roofline fractions are read against, next
 * to the published peaks. Not part of the verification path; libasv_microbench.so is a
 * separate library. Each call enqueues one kernel on `stream` (a hipStream_t) and returns 0,
 * or -1 for invalid arguments, -3 if the launch fails.
 */
#ifndef ASV_MICROBENCH_H_
#define ASV_MICROBENCH_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Streaming read of `bytes` bytes of device memory at `buf` (16-byte aligned, bytes a multiple
 * of 16): `grid` workgroups of 256 threads, each reading one contiguous chunk with 16-byte
 * loads, eight in flight per lane, folded into one word written to sink[workgroup] only when
 * it equals a constant that random data never produce (so the loads cannot be removed).
 * sink: [grid] device words. Bytes moved: `bytes`. */
int asvb_stream_read(const void *buf, uint64_t bytes, uint32_t *sink, int32_t grid,
                     void *stream);

/* The same read with the non-temporal hint on every load, interleaved across workgroups
 * (round k of workgroup g reads 16-byte words (k grid + g) 1024 .. + 1023): the fastest plain
 * read of HBM measured on this GPU. Unlike asvb_stream_read it does not fill the caches, so it
 * is no cache flush. Same arguments and checks. */
int asvb_stream_read_nt(const void *buf, uint64_t bytes, uint32_t *sink, int32_t grid,
                        void *stream);

/* Dense bf16 MFMA loop: `grid` workgroups of 256 threads; each wave runs `iters` rounds of
 * eight independent v_mfma_f32_32x32x16_bf16 on register operands (no memory traffic) and
 * writes one float per lane to sink[(workgroup * 256) + thread] at the end.
 * sink: [grid * 256] device floats. FLOPs: grid * 4 * iters * 8 * 32768. */
int asvb_mfma_loop(float *sink, int32_t iters, int32_t grid, void *stream);

/* LDS read-pattern probe: `grid` workgroups of 256 threads fill a 16 KB LDS buffer of 1024
 * 16-byte units, then every wave reads unit unit_of_lane[lane] % 1024 (unit_of_lane: 64 device
 * ints) with ds_read_b128, `iters` times, and each thread writes one word to
 * sink[(workgroup * 256) + thread]. The dispatch's hardware counters (SQ_INSTS_LDS,
 * SQ_LDS_BANK_CONFLICT) then give the bank-conflict cycles of that lane pattern.
 * sink: [grid * 256] device words. */
int asvb_lds_read(const int32_t *unit_of_lane, int32_t iters, uint32_t *sink, int32_t grid,
                  void *stream);

#ifdef __cplusplus
}
#endif

#endif /* ASV_MICROBENCH_H_ */
