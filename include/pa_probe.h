/*
 * pa_probe.h -- HBM read-stream probe of libpagedattn.so (measurement aid).
 *
 * Decode attention must read every cached K/V byte once per step (MoE-Lens
 * Sec. 5.3: each iteration reads the whole KV cache), so its ceiling is the
 * rate at which the GPU streams that access pattern from HBM.  This entry
 * point reads a buffer with the attention kernels' load pattern and nothing
 * else, so a benchmark can time what the pattern itself reaches: 4 KiB slices
 * read by waves of 64 lanes x 16 bytes x 4 loads, eight waves per workgroup,
 * two slices in flight per wave, a persistent grid splitting the slice list
 * into equal contiguous ranges.
 */
#ifndef PA_PROBE_H
#define PA_PROBE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Read n_chunks chunks of chunk_bytes (4096 times a power of two, at most
 * 4 GiB) from buf.
 *   buf            device buffer, read
 *   chunk_offsets  device int64 [n_chunks]: byte offset of each chunk in buf
 *                  (each chunk must lie inside the caller's buffer; the
 *                  probe does not check), or NULL for consecutive chunks
 *                  starting at offset 0
 *   grid           persistent workgroups (1 .. 65535); the chunks' 4 KiB
 *                  slices are split into grid equal contiguous ranges, and
 *                  the waves of a workgroup take consecutive slices, so one
 *                  32 KiB chunk is read by one workgroup at a time
 *   waves          waves per workgroup, 4 or 8
 *   depth          slices in flight per wave: 2 (the next slice's loads go
 *                  out before the current one is folded, as in the decode
 *                  kernels' two-tile ring) or 1 (each slice waited for
 *                  before the next is loaded)
 *   non_temporal   1: loads with the non-temporal cache policy (as the
 *                  decode kernels load K/V), 0: default policy
 *   sink           device uint32 [grid * 64 * waves], written (a fold of the
 *                  bytes read, so the loads cannot be elided)
 * Enqueued on `stream`; returns without synchronising.
 * Errors: PA_EINVAL (-1) for a null buffer or sink, chunk_bytes not 4096
 * times a power of two up to 2^20, n_chunks < 0, grid out of range, waves not 4
 * or 8 or depth not 1 or 2; PA_EHIP (-4)
 * for a launch error. */
int pa_read_probe(const void *buf, int64_t chunk_bytes, const int64_t *chunk_offsets, int64_t n_chunks,
                  int32_t grid, int32_t waves, int32_t depth, int32_t non_temporal, uint32_t *sink,
                  hipStream_t stream);

/* Issue-overlap probe: how much vector-ALU work runs while the matrix cores
 * work (the prefill kernel's step time depends on it).  One launch of `grid`
 * workgroups of `waves` waves; each wave runs `iters` iterations of four
 * independent bf16 matrix products (v_mfma_f32_32x32x16_bf16 when big_mfma,
 * else v_mfma_f32_16x16x32_bf16; four accumulator chains), each with
 * `valu_per_mfma` independent vector instructions (fp32 FMAs, or v_exp_f32
 * when exp2 is non-zero) that the compiler interleaves with them.
 *   mode 0  every wave runs both
 *   mode 1  products only         mode 2  vector work only
 *   mode 3  the first waves/2 waves run the products, the others (which
 *           share their SIMDs) the vector work
 * Each product is followed by its vector instructions in program order.
 *   sink    device float [grid * 64 * waves], every element written (keeps
 *           the work alive; its values are the lanes' sums of their
 *           accumulators and vector registers)
 *   cycles  device uint64 [grid * waves] or NULL: shader-clock cycles
 *           (s_memtime) of each wave's loop, element x * waves + w for wave
 *           w of workgroup x
 * Errors: -1 for a null sink, waves not in {1, 2, 4, 8}, iters < 1, grid
 * outside 1..65535, mode outside 0..3, mode 3 with one wave, or
 * valu_per_mfma not in {0, 1, 2, 3, 4, 6, 8, 16}; -4 for a launch error. */
int pa_issue_probe(int32_t grid, int32_t waves, int32_t iters, int32_t big_mfma, int32_t valu_per_mfma,
                   int32_t exp2, int32_t mode, float *sink, uint64_t *cycles, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* PA_PROBE_H */
