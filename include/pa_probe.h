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

/* Read n_chunks chunks of chunk_bytes (a multiple of 4096) from buf.
 *   buf            device buffer, read
 *   chunk_offsets  device int64 [n_chunks]: byte offset of each chunk in buf
 *                  (each chunk must lie inside the caller's buffer; the
 *                  probe does not check), or NULL for consecutive chunks
 *                  starting at offset 0
 *   grid           persistent workgroups (1 .. 65535); the chunks' 4 KiB
 *                  slices are split into grid equal contiguous ranges, and
 *                  the 8 waves of a workgroup take consecutive slices, so
 *                  one 32 KiB chunk is read by one workgroup at a time
 *   non_temporal   1: loads with the non-temporal cache policy (as the
 *                  decode kernels load K/V), 0: default policy
 *   sink           device uint32 [grid * 512], written (a fold of the bytes
 *                  read, so the loads cannot be elided)
 * Enqueued on `stream`; returns without synchronising.
 * Errors: PA_EINVAL (-1) for a null buffer or sink, chunk_bytes not a
 * positive multiple of 4096, n_chunks < 0 or grid out of range; PA_EHIP (-4)
 * for a launch error. */
int pa_read_probe(const void *buf, int64_t chunk_bytes, const int64_t *chunk_offsets, int64_t n_chunks,
                  int32_t grid, int32_t non_temporal, uint32_t *sink, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* PA_PROBE_H */
