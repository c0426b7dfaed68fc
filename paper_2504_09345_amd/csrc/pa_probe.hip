// HBM read-stream probe: the decode kernels' load pattern with no arithmetic
// (declared in pa_probe.h).  Each wave reads 4 KiB slices with four 16-byte
// raw buffer loads per lane (one 1 KiB row of 64 lanes per load, fully
// coalesced), keeping the next slice's loads in flight while it folds the
// current one, exactly as the attention kernels' two-tile ring does.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pa_probe.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = 8;
constexpr int kSlice = 4096;

template <int POLICY>
__device__ __forceinline__ void load_slice(const uint8_t* p, int lane, u32x4 (&r)[4]) {
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(p), (short)0, kSlice, 0x00020000);
#pragma unroll
  for (int i = 0; i < 4; ++i) r[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, lane * 16, i * 1024, POLICY);
}

template <int POLICY>
__global__ __launch_bounds__(64 * kWaves) void read_probe_kernel(const uint8_t* buf, const int64_t* offs,
                                                                 int64_t slices_per_chunk, int64_t n_slices,
                                                                 uint32_t* sink) {
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t G = gridDim.x, x = blockIdx.x;
  const int64_t s0 = n_slices * x / G, s1 = n_slices * (x + 1) / G;
  auto addr = [&](int64_t j) -> const uint8_t* {
    const int64_t c = j / slices_per_chunk, sub = j - c * slices_per_chunk;
    const int64_t base = offs != nullptr ? offs[c] : c * slices_per_chunk * kSlice;
    return buf + base + sub * kSlice;
  };
  uint32_t acc = 0;
  u32x4 a[4], b[4];
  int64_t j = s0 + w;
  if (j < s1) load_slice<POLICY>(addr(j), lane, a);
  for (; j < s1; j += 2 * kWaves) {
    const int64_t jn = j + kWaves;
    if (jn < s1) load_slice<POLICY>(addr(jn), lane, b);
#pragma unroll
    for (int i = 0; i < 4; ++i) acc ^= a[i].x ^ a[i].y ^ a[i].z ^ a[i].w;
    if (jn >= s1) break;
    const int64_t jm = jn + kWaves;
    if (jm < s1) load_slice<POLICY>(addr(jm), lane, a);
#pragma unroll
    for (int i = 0; i < 4; ++i) acc ^= b[i].x ^ b[i].y ^ b[i].z ^ b[i].w;
  }
  sink[x * 64 * kWaves + threadIdx.x] = acc;
}

}  // namespace

extern "C" int pa_read_probe(const void* buf, int64_t chunk_bytes, const int64_t* chunk_offsets,
                             int64_t n_chunks, int32_t grid, int32_t non_temporal, uint32_t* sink,
                             hipStream_t stream) {
  if (buf == nullptr || sink == nullptr || chunk_bytes <= 0 || chunk_bytes % kSlice != 0 || n_chunks < 0 ||
      grid < 1 || grid > 65535)
    return -1;
  const int64_t spc = chunk_bytes / kSlice;
  const uint8_t* p = static_cast<const uint8_t*>(buf);
  if (non_temporal)
    read_probe_kernel<2><<<dim3(grid), dim3(64 * kWaves), 0, stream>>>(p, chunk_offsets, spc, spc * n_chunks, sink);
  else
    read_probe_kernel<0><<<dim3(grid), dim3(64 * kWaves), 0, stream>>>(p, chunk_offsets, spc, spc * n_chunks, sink);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}
