// Gather-trace instantiations of the stream-K decode kernel: the same kernel,
// which also records the pool row of every token it loads (the block-table
// gather checked bit for bit against the oracle), plus the fill kernel that
// sets the trace's starting state.
#include "pa_stream_kernel.h"

namespace pa {

template const void* stream_pick<uint16_t, 128, true>(int, int);

__global__ __launch_bounds__(256) void fill_i64_kernel(int64_t* p, int64_t n, int64_t value) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) p[i] = value;
}

hipError_t launch_fill_i64(int64_t* p, int64_t n, int64_t value, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = (n + 255) / 256;
  fill_i64_kernel<<<dim3((unsigned)(blocks < 4096 ? blocks : 4096)), dim3(256), 0, st>>>(p, n, value);
  return hipGetLastError();
}

}  // namespace pa
