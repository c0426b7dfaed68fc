// Gather-trace instantiations of the stream-K decode kernel for bf16 with
// head_dim 64 and for fp32 (see pa_trace.hip).
#include "pa_stream_kernel.h"

namespace pa {

template const void* stream_pick<uint16_t, 64, true>(int, int);
template const void* stream_pick<float, 128, true>(int, int);
template const void* stream_pick<float, 64, true>(int, int);

}  // namespace pa
