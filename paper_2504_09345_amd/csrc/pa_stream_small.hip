// Stream-K decode kernels for bf16 with head_dim 64 and for fp32 (the
// matrix-core variant covers bf16 with head_dim 128 in pa_stream.hip).
#include "pa_stream_kernel.h"

namespace pa {

template const void* stream_pick<uint16_t, 64, false>(int, int);
template const void* stream_pick<float, 128, false>(int, int);
template const void* stream_pick<float, 64, false>(int, int);

}  // namespace pa
