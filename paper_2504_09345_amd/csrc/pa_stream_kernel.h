// The stream-K decode kernel template and its picker by GQA group size s and
// waves per workgroup W (design in pa_stream.hip).  Each (element type, head
// dim, trace) combination is instantiated in one translation unit.
#pragma once

#include "pa_stream_body.h"

namespace pa {

template <typename T, int D, int S, int W, int NBUF, bool MF, bool TR>
__global__ __launch_bounds__(64 * W) void stream_kernel(StreamArgs a) {
  __shared__ StreamSmem<W, MF> sm;
  stream_body<T, D, S, W, NBUF, MF, TR>(a, sm, blockIdx.x, gridDim.x);
}

template <typename T, int D, int S, bool TR>
const void* stream_pick_w(int W) {
  constexpr bool mf = kStreamMfma && sizeof(T) == 2 && D == 128;
  switch (W) {
    case 1: return reinterpret_cast<const void*>(&stream_kernel<T, D, S, 1, kStreamRing, mf, TR>);
    case 2: return reinterpret_cast<const void*>(&stream_kernel<T, D, S, 2, kStreamRing, mf, TR>);
    case 4: return reinterpret_cast<const void*>(&stream_kernel<T, D, S, 4, kStreamRing, mf, TR>);
    case 8: return reinterpret_cast<const void*>(&stream_kernel<T, D, S, 8, kStreamRing, mf, TR>);
  }
  return nullptr;
}

template <typename T, int D, bool TR>
const void* stream_pick(int s, int W) {
  switch (s) {
    case 1: return stream_pick_w<T, D, 1, TR>(W);
    case 2: return stream_pick_w<T, D, 2, TR>(W);
    case 4: return stream_pick_w<T, D, 4, TR>(W);
    case 6: return stream_pick_w<T, D, 6, TR>(W);
    case 8: return stream_pick_w<T, D, 8, TR>(W);
  }
  return nullptr;
}

}  // namespace pa
