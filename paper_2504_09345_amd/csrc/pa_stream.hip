// Persistent stream-K paged GQA attention for gfx950 (decode rows).
//
// Same arithmetic as the split-K kernel (QK dot products, online softmax,
// PV scaled vector adds over bf16 KV in fp32: MoE-Lens Sec. 5.3 Eq. 6 and
// Sec. 6.6; paged KV through a block table: Sec. 5.5; GQA groups: Sec. 2), with
// a different division of work built for one GPU's HBM:
//
//  * Work units are (row, head block, page): a head block is W consecutive KV
//    heads, handled by the W waves of one workgroup in lockstep, so a
//    workgroup reading one page reads W adjacent 4 KiB head tiles (32 KiB
//    contiguous at W = 8) for K and for V.
//  * A persistent grid of G workgroups splits the U units of the whole batch
//    into G contiguous, equal ranges (stream-K): every workgroup streams the
//    same number of bytes whatever the mix of context lengths, with no empty
//    or short workgroups and one setup per workgroup instead of one per split.
//  * A (row, head) item that lies inside one range is finished in place.  An
//    item cut by a range boundary leaves partial (o, m, l) records, at most
//    two per workgroup ("head": the range starts inside the item, "tail": the
//    item continues past the range).  Each part counts its arrival at the
//    item's counter once its record is stored; the last part to arrive merges
//    every record in range order (deterministic, no float atomics, and no
//    workgroup ever waits for another): one launch per call.  A range whose
//    last item has one other part that has already counted merges it from
//    registers with that part's record, in the same order and arithmetic.
//
// Per workgroup: prefix sums of page counts over all rows (LDS), then a unit
// table for its range (page id and flags per unit, LDS), then the units in
// order, with a workgroup barrier per unit to keep the waves in step.  With
// the matrix-core fold (bf16, head dim 128) each wave loads a unit's K and V
// tiles half a unit apart, one register set each; otherwise it runs a ring
// of NBUF whole-tile register buffers, as the split kernel's inner loop does.
#include "pa_stream_kernel.h"

namespace pa {

// Kernels of the other (element type, head dim) combinations and the trace
// instantiations are compiled in their own translation units.
extern template const void* stream_pick<uint16_t, 64, false>(int, int);
extern template const void* stream_pick<float, 128, false>(int, int);
extern template const void* stream_pick<float, 64, false>(int, int);
extern template const void* stream_pick<uint16_t, 128, true>(int, int);
extern template const void* stream_pick<uint16_t, 64, true>(int, int);
extern template const void* stream_pick<float, 128, true>(int, int);
extern template const void* stream_pick<float, 64, true>(int, int);
template const void* stream_pick<uint16_t, 128, false>(int, int);

static const void* stream_kernel_fn(int dtype, int D, int s, int W, bool trace) {
  if (dtype == 0 && D == 128) return trace ? stream_pick<uint16_t, 128, true>(s, W) : stream_pick<uint16_t, 128, false>(s, W);
  if (dtype == 0 && D == 64) return trace ? stream_pick<uint16_t, 64, true>(s, W) : stream_pick<uint16_t, 64, false>(s, W);
  if (dtype == 1 && D == 128) return trace ? stream_pick<float, 128, true>(s, W) : stream_pick<float, 128, false>(s, W);
  if (dtype == 1 && D == 64) return trace ? stream_pick<float, 64, true>(s, W) : stream_pick<float, 64, false>(s, W);
  return nullptr;
}

hipError_t launch_stream(int dtype, int D, int s, int W, const StreamArgs& a, int G, hipStream_t st,
                         KernelEvents ev) {
  const void* fn = stream_kernel_fn(dtype, D, s, W, a.trace != nullptr);
  if (fn == nullptr || G <= 0) return hipErrorInvalidValue;
  void* args[] = {const_cast<StreamArgs*>(&a)};
  hipError_t e = hipExtLaunchKernel(fn, dim3(G), dim3(64 * W), args, 0, st, ev.start, ev.stop, 0);
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

int stream_occupancy(int dtype, int D, int s, int W) {
  const void* fn = stream_kernel_fn(dtype, D, s, W, false);
  if (fn == nullptr) return 0;
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, 64 * W, 0) != hipSuccess) return 0;
  return n;
}

}  // namespace pa
