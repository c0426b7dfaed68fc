// Mixed batch in one launch: the decode rows' stream-K workgroups and the
// chunked-prefill workgroups share one grid, one workgroup per CU.
//
// Decode attention is HBM-bound and streams fastest on about three quarters
// of the CUs (fewer requests in flight keep HBM in its efficient range);
// prefill is matrix-core bound.  Giving the decode rows G_dec workgroups and
// the prefill chunks the remaining CUs runs the two side by side instead of
// one after the other.  Workgroups [0, G_dec) run the stream-K body over the
// decode units exactly as the stream kernel would with a grid of G_dec
// (including the merge of cut items); workgroups [G_dec, grid) run the
// prefill body with a grid of grid - G_dec.  No workgroup waits on another
// (a cut decode item is merged by whichever of its parts finishes last), so
// the split is correct whatever the residency and dispatch order.  The two
// bodies' LDS layouts share one union.
#include "pa_prefill_body.h"
#include "pa_stream_body.h"

namespace pa {

namespace {

constexpr int kMixedW = 8;  // decode waves per workgroup = prefill waves
static_assert(64 * kMixedW == kPfThreads, "decode and prefill workgroups must match");

union MixedSmem {
  StreamSmem<kMixedW, true> dec;
  struct {
    PrefillSmem smem;
    int32_t cum[kStreamMaxRows + 1];
  } pf;
};

template <int S, bool TR>
__global__ __launch_bounds__(64 * kMixedW) void mixed_kernel(StreamArgs sa, PrefillArgs pa_, int G_dec) {
  __shared__ MixedSmem sm;
  if ((int)blockIdx.x < G_dec)
    stream_body<uint16_t, mfma::kD, S, kMixedW, kStreamRing, true, TR, false>(sa, sm.dec, blockIdx.x, G_dec);
  else
    prefill_body<mfma::kD, S, TR>(pa_, sm.pf.smem, sm.pf.cum, blockIdx.x - G_dec, gridDim.x - G_dec);
}

template <bool TR>
const void* mixed_pick(int s) {
  switch (s) {
    case 1: return reinterpret_cast<const void*>(&mixed_kernel<1, TR>);
    case 2: return reinterpret_cast<const void*>(&mixed_kernel<2, TR>);
    case 4: return reinterpret_cast<const void*>(&mixed_kernel<4, TR>);
    case 6: return reinterpret_cast<const void*>(&mixed_kernel<6, TR>);
    case 8: return reinterpret_cast<const void*>(&mixed_kernel<8, TR>);
  }
  return nullptr;
}

// trace: the gather-trace instantiation (also records the rows it loads)
const void* mixed_fn(int s, bool trace = false) { return trace ? mixed_pick<true>(s) : mixed_pick<false>(s); }

}  // namespace

bool mixed_supported(int dtype, int D, int s, int W) {
  return kStreamMfma && dtype == 0 && D == mfma::kD && W == kMixedW && mixed_fn(s) != nullptr;
}

hipError_t launch_mixed(int s, const StreamArgs& sa, const PrefillArgs& pa_, int G_dec, int G, hipStream_t st,
                        KernelEvents ev) {
  const void* fn = mixed_fn(s, sa.trace != nullptr);
  if (fn == nullptr || G_dec <= 0 || G <= G_dec) return hipErrorInvalidValue;
  StreamArgs a0 = sa;
  PrefillArgs a1 = pa_;
  int g = G_dec;
  void* args[] = {&a0, &a1, &g};
  hipError_t e = hipExtLaunchKernel(fn, dim3(G), dim3(64 * kMixedW), args, 0, st, ev.start, ev.stop, 0);
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

}  // namespace pa
