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
//    item continues past the range); the fixup kernel merges them in a fixed
//    order (deterministic, no atomics).
//
// Per workgroup: prefix sums of page counts over all rows (LDS), then a unit
// table for its range (page id and flags per unit, LDS), then each wave runs
// a ring of NBUF register tile buffers over the units, exactly as in the
// split kernel's inner loop, with a workgroup barrier per unit to keep the
// waves in step.
#include "pa_stream_body.h"

namespace pa {

template <typename T, int D, int S, int W, int NBUF, bool MF>
__global__ __launch_bounds__(64 * W) void stream_kernel(StreamArgs a) {
  __shared__ StreamSmem<W, MF> sm;
  stream_body<T, D, S, W, NBUF, MF>(a, sm, blockIdx.x, gridDim.x);
}

// Fixup: merge the partial records of every (row, KV head) item that a range
// boundary cut; write zeros for empty rows and NaN for contract violations.
// One wave per (row, KV head); records are merged in workgroup order.
template <typename T, int D, int S, int W>
__global__ __launch_bounds__(256) void stream_fixup_kernel(StreamArgs a, int G) {
  constexpr int E = S * D / 64;  // elements per lane
  const int lane = threadIdx.x & 63;
  const int64_t item = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (item >= (int64_t)a.B * a.H_kv) return;
  const int r = (int)(item / a.H_kv), g = (int)(item % a.H_kv);
  const int hb = g / W, w = g % W;
  int qrow, nv;
  const int status = seq_decode_row(a.query_start_loc, a.context_lens, a.max_context_len, r, qrow, nv);
  if (status == 0) return;
  T* out = reinterpret_cast<T*>(a.out) + ((int64_t)qrow * a.H_q + (int64_t)g * S) * D;
  const int np = status == 1 ? (nv + kPage - 1) / kPage : 0;
  if (status < 0 || np > (int)a.bt_stride || np == 0) {
    const float fill = (status < 0 || np > (int)a.bt_stride) ? NAN : 0.0f;
#pragma unroll
    for (int e = 0; e < E; ++e) store_out<T>(out + lane * E + e, fill);
    return;
  }
  const int64_t U = (int64_t)a.nb * a.ws_cum[a.B];
  const int64_t s = (int64_t)a.nb * a.ws_cum[r] + (int64_t)hb * np, e_last = s + np - 1;
  const int64_t wg_first = ((s + 1) * G - 1) / U, wg_last = ((e_last + 1) * G - 1) / U;
  if (wg_first == wg_last) return;  // finished in place by the attention kernel

  float M[S], L[S], acc[E];
#pragma unroll
  for (int j = 0; j < S; ++j) { M[j] = kMInit; L[j] = 0.0f; }
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.0f;
  // pass 1: maxima
  for (int64_t x = wg_first; x <= wg_last; ++x) {
    if (U * x / G == U * (x + 1) / G) continue;  // empty range wrote nothing
    const int64_t slot = (x * 2 + (x == wg_first ? 1 : 0)) * W + w;
#pragma unroll
    for (int j = 0; j < S; ++j) M[j] = fmaxf(M[j], a.ws_ml[slot * S * 2 + j * 2]);
  }
  // pass 2: weighted sums
  for (int64_t x = wg_first; x <= wg_last; ++x) {
    if (U * x / G == U * (x + 1) / G) continue;
    const int64_t slot = (x * 2 + (x == wg_first ? 1 : 0)) * W + w;
    float c[S];
#pragma unroll
    for (int j = 0; j < S; ++j) {
      c[j] = fast_exp2(a.ws_ml[slot * S * 2 + j * 2] - M[j]);
      L[j] = fmaf(a.ws_ml[slot * S * 2 + j * 2 + 1], c[j], L[j]);
    }
    const float* o = a.ws_o + slot * S * D;
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int idx = lane * E + e;
      acc[e] = fmaf(o[idx], c[idx / D], acc[e]);
    }
  }
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int idx = lane * E + e;
    store_out<T>(out + idx, acc[e] / L[idx / D]);
  }
}

// ---- launchers -----------------------------------------------------------

template <typename T, int D, int S, int W>
static const void* stream_fn() {
  constexpr bool mf = kStreamMfma && sizeof(T) == 2 && D == 128;
  return reinterpret_cast<const void*>(&stream_kernel<T, D, S, W, kStreamRing, mf>);
}

template <typename T, int D, int S>
static const void* pick_w(int W) {
  switch (W) {
    case 1: return stream_fn<T, D, S, 1>();
    case 2: return stream_fn<T, D, S, 2>();
    case 4: return stream_fn<T, D, S, 4>();
    case 8: return stream_fn<T, D, S, 8>();
  }
  return nullptr;
}

template <typename T, int D>
static const void* pick_s(int s, int W) {
  switch (s) {
    case 1: return pick_w<T, D, 1>(W);
    case 2: return pick_w<T, D, 2>(W);
    case 4: return pick_w<T, D, 4>(W);
    case 6: return pick_w<T, D, 6>(W);
    case 8: return pick_w<T, D, 8>(W);
  }
  return nullptr;
}

const void* stream_kernel_fn(int dtype, int D, int s, int W) {
  if (dtype == 0 && D == 128) return pick_s<uint16_t, 128>(s, W);
  if (dtype == 0 && D == 64) return pick_s<uint16_t, 64>(s, W);
  if (dtype == 1 && D == 128) return pick_s<float, 128>(s, W);
  if (dtype == 1 && D == 64) return pick_s<float, 64>(s, W);
  return nullptr;
}

template <typename T, int D, int S, int W>
static void launch_fixup(const StreamArgs& a, int G, hipStream_t st) {
  const int64_t items = (int64_t)a.B * a.H_kv;
  stream_fixup_kernel<T, D, S, W><<<dim3((unsigned)((items + 3) / 4)), dim3(256), 0, st>>>(a, G);
}

template <typename T, int D, int S>
static bool fixup_w(int W, const StreamArgs& a, int G, hipStream_t st) {
  switch (W) {
    case 1: launch_fixup<T, D, S, 1>(a, G, st); return true;
    case 2: launch_fixup<T, D, S, 2>(a, G, st); return true;
    case 4: launch_fixup<T, D, S, 4>(a, G, st); return true;
    case 8: launch_fixup<T, D, S, 8>(a, G, st); return true;
  }
  return false;
}

template <typename T, int D>
static bool fixup_s(int s, int W, const StreamArgs& a, int G, hipStream_t st) {
  switch (s) {
    case 1: return fixup_w<T, D, 1>(W, a, G, st);
    case 2: return fixup_w<T, D, 2>(W, a, G, st);
    case 4: return fixup_w<T, D, 4>(W, a, G, st);
    case 6: return fixup_w<T, D, 6>(W, a, G, st);
    case 8: return fixup_w<T, D, 8>(W, a, G, st);
  }
  return false;
}

hipError_t launch_stream(int dtype, int D, int s, int W, const StreamArgs& a, int G, hipStream_t st,
                         KernelEvents ev) {
  const void* fn = stream_kernel_fn(dtype, D, s, W);
  if (fn == nullptr || G <= 0) return hipErrorInvalidValue;
  void* args[] = {const_cast<StreamArgs*>(&a)};
  hipError_t e = hipExtLaunchKernel(fn, dim3(G), dim3(64 * W), args, 0, st, ev.start, ev.stop, 0);
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

hipError_t launch_stream_fixup(int dtype, int D, int s, int W, const StreamArgs& a, int G, hipStream_t st) {
  if (a.B == 0) return hipSuccess;
  bool ok = false;
  if (dtype == 0 && D == 128) ok = fixup_s<uint16_t, 128>(s, W, a, G, st);
  else if (dtype == 0 && D == 64) ok = fixup_s<uint16_t, 64>(s, W, a, G, st);
  else if (dtype == 1 && D == 128) ok = fixup_s<float, 128>(s, W, a, G, st);
  else if (dtype == 1 && D == 64) ok = fixup_s<float, 64>(s, W, a, G, st);
  if (!ok) return hipErrorInvalidValue;
  return hipGetLastError();
}

int stream_occupancy(int dtype, int D, int s, int W) {
  const void* fn = stream_kernel_fn(dtype, D, s, W);
  if (fn == nullptr) return 0;
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, 64 * W, 0) != hipSuccess) return 0;
  return n;
}

}  // namespace pa
