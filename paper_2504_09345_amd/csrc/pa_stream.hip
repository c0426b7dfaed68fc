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
#include "pa_device.h"
#include "pa_kernels.h"
#include "pa_tile.h"

namespace pa {

// info word of a unit: valid tokens (5 bits) | item start | item end | head
// block (6 bits) | q/out row (19 bits)
__device__ __forceinline__ int info_valid(int i) { return i & 31; }
__device__ __forceinline__ bool info_start(int i) { return (i >> 5) & 1; }
__device__ __forceinline__ bool info_end(int i) { return (i >> 6) & 1; }
__device__ __forceinline__ int info_hb(int i) { return (i >> 7) & 63; }
__device__ __forceinline__ int info_row(int i) { return (int)((unsigned)i >> 13); }

template <typename T, int D, int S, int W, int NBUF, bool MF>
__global__ __launch_bounds__(64 * W) void stream_kernel(StreamArgs a) {
  using Sh = DecodeShape<T, D, S>;
  constexpr int NT = 64 * W;
  __shared__ int32_t s_cum[kStreamMaxRows + 1];
  __shared__ uint8_t s_tail[kStreamMaxRows];
  __shared__ int32_t s_page[kStreamMaxUnits];
  __shared__ int32_t s_info[kStreamMaxUnits];
  __shared__ int32_t s_scan[NT];

  const int tid = threadIdx.x;
  const int R = a.B;  // items are sequences

  // 1. pages per sequence and their prefix sums (every workgroup, redundantly)
  {
    const int per = (R + NT - 1) / NT;
    const int r0 = min(R, tid * per), r1 = min(R, r0 + per);
    int local = 0;
    for (int r = r0; r < r1; ++r) {
      int row, nv;
      int np = seq_decode_row(a.query_start_loc, a.context_lens, a.max_context_len, r, row, nv) == 1
                   ? (nv + kPage - 1) / kPage : 0;
      if (np > (int)a.bt_stride) np = 0;  // contract violation: the fixup writes NaN
      s_tail[r] = (uint8_t)(np ? nv - (np - 1) * kPage : 0);
      s_cum[r] = local;
      local += np;
    }
    const int off = block_exclusive_scan<NT>(local, s_scan);
    for (int r = r0; r < r1; ++r) s_cum[r] += off;
    if (tid == NT - 1) s_cum[R] = off + local;
    __syncthreads();
  }
  const int64_t U = (int64_t)a.nb * s_cum[R];
  if (blockIdx.x == 0)
    for (int r = tid; r <= R; r += NT) a.ws_cum[r] = s_cum[r];
  const int64_t G = gridDim.x;
  const int64_t u0 = U * blockIdx.x / G, u1 = U * (blockIdx.x + 1) / G;
  const int n_units = (int)(u1 - u0);
  if (n_units <= 0) return;

  // 2. unit table of this range
  const BlockTable bt{a.block_table, a.bt_stride};
  for (int i = tid; i < n_units; i += NT) {
    const int64_t u = u0 + i;
    int lo = 0, hi = R - 1;  // largest r with nb * cum[r] <= u (a non-empty sequence)
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if ((int64_t)a.nb * s_cum[mid] <= u) lo = mid; else hi = mid - 1;
    }
    const int r = lo;
    const int np = s_cum[r + 1] - s_cum[r];
    const int rem = (int)(u - (int64_t)a.nb * s_cum[r]);
    const int hb = rem / np, p = rem - hb * np;
    const int qrow = a.query_start_loc != nullptr ? a.query_start_loc[r] : r;
    s_page[i] = bt.page(r, p);
    const int valid = p == np - 1 ? (int)s_tail[r] : kPage;
    s_info[i] = valid | (p == 0) << 5 | (p == np - 1) << 6 | hb << 7 | qrow << 13;
  }
  __syncthreads();

  // 3. stream the units: wave w handles KV head hb * W + w of every unit
  const int lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int dl = lane % Sh::LPT, row = lane / Sh::LPT;
  const int lane_off = lane * 16;
  const T* kp = reinterpret_cast<const T*>(a.k_pages);
  const T* vp = reinterpret_cast<const T*>(a.v_pages);
  const T* qbase = reinterpret_cast<const T*>(a.q);

  DecodeState<T, D, S> st;
  mfma::State<S> ms;  // matrix-core variant (bf16, D = 128)
  __shared__ __attribute__((aligned(16))) uint8_t s_kv[MF ? W : 1][MF ? 2 * mfma::kTile : 16];
  bool head_partial = false;

  auto issue = [&](u32x4 (&kr)[Sh::NI], u32x4 (&vr)[Sh::NI], int k) {
    int valid = 0;
    int64_t off = 0;
    if (k < n_units) {
      const int page = __builtin_amdgcn_readfirstlane(s_page[k]);
      const int info = __builtin_amdgcn_readfirstlane(s_info[k]);
      off = tile_offset(page, info_hb(info) * W + w, a.H_kv, D);
      valid = info_valid(info);
    }
    issue_tile<Sh::NI>(tile_rsrc<T, D>(kp + off, valid), tile_rsrc<T, D>(vp + off, valid), lane_off, kr, vr);
  };

  u32x4 kr[NBUF][Sh::NI], vr[NBUF][Sh::NI];
#pragma unroll
  for (int u = 0; u + 1 < NBUF; ++u) issue(kr[u], vr[u], u);
  for (int base = 0; base < n_units; base += NBUF) {
#pragma unroll
    for (int u = 0; u < NBUF; ++u) {
      // Lockstep: without a barrier the older wave of each SIMD runs ahead,
      // waves 0..3 finish ~30% before waves 4..7, and those then stream the
      // rest alone with half the loads in flight.  In step, the W waves also
      // issue the W adjacent head tiles of a page together.
      __syncthreads();
      const int k = base + u;
      int info = 0;
      if (k < n_units) {
        info = __builtin_amdgcn_readfirstlane(s_info[k]);
        if (info_start(info) || k == 0) {  // a new (row, head) item: its queries
          head_partial = !info_start(info);
          const int g = info_hb(info) * W + w;
          const T* qg = qbase + ((int64_t)info_row(info) * a.H_q + (int64_t)g * S) * D;
          if constexpr (MF) {
            mfma::begin_item<S>(ms, reinterpret_cast<const uint16_t*>(qg), lane);
          } else {
            const T* qp = qg + dl * Sh::VEC;
#pragma unroll
            for (int j = 0; j < S; ++j) {
              st.q[j] = *reinterpret_cast<const u32x4*>(qp + j * D);
              st.m[j] = kMInit;
              st.l[j] = 0.0f;
#pragma unroll
              for (int e = 0; e < Sh::VEC; ++e) st.o[j][e] = 0.0f;
            }
          }
        }
      }
      issue(kr[(u + NBUF - 1) % NBUF], vr[(u + NBUF - 1) % NBUF], k + NBUF - 1);
      if (k < n_units) {
        if constexpr (MF)
          mfma::fold<S>(ms, kr[u], vr[u], s_kv[w], lane, info_valid(info), a.scale_log2);
        else
          fold_tile<T, D, S>(st, kr[u], vr[u], row, info_valid(info), a.scale_log2);
        const bool tail_partial = k == n_units - 1 && !info_end(info);
        if (info_end(info) || k == n_units - 1) {
          const int r = info_row(info);
          const int g = info_hb(info) * W + w;
          T* outp = reinterpret_cast<T*>(a.out) + ((int64_t)r * a.H_q + (int64_t)g * S) * D;
          const int64_t slot = ((int64_t)blockIdx.x * 2 + (head_partial ? 0 : 1)) * W + w;
          if constexpr (MF) {
            if (!head_partial && !tail_partial)
              mfma::finish<S, T>(ms, lane, outp);
            else
              mfma::partial<S>(ms, lane, a.ws_o + slot * S * D, a.ws_ml + slot * S * 2);
          } else {
            if (!head_partial && !tail_partial)
              finish_rows<T, D, S>(st, row, dl, outp);
            else
              partial_rows<T, D, S>(st, row, dl, lane, a.ws_o + slot * S * D, a.ws_ml + slot * S * 2);
          }
        }
      }
    }
  }
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

hipError_t launch_stream(int dtype, int D, int s, int W, const StreamArgs& a, int G, hipStream_t st) {
  const void* fn = stream_kernel_fn(dtype, D, s, W);
  if (fn == nullptr || G <= 0) return hipErrorInvalidValue;
  void* args[] = {const_cast<StreamArgs*>(&a)};
  hipError_t e = hipLaunchKernel(fn, dim3(G), dim3(64 * W), args, 0, st);
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
