// Body of the persistent stream-K decode workgroup, shared by the stream-K
// kernel and the mixed prefill + decode kernel (see pa_stream.hip for the
// design).
#pragma once

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

// LDS of one stream-K workgroup.
template <int W, bool MF>
struct StreamSmem {
  int32_t cum[kStreamMaxRows + 1];  // page prefix sums over rows
  uint8_t tail[kStreamMaxRows];     // valid tokens of each row's last page
  int32_t page[kStreamMaxUnits];    // unit table of the range: page id
  int32_t info[kStreamMaxUnits];    //   and info word
  int32_t scan[64 * W];
  __attribute__((aligned(16))) uint8_t kv[MF ? W : 1][MF ? 2 * mfma::kTile : 16];  // per-wave tile staging
};

// The stream-K decode workgroup `bid` of a grid of G (see pa_stream.hip).
template <typename T, int D, int S, int W, int NBUF, bool MF>
__device__ __forceinline__ void stream_body(const StreamArgs& a, StreamSmem<W, MF>& sm, int bid, int G_) {
  using Sh = DecodeShape<T, D, S>;
  constexpr int NT = 64 * W;
  int32_t* s_cum = sm.cum;
  uint8_t* s_tail = sm.tail;
  int32_t* s_page = sm.page;
  int32_t* s_info = sm.info;
  int32_t* s_scan = sm.scan;

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
  if (bid == 0)
    for (int r = tid; r <= R; r += NT) a.ws_cum[r] = s_cum[r];
  const int64_t G = G_;
  const int64_t u0 = U * bid / G, u1 = U * (bid + 1) / G;
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
  auto& s_kv = sm.kv;
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
          const int64_t slot = ((int64_t)bid * 2 + (head_partial ? 0 : 1)) * W + w;
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

}  // namespace pa
