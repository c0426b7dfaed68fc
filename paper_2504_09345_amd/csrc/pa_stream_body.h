// Body of the persistent stream-K decode workgroup, shared by the stream-K
// kernel and the mixed prefill + decode kernel (see pa_stream.hip for the
// design).
#pragma once

#include <type_traits>

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

// Merge the partial records of item (row r, KV head g) held by ranges
// wg_first .. wg_last (record slot 1 of wg_first, slot 0 of the others; empty
// ranges wrote nothing) and write the output row: one wave, E elements per
// lane, records merged in range order.  Every part of the item stores its
// record before it counts its arrival, and whichever part arrives last runs
// this merge over all the records, so the result does not depend on which
// range merges.  When a lane's E elements lie in one head (D a multiple of
// E), the lane keeps only that head's running (M, L); the arithmetic of each
// element is the same either way.
template <typename T, int D, int S, int W>
__device__ __forceinline__ void merge_item(const StreamArgs& a, int64_t U, int64_t G, int64_t wg_first,
                                           int64_t wg_last, int w, int lane, T* out) {
  constexpr int E = S * D / 64;  // elements per lane
  constexpr bool kOneHead = D % E == 0;
  constexpr int NH = kOneHead ? 1 : S;  // heads whose (M, L) the lane keeps
  const int h0 = kOneHead ? lane * E / D : 0;
  float M[NH], L[NH], acc[E];
#pragma unroll
  for (int j = 0; j < NH; ++j) { M[j] = kMInit; L[j] = 0.0f; }
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.0f;
  // pass 1: maxima
  for (int64_t x = wg_first; x <= wg_last; ++x) {
    if (U * x / G == U * (x + 1) / G) continue;  // empty range wrote nothing
    const int64_t slot = (x * 2 + (x == wg_first ? 1 : 0)) * W + w;
#pragma unroll
    for (int j = 0; j < NH; ++j) M[j] = fmaxf(M[j], load_dev(a.ws_ml + slot * S * 2 + (h0 + j) * 2));
  }
  // pass 2: weighted sums
  for (int64_t x = wg_first; x <= wg_last; ++x) {
    if (U * x / G == U * (x + 1) / G) continue;
    const int64_t slot = (x * 2 + (x == wg_first ? 1 : 0)) * W + w;
    float c[NH];
#pragma unroll
    for (int j = 0; j < NH; ++j) {
      float m, l;
      load_dev2(a.ws_ml + slot * S * 2 + (h0 + j) * 2, m, l);
      c[j] = fast_exp2(m - M[j]);
      L[j] = fmaf(l, c[j], L[j]);
    }
    const float* o = a.ws_o + slot * S * D;
    float v[E];
    if constexpr (E % 2 == 0) {
#pragma unroll
      for (int e = 0; e < E; e += 2) load_dev2(o + lane * E + e, v[e], v[e + 1]);
    } else {
#pragma unroll
      for (int e = 0; e < E; ++e) v[e] = load_dev(o + lane * E + e);
    }
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int idx = lane * E + e;
      acc[e] = fmaf(v[e], c[idx / D - h0], acc[e]);
    }
  }
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int idx = lane * E + e;
    store_out<T>(out + idx, acc[e] / L[idx / D - h0]);
  }
}

// The record of an item's other part, loaded ahead of merge_held: (M, L) and
// the unnormalised O of this lane's head column in the matrix-core layout
// (lanes of heads >= S load nothing).
template <int S>
struct HeldRecord {
  float m = 0.0f, l = 0.0f;
  float o[mfma::kD / 16][4] = {};
};
template <int S>
__device__ __forceinline__ void load_held(HeldRecord<S>& r, const float* o, const float* ml, int lane) {
  const int n = lane & 15, G = lane >> 4;
  if (n < S) {
    load_dev2(ml + n * 2, r.m, r.l);
#pragma unroll
    for (int mb = 0; mb < mfma::kD / 16; ++mb) {
      load_dev2(o + n * mfma::kD + mb * 16 + 4 * G, r.o[mb][0], r.o[mb][1]);
      load_dev2(o + n * mfma::kD + mb * 16 + 4 * G + 2, r.o[mb][2], r.o[mb][3]);
    }
  }
}

// merge_item for an item of two parts whose first part is this wave's
// matrix-core state (its record never stored) and whose second part is the
// record r: the same operations in the same order as merge_item over the two
// records, so the output bits do not depend on which of the two parts merged.
template <typename T, int S>
__device__ __forceinline__ void merge_held(const mfma::State<S>& st, const HeldRecord<S>& r, int lane, T* out) {
  const float l0 = mfma::total_l(st);  // (every lane: a cross-lane sum)
  const int n = lane & 15, G = lane >> 4;
  if (n < S) {
    const float M = fmaxf(fmaxf(kMInit, st.m), r.m);
    const float c0 = fast_exp2(st.m - M), c1 = fast_exp2(r.m - M);
    const float L = fmaf(r.l, c1, fmaf(l0, c0, 0.0f));
#pragma unroll
    for (int mb = 0; mb < mfma::kD / 16; ++mb) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        store_out<T>(out + n * mfma::kD + mb * 16 + 4 * G + i,
                     fmaf(r.o[mb][i], c1, fmaf(st.acc[mb][i], c0, 0.0f)) / L);
    }
  }
}

// Count one part's arrival at an item's counter and return the parts counted
// so far, this one included.  The counter's upper 48 bits carry the call's
// token and its lower 16 bits the count: a counter left by an earlier call
// (or found in a fresh workspace) holds another token and starts over at 1.
// The first compare-and-swap guesses that the other parts (parts - 1) have
// all arrived, so the last part, which goes on to merge, usually needs one
// round trip; a wrong guess returns the counter's value and the loop goes on
// from it.  It only repeats when another part of the same item changed the
// counter in between, so it ends after at most as many rounds as the item
// has parts, plus the guess; nothing here waits for another workgroup.
__device__ __forceinline__ int arrive_count(unsigned long long* ctr, unsigned long long token, int parts) {
  const unsigned long long tag = (token & 0xffffffffffffull) << 16;
  unsigned long long old = tag | (unsigned long long)(parts - 1);
  for (;;) {
    const unsigned long long base = (old & ~0xffffull) == tag ? old : tag;
    if (__hip_atomic_compare_exchange_strong(ctr, &old, base + 1, __ATOMIC_RELAXED, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT))
      return (int)((base + 1) & 0xffffull);
  }
}

// Range (of G equal ranges over U units) that holds unit e: the largest x
// with floor(U x / G) <= e.
__device__ __forceinline__ int64_t range_of(int64_t e, int64_t U, int64_t G) { return ((e + 1) * G - 1) / U; }

// Sequence of unit u: the largest r with nb * cum[r] <= u (a non-empty one).
__device__ __forceinline__ int info_row_seq(const int32_t* cum, int R, int nb, int64_t u) {
  int lo = 0, hi = R - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if ((int64_t)nb * cum[mid] <= u) lo = mid; else hi = mid - 1;
  }
  return lo;
}

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

// Codes in s_tail for rows without units (a row with units holds 1 .. 16,
// the tokens in its last page).
constexpr uint8_t kRowZeros = 0x20, kRowNaN = 0x40;

// The stream-K decode workgroup `bid` of a grid of G (see pa_stream.hip).
// TR: gather-trace instantiation (records every loaded token's pool row in
// a.trace besides computing the attention).  SPLIT: with the matrix-core
// fold, load K and V half a unit apart (the decode-only kernel); without it,
// through the ring of NBUF whole tiles (the mixed kernel, whose decode
// workgroups share HBM with prefill workgroups and need the longer lead).
template <typename T, int D, int S, int W, int NBUF, bool MF, bool TR = false, bool SPLIT = kStreamSplitKV>
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
      const int status = seq_decode_row(a.query_start_loc, a.context_lens, a.max_context_len, r, row, nv);
      int np = status == 1 ? (nv + kPage - 1) / kPage : 0;
      const bool bad = status < 0 || np > (int)a.bt_stride;  // contract violation: a NaN row (below)
      if (bad) np = 0;
      // tokens in the last page, or for a row without units what its output
      // gets: kRowZeros (empty decode context), kRowNaN (violation), 0 (none)
      s_tail[r] = (uint8_t)(np ? nv - (np - 1) * kPage : bad ? kRowNaN : status == 1 ? kRowZeros : 0);
      s_cum[r] = local;
      local += np;
    }
    const int off = block_exclusive_scan<NT>(local, s_scan);
    for (int r = r0; r < r1; ++r) s_cum[r] += off;
    if (tid == NT - 1) s_cum[R] = off + local;
    __syncthreads();
  }
  const int64_t U = (int64_t)a.nb * s_cum[R];
  const int64_t G = G_;
  // Rows without units: zeros for an empty decode context, NaN for a contract
  // violation (flagged in s_tail above); rows r = bid (mod G) are this
  // workgroup's to write.
  for (int r = bid; r < R; r += G_) {
    if (s_cum[r + 1] != s_cum[r]) continue;  // the row has units
    const int code = s_tail[r];
    if (code != kRowZeros && code != kRowNaN) continue;
    const int qrow = a.query_start_loc != nullptr ? a.query_start_loc[r] : r;
    const float fill = code == kRowNaN ? NAN : 0.0f;
    T* o = reinterpret_cast<T*>(a.out) + (int64_t)qrow * a.H_q * D;
    for (int i = tid; i < a.H_q * D; i += NT) store_out<T>(o + i, fill);
  }
  const int64_t u0 = U * bid / G, u1 = U * (bid + 1) / G;
  const int n_units = (int)(u1 - u0);
  if (n_units <= 0) return;

  // 2. unit table of this range
  const BlockTable bt{a.block_table, a.bt_stride};
  for (int i = tid; i < n_units; i += NT) {
    const int64_t u = u0 + i;
    const int r = info_row_seq(s_cum, R, a.nb, u);
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

  // Element offset and live tokens of unit k's tile for this wave (a null
  // tile past the range); the trace instantiation records the tile's rows.
  auto unit_tile = [&](int k, int64_t& off, int& valid, bool record) {
    valid = 0;
    off = 0;
    if (k < n_units) {
      const int page = __builtin_amdgcn_readfirstlane(s_page[k]);
      const int info = __builtin_amdgcn_readfirstlane(s_info[k]);
      off = tile_offset(page, info_hb(info) * W + w, a.H_kv, D);
      valid = info_valid(info);
      if constexpr (TR) {
        if (record) {
          // (sequence, head block, page) of the unit, from the unit's index
          const int r = info_row_seq(s_cum, R, a.nb, u0 + k);
          const int np = s_cum[r + 1] - s_cum[r];
          const int rem = (int)(u0 + k - (int64_t)a.nb * s_cum[r]);
          const int hb = rem / np, p = rem - hb * np;
          if (lane < valid)
            trace_put(a.trace, ((int64_t)(hb * W + w) * R + r) * (a.bt_stride * kPage) + p * kPage + lane,
                      off / D + lane);
        }
      }
    }
  };
  auto issue = [&](u32x4 (&kr)[Sh::NI], u32x4 (&vr)[Sh::NI], int k) {
    int64_t off;
    int valid;
    unit_tile(k, off, valid, true);
    issue_tile<Sh::NI>(tile_rsrc<T, D>(kp + off, valid), tile_rsrc<T, D>(vp + off, valid), lane_off, kr, vr);
  };

  // Items cut by range boundaries.  Every part (the item's first part ends
  // its range; a later part starts one) stores its partial record, then
  // counts its arrival at the item's counter; the part that arrives last
  // merges all the records in range order and writes the output.  Nothing
  // waits on another workgroup, so the result and the kernel's completion do
  // not depend on how many workgroups are resident or in which order they
  // run.  Records travel through device-coherent stores and loads; a part
  // counts itself only once its record stores have completed.
  auto arrive = [&](int64_t x0, int64_t x1, int qrow, int g) {
    int parts = 0;
    for (int64_t x = x0; x <= x1; ++x) parts += U * x / G != U * (x + 1) / G ? 1 : 0;
    int got = 0;
    if (lane == 0) got = arrive_count(a.ws_flag + x0 * W + w, a.token, parts);
    got = __builtin_amdgcn_readfirstlane(got);
    if (got == parts) {
      T* outp = reinterpret_cast<T*>(a.out) + ((int64_t)qrow * a.H_q + (int64_t)g * S) * D;
      merge_item<T, D, S, W>(a, U, G, x0, x1, w, lane, outp);
    }
  };

  // A part whose record is stored at unit k < n_units - 1 counts its arrival
  // one unit later, once the loads issued after the record are the only ones
  // outstanding: waiting for the record stores then does not drain the tile
  // loads in flight (the vector-memory counter retires loads and stores in
  // issue order).
  bool pending = false;  // (wave-uniform) an arrival to count at the next unit
  int64_t pend_x0 = 0, pend_x1 = 0;
  int pend_row = 0, pend_g = 0;

  // Range-end merge from registers (the matrix-core split loop sets these):
  // the item ending the range has one other part, which has counted, and
  // its record is in held_rec.
  bool held_now = false;
  HeldRecord<S> held_rec;

  // Start of unit k, every wave in step (without the barrier the older wave
  // of each SIMD runs ahead, waves 0..3 finish ~30% before waves 4..7, and
  // those then stream the rest alone with half the loads in flight; in step,
  // the W waves also issue the W adjacent head tiles of a page together).
  // A new (row, head) item loads its queries.  Returns the unit's info word.
  auto begin_unit = [&](int k) {
    __syncthreads();
    int info = 0;
    if (k < n_units) {
      info = __builtin_amdgcn_readfirstlane(s_info[k]);
      if (info_start(info) || k == 0) {
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
    return info;
  };
  // End of unit k (k < n_units): an item that ends here is finished in place
  // when it lies wholly in the range; a part cut by the range stores its
  // record and counts its arrival (at the next unit, or now at the range's
  // last unit).
  auto end_unit = [&](int k, int info) {
    const bool tail_partial = k == n_units - 1 && !info_end(info);
    if (info_end(info) || k == n_units - 1) {
      const int r = info_row(info);
      const int g = info_hb(info) * W + w;
      T* outp = reinterpret_cast<T*>(a.out) + ((int64_t)r * a.H_q + (int64_t)g * S) * D;
      if (!head_partial && !tail_partial) {  // the whole item in this range
        if constexpr (MF)
          mfma::finish<S, T>(ms, lane, outp);
        else
          finish_rows<T, D, S>(st, row, dl, outp);
      } else {  // (workgroup-uniform, but for merge_held)
        if constexpr (MF) {
          if (held_now && k == n_units - 1) {  // (wave-uniform)
            merge_held<T, S>(ms, held_rec, lane, outp);
            return;
          }
        }
        const int64_t slot = ((int64_t)bid * 2 + (head_partial ? 0 : 1)) * W + w;
        if constexpr (MF)
          mfma::partial<S>(ms, lane, a.ws_o + slot * S * D, a.ws_ml + slot * S * 2);
        else
          partial_rows<T, D, S>(st, row, dl, lane, a.ws_o + slot * S * D, a.ws_ml + slot * S * 2);
        // the item's first and last units, and the ranges holding them
        const int rr = info_row_seq(s_cum, R, a.nb, u0 + k);
        const int np = s_cum[rr + 1] - s_cum[rr];
        const int64_t e_first = (int64_t)a.nb * s_cum[rr] + (int64_t)info_hb(info) * np;
        pend_x0 = range_of(e_first, U, G);
        pend_x1 = range_of(e_first + np - 1, U, G);
        pend_row = r;
        pend_g = g;
        if (k + 1 < n_units) {
          pending = true;  // counted at the next unit
        } else {
          __builtin_amdgcn_s_waitcnt(0);  // the record stores have completed
          arrive(pend_x0, pend_x1, pend_row, pend_g);
        }
      }
    }
  };
  // (wait: the s_waitcnt encoding that leaves only the loads just issued
  // outstanding, as a std::integral_constant)
  auto arrive_pending = [&](auto wait) {
    if (pending) {  // wave-uniform
      pending = false;
      __builtin_amdgcn_s_waitcnt(decltype(wait)::value);
      arrive(pend_x0, pend_x1, pend_row, pend_g);
    }
  };

  if constexpr (MF && SPLIT) {
    // Matrix-core fold: a unit's K and V loads go out half a unit apart.  The
    // K loads of unit k + 1 (after the queries of the item it starts, if it
    // starts one) follow unit k's QK half, and its V loads follow unit k's PV
    // half, before the unit's end (an output, or a record and maybe a merge);
    // each is waited for about a unit after it was issued, so about one K and
    // one V tile (8 KiB) are in flight per wave instead of two whole tiles,
    // and one register set of each suffices.  These loads are issued as
    // inline assembly, which the compiler's wait counting does not see (its
    // own counting, across the merge paths, waited for every load at each
    // unit), and are waited for explicitly: when unit k + 1's QK half starts,
    // its V loads (NI instructions) went out after its K loads and queries,
    // and when unit k's PV half starts, unit k + 1's K loads went out after
    // unit k's V loads, so vmcnt(NI) suffices at both points whatever else
    // (records, merges, outputs) went out in between.
    static_assert(Sh::NI < 16, "vmcnt range");
    const int n_q = lane & 15, g_q = lane >> 4;
    auto load_queries = [&](int info) {
      const int g = info_hb(info) * W + w;
      const T* qg = qbase + ((int64_t)info_row(info) * a.H_q + (int64_t)g * S) * D;
      // lane (n, G): row n of the group (zeros past the S rows), dims
      // 32 s + 8 G .. +8 of Q^T operand s
      asm_issue<mfma::kD / 32, 64>(scalar_rsrc(qg, S * D * 2), (n_q * D + g_q * 8) * 2, ms.qt);
    };
    auto tile_k = [&](int k, u32x4 (&x)[Sh::NI]) {
      int64_t off;
      int valid;
      unit_tile(k, off, valid, true);
      asm_issue<Sh::NI>(scalar_rsrc(kp + off, valid * D * (int)sizeof(T)), lane_off, x);
    };
    auto tile_v = [&](int k, u32x4 (&x)[Sh::NI]) {
      int64_t off;
      int valid;
      unit_tile(k, off, valid, false);
      asm_issue<Sh::NI>(scalar_rsrc(vp + off, valid * D * (int)sizeof(T)), lane_off, x);
    };
    //
    // The range's last item, when cut by the range's end, usually finishes
    // last: its other part started the next range and counted long before.
    // If that item has two parts (it ends in the next range), its counter is
    // loaded (inline assembly too) when the next-to-last unit's QK half
    // starts, older than the K loads of the last unit, so the waits above
    // cover it unchanged; it is looked at when the last unit starts; if the
    // other part has counted, its record is loaded then, and the last unit
    // ends by merging from registers (merge_held): no record stored, no
    // arrival counted (every other part has counted, so no part reads the
    // counter again in this call), the record's latency hidden behind the
    // unit's fold.  With a single unit the counter load goes out between
    // its K and V loads.
    bool held = false;  // (wave-uniform) the range's last item qualifies
    {
      const int info_l = __builtin_amdgcn_readfirstlane(s_info[n_units - 1]);
      if (!info_end(info_l)) {
        const int rr = info_row_seq(s_cum, R, a.nb, u1 - 1);
        const int np = s_cum[rr + 1] - s_cum[rr];
        const int64_t e_first = (int64_t)a.nb * s_cum[rr] + (int64_t)info_hb(info_l) * np;
        held = e_first >= u0 && range_of(e_first + np - 1, U, G) == bid + 1;
      }
    }
    const unsigned long long* ctr_p = a.ws_flag + (int64_t)bid * W + w;
    const unsigned long long counted = ((a.token & 0xffffffffffffull) << 16) | 1ull;  // one part counted
    u32x2_t ctr = u32x2_t{0u, 0u};

    u32x4 kc[Sh::NI], vc[Sh::NI];
    load_queries(__builtin_amdgcn_readfirstlane(s_info[0]));
    tile_k(0, kc);
    if (held && n_units == 1) asm_load_dev(ctr_p, ctr);
    tile_v(0, vc);
    for (int k = 0; k < n_units; ++k) {
      __syncthreads();  // lockstep, as in begin_unit
      const int info = __builtin_amdgcn_readfirstlane(s_info[k]);
      if (info_start(info) || k == 0) {
        head_partial = !info_start(info);
        mfma::reset<S>(ms);
      }
      vm_wait<Sh::NI>(kc);  // K of unit k and the queries (issued before it)
      vm_wait<Sh::NI>(ms.qt);
      if (held && k + 2 == n_units) asm_load_dev(ctr_p, ctr);
      if (held && k == n_units - 1) {
        vm_wait<Sh::NI>(ctr);  // (issued before unit k's V loads)
        held_now = __builtin_amdgcn_readfirstlane(ctr.x) == (uint32_t)counted &&
                   __builtin_amdgcn_readfirstlane(ctr.y) == (uint32_t)(counted >> 32);
        if (held_now) {
          const int64_t slot = ((int64_t)(bid + 1) * 2 + 0) * W + w;
          load_held<S>(held_rec, a.ws_o + slot * S * D, a.ws_ml + slot * S * 2, lane);
        }
      }
      mfma::s16x4_t phi, plo;
      mfma::fold_qk<S>(ms, kc, s_kv[w], lane, info_valid(info), a.scale_log2, phi, plo);
      if (k + 1 < n_units) {  // the queries are free once the QK half is done
        const int next = __builtin_amdgcn_readfirstlane(s_info[k + 1]);
        if (info_start(next)) load_queries(next);
      }
      tile_k(k + 1, kc);
      arrive_pending(std::integral_constant<int, (Sh::NI & 15) | (7 << 4) | (15 << 8)>{});
      vm_wait<Sh::NI>(vc);  // V of unit k
      mfma::fold_pv<S>(ms, vc, s_kv[w], lane, phi, plo);
      tile_v(k + 1, vc);
      end_unit(k, info);
    }
    __builtin_amdgcn_s_waitcnt(0);  // the last (null) tiles' loads
  } else {
    // A ring of NBUF register tiles: the tile of unit k + NBUF - 1 is issued
    // at the start of unit k.
    constexpr int kRingLoads = 2 * Sh::NI;  // load instructions of one issue()
    constexpr int kWaitRing = (kRingLoads & 15) | (7 << 4) | (15 << 8) | ((kRingLoads >> 4) << 14);
    static_assert(kRingLoads < 64, "vmcnt range");
    u32x4 kr[NBUF][Sh::NI], vr[NBUF][Sh::NI];
#pragma unroll
    for (int u = 0; u + 1 < NBUF; ++u) issue(kr[u], vr[u], u);
    for (int base = 0; base < n_units; base += NBUF) {
#pragma unroll
      for (int u = 0; u < NBUF; ++u) {
        const int k = base + u;
        const int info = begin_unit(k);
        issue(kr[(u + NBUF - 1) % NBUF], vr[(u + NBUF - 1) % NBUF], k + NBUF - 1);
        arrive_pending(std::integral_constant<int, kWaitRing>{});
        if (k < n_units) {
          if constexpr (MF)
            mfma::fold<S>(ms, kr[u], vr[u], s_kv[w], lane, info_valid(info), a.scale_log2);
          else
            fold_tile<T, D, S>(st, kr[u], vr[u], row, info_valid(info), a.scale_log2);
          end_unit(k, info);
        }
      }
    }
  }
}

}  // namespace pa
