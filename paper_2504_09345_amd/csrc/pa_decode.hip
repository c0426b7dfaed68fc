// Split-K paged GQA decode attention for gfx950 (CDNA4, wave64).
//
// What it computes: for each sequence b and query head h, softmax(scale *
// q.K^T) V over the sequence's cached tokens, with K/V gathered page by page
// through the block table (paged KV, MoE-Lens Sec. 5.5) and the s query heads
// of a GQA group sharing their KV head (Sec. 2).  The paper's CPU kernel is a
// flash-attention style loop of dot products and scaled vector adds over
// bf16 KV up-converted to fp32 (Sec. 5.3 Eq. 6, Sec. 6.6); this kernel keeps
// that arithmetic (fp32 accumulate, online softmax) and maps it to a GPU.
//
// Mapping.  A workgroup of kDecodeWaves waves owns (split, kv head g, seq b):
// a range of up to pages_per_split pages, dealt to its waves round-robin.  A
// (page, g) tile is 16 tokens x D contiguous elements (4 KiB at D = 128 bf16);
// a wave reads it with NI wave-wide 16-byte-per-lane loads (1 KiB each, fully
// coalesced).  Lane l holds VEC consecutive dims of token (l / LPT) + TPI * i.
// All s query heads of the group are processed by the same wave from those
// registers, so each K/V byte is fetched from HBM once and used s times
// without an LDS round trip.
//   QK:  per-lane partial dot products (v_dot2 on packed bf16) reduced over the
//        LPT lanes of a token with DPP.
//   softmax: online, per (lane row, head): each row of LPT lanes keeps its own
//        running max / sum over the tokens it owns; rows and waves are merged
//        once at the end of the split (log-sum-exp merge).
//   PV:  per-lane FMA into VEC fp32 accumulators per head.
// A sequence that needs one split writes the normalised output; otherwise the
// split writes (o unnormalised, m, l) to the workspace and the reduction
// kernel merges the splits.
#include "pa_device.h"
#include "pa_kernels.h"
#include "pa_tile.h"

namespace pa {

// TR: gather-trace instantiation (records every loaded token's pool row in
// a.trace besides computing the attention).
template <typename T, int D, int S, int WAVES, int NBUF, bool TR>
__global__ __launch_bounds__(64 * WAVES) void decode_kernel(DecodeArgs a) {
  using Sh = DecodeShape<T, D, S>;
  constexpr int NT = 64 * WAVES;
  __shared__ float sm_o[WAVES][S][D];
  __shared__ float sm_ml[WAVES][S][2];

  const int split = blockIdx.x % a.n_split_slots;
  const int rest = blockIdx.x / a.n_split_slots;
  const int g = rest % a.H_kv, row_idx = rest / a.H_kv;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: keep it scalar
  int b, ctx;  // ctx: keys this row sees
  const bool ok = row_context(a.query_start_loc, a.context_lens, a.B, a.max_context_len, row_idx, b, ctx);
  if (a.skip_single_rows && a.query_start_loc[b + 1] - a.query_start_loc[b] == 1) return;
  const int n_pages = ok ? (ctx + kPage - 1) / kPage : 0;
  const int pps = a.pages_per_split;
  const int p0 = split * pps;
  T* out = reinterpret_cast<T*>(a.out);
  const int64_t out_base = ((int64_t)row_idx * a.H_q + (int64_t)g * S) * D;

  // Contract violations (negative length, a chunk longer than its context, or
  // more pages than the block-table row / the grid can hold) are reported as
  // NaN output, never read past.
  const bool bad = !ok || n_pages > (int)a.bt_stride || n_pages > a.n_split_slots * pps;
  if (bad || n_pages == 0) {
    if (split == 0)
      for (int idx = threadIdx.x; idx < S * D; idx += NT) store_out<T>(out + out_base + idx, bad ? NAN : 0.0f);
    return;
  }
  if (p0 >= n_pages) return;
  const int p1 = min(p0 + pps, n_pages);
  const bool single = n_pages <= pps;

  // Pages of this wave: p0 + wave + WAVES * k, k < my_n; lane k holds entry k.
  const int my_n = max(0, (p1 - p0 - wave + WAVES - 1) / WAVES);
  const BlockTable bt{a.block_table, a.bt_stride};
  const int32_t bt_lane = lane < my_n ? bt.page(b, p0 + wave + WAVES * lane) : 0;

  DecodeState<T, D, S> st;
  const int dl = lane % Sh::LPT, row = lane / Sh::LPT;
  {
    const T* qp = reinterpret_cast<const T*>(a.q) + out_base + dl * Sh::VEC;
#pragma unroll
    for (int j = 0; j < S; ++j) st.q[j] = *reinterpret_cast<const u32x4*>(qp + j * D);
  }
#pragma unroll
  for (int j = 0; j < S; ++j) {
    st.m[j] = kMInit;
    st.l[j] = 0.0f;
#pragma unroll
    for (int e = 0; e < Sh::VEC; ++e) st.o[j][e] = 0.0f;
  }

  const T* kp = reinterpret_cast<const T*>(a.k_pages);
  const T* vp = reinterpret_cast<const T*>(a.v_pages);
  const int lane_off = lane * 16;

  // Ring of NBUF register tile buffers: while tile k is folded, the loads of
  // tiles k+1 .. k+NBUF-1 are in flight.  Loads are issued unconditionally;
  // a tile index past the wave's pages gets a null descriptor (zeros, no
  // memory access), so the number of outstanding loads is the same on every
  // path and the wait before each fold is a fixed count.
  auto issue = [&](u32x4 (&kr)[Sh::NI], u32x4 (&vr)[Sh::NI], int kk) {
    int valid = 0;
    int64_t off = 0;
    if (kk < my_n) {
      const int p = p0 + wave + WAVES * kk;
      const int32_t page = __builtin_amdgcn_readlane(bt_lane, kk);
      off = tile_offset(page, g, a.H_kv, D);
      valid = min(kPage, ctx - p * kPage);
      if constexpr (TR) {
        if (lane < valid)
          trace_put(a.trace, ((int64_t)g * a.B + b) * (a.bt_stride * kPage) + p * kPage + lane, off / D + lane);
      }
    }
    issue_tile<Sh::NI>(tile_rsrc<T, D>(kp + off, valid), tile_rsrc<T, D>(vp + off, valid), lane_off, kr, vr);
  };
  auto fold = [&](const u32x4 (&kr)[Sh::NI], const u32x4 (&vr)[Sh::NI], int kk) {
    if (kk < my_n) {
      const int p = p0 + wave + WAVES * kk;
      fold_tile<T, D, S>(st, kr, vr, row, min(kPage, ctx - p * kPage), a.scale_log2);
    }
  };

  u32x4 kr[NBUF][Sh::NI], vr[NBUF][Sh::NI];
#pragma unroll
  for (int u = 0; u + 1 < NBUF; ++u) issue(kr[u], vr[u], u);
  for (int base = 0; base < my_n; base += NBUF) {
#pragma unroll
    for (int u = 0; u < NBUF; ++u) {
      issue(kr[(u + NBUF - 1) % NBUF], vr[(u + NBUF - 1) % NBUF], base + u + NBUF - 1);
      fold(kr[u], vr[u], base + u);
    }
  }

  // Merge the token rows of the wave (log-sum-exp), then the waves via LDS.
#pragma unroll
  for (int j = 0; j < S; ++j) {
    const float M = across_groups_max<Sh::LPT>(st.m[j]);
    const float w = fast_exp2(st.m[j] - M);
    const float L = across_groups_sum<Sh::LPT>(st.l[j] * w);
#pragma unroll
    for (int e = 0; e < Sh::VEC; ++e) {
      const float oe = across_groups_sum<Sh::LPT>(st.o[j][e] * w);
      if (row == 0) sm_o[wave][j][dl * Sh::VEC + e] = oe;
    }
    if (lane == 0) {
      sm_ml[wave][j][0] = M;
      sm_ml[wave][j][1] = L;
    }
  }
  __syncthreads();

  const int64_t ws_row = ((int64_t)row_idx * a.H_q + (int64_t)g * S) * a.n_split_slots + split;
  for (int idx = threadIdx.x; idx < S * D; idx += NT) {
    const int j = idx / D, d = idx % D;
    float M = sm_ml[0][j][0];
#pragma unroll
    for (int w = 1; w < WAVES; ++w) M = fmaxf(M, sm_ml[w][j][0]);
    float L = 0.0f, O = 0.0f;
#pragma unroll
    for (int w = 0; w < WAVES; ++w) {
      const float c = fast_exp2(sm_ml[w][j][0] - M);
      L = fmaf(sm_ml[w][j][1], c, L);
      O = fmaf(sm_o[w][j][d], c, O);
    }
    if (single) {
      store_out<T>(out + out_base + idx, O / L);
    } else {
      const int64_t r = ws_row + (int64_t)j * a.n_split_slots;  // row (b, g*S+j, split)
      a.ws_o[r * D + d] = O;
      if (d == 0) {
        a.ws_ml[r * 2] = M;
        a.ws_ml[r * 2 + 1] = L;
      }
    }
  }
}

// Log-sum-exp merge of the split partials of one (sequence, query head) per
// wave: M = max_i m_i, L = sum_i l_i 2^(m_i - M), out = sum_i o_i 2^(m_i - M) / L.
// Deterministic (fixed order, no atomics).
template <typename T, int D>
__global__ __launch_bounds__(256) void reduce_kernel(ReduceArgs a) {
  constexpr int E = D / 64;
  const int lane = threadIdx.x & 63;
  const int item = blockIdx.x * 4 + (threadIdx.x >> 6);  // row * H_q + h
  if (item >= a.rows * a.H_q) return;
  int b, ctx;
  if (!row_context(a.query_start_loc, a.context_lens, a.B, a.max_context_len, item / a.H_q, b, ctx)) return;
  if (a.skip_single_rows && a.query_start_loc[b + 1] - a.query_start_loc[b] == 1) return;
  const int n_pages = (ctx + kPage - 1) / kPage;
  const int n_splits = (n_pages + a.pages_per_split - 1) / a.pages_per_split;
  if (n_splits <= 1 || n_splits > a.n_split_slots) return;  // written by the attention kernel
  const float* ml = a.ws_ml + (int64_t)item * a.n_split_slots * 2;
  const float* o = a.ws_o + (int64_t)item * a.n_split_slots * D;
  float M = kMInit;
  for (int i = lane; i < n_splits; i += 64) M = fmaxf(M, ml[2 * i]);
  M = across_groups_max<1>(M);
  float L = 0.0f, acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.0f;
  for (int i = 0; i < n_splits; ++i) {
    const float c = fast_exp2(ml[2 * i] - M);
    L = fmaf(ml[2 * i + 1], c, L);
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] = fmaf(o[(int64_t)i * D + lane * E + e], c, acc[e]);
  }
  T* out = reinterpret_cast<T*>(a.out) + (int64_t)item * D;
#pragma unroll
  for (int e = 0; e < E; ++e) store_out<T>(out + lane * E + e, acc[e] / L);
}

// ---- launchers -----------------------------------------------------------

template <typename T, int D, bool TR>
static const void* decode_pick(int s) {
  switch (s) {
    case 1: return reinterpret_cast<const void*>(&decode_kernel<T, D, 1, kDecodeWaves, kDecodeRing, TR>);
    case 2: return reinterpret_cast<const void*>(&decode_kernel<T, D, 2, kDecodeWaves, kDecodeRing, TR>);
    case 4: return reinterpret_cast<const void*>(&decode_kernel<T, D, 4, kDecodeWaves, kDecodeRing, TR>);
    case 6: return reinterpret_cast<const void*>(&decode_kernel<T, D, 6, kDecodeWaves, kDecodeRing, TR>);
    case 8: return reinterpret_cast<const void*>(&decode_kernel<T, D, 8, kDecodeWaves, kDecodeRing, TR>);
  }
  return nullptr;
}

template <typename T, int D>
static const void* decode_fn(int s, bool trace) { return trace ? decode_pick<T, D, true>(s) : decode_pick<T, D, false>(s); }

hipError_t launch_decode(int dtype, int D, int s, const DecodeArgs& a, int rows, hipStream_t st, KernelEvents ev) {
  const void* fn = nullptr;
  const bool tr = a.trace != nullptr;
  if (dtype == 0 && D == 128) fn = decode_fn<uint16_t, 128>(s, tr);
  else if (dtype == 0 && D == 64) fn = decode_fn<uint16_t, 64>(s, tr);
  else if (dtype == 1 && D == 128) fn = decode_fn<float, 128>(s, tr);
  else if (dtype == 1 && D == 64) fn = decode_fn<float, 64>(s, tr);
  if (fn == nullptr) return hipErrorInvalidValue;
  const int64_t n = (int64_t)rows * a.H_kv * a.n_split_slots;
  if (n == 0) return hipSuccess;
  if (n > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  DecodeArgs a0 = a;
  void* args[] = {&a0};
  hipError_t e = hipExtLaunchKernel(fn, dim3((unsigned)n), dim3(64 * kDecodeWaves), args, 0, st, ev.start, ev.stop, 0);
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

hipError_t launch_reduce(int dtype, int D, const ReduceArgs& a, hipStream_t st) {
  const dim3 grid((unsigned)(((int64_t)a.rows * a.H_q + 3) / 4)), block(256);
  if (grid.x == 0) return hipSuccess;
  if (dtype == 0 && D == 128) reduce_kernel<uint16_t, 128><<<grid, block, 0, st>>>(a);
  else if (dtype == 0 && D == 64) reduce_kernel<uint16_t, 64><<<grid, block, 0, st>>>(a);
  else if (dtype == 1 && D == 128) reduce_kernel<float, 128><<<grid, block, 0, st>>>(a);
  else if (dtype == 1 && D == 64) reduce_kernel<float, 64><<<grid, block, 0, st>>>(a);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace pa
