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

namespace pa {

template <typename T, int D, int S>
struct DecodeShape {
  static constexpr int VEC = 16 / (int)sizeof(T);  // elements per 16-byte lane load
  static constexpr int LPT = D / VEC;              // lanes per token row
  static constexpr int TPI = 64 / LPT;             // token rows per wave-wide load
  static constexpr int NI = kPage / TPI;           // loads per 16-token tile
  static_assert(LPT >= 2 && LPT <= 32 && 64 % LPT == 0 && kPage % TPI == 0, "unsupported shape");
};

// Partial dot product of the lane's VEC query elements with VEC key elements.
__device__ __forceinline__ float lane_dot(const u32x4& q, const u32x4& k, uint16_t) {
  float acc = 0.0f;
  acc = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(q.x), as_bf16x2(k.x), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(q.y), as_bf16x2(k.y), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(q.z), as_bf16x2(k.z), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(q.w), as_bf16x2(k.w), acc, false);
  return acc;
}
__device__ __forceinline__ float lane_dot(const u32x4& q, const u32x4& k, float) {
  float acc = __uint_as_float(q.x) * __uint_as_float(k.x);
  acc = fmaf(__uint_as_float(q.y), __uint_as_float(k.y), acc);
  acc = fmaf(__uint_as_float(q.z), __uint_as_float(k.z), acc);
  acc = fmaf(__uint_as_float(q.w), __uint_as_float(k.w), acc);
  return acc;
}

// Widen the lane's VEC value elements to fp32.
__device__ __forceinline__ void widen(const u32x4& v, float* f, uint16_t) {
  f[0] = bf16_lo(v.x); f[1] = bf16_hi(v.x);
  f[2] = bf16_lo(v.y); f[3] = bf16_hi(v.y);
  f[4] = bf16_lo(v.z); f[5] = bf16_hi(v.z);
  f[6] = bf16_lo(v.w); f[7] = bf16_hi(v.w);
}
__device__ __forceinline__ void widen(const u32x4& v, float* f, float) {
  f[0] = __uint_as_float(v.x); f[1] = __uint_as_float(v.y);
  f[2] = __uint_as_float(v.z); f[3] = __uint_as_float(v.w);
}

template <typename T, int D, int S>
struct DecodeState {
  using Sh = DecodeShape<T, D, S>;
  u32x4 q[S];                  // lane's slice of the s query vectors (raw)
  float o[S][Sh::VEC];         // unnormalised output slice per head
  float m[S], l[S];            // running max (log2 units) and sum per head
};

// One (page, g) tile: NI K loads and NI V loads per lane.
template <typename T, int D, int S>
__device__ __forceinline__ void load_tile(const T* __restrict__ kp, const T* __restrict__ vp,
                                          int64_t tile, int lane, u32x4 (&k)[DecodeShape<T, D, S>::NI],
                                          u32x4 (&v)[DecodeShape<T, D, S>::NI]) {
  using Sh = DecodeShape<T, D, S>;
  const u32x4* kt = reinterpret_cast<const u32x4*>(kp + tile) + lane;
  const u32x4* vt = reinterpret_cast<const u32x4*>(vp + tile) + lane;
#pragma unroll
  for (int i = 0; i < Sh::NI; ++i) k[i] = __builtin_nontemporal_load(kt + 64 * i);
#pragma unroll
  for (int i = 0; i < Sh::NI; ++i) v[i] = __builtin_nontemporal_load(vt + 64 * i);
}

// Fold one tile into the running state.  MASKED: tokens at or past `ctx`
// (only in a sequence's last page) get logit -inf and value 0, so whatever
// bytes the unused slots hold (even NaN) cannot reach the result.
template <typename T, int D, int S, bool MASKED>
__device__ __forceinline__ void process_tile(DecodeState<T, D, S>& st,
                                             const u32x4 (&k)[DecodeShape<T, D, S>::NI],
                                             u32x4 (&v)[DecodeShape<T, D, S>::NI], int row,
                                             int first_token, int ctx, float scale_log2) {
  using Sh = DecodeShape<T, D, S>;
  float x[S][Sh::NI];
#pragma unroll
  for (int i = 0; i < Sh::NI; ++i)
#pragma unroll
    for (int j = 0; j < S; ++j) x[j][i] = lane_dot(st.q[j], k[i], T());
#pragma unroll
  for (int i = 0; i < Sh::NI; ++i)
#pragma unroll
    for (int j = 0; j < S; ++j) x[j][i] = group_sum<Sh::LPT>(x[j][i]) * scale_log2;
  if constexpr (MASKED) {
#pragma unroll
    for (int i = 0; i < Sh::NI; ++i) {
      const bool dead = first_token + row + Sh::TPI * i >= ctx;
#pragma unroll
      for (int j = 0; j < S; ++j) x[j][i] = dead ? -INFINITY : x[j][i];
      v[i].x = dead ? 0u : v[i].x;
      v[i].y = dead ? 0u : v[i].y;
      v[i].z = dead ? 0u : v[i].z;
      v[i].w = dead ? 0u : v[i].w;
    }
  }
  float vf[Sh::NI][Sh::VEC];
#pragma unroll
  for (int i = 0; i < Sh::NI; ++i) widen(v[i], vf[i], T());
#pragma unroll
  for (int j = 0; j < S; ++j) {
    float mx = x[j][0];
#pragma unroll
    for (int i = 1; i < Sh::NI; ++i) mx = fmaxf(mx, x[j][i]);
    const float mnew = fmaxf(st.m[j], mx);
    const float alpha = fast_exp2(st.m[j] - mnew);
    st.m[j] = mnew;
    float p[Sh::NI];
    float psum = 0.0f;
#pragma unroll
    for (int i = 0; i < Sh::NI; ++i) {
      p[i] = fast_exp2(x[j][i] - mnew);
      psum += p[i];
    }
    st.l[j] = fmaf(st.l[j], alpha, psum);
#pragma unroll
    for (int e = 0; e < Sh::VEC; ++e) {
      float acc = st.o[j][e] * alpha;
#pragma unroll
      for (int i = 0; i < Sh::NI; ++i) acc = fmaf(p[i], vf[i][e], acc);
      st.o[j][e] = acc;
    }
  }
}

// Sequence b and visible-key count n_vis of query row `row`.  Decode: row = b
// and all ctx keys are visible.  Varlen: b is the largest sequence with
// query_start_loc[b] <= row, and row r of a chunk of length L sees keys
// 0 .. ctx - L + r.  Returns false when the row breaks the call's contract
// (negative length, a context above max_context_len, a chunk longer than its
// context); such rows are written as NaN by the attention kernel and left
// alone by the reduction.
__device__ __forceinline__ bool row_context(const int32_t* __restrict__ qsl,
                                            const int32_t* __restrict__ context_lens, int B,
                                            int max_context_len, int row, int& b, int& n_vis) {
  if (qsl == nullptr) {
    b = row;
    n_vis = context_lens[row];
    return n_vis >= 0 && n_vis <= max_context_len;
  }
  int lo = 0, hi = B - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (qsl[mid] <= row) lo = mid; else hi = mid - 1;
  }
  b = lo;
  const int ctx = context_lens[b];
  const int L = qsl[b + 1] - qsl[b];
  n_vis = ctx - L + (row - qsl[b]) + 1;
  return ctx >= 0 && ctx <= max_context_len && n_vis >= 1;
}

template <typename T, int D, int S, int WAVES>
__global__ __launch_bounds__(64 * WAVES) void decode_kernel(DecodeArgs a) {
  using Sh = DecodeShape<T, D, S>;
  constexpr int NT = 64 * WAVES;
  __shared__ float sm_o[WAVES][S][D];
  __shared__ float sm_ml[WAVES][S][2];

  const int split = blockIdx.x % a.n_split_slots;
  const int rest = blockIdx.x / a.n_split_slots;
  const int g = rest % a.H_kv, row_idx = rest / a.H_kv;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  int b, ctx;  // ctx: keys this row sees
  const bool ok = row_context(a.query_start_loc, a.context_lens, a.B, a.max_context_len, row_idx, b, ctx);
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
  const int last_page = n_pages - 1;
  const bool ragged = (ctx % kPage) != 0;

  auto tile_of = [&](int kk) {
    const int32_t page = __builtin_amdgcn_readlane(bt_lane, kk);
    return tile_offset(page, g, a.H_kv, D);
  };
  auto fold = [&](const u32x4 (&kr)[Sh::NI], u32x4 (&vr)[Sh::NI], int kk) {
    const int p = p0 + wave + WAVES * kk;
    if (ragged && p == last_page)
      process_tile<T, D, S, true>(st, kr, vr, row, p * kPage, ctx, a.scale_log2);
    else
      process_tile<T, D, S, false>(st, kr, vr, row, p * kPage, ctx, a.scale_log2);
  };

  // Two register buffers: the next tile's loads are in flight while the
  // current one is folded.
  u32x4 kA[Sh::NI], vA[Sh::NI], kB[Sh::NI], vB[Sh::NI];
  if (my_n > 0) load_tile<T, D, S>(kp, vp, tile_of(0), lane, kA, vA);
  for (int kk = 0; kk < my_n; kk += 2) {
    if (kk + 1 < my_n) load_tile<T, D, S>(kp, vp, tile_of(kk + 1), lane, kB, vB);
    fold(kA, vA, kk);
    if (kk + 1 < my_n) {
      if (kk + 2 < my_n) load_tile<T, D, S>(kp, vp, tile_of(kk + 2), lane, kA, vA);
      fold(kB, vB, kk + 1);
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

// Gather trace: rows_out[row_start[b] + t] = pool row of token t of sequence b,
// through the same BlockTable / pool_row functions the attention kernels use.
__global__ __launch_bounds__(256) void gather_trace_kernel(BlockTable bt, const int32_t* context_lens,
                                                           const int64_t* row_start, int64_t* rows_out) {
  const int b = blockIdx.y;
  const int t = blockIdx.x * 256 + threadIdx.x;
  const int ctx = context_lens[b];
  if (t >= ctx) return;
  // a context longer than the block-table row is a contract violation: -1
  rows_out[row_start[b] + t] = t / kPage < bt.stride ? pool_row(bt.page(b, t / kPage), t) : -1;
}

// ---- launchers -----------------------------------------------------------

template <typename T, int D>
static hipError_t decode_s(int s, const DecodeArgs& a, int rows, hipStream_t st) {
  const int64_t n = (int64_t)rows * a.H_kv * a.n_split_slots;
  if (n == 0) return hipSuccess;
  if (n > 0x7fffffffLL) return hipErrorInvalidConfiguration;
  const dim3 grid((unsigned)n), block(64 * kDecodeWaves);
  switch (s) {
    case 1: decode_kernel<T, D, 1, kDecodeWaves><<<grid, block, 0, st>>>(a); break;
    case 2: decode_kernel<T, D, 2, kDecodeWaves><<<grid, block, 0, st>>>(a); break;
    case 4: decode_kernel<T, D, 4, kDecodeWaves><<<grid, block, 0, st>>>(a); break;
    case 6: decode_kernel<T, D, 6, kDecodeWaves><<<grid, block, 0, st>>>(a); break;
    case 8: decode_kernel<T, D, 8, kDecodeWaves><<<grid, block, 0, st>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_decode(int dtype, int D, int s, const DecodeArgs& a, int rows, hipStream_t st) {
  if (dtype == 0 && D == 128) return decode_s<uint16_t, 128>(s, a, rows, st);
  if (dtype == 0 && D == 64) return decode_s<uint16_t, 64>(s, a, rows, st);
  if (dtype == 1 && D == 128) return decode_s<float, 128>(s, a, rows, st);
  if (dtype == 1 && D == 64) return decode_s<float, 64>(s, a, rows, st);
  return hipErrorInvalidValue;
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

hipError_t launch_gather_trace(const int32_t* block_table, int64_t bt_stride,
                               const int32_t* context_lens, const int64_t* row_start, int B,
                               int max_context_len, int64_t* rows_out, hipStream_t st) {
  if (B == 0 || max_context_len == 0) return hipSuccess;
  const dim3 grid((max_context_len + 255) / 256, B), block(256);
  gather_trace_kernel<<<grid, block, 0, st>>>(BlockTable{block_table, bt_stride}, context_lens,
                                              row_start, rows_out);
  return hipGetLastError();
}

}  // namespace pa
