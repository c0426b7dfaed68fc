// KV append: the cache write that precedes attention.
//
// A token's K/V are in the paged cache when attention reads them (MoE-Lens
// Sec. 6.4: the task receiving a decode token's pre-attention K/V stores it in
// the KV cache, then attends; Sec. 5.5 paging).  Sequence b appends L_b new
// tokens at the last L_b positions of its context: row query_start_loc[b] + j
// goes to position context_lens[b] - L_b + j (decode layout: row b, position
// context_lens[b] - 1, nothing for an empty context).  Each (row, KV head)
// vector of D elements lands in slot position % 16 of page
// block_table[b][position / 16], KV head g.
//
// One wave per new row: the row's sequence, position and page are found once
// (wave-uniform; a varlen row's sequence by a binary search over
// query_start_loc, staged in LDS), then each lane moves 16-byte chunks of K
// and V, consecutive lanes covering a (row, head) vector's contiguous bytes on
// both the read and the write side.  Per appended token it reads and writes
// H_kv * D * 2 elements; at decode batch sizes that is a few MiB, and the
// kernel's time is its launch and its chain of dependent reads.
#include "pa_device.h"
#include "pa_kernels.h"

namespace pa {

namespace {

constexpr int kAppendWaves = 4;  // rows per workgroup pass (one wave per row)
constexpr int kAppendMaxGrid = 2048;
constexpr int kAppendMaxLdsSeqs = 16383;  // query_start_loc staged in LDS up to this many sequences

// LDS_QSL: varlen rows find their sequence by a binary search over
// query_start_loc staged in LDS (one cooperative read per workgroup) rather
// than over global memory (one dependent read per search step).
template <bool LDS_QSL>
__global__ __launch_bounds__(64 * kAppendWaves) void kv_append_kernel(AppendArgs a) {
  extern __shared__ int32_t s_qsl[];  // [B + 1] when LDS_QSL
  if constexpr (LDS_QSL) {
    // four independent reads per thread and pass (the entries past B read as
    // entry B, the last valid one, and are not stored)
    constexpr int NT = 64 * kAppendWaves;
    for (int i0 = threadIdx.x; i0 <= a.B; i0 += 4 * NT) {
      int32_t v[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = a.query_start_loc[min(i0 + u * NT, a.B)];
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (i0 + u * NT <= a.B) s_qsl[i0 + u * NT] = v[u];
    }
    __syncthreads();
  }
  const int32_t* qsl = LDS_QSL ? s_qsl : a.query_start_loc;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int CH = a.row_bytes / 16;  // 16-byte chunks per (row, head) vector
  const int n = a.H_kv * CH;        // chunks per row (all KV heads)
  const BlockTable bt{a.block_table, a.bt_stride};
  for (int row = blockIdx.x * kAppendWaves + wave; row < a.rows; row += gridDim.x * kAppendWaves) {
    // The row's first 128 chunks of K and V are loaded before the lookups:
    // they depend on the row alone, so their latency overlaps the chain
    // sequence -> position -> page (two dependent reads) instead of
    // following it.
    const uint8_t* ks = a.k_new + (int64_t)row * n * 16;
    const uint8_t* vs = a.v_new + (int64_t)row * n * 16;
    u32x4 kv[2], vv[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = lane + 64 * i;
      if (c < n) {
        kv[i] = *reinterpret_cast<const u32x4*>(ks + c * 16);
        vv[i] = *reinterpret_cast<const u32x4*>(vs + c * 16);
      }
    }
    // the row's sequence b, its chunk length L and its index j in the chunk
    // (wave-uniform)
    int b, L, j;
    if (a.query_start_loc != nullptr) {
      int lo = 0, hi = a.B - 1;  // largest b with query_start_loc[b] <= row
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (qsl[mid] <= row) lo = mid; else hi = mid - 1;
      }
      b = lo;
      L = qsl[b + 1] - qsl[b];
      j = row - qsl[b];
    } else {
      b = row;
      L = a.context_lens[b] > 0 ? 1 : 0;
      j = 0;
    }
    const int C = a.context_lens[b];
    // contract violations write nothing
    if (j < 0 || j >= L || L > C || C > a.max_context_len) continue;
    const int pos = C - L + j;
    if (pos / kPage >= a.bt_stride) continue;
    const int32_t page = bt.page(b, pos / kPage);
    if (page < 0 || page >= a.num_pages) continue;
    // [page][g][slot] vectors of the pool: head g's vector starts at
    // ((page * H_kv + g) * 16 + slot) * row_bytes
    const int64_t dst0 = ((int64_t)page * a.H_kv * kPage + (pos & (kPage - 1))) * a.row_bytes;
    auto dst = [&](int c) {
      const int g = c / CH, cc = c - g * CH;
      return dst0 + (int64_t)g * kPage * a.row_bytes + cc * 16;
    };
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int c = lane + 64 * i;
      if (c < n) {
        *reinterpret_cast<u32x4*>(a.k_pages + dst(c)) = kv[i];
        *reinterpret_cast<u32x4*>(a.v_pages + dst(c)) = vv[i];
      }
    }
    for (int c = lane + 128; c < n; c += 64) {  // rows wider than 128 chunks
      const u32x4 k1 = *reinterpret_cast<const u32x4*>(ks + c * 16);
      const u32x4 v1 = *reinterpret_cast<const u32x4*>(vs + c * 16);
      *reinterpret_cast<u32x4*>(a.k_pages + dst(c)) = k1;
      *reinterpret_cast<u32x4*>(a.v_pages + dst(c)) = v1;
    }
  }
}

}  // namespace

hipError_t launch_kv_append(const AppendArgs& a, hipStream_t st) {
  if (a.rows == 0) return hipSuccess;
  const int blocks = (a.rows + kAppendWaves - 1) / kAppendWaves;
  const int grid = blocks < kAppendMaxGrid ? blocks : kAppendMaxGrid;
  if (a.query_start_loc != nullptr && a.B <= kAppendMaxLdsSeqs)
    kv_append_kernel<true><<<grid, 64 * kAppendWaves, (size_t)(a.B + 1) * sizeof(int32_t), st>>>(a);
  else
    kv_append_kernel<false><<<grid, 64 * kAppendWaves, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace pa
