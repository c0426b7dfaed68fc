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
// (wave-uniform), then each lane moves 16-byte chunks of K and V, consecutive
// lanes covering a (row, head) vector's contiguous bytes on both the read and
// the write side.  The kernel is HBM-bound: per appended token it reads and
// writes H_kv * D * 2 elements.
#include "pa_device.h"
#include "pa_kernels.h"

namespace pa {

namespace {

constexpr int kAppendWaves = 4;  // rows per workgroup pass (one wave per row)
constexpr int kAppendMaxGrid = 2048;

__global__ __launch_bounds__(64 * kAppendWaves) void kv_append_kernel(AppendArgs a) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int CH = a.row_bytes / 16;  // 16-byte chunks per (row, head) vector
  const int n = a.H_kv * CH;        // chunks per row (all KV heads)
  const BlockTable bt{a.block_table, a.bt_stride};
  for (int row = blockIdx.x * kAppendWaves + wave; row < a.rows; row += gridDim.x * kAppendWaves) {
    // the row's sequence b, its chunk length L and its index j in the chunk
    // (wave-uniform)
    int b, L, j;
    if (a.query_start_loc != nullptr) {
      int lo = 0, hi = a.B - 1;  // largest b with query_start_loc[b] <= row
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (a.query_start_loc[mid] <= row) lo = mid; else hi = mid - 1;
      }
      b = lo;
      L = a.query_start_loc[b + 1] - a.query_start_loc[b];
      j = row - a.query_start_loc[b];
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
    const uint8_t* ks = a.k_new + (int64_t)row * n * 16;
    const uint8_t* vs = a.v_new + (int64_t)row * n * 16;
    // [page][g][slot] vectors of the pool: head g's vector starts at
    // ((page * H_kv + g) * 16 + slot) * row_bytes
    const int64_t dst0 = ((int64_t)page * a.H_kv * kPage + (pos & (kPage - 1))) * a.row_bytes;
    for (int c = lane; c < n; c += 64) {
      const int g = c / CH, cc = c - g * CH;
      const int64_t dst = dst0 + (int64_t)g * kPage * a.row_bytes + cc * 16;
      const u32x4 kv = *reinterpret_cast<const u32x4*>(ks + c * 16);
      const u32x4 vv = *reinterpret_cast<const u32x4*>(vs + c * 16);
      *reinterpret_cast<u32x4*>(a.k_pages + dst) = kv;
      *reinterpret_cast<u32x4*>(a.v_pages + dst) = vv;
    }
  }
}

}  // namespace

hipError_t launch_kv_append(const AppendArgs& a, hipStream_t st) {
  if (a.rows == 0) return hipSuccess;
  const int blocks = (a.rows + kAppendWaves - 1) / kAppendWaves;
  const int grid = blocks < kAppendMaxGrid ? blocks : kAppendMaxGrid;
  kv_append_kernel<<<grid, 64 * kAppendWaves, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace pa
