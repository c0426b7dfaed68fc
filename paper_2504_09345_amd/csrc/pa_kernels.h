// Host-side launchers of the gfx950 kernels (internal to libpagedattn.so).
#pragma once

#include <hip/hip_ext.h>

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pa {

// Arguments of the split-K attention kernel.  Flat grid of
// n_split_slots * H_kv * rows workgroups; workgroup id = (row * H_kv + g) *
// n_split_slots + split attends the s = H_q / H_kv query heads of KV head g
// for query row `row` over pages [split * pages_per_split, +pages_per_split)
// of the keys that row may see.  Decode: row = sequence.  Varlen: the row's
// sequence is found in query_start_loc and its causal limit applied.
struct DecodeArgs {
  const void* q;             // [rows][H_q][D]
  const void* k_pages;       // [num_pages][H_kv][16][D]
  const void* v_pages;
  const int32_t* block_table;
  const int32_t* context_lens;
  const int32_t* query_start_loc;  // [B+1] for varlen, nullptr for decode
  void* out;                 // [rows][H_q][D]
  float* ws_o;               // [rows][H_q][n_split_slots][D] partial outputs (unnormalised)
  float* ws_ml;              // [rows][H_q][n_split_slots][2] (running max in log2 units, sum)
  int64_t bt_stride;         // max_pages_per_seq
  float scale_log2;          // scale * log2(e)
  int B;                     // sequences
  int max_context_len;       // declared bound; longer contexts are flagged
  int H_q, H_kv;
  int pages_per_split;
  int n_split_slots;
  int skip_single_rows;      // varlen: leave one-row sequences to the stream kernel
  int64_t* trace;            // gather-trace launches only (see StreamArgs), else nullptr
};

struct ReduceArgs {
  const float* ws_o;
  const float* ws_ml;
  const int32_t* context_lens;
  const int32_t* query_start_loc;  // nullptr for decode
  void* out;
  int B, rows, H_q;
  int max_context_len;
  int pages_per_split;
  int n_split_slots;
  int skip_single_rows;
};

// Arguments of the persistent stream-K kernel.  Items are
// (sequence, KV head); for varlen calls only sequences with exactly one
// query row are taken (chunked prefill rows go to the per-row kernel).
struct StreamArgs {
  const void* q;
  const void* k_pages;
  const void* v_pages;
  const int32_t* block_table;
  const int32_t* context_lens;
  const int32_t* query_start_loc;  // nullptr for decode
  void* out;
  float* ws_o;       // [G][2][W][s][D] partial outputs (slot 0 head, 1 tail)
  float* ws_ml;      // [G][2][W][s][2]
  unsigned long long* ws_flag;  // [G][W] arrival counters of cut items, keyed by the item's first range
  unsigned long long token;     // tag of this call (never 0; differs from every earlier call's)
  int64_t bt_stride;
  float scale_log2;
  int B, H_q, H_kv, max_context_len;
  int nb;            // head blocks = H_kv / W
  // Gather trace (nullptr in attention calls): [H_kv][B][bt_stride * 16]
  // int64, the pool row ((page * H_kv + g) * 16 + slot) each loaded token came
  // from; launched through the trace instantiations of the kernels.
  int64_t* trace;
};

constexpr int kStreamMaxRows = 8192;    // sequences per call on the stream path
constexpr int kStreamMaxUnits = 2048;   // units per workgroup range (LDS unit table)
constexpr int kStreamMaxGrid = 1024;    // persistent workgroups (partial-record space)
#ifndef PA_STREAM_RING
#define PA_STREAM_RING 2
#endif
constexpr int kStreamRing = PA_STREAM_RING;
#ifndef PA_STREAM_SPLIT_KV
#define PA_STREAM_SPLIT_KV 1
#endif
// Stream-K kernel with the matrix-core fold: load a unit's K and V tiles
// half a unit apart (about one tile of each in flight per wave) rather than
// through the NBUF ring.  The mixed kernel keeps the ring.
constexpr bool kStreamSplitKV = PA_STREAM_SPLIT_KV != 0;
#ifndef PA_STREAM_MAX_WAVES
#define PA_STREAM_MAX_WAVES 8
#endif
constexpr int kStreamMaxWaves = PA_STREAM_MAX_WAVES;  // waves (KV heads) per stream workgroup
#ifndef PA_STREAM_MFMA
#define PA_STREAM_MFMA 1
#endif
constexpr bool kStreamMfma = PA_STREAM_MFMA != 0;  // bf16 D = 128 tiles on the matrix cores

// Optional events bracketing one kernel's execution (hipExtLaunchKernel's
// start/stop events: taken when the kernel starts and ends, not when the
// stream reaches the launch).  Null members record nothing.
struct KernelEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};

hipError_t launch_stream(int dtype, int D, int s, int W, const StreamArgs& a, int G, hipStream_t st,
                         KernelEvents ev = {});
int stream_occupancy(int dtype, int D, int s, int W);  // workgroups per CU, 0 on error
// Stream-K kernel for (element type, head dim, trace): pick by s and W (one
// translation unit per combination, compiled in parallel).
template <typename T, int D, bool TR> const void* stream_pick(int s, int W);

// Arguments of the MFMA chunked-prefill kernel (bf16, head_dim 128): the rows
// of every sequence with a chunk of L > 1 query rows.
struct PrefillArgs {
  const void* q;
  const void* k_pages;
  const void* v_pages;
  const int32_t* block_table;
  const int32_t* context_lens;
  const int32_t* query_start_loc;
  void* out;
  int64_t bt_stride;
  float scale_log2;
  int B, H_q, H_kv, max_context_len;
  int64_t* trace;  // gather-trace launches only (see StreamArgs), else nullptr
};

bool prefill_supported(int dtype, int D, int s);

// Mixed batch in one launch: G_dec stream-K decode workgroups and G - G_dec
// prefill workgroups (bf16, head_dim 128, W = 8 decode waves).
bool mixed_supported(int dtype, int D, int s, int W);
hipError_t launch_mixed(int s, const StreamArgs& sa, const PrefillArgs& pa, int G_dec, int G, hipStream_t st,
                        KernelEvents ev = {});
int prefill_occupancy(int s, int B);  // workgroups per CU, 0 on error
hipError_t launch_prefill(int s, const PrefillArgs& a, int G, hipStream_t st, KernelEvents ev = {});

// Arguments of the KV-append (cache write) kernel.  query_start_loc == nullptr
// is the decode layout (row b appends position context_lens[b] - 1).
struct AppendArgs {
  const uint8_t* k_new;
  const uint8_t* v_new;
  uint8_t* k_pages;
  uint8_t* v_pages;
  const int32_t* block_table;
  const int32_t* context_lens;
  const int32_t* query_start_loc;
  int64_t bt_stride;
  int B, rows, H_kv, row_bytes, num_pages, max_context_len;
};

hipError_t launch_kv_append(const AppendArgs& a, hipStream_t st);

// dtype: 0 bf16, 1 fp32.  Return hipSuccess or the launch error.
hipError_t launch_decode(int dtype, int D, int s, const DecodeArgs& a, int rows, hipStream_t st,
                         KernelEvents ev = {});
hipError_t launch_reduce(int dtype, int D, const ReduceArgs& a, hipStream_t st);
// Fill n int64 entries with `value` (the gather trace's starting state).
hipError_t launch_fill_i64(int64_t* p, int64_t n, int64_t value, hipStream_t st);

// Maximum pages a workgroup's split may span (block-table entries are held one
// per lane of each wave).
#ifndef PA_DECODE_WAVES
#define PA_DECODE_WAVES 4
#endif
#ifndef PA_DECODE_RING
#define PA_DECODE_RING 2
#endif
constexpr int kDecodeWaves = PA_DECODE_WAVES;  // waves per workgroup sharing one split
constexpr int kDecodeRing = PA_DECODE_RING;    // register tile buffers per wave
constexpr int kMaxPagesPerSplit = 64 * kDecodeWaves;

}  // namespace pa
