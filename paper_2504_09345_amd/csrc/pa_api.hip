// C ABI of libpagedattn.so: host-side validation, launch planning and
// dispatch.  Validation runs before any HIP call, so a rejected call enqueues
// nothing and is testable without a GPU.  The library allocates nothing; its
// only state between calls is the counter that tags each call's range flags.
#include <climits>
#include <math.h>
#include <stddef.h>
#include <stdint.h>

#include <atomic>
#include <chrono>
#include <mutex>

#include "pa_kernels.h"
#include "pa_sched.h"
#include "pagedattn.h"

namespace {

// Split-K granule of the per-row path when the caller leaves it to the
// library: 128 pages = 2048 tokens per workgroup (32 pages per wave).
constexpr int kDefaultPagesPerSplit = 128;

// Share of the CUs that run the persistent stream-K decode grid.
#ifndef PA_STREAM_CU_NUM
#define PA_STREAM_CU_NUM 13
#endif
#ifndef PA_STREAM_CU_DEN
#define PA_STREAM_CU_DEN 16
#endif
constexpr int kStreamCuNum = PA_STREAM_CU_NUM, kStreamCuDen = PA_STREAM_CU_DEN;
// share of the CUs the mixed launch gives the prefill chunks
#ifndef PA_MIXED_PF_NUM
#define PA_MIXED_PF_NUM 1
#endif
#ifndef PA_MIXED_PF_DEN
#define PA_MIXED_PF_DEN 4
#endif

struct Plan {
  int s = 0;
  int rows = 0;
  // stream-K path (decode rows)
  bool stream = false;
  int W = 0, nb = 0;
  int64_t g_min = 0;  // persistent workgroups needed to keep every range within the LDS unit table
  size_t st_o = 0, st_ml = 0, st_cum = 0;
  // MFMA prefill path (chunk rows of a varlen call)
  bool prefill = false;
  // split-K path (all rows of a decode call that the stream path cannot take,
  // or the chunked-prefill rows of a varlen call the MFMA path cannot take)
  bool split = false;
  int pps = 0;
  int n_split_slots = 0;
  size_t sp_o = 0, sp_ml = 0;
  size_t ws_bytes = 0;
};

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

bool group_supported(int s) { return s == 1 || s == 2 || s == 4 || s == 6 || s == 8; }

int plan(const pa_dims_t* d, bool varlen, Plan* p) {
  if (d == nullptr || p == nullptr) return PA_EINVAL;
  if (d->num_seqs < 0 || d->num_q_heads <= 0 || d->num_kv_heads <= 0 || d->num_pages < 0 ||
      d->max_pages_per_seq < 0 || d->max_context_len < 0 || d->pages_per_split < 0)
    return PA_EINVAL;
  if (d->num_q_heads % d->num_kv_heads != 0) return PA_EINVAL;
  if (d->dtype != PA_BF16 && d->dtype != PA_FP32) return PA_ENOTSUP;
  if (d->head_dim != 64 && d->head_dim != 128) return PA_ENOTSUP;
  if (d->page_size != 16) return PA_ENOTSUP;
  const int s = d->num_q_heads / d->num_kv_heads;
  if (!group_supported(s)) return PA_ENOTSUP;
  const int64_t max_pages = ((int64_t)d->max_context_len + 15) / 16;
  if (max_pages > d->max_pages_per_seq) return PA_EINVAL;
  if (d->pages_per_split > pa::kMaxPagesPerSplit) return PA_EINVAL;
  int rows;
  if (varlen) {
    if (d->num_q_rows < 0 || d->max_q_len < 0) return PA_EINVAL;
    if (d->num_q_rows > 0 && (d->max_q_len < 1 || d->num_seqs == 0)) return PA_EINVAL;
    if (d->max_q_len > d->max_context_len && d->num_q_rows > 0) return PA_EINVAL;
    rows = d->num_q_rows;
  } else {
    if (!(d->num_q_rows == 0 || d->num_q_rows == d->num_seqs)) return PA_EINVAL;
    if (!(d->max_q_len == 0 || d->max_q_len == 1)) return PA_EINVAL;
    rows = d->num_seqs;
  }
  p->s = s;
  p->rows = rows;

  // stream-K: W = widest power of two <= 8 dividing H_kv waves per workgroup
  p->W = (d->num_kv_heads % 8 == 0 && pa::kStreamMaxWaves >= 8) ? 8
         : (d->num_kv_heads % 4 == 0 && pa::kStreamMaxWaves >= 4) ? 4
         : (d->num_kv_heads % 2 == 0 && pa::kStreamMaxWaves >= 2) ? 2 : 1;
  p->nb = d->num_kv_heads / p->W;
  const int64_t u_max = (int64_t)p->nb * d->num_seqs * max_pages;
  p->g_min = (u_max + pa::kStreamMaxUnits - 1) / pa::kStreamMaxUnits;
  // an explicit split granule asks for the split-K path
  p->stream = d->pages_per_split == 0 && d->num_seqs <= pa::kStreamMaxRows && p->nb < 64 &&
              rows < (1 << 19) && p->g_min <= pa::kStreamMaxGrid;
  if (p->stream) {
    const size_t recs = (size_t)pa::kStreamMaxGrid * 2 * p->W * s;  // (workgroup, slot, wave, head)
    p->st_o = align256(recs * (size_t)d->head_dim * sizeof(float));
    p->st_ml = align256(recs * 2 * sizeof(float));
    // arrival counters of cut items: one per (first range, wave)
    p->st_cum = align256((size_t)pa::kStreamMaxGrid * p->W * sizeof(unsigned long long));
  }
  // chunked-prefill rows of a varlen call: MFMA kernel (bf16, head_dim 128)
  p->prefill = varlen && p->stream && pa::prefill_supported(d->dtype, d->head_dim, s);
  // split-K for whatever the stream and prefill paths do not take: in a
  // varlen call, chunk rows the MFMA kernel cannot take (there are none when
  // max_q_len <= 1: every row is then a decode row, which the stream kernel
  // takes)
  p->split = varlen ? (rows > 0 && !p->prefill && (d->max_q_len > 1 || !p->stream)) : !p->stream;
  p->pps = d->pages_per_split > 0 ? d->pages_per_split : kDefaultPagesPerSplit;
  p->n_split_slots = (int)((max_pages + p->pps - 1) / p->pps);
  if (p->n_split_slots < 1) p->n_split_slots = 1;
  if (p->split) {
    if ((int64_t)rows * d->num_kv_heads * p->n_split_slots > 0x7fffffffLL) return PA_ENOTSUP;
    if (p->n_split_slots > 1) {
      const size_t items = (size_t)rows * (size_t)d->num_q_heads * (size_t)p->n_split_slots;
      p->sp_o = align256(items * (size_t)d->head_dim * sizeof(float));
      p->sp_ml = align256(items * 2 * sizeof(float));
    }
  }
  if (rows == 0) {  // nothing to launch, nothing to hold
    p->stream = p->split = p->prefill = false;
    p->st_o = p->st_ml = p->st_cum = p->sp_o = p->sp_ml = 0;
  }
  p->ws_bytes = p->st_o + p->st_ml + p->st_cum + p->sp_o + p->sp_ml;
  return PA_OK;
}

// Tag of one call's arrival counters in the workspace: process-wide, never 0
// and never repeated, so counters left in a reused workspace by earlier calls
// (or found in a fresh one) do not match.  This counter is the library's only
// state besides the fixed scratch below; it does not influence any result.
unsigned long long next_token() {
  static std::atomic<unsigned long long> counter{
      0x9e3779b97f4a7c15ull ^
      (unsigned long long)std::chrono::steady_clock::now().time_since_epoch().count()};
  unsigned long long t = counter.fetch_add(1, std::memory_order_relaxed) + 1;
  return t != 0 ? t : counter.fetch_add(1, std::memory_order_relaxed) + 1;
}

// Fixed device scratch of paged_attn_varlen_noalloc: the workspace of a call
// made by a caller that cannot allocate.  Every GPU that runs the library
// holds its own copy for the life of the process.  Host code never passes
// the array's name to a kernel (on the host it is only a stand-in for the
// symbol): it uses the device address that hipGetSymbolAddress returns, taken
// once per device with that device current.
constexpr size_t kScratchBytes = (size_t)32 << 20;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_addr[kMaxDevices];
std::mutex g_scratch_mu;

// Device address of the current device's scratch (set up on the first call
// on that device).
int scratch_address(void** addr) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return PA_EHIP;
  void* p = g_scratch_addr[dev].load(std::memory_order_acquire);
  if (p == nullptr) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_addr[dev].load(std::memory_order_relaxed);
    if (p == nullptr) {
      if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return PA_EHIP;
      g_scratch_addr[dev].store(p, std::memory_order_release);
    }
  }
  *addr = p;
  return PA_OK;
}

void record(hipEvent_t ev, hipStream_t st) {
  if (ev != nullptr) (void)hipEventRecord(ev, st);
}

// Host checks of an attention call's arguments (after plan()).
int check_args(const Plan& p, bool varlen, const void* q, const void* k_pages, const void* v_pages,
               const int32_t* block_table, const int32_t* context_lens, const int32_t* query_start_loc,
               float scale, const void* out) {
  if (!isfinite(scale) || !(scale > 0.0f)) return PA_EINVAL;
  if (p.rows > 0) {
    if (!q || !k_pages || !v_pages || !block_table || !context_lens || !out) return PA_EINVAL;
    if (varlen && !query_start_loc) return PA_EINVAL;
  }
  return PA_OK;
}

// One attention call.  trace: nullptr, or the gather trace's array (the
// kernels' trace instantiations then also record every loaded token's row).
int run(const void* q, const void* k_pages, const void* v_pages, const int32_t* block_table,
        const int32_t* context_lens, const int32_t* query_start_loc, float scale, void* out,
        const pa_dims_t* dims, void* workspace, size_t workspace_bytes, hipStream_t stream,
        const pa_timing_t* timing, bool varlen, int64_t* trace = nullptr, bool fixed_scratch = false) {
  Plan p;
  int rc = plan(dims, varlen, &p);
  if (rc != PA_OK) return rc;
  rc = check_args(p, varlen, q, k_pages, v_pages, block_table, context_lens, query_start_loc, scale, out);
  if (rc != PA_OK) return rc;
  // A caller's workspace must hold pa_workspace_size() bytes (sized for the
  // largest grid); the fixed scratch of the no-allocation entry only needs
  // what this call's grid uses (checked below, once the grid is known).
  if (!fixed_scratch && p.ws_bytes > 0 && (workspace == nullptr || workspace_bytes < p.ws_bytes))
    return PA_ENOSPC;
  if (p.rows > 0 && p.split == false && p.stream == false) return PA_ENOTSUP;

  const hipEvent_t ev_begin = timing ? timing->attn_begin : nullptr;
  const hipEvent_t ev_attn = timing ? timing->attn_end : nullptr;
  const hipEvent_t ev_reduce = timing ? timing->reduce_end : nullptr;
  if (p.rows == 0) {
    record(ev_begin, stream);
    record(ev_attn, stream);
    record(ev_reduce, stream);
    return PA_OK;
  }

  char* ws = static_cast<char*>(workspace);
  hipError_t e = hipSuccess;
  pa::StreamArgs sa{};
  int G = 0;
  if (p.stream) {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return PA_EHIP;
    const int per_cu = pa::stream_occupancy(dims->dtype, dims->head_dim, p.s, p.W);
    if (per_cu <= 0) return PA_EHIP;
    // 13/16 of the CUs (208 of 256 on MI355X, 26 per XCD) stream faster than
    // all of them: fewer requests in flight keep HBM in its efficient range.
    // Back-to-back launches (measured as a sustained loop, MI355X): Mixtral
    // batch 256 213-214 us per launch at 208 workgroups, 214-217 at 192, 218
    // at 256, 231 at 160; DBRX and 32k contexts within 0.5 % from 192 to 208,
    // 1-2 % slower at 256.
    // A batch whose ranges would overflow the LDS unit table takes more
    // workgroups (up to kStreamMaxGrid), even beyond one wave of resident
    // workgroups: no workgroup waits for another, so any residency works.
    int64_t g = (int64_t)per_cu * cus * kStreamCuNum / kStreamCuDen;
    if (g < 1) g = 1;
    if (g < p.g_min) g = p.g_min;
    if (g > pa::kStreamMaxGrid) g = pa::kStreamMaxGrid;
    G = (int)g;
    // workspace layout of this call: records and counters of G ranges, then
    // the split-K partials (a caller's workspace, sized for kStreamMaxGrid
    // ranges, always holds it)
    const size_t recs = (size_t)G * 2 * p.W * p.s;
    p.st_o = align256(recs * (size_t)dims->head_dim * sizeof(float));
    p.st_ml = align256(recs * 2 * sizeof(float));
    p.st_cum = align256((size_t)G * p.W * sizeof(unsigned long long));
    sa.q = q;
    sa.k_pages = k_pages;
    sa.v_pages = v_pages;
    sa.block_table = block_table;
    sa.context_lens = context_lens;
    sa.query_start_loc = varlen ? query_start_loc : nullptr;
    sa.out = out;
    sa.ws_o = reinterpret_cast<float*>(ws);
    sa.ws_ml = reinterpret_cast<float*>(ws + p.st_o);
    sa.ws_flag = reinterpret_cast<unsigned long long*>(ws + p.st_o + p.st_ml);
    sa.token = next_token();
    sa.bt_stride = dims->max_pages_per_seq;
    sa.scale_log2 = scale * 1.4426950408889634f;
    sa.B = dims->num_seqs;
    sa.H_q = dims->num_q_heads;
    sa.H_kv = dims->num_kv_heads;
    sa.max_context_len = dims->max_context_len;
    sa.nb = p.nb;
    sa.trace = trace;
  }
  if (p.st_o + p.st_ml + p.st_cum + p.sp_o + p.sp_ml > workspace_bytes) return PA_ENOSPC;
  // Mixed batch: decode and prefill workgroups side by side in one launch,
  // unless the chunk rows outweigh the decode rows.  A decode row streams its
  // whole KV (HBM-bound); a chunk row costs about s/80 of that on the matrix
  // cores at equal context (Mixtral shapes: 4,096 chunk rows took 151 us on
  // all CUs against 660 us for 512 decode rows).  Past half the decode work,
  // a quarter of the CUs would hold the launch up; the kernels then run one
  // after the other, prefill on every CU.
  const int64_t chunk_rows = (int64_t)dims->num_q_rows - dims->num_seqs;
  // Every sequence carrying max_q_len > 1 rows (the rows add up to
  // num_seqs * max_q_len) leaves no decode row: the stream-K kernel, which
  // takes only one-row sequences, would find no work and is not launched.
  const bool no_decode_rows = p.prefill && dims->max_q_len > 1 &&
                              (int64_t)dims->max_q_len * dims->num_seqs == dims->num_q_rows;
  const bool launch_stream = p.stream && dims->num_seqs > 0 && !no_decode_rows;
  const bool mixed = launch_stream && p.prefill &&
                     chunk_rows * p.s <= (int64_t)40 * dims->num_seqs &&
                     pa::mixed_supported(dims->dtype, dims->head_dim, p.s, p.W);
  // attention kernels in launch order: stream-K (or mixed), prefill, split-K;
  // the timing events bracket the first one's start and the last one's end
  // (rows > 0 here, so every planned kernel launches)
  const int n_attn = (launch_stream && !mixed ? 1 : 0) + (p.prefill ? 1 : 0) + (p.split ? 1 : 0);
  int n_launched = 0;
  auto next_events = [&]() {
    pa::KernelEvents k;
    k.start = n_launched == 0 ? ev_begin : nullptr;
    k.stop = n_launched == n_attn - 1 ? ev_attn : nullptr;
    ++n_launched;
    return k;
  };
  if (launch_stream && !mixed) {
    e = pa::launch_stream(dims->dtype, dims->head_dim, p.s, p.W, sa, G, stream, next_events());
    if (e != hipSuccess) return PA_EHIP;
  }
  if (p.prefill) {
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      return PA_EHIP;
    pa::PrefillArgs pf{};
    pf.q = q;
    pf.k_pages = k_pages;
    pf.v_pages = v_pages;
    pf.block_table = block_table;
    pf.context_lens = context_lens;
    pf.query_start_loc = query_start_loc;
    pf.out = out;
    pf.bt_stride = dims->max_pages_per_seq;
    pf.scale_log2 = scale * 1.4426950408889634f;
    pf.B = dims->num_seqs;
    pf.H_q = dims->num_q_heads;
    pf.H_kv = dims->num_kv_heads;
    pf.max_context_len = dims->max_context_len;
    pf.trace = trace;
    if (mixed) {
      // a quarter of the CUs for the chunks, the rest (at most the decode
      // grid) for the decode rows: one grid of one workgroup per CU
      // (measured on the mixed Mixtral batch: splits 176..208 / 48..80 of the
      // 256 CUs are within 2 % of 192 / 64)
      const int g_pf = cus * PA_MIXED_PF_NUM / PA_MIXED_PF_DEN > 0 ? cus * PA_MIXED_PF_NUM / PA_MIXED_PF_DEN : 1;
      const int g_dec = G < cus - g_pf ? G : (cus - g_pf > p.g_min ? cus - g_pf : (int)p.g_min);
      e = pa::launch_mixed(p.s, sa, pf, g_dec, g_dec + g_pf, stream, next_events());
    } else {
      const int per_cu = pa::prefill_occupancy(p.s, dims->num_seqs);
      if (per_cu <= 0) return PA_EHIP;
      e = pa::launch_prefill(p.s, pf, per_cu * cus, stream, next_events());
    }
    if (e != hipSuccess) return PA_EHIP;
  }
  pa::DecodeArgs a{};
  if (p.split) {
    char* sp = ws + p.st_o + p.st_ml + p.st_cum;
    a.q = q;
    a.k_pages = k_pages;
    a.v_pages = v_pages;
    a.block_table = block_table;
    a.context_lens = context_lens;
    a.query_start_loc = varlen ? query_start_loc : nullptr;
    a.out = out;
    a.ws_o = p.sp_o ? reinterpret_cast<float*>(sp) : nullptr;
    a.ws_ml = p.sp_o ? reinterpret_cast<float*>(sp + p.sp_o) : nullptr;
    a.bt_stride = dims->max_pages_per_seq;
    a.scale_log2 = scale * 1.4426950408889634f;
    a.B = dims->num_seqs;
    a.max_context_len = dims->max_context_len;
    a.H_q = dims->num_q_heads;
    a.H_kv = dims->num_kv_heads;
    a.pages_per_split = p.pps;
    a.n_split_slots = p.n_split_slots;
    a.skip_single_rows = p.stream ? 1 : 0;
    a.trace = trace;
    e = pa::launch_decode(dims->dtype, dims->head_dim, p.s, a, p.rows, stream, next_events());
    if (e != hipSuccess) return PA_EHIP;
  }
  if (n_launched == 0) {  // (cannot happen with rows > 0; keeps the events consistent)
    record(ev_begin, stream);
    record(ev_attn, stream);
  }
  if (p.split && p.n_split_slots > 1) {
    pa::ReduceArgs r{};
    r.ws_o = a.ws_o;
    r.ws_ml = a.ws_ml;
    r.context_lens = context_lens;
    r.query_start_loc = a.query_start_loc;
    r.out = out;
    r.B = dims->num_seqs;
    r.rows = p.rows;
    r.H_q = dims->num_q_heads;
    r.max_context_len = dims->max_context_len;
    r.pages_per_split = p.pps;
    r.n_split_slots = p.n_split_slots;
    r.skip_single_rows = a.skip_single_rows;
    e = pa::launch_reduce(dims->dtype, dims->head_dim, r, stream);
    if (e != hipSuccess) return PA_EHIP;
  }
  record(ev_reduce, stream);
  return PA_OK;
}

}  // namespace

extern "C" {

int pa_workspace_size(const pa_dims_t* dims, size_t* bytes) {
  if (bytes == nullptr) return PA_EINVAL;
  // The workspace depends on the number of query rows only: a call whose
  // dims carry chunked rows (max_q_len > 1 or num_q_rows != num_seqs) is
  // planned as varlen, any other as decode (they coincide when all L_b = 1).
  Plan p;
  const bool varlen = dims != nullptr &&
                      (dims->max_q_len > 1 || (dims->num_q_rows != 0 && dims->num_q_rows != dims->num_seqs));
  int rc = plan(dims, varlen, &p);
  if (rc != PA_OK) return rc;
  *bytes = p.ws_bytes;
  return PA_OK;
}

int paged_attn(const void* q, const void* k_pages, const void* v_pages, const int32_t* block_table,
               const int32_t* context_lens, float scale, void* out, const pa_dims_t* dims,
               void* workspace, size_t workspace_bytes, hipStream_t stream,
               const pa_timing_t* timing) {
  return run(q, k_pages, v_pages, block_table, context_lens, nullptr, scale, out, dims, workspace,
             workspace_bytes, stream, timing, false);
}

int paged_attn_varlen(const void* q, const void* k_pages, const void* v_pages,
                      const int32_t* block_table, const int32_t* context_lens,
                      const int32_t* query_start_loc, float scale, void* out,
                      const pa_dims_t* dims, void* workspace, size_t workspace_bytes,
                      hipStream_t stream, const pa_timing_t* timing) {
  return run(q, k_pages, v_pages, block_table, context_lens, query_start_loc, scale, out, dims,
             workspace, workspace_bytes, stream, timing, true);
}

int paged_attn_varlen_noalloc(const void* q, const void* k_pages, const void* v_pages,
                              const int32_t* block_table, const int32_t* context_lens,
                              const int32_t* query_start_loc, float scale, void* out,
                              const pa_dims_t* dims, hipStream_t stream, const pa_timing_t* timing) {
  Plan p;  // host validation before the first device call
  int rc = plan(dims, true, &p);
  if (rc != PA_OK) return rc;
  rc = check_args(p, true, q, k_pages, v_pages, block_table, context_lens, query_start_loc, scale, out);
  if (rc != PA_OK) return rc;
  if (p.rows == 0)
    return run(q, k_pages, v_pages, block_table, context_lens, query_start_loc, scale, out, dims, nullptr, 0,
               stream, timing, true);
  void* ws = nullptr;
  rc = scratch_address(&ws);
  if (rc != PA_OK) return rc;
  return run(q, k_pages, v_pages, block_table, context_lens, query_start_loc, scale, out, dims, ws,
             kScratchBytes, stream, timing, true, nullptr, true);
}

int pa_gather_trace(const void* q, const void* k_pages, const void* v_pages, const int32_t* block_table,
                    const int32_t* context_lens, const int32_t* query_start_loc, float scale, void* out,
                    const pa_dims_t* dims, void* workspace, size_t workspace_bytes, int64_t* rows_out,
                    hipStream_t stream) {
  const bool varlen = query_start_loc != nullptr;
  Plan p;
  int rc = plan(dims, varlen, &p);
  if (rc != PA_OK) return rc;
  if (p.rows == 0) return run(q, k_pages, v_pages, block_table, context_lens, query_start_loc, scale, out, dims,
                              workspace, workspace_bytes, stream, nullptr, varlen);
  if (rows_out == nullptr) return PA_EINVAL;
  const int64_t n = (int64_t)dims->num_kv_heads * dims->num_seqs * dims->max_pages_per_seq * 16;
  // the attention call's own validation runs before anything is enqueued
  if (!isfinite(scale) || !(scale > 0.0f)) return PA_EINVAL;
  if (!q || !k_pages || !v_pages || !block_table || !context_lens || !out) return PA_EINVAL;
  if (p.ws_bytes > 0 && (workspace == nullptr || workspace_bytes < p.ws_bytes)) return PA_ENOSPC;
  if (pa::launch_fill_i64(rows_out, n, -1, stream) != hipSuccess) return PA_EHIP;
  return run(q, k_pages, v_pages, block_table, context_lens, query_start_loc, scale, out, dims, workspace,
             workspace_bytes, stream, nullptr, varlen, rows_out);
}

int pa_kv_append(const void* k_new, const void* v_new, const int32_t* block_table,
                 const int32_t* context_lens, const int32_t* query_start_loc, void* k_pages,
                 void* v_pages, const pa_dims_t* dims, hipStream_t stream) {
  if (dims == nullptr) return PA_EINVAL;
  const pa_dims_t* d = dims;
  if (d->num_seqs < 0 || d->num_kv_heads <= 0 || d->num_pages < 0 || d->max_pages_per_seq < 0 ||
      d->max_context_len < 0)
    return PA_EINVAL;
  if (d->dtype != PA_BF16 && d->dtype != PA_FP32) return PA_ENOTSUP;
  if (d->head_dim != 64 && d->head_dim != 128) return PA_ENOTSUP;
  if (d->page_size != 16) return PA_ENOTSUP;
  if (((int64_t)d->max_context_len + 15) / 16 > d->max_pages_per_seq) return PA_EINVAL;
  int rows;
  if (query_start_loc != nullptr) {
    if (d->num_q_rows < 0) return PA_EINVAL;
    if (d->num_q_rows > 0 && d->num_seqs == 0) return PA_EINVAL;
    rows = d->num_q_rows;
  } else {
    if (d->num_q_rows != 0 && d->num_q_rows != d->num_seqs) return PA_EINVAL;
    rows = d->num_seqs;
  }
  if (rows == 0) return PA_OK;
  if (!k_new || !v_new || !block_table || !context_lens || !k_pages || !v_pages) return PA_EINVAL;
  pa::AppendArgs a;
  a.k_new = static_cast<const uint8_t*>(k_new);
  a.v_new = static_cast<const uint8_t*>(v_new);
  a.k_pages = static_cast<uint8_t*>(k_pages);
  a.v_pages = static_cast<uint8_t*>(v_pages);
  a.block_table = block_table;
  a.context_lens = context_lens;
  a.query_start_loc = query_start_loc;
  a.bt_stride = d->max_pages_per_seq;
  a.B = d->num_seqs;
  a.rows = rows;
  a.H_kv = d->num_kv_heads;
  a.row_bytes = d->head_dim * (d->dtype == PA_BF16 ? 2 : 4);
  a.num_pages = d->num_pages;
  a.max_context_len = d->max_context_len;
  return pa::launch_kv_append(a, stream) == hipSuccess ? PA_OK : PA_EHIP;
}

int pa_schedule_step(const pa_sched_state_t* state, int32_t n_real, const int32_t* new_seq,
                     const int32_t* new_prompt, const int32_t* new_fin, int32_t n_new,
                     int32_t* query_start_loc, int32_t* finished_out, int32_t* info, hipStream_t stream) {
  if (state == nullptr) return PA_EINVAL;
  const pa_sched_state_t& st = *state;
  if (st.num_slots <= 0 || st.num_pages < 0 || st.max_pages_per_seq <= 0 || st.queue_cap <= st.num_slots ||
      n_real < 0 || n_new < 0)
    return PA_EINVAL;
  if (st.num_slots > pa::kSchedMaxSlots) return PA_ENOTSUP;
  // token and page counts of a step stay within int32
  if ((int64_t)st.num_slots * (st.max_pages_per_seq + 1) * 16 > INT32_MAX) return PA_EINVAL;
  if (!st.free_pages && st.num_pages > 0) return PA_EINVAL;
  if (!st.hdr || !st.queue_seq || !st.queue_tok || !st.queue_fin || !st.slot_seq || !st.slot_order ||
      !st.slot_fin || !st.context_lens || !st.block_table || !query_start_loc || !finished_out || !info)
    return PA_EINVAL;
  if (n_new > 0 && (!new_seq || !new_prompt || !new_fin)) return PA_EINVAL;
  pa::SchedArgs a;
  a.free_pages = st.free_pages;
  a.hdr = st.hdr;
  a.queue_seq = st.queue_seq;
  a.queue_tok = st.queue_tok;
  a.queue_fin = st.queue_fin;
  a.slot_seq = st.slot_seq;
  a.slot_order = st.slot_order;
  a.slot_fin = st.slot_fin;
  a.context_lens = st.context_lens;
  a.block_table = st.block_table;
  a.S = st.num_slots;
  a.P = st.num_pages;
  a.MP = st.max_pages_per_seq;
  a.Q = st.queue_cap;
  a.n_real = n_real;
  a.new_seq = new_seq;
  a.new_prompt = new_prompt;
  a.new_fin = new_fin;
  a.n_new = n_new;
  a.query_start_loc = query_start_loc;
  a.finished_out = finished_out;
  a.info = info;
  return pa::launch_sched(a, stream) == hipSuccess ? PA_OK : PA_EHIP;
}

const char* pa_strerror(int code) {
  switch (code) {
    case PA_OK: return "success";
    case PA_EINVAL: return "invalid argument (null pointer, negative or inconsistent size)";
    case PA_ENOTSUP: return "unsupported configuration (head_dim, page_size, dtype or GQA group size)";
    case PA_ENOSPC: return "workspace smaller than pa_workspace_size() (or the call needs more than the no-allocation entry's fixed scratch)";
    case PA_EHIP: return "HIP kernel launch failed";
    default: return "unknown error code";
  }
}

}  // extern "C"
