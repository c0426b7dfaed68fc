// Causal chunked-prefill rows on MFMA (gfx950), sharing a varlen call with the
// decode rows.
//
// A sequence with context C issuing a chunk of L > 1 query rows has the
// chunk's own K/V already in its pages (the library's reading of the
// paper's GPU prefill, MoE-Lens Sec. 6.4); row j sits at position C - L + j
// and attends to keys 0 .. C - L + j (Sec. 2 GQA groups, Sec. 5.5 paged KV).
// Unlike a decode row, a chunk reuses every K/V page across many query rows,
// so the contraction is dense enough for the matrix cores.
//
// Work item: (sequence, KV head g, block of PB chunk positions).  The block's
// M = PB * s query rows (position-major, the s heads of group g) are split
// over 8 waves of two 16-row MFMA blocks each (256 rows), so every operand
// read from LDS feeds two matrix products.  Per step of two 16-key pages:
//   S^T[key][row] = K . Q^T   (v_mfma_f32_16x16x32_bf16 per page, K as the A
//                  operand)
//   online softmax per row (each lane owns one row and 8 of its keys)
//   O^T[dim][row] += V^T . P^T (one v_mfma_f32_16x16x32_f16 over the step's
//                  keys: P rounded to fp16, V staged in LDS as fp16)
// fp16 keeps 11 significant bits against bf16's 8, so P's rounding error is
// 2^-11 relative (bf16 P alone missed the relative tolerance; fp16 P adds a
// tenth of what the bf16 rounding of the output costs), and bf16 V converts
// to fp16 exactly for magnitudes in [2^-17, 2^16).  An item whose V holds a
// value of 2^16 or more (or inf / NaN; in fp16 each makes every row of the
// item non-finite), or whose output rows have an RMS below 2^-14 (where
// fp16's subnormal V could matter), is computed again in a bf16 pass: V as
// loaded, P as its bf16 high and low parts in two v_mfma_f32_16x16x32_bf16
// (fp32-level accuracy).  Both conditions are read off the first pass's
// output rows.
// Computing the transposed products keeps "lane l % 16 = query row" in every
// accumulator, so the softmax statistics, the P operand and the O rescale all
// stay in the lane that owns the row: no register transposes.
// The pages' K and V tiles are staged in LDS once per workgroup, two pages
// per synchronised step, and read by all 8 waves, both with 16-byte chunks
// XOR-swizzled by key (conflict-free operand reads); each lane's PV operand
// (4 keys of one dim) is one ds_read_b64_tr_b16 from the [key][dim] V tile.
// The step loop is software-pipelined: the QK products of step t + 1 are
// issued before the softmax and PV of step t, so the matrix cores and the
// VALU work side by side.  Global loads run up to four steps ahead through two
// register sets and a three-step LDS ring, and the item's block-table
// entries are read from an LDS window.
// A persistent grid walks the items in a snake order (item x and 2G-1-x per
// workgroup) so early and late causal blocks pair up.
#include "pa_prefill_body.h"

namespace pa {

template <int D, int S, bool TR>
__global__ __launch_bounds__(kPfThreads) void prefill_kernel(PrefillArgs a) {
  __shared__ PrefillSmem sm;
  extern __shared__ int32_t s_cum[];  // [B + 1] prefix of items per sequence
  prefill_body<D, S, TR>(a, sm, s_cum, blockIdx.x, gridDim.x);
}

template <bool TR>
static const void* prefill_pick(int s) {
  switch (s) {
    case 1: return reinterpret_cast<const void*>(&prefill_kernel<128, 1, TR>);
    case 2: return reinterpret_cast<const void*>(&prefill_kernel<128, 2, TR>);
    case 4: return reinterpret_cast<const void*>(&prefill_kernel<128, 4, TR>);
    case 6: return reinterpret_cast<const void*>(&prefill_kernel<128, 6, TR>);
    case 8: return reinterpret_cast<const void*>(&prefill_kernel<128, 8, TR>);
  }
  return nullptr;
}

// trace: the gather-trace instantiation (also records the rows it loads)
static const void* prefill_fn(int s, bool trace = false) { return trace ? prefill_pick<true>(s) : prefill_pick<false>(s); }

bool prefill_supported(int dtype, int D, int s) { return dtype == 0 && D == 128 && prefill_fn(s) != nullptr; }

int prefill_occupancy(int s, int B) {
  const void* fn = prefill_fn(s);
  if (fn == nullptr) return 0;
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, kPfThreads, (size_t)(B + 1) * sizeof(int32_t)) != hipSuccess)
    return 0;
  return n;
}

hipError_t launch_prefill(int s, const PrefillArgs& a, int G, hipStream_t st, KernelEvents ev) {
  const void* fn = prefill_fn(s, a.trace != nullptr);
  if (fn == nullptr || G <= 0) return hipErrorInvalidValue;
  void* args[] = {const_cast<PrefillArgs*>(&a)};
  hipError_t e = hipExtLaunchKernel(fn, dim3(G), dim3(kPfThreads), args, (size_t)(a.B + 1) * sizeof(int32_t), st,
                                    ev.start, ev.stop, 0);
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

}  // namespace pa
