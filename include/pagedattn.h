/*
 * pagedattn.h -- C ABI of the MI355X (gfx950) paged-KV grouped-query
 * attention library (libpagedattn.so).
 *
 * The operation is the decode-step attention of MoE-Lens (arXiv 2504.09345):
 * every sequence of a batch attends with its query heads to its own cached
 * keys and values, which live in fixed-size blocks of token slots addressed
 * through a per-sequence block table (Sec. 5.5, the paged-KV assumption of
 * the Stage-2 model).  A group of s = H_q / H_kv query heads shares one KV head
 * (grouped-query attention, Sec. 2); query head h reads KV head h / s.  KV is
 * stored in bf16 and the arithmetic runs in fp32 as dot products q.k and
 * scaled vector adds over V (Sec. 5.3, Eq. 6 and the text after it).  The new
 * token's K/V are already in the cache when decode attention runs (Sec. 6.4,
 * compute-graph division), so a context length counts the current token.
 * The varlen entry adds causal prefill chunks that share the launch with the
 * decode rows (the paper prefills on the GPU, Sec. 6.4; chunking is this
 * library's reading: a chunk's own K/V are already in its pages).
 *
 * Result, per sequence b, query row r of its chunk of length L (decode: L = 1,
 * r = 0) and query head h, with C = context_lens[b] and g = h / s:
 *   x_t = scale * dot(q[row][h], K[t])           for t = 0 .. C - L + r
 *   out[row][h] = sum_t softmax(x)_t * V[t]
 * where K[t] / V[t] is slot t % P of page block_table[b][t / P], KV head g.
 * A row that sees no key (C = 0) produces zeros.
 *
 * Conventions for every entry point
 *   - All array pointers are DEVICE pointers (HBM), except where a name ends
 *     in _host.  The caller owns every buffer; the library allocates nothing.
 *     Its only state between calls is a process-wide counter that tags each
 *     call's use of the workspace (it never changes a result).  Calls on
 *     different streams may overlap as long as their output and workspace
 *     buffers do not.
 *   - Work is enqueued on `stream` (NULL = the null stream) and the call
 *     returns without synchronising.  Faults inside kernels (for example a
 *     block-table entry outside the pool) surface at the caller's next
 *     synchronisation; the hot path does not range-check page indices.
 *   - Argument validation happens on the host before any HIP call; a
 *     validation failure enqueues nothing.
 *   - Return value: PA_OK (0) or a negative error code (see pa_strerror).
 *
 * Layouts (row-major, element type given by dims->dtype for q/k/v/out):
 *   q, out        [num_q_rows][num_q_heads][head_dim]
 *                 (decode: num_q_rows = num_seqs, row b belongs to sequence b)
 *   k_pages,
 *   v_pages       [num_pages][num_kv_heads][page_size][head_dim]
 *                 one (page, kv head) tile is page_size*head_dim contiguous
 *                 elements (4 KiB at 16 x 128 bf16)
 *   block_table   int32 [num_seqs][max_pages_per_seq]; entries at or beyond
 *                 ceil(context_lens[b] / page_size) are never read
 *   context_lens  int32 [num_seqs], 0 <= context_lens[b] <= max_context_len
 *   query_start_loc int32 [num_seqs + 1] (varlen only): sequence b owns rows
 *                 query_start_loc[b] .. query_start_loc[b+1]-1, with
 *                 query_start_loc[0] = 0 and
 *                 1 <= L_b = query_start_loc[b+1]-query_start_loc[b]
 *                    <= min(max_q_len, context_lens[b])  (or L_b = 0 when
 *                 context_lens[b] = 0)
 */
#ifndef PAGEDATTN_H
#define PAGEDATTN_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Error codes. */
enum {
  PA_OK = 0,
  PA_EINVAL = -1,  /* null pointer, negative or inconsistent size */
  PA_ENOTSUP = -2, /* head_dim, page_size, dtype or GQA group size not compiled */
  PA_ENOSPC = -3,  /* workspace smaller than pa_workspace_size() */
  PA_EHIP = -4     /* a HIP launch reported an error (hipGetLastError) */
};

/* Element type of q, k_pages, v_pages and out (all four share it).  bf16 is
 * stored as raw 16-bit patterns; out is rounded to nearest even from fp32. */
typedef enum { PA_BF16 = 0, PA_FP32 = 1 } pa_dtype_t;

/* Problem description (host memory, read during the call only).
 * Supported: head_dim 64 or 128; page_size 16; GQA group size
 * s = num_q_heads / num_kv_heads in {1, 2, 4, 6, 8}; dtype bf16 or fp32. */
typedef struct pa_dims {
  int32_t num_seqs;          /* B >= 0                                      */
  int32_t num_q_heads;       /* H_q > 0, a multiple of num_kv_heads         */
  int32_t num_kv_heads;      /* H_kv > 0                                    */
  int32_t head_dim;          /* D                                           */
  int32_t page_size;         /* token slots per page, must be 16            */
  int32_t num_pages;         /* pages in the pool                           */
  int32_t max_pages_per_seq; /* block_table row stride, >= ceil(max_context_len / 16) */
  int32_t max_context_len;   /* upper bound on context_lens[], sizes the grid */
  int32_t pages_per_split;   /* 0: library choice (persistent stream-K kernel
                                where the batch fits it); > 0: per-row split-K
                                kernel with this many pages per workgroup      */
  int32_t dtype;             /* pa_dtype_t                                  */
  int32_t num_q_rows;        /* varlen: total query rows; decode: 0 or num_seqs */
  int32_t max_q_len;         /* varlen: bound on any chunk length; decode: 0 or 1 */
} pa_dims_t;

/* Optional timing hooks: when a pa_timing_t* is passed and an event is
 * non-NULL, it is recorded for the call: attn_begin when the first attention
 * kernel starts executing and attn_end when the last attention kernel ends
 * (both taken by the kernel launches themselves, so their difference is the
 * kernels' own duration), and reduce_end on the call's stream after the
 * kernel that merges split partial results (recorded even when none was
 * needed). */
typedef struct pa_timing {
  hipEvent_t attn_begin;
  hipEvent_t attn_end;
  hipEvent_t reduce_end;
} pa_timing_t;

/* Bytes of device workspace a paged_attn / paged_attn_varlen call with these
 * dims needs: partial outputs and softmax statistics of items split across
 * workgroups, and the arrival counters of those items.  Writes 0 when no
 * workspace is needed.  A call whose dims carry chunked rows (max_q_len > 1 or
 * num_q_rows != num_seqs) is sized as varlen.  Host only; no HIP call.
 * Errors: PA_EINVAL / PA_ENOTSUP as for paged_attn. */
int pa_workspace_size(const pa_dims_t *dims, size_t *bytes);

/* Decode attention: one query row per sequence (Sec. 6.6 computes exactly
 * this on the CPU).  Here: a persistent stream-K kernel over equal ranges of
 * (sequence, KV-head block, page) units whose workgroups also merge the
 * items cut by range boundaries (one launch: the last part of a cut item to
 * finish merges it, so no workgroup ever waits for another); with
 * pages_per_split > 0, or more than 8192 sequences, a per-row split-K kernel
 * plus a reduction kernel.  Both are deterministic (no float atomics; merges
 * run in a fixed order).
 *   q            [num_seqs][H_q][D]        device, read
 *   k_pages,
 *   v_pages      pool, see layouts above   device, read
 *   block_table, context_lens              device, read
 *   scale        multiplies every dot product (typically 1/sqrt(D)); must be
 *                finite and > 0 (PA_EINVAL otherwise)
 *   out          [num_seqs][H_q][D]        device, written
 *   workspace    device scratch of at least pa_workspace_size() bytes (may
 *                be NULL when that size is 0); contents are overwritten
 *   timing       optional events, may be NULL
 * Errors: PA_EINVAL, PA_ENOTSUP, PA_ENOSPC, PA_EHIP. */
int paged_attn(const void *q, const void *k_pages, const void *v_pages,
               const int32_t *block_table, const int32_t *context_lens, float scale,
               void *out, const pa_dims_t *dims, void *workspace, size_t workspace_bytes,
               hipStream_t stream, const pa_timing_t *timing);

/* Mixed batch: causal prefill chunks and decode rows in one call.  Decode
 * rows take the stream-K kernel; chunk rows (L_b > 1) take an MFMA kernel
 * (bf16, head_dim 128) or, otherwise, the per-row split-K kernel.  The MFMA
 * kernel forms P.V with P rounded to fp16 (relative error 2^-11) and V in
 * fp16 (exact for bf16 magnitudes in [2^-17, 2^16)); a chunk block whose V
 * leaves that range (or holds inf / NaN), or whose output rows have an RMS
 * below 2^-14, is computed again with fp32-level P.V.  When every sequence
 * has max_q_len > 1 rows, only the chunk kernel runs.
 * Same as paged_attn, with q/out of [num_q_rows][H_q][D] and the device array
 * query_start_loc (see layouts).  Row j of a chunk of length L in a sequence
 * of context C attends to positions 0 .. C - L + j.  dims->num_q_rows must
 * equal query_start_loc[num_seqs] and dims->max_q_len bound every L_b.
 * Errors: PA_EINVAL, PA_ENOTSUP, PA_ENOSPC, PA_EHIP. */
int paged_attn_varlen(const void *q, const void *k_pages, const void *v_pages,
                      const int32_t *block_table, const int32_t *context_lens,
                      const int32_t *query_start_loc, float scale, void *out,
                      const pa_dims_t *dims, void *workspace, size_t workspace_bytes,
                      hipStream_t stream, const pa_timing_t *timing);

/* No-allocation variant of paged_attn_varlen, for callers that cannot
 * allocate device memory or pass a workspace: code recorded under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  Same
 * arguments, layouts, results and errors as paged_attn_varlen, without the
 * workspace: the partial records and arrival counters live in a fixed
 * 32 MiB array of device memory inside the library (one per GPU, held until
 * the process ends; its address is taken on the first call on each device).
 * The call allocates nothing.
 *   - A call that needs more than the 32 MiB returns PA_ENOSPC and enqueues
 *     nothing.  The stream-K decode rows need 66.5 KiB per workgroup of the
 *     grid at s = 8 (33 KiB at s = 4, 208 workgroups on MI355X: ~7 MB);
 *     chunk rows that take the per-row split-K kernel (fp32, head_dim 64)
 *     need rows x H_q x splits x (D + 2) x 4 bytes.
 *   - Every call on one GPU shares that GPU's array and leaves its contents
 *     behind (the arrival counters are tagged per call, so nothing needs
 *     clearing): calls that overlap in time on one GPU (other streams,
 *     other threads) race on it and must be serialised by the caller.
 *   - Decode-only callers pass query_start_loc = {0, 1, ..., num_seqs} with
 *     num_q_rows = num_seqs and max_q_len = 1, which runs exactly the kernels
 *     of paged_attn.
 * Errors: as paged_attn_varlen; PA_EHIP also when the scratch's device
 * address cannot be taken. */
int paged_attn_varlen_noalloc(const void *q, const void *k_pages, const void *v_pages,
                              const int32_t *block_table, const int32_t *context_lens,
                              const int32_t *query_start_loc, float scale, void *out,
                              const pa_dims_t *dims, hipStream_t stream, const pa_timing_t *timing);

/* Block-table gather trace (Sec. 5.5 paging; Sec. 2 GQA): the same call as
 * paged_attn (query_start_loc == NULL) or paged_attn_varlen (otherwise), run
 * through instantiations of the very same kernels that also record, for every
 * token they load, the pool row its K and V came from.  `out` is written
 * exactly as the attention call writes it.  The record is taken from the
 * element offset each kernel hands to its tile loads, so it checks the
 * kernels' own block-table gather (the stream-K unit table, the prefill
 * kernel's block-table window, the split-K kernel's per-lane entries), not a
 * separate address function.
 *   rows_out  int64 device array [num_kv_heads][num_seqs][max_pages_per_seq * 16],
 *             filled by the call: entry (g, b, t) is the row
 *             (page * num_kv_heads + g) * 16 + t % 16 of the
 *             [num_pages][num_kv_heads][16] pool, page = block_table[b][t / 16],
 *             from which some kernel loaded token t of sequence b for KV head
 *             g; -1 where no kernel loaded the token (t >= context_lens[b]),
 *             -2 where two loads of the token came from different rows.
 * Other arguments, layouts, workspace and errors as for paged_attn /
 * paged_attn_varlen (rows_out == NULL with query rows: PA_EINVAL).  Meant
 * for tests: the trace instantiations run somewhat slower than the
 * attention kernels. */
int pa_gather_trace(const void *q, const void *k_pages, const void *v_pages,
                    const int32_t *block_table, const int32_t *context_lens,
                    const int32_t *query_start_loc, float scale, void *out,
                    const pa_dims_t *dims, void *workspace, size_t workspace_bytes,
                    int64_t *rows_out, hipStream_t stream);

/* KV append: store the new tokens' keys and values into the paged cache, the
 * step right before attention (Sec. 6.4: the task that receives a decode
 * token's pre-attention K/V stores it in the KV cache, then attends; Sec. 5.5
 * paging).  Sequence b appends L_b tokens at the LAST L_b positions of its
 * context, so context_lens already counts them (the same convention as the
 * attention calls):
 *   - query_start_loc != NULL: rows query_start_loc[b] .. query_start_loc[b+1]-1,
 *     row query_start_loc[b] + j at position context_lens[b] - L_b + j;
 *     dims->num_q_rows rows in total;
 *   - query_start_loc == NULL (decode): row b at position context_lens[b] - 1,
 *     nothing for context_lens[b] = 0; dims->num_seqs rows.
 * Row r, KV head g (D elements) is copied bit for bit into KV head g of slot
 * position % page_size of page block_table[b][position / page_size].
 *   k_new, v_new     [rows][num_kv_heads][head_dim]   device, read
 *   k_pages, v_pages pool, see layouts above         device, updated in place
 *   block_table, context_lens, query_start_loc       device, read
 * Uses num_seqs, num_kv_heads, head_dim, page_size, num_pages,
 * max_pages_per_seq, max_context_len, dtype and (varlen) num_q_rows of dims.
 * A sequence whose chunk is longer than its context, whose context exceeds
 * max_context_len, or whose written page entry lies outside [0, num_pages) is
 * not written (nothing outside the pool is ever touched).  Rows of different
 * calls on one stream are written in call order; the caller runs attention on
 * the same stream after this call.
 * Errors: PA_EINVAL, PA_ENOTSUP, PA_EHIP. */
int pa_kv_append(const void *k_new, const void *v_new, const int32_t *block_table,
                 const int32_t *context_lens, const int32_t *query_start_loc, void *k_pages,
                 void *v_pages, const pa_dims_t *dims, hipStream_t stream);

/* Scheduler step: the GPU-resident page allocator and block-table builder of
 * the Resource-Aware Scheduler (Sec. 6.2).  A prefill scheduler holds a queue
 * of sequences waiting for their prompt pass; a decode scheduler estimates the
 * 16-token pages its sequences' next tokens need, garbage-collects finished
 * sequences and, when pages run short, preempts the newest decode sequences,
 * which re-enter the queue ahead of new arrivals and prefill their whole
 * context again while admission pauses (preemption mode).  Otherwise the
 * prefill scheduler admits queue-head sequences while their tokens fit what
 * the pass has left after the decode rows (normal mode).  Both keep their
 * state in device memory; one call is one kernel launch.
 *
 * State (all int32 device arrays, updated in place; page size 16):
 *   free_pages   [num_pages]  stack of free page indices, entries
 *                0 .. hdr[0]-1, top = hdr[0]-1
 *   hdr          [4]  free count, next admission order, queue head, queue
 *                length
 *   queue_seq, queue_tok, queue_fin  [queue_cap]  circular queue from the
 *                head: logical id, tokens to prefill, finish length
 *   slot_seq     [num_slots]  logical id in the batch slot, -1 = empty
 *   slot_order   [num_slots]  admission order (larger = newer)
 *   slot_fin     [num_slots]  context length at which the sequence finishes
 *   context_lens [num_slots]  tokens in the cache, counting this pass's
 *   block_table  [num_slots][max_pages_per_seq]
 * A fresh state: free_pages = 0 .. num_pages-1, hdr = {num_pages, 0, 0, 0},
 * slot_seq all -1 (the other arrays any value).  context_lens, block_table
 * and query_start_loc are the attention calls' arguments for the pass, with
 * the slot as the sequence index (num_seqs = num_slots): an admitted slot's
 * chunk is its whole context, a decode slot's chunk is one row.
 *
 * One step, in this order (slot order = ascending slot index):
 *   0. arrivals i = 0 .. n_new-1 (new_seq, new_prompt, new_fin: device
 *      arrays) with 1 <= new_prompt[i] <= new_fin[i] <= 16*max_pages_per_seq
 *      join the queue tail in order while the queue length stays below
 *      queue_cap - num_slots; others are dropped;
 *   1. slots with context_lens >= slot_fin finish: their ids go to
 *      finished_out in slot order, their pages are pushed (slot order, page
 *      order), slot_seq = -1, context_lens = 0;
 *   2. a remaining slot needs a page iff context_lens % 16 == 0;
 *   3. if more pages are needed than free: preempt the slots with the
 *      largest admission orders, the fewest that make the rest fit; push their
 *      pages (slot order); they enter the queue ahead of the head, lowest slot
 *      first, with tokens = their context; no admission this step;
 *   4. each remaining slot (slot order) pops its page if needed, and its
 *      context grows by 1;
 *   5. in normal mode admit queue-head entries while the running token sum
 *      stays <= n_real - (decode slots of step 4), their pages fit the free
 *      stack and empty slots remain; the r-th admitted takes the r-th lowest
 *      empty slot, order hdr[1] + r, context = its tokens, and pops its pages
 *      in page order;
 *   6. query_start_loc [num_slots + 1] = prefix sum of the rows (1 per decode
 *      slot, the context per admitted slot, 0 otherwise).
 * info (device, int32 [8]) = {mode (0 normal, 1 preemption, -1 state
 * rejected), finished, preempted, admitted, decode slots, arrivals accepted,
 * free pages after, total rows}.  finished_out has num_slots entries.
 *
 * The kernel first checks that the state is one a step can produce: header
 * fields in range, 1 <= context_lens <= 16*max_pages_per_seq and slot_fin <=
 * 16*max_pages_per_seq for occupied slots, queued entries with
 * 1 <= tokens <= finish <= 16*max_pages_per_seq, pages free plus held <=
 * num_pages, queued plus occupied <= queue_cap.  On failure it writes
 * info = {-1, 0, ...} and changes nothing else.  Page indices themselves are
 * only copied, never used as addresses, and are not range-checked; admission
 * orders of occupied slots must be distinct (every step keeps them so).
 * Errors (host-side, nothing enqueued): PA_EINVAL (null pointer, num_slots
 * <= 0, queue_cap <= num_slots, negative sizes, or num_slots *
 * (max_pages_per_seq + 1) * 16 beyond int32), PA_ENOTSUP (num_slots > 8192),
 * PA_EHIP. */
typedef struct {
  int32_t *free_pages;
  int32_t *hdr;
  int32_t *queue_seq;
  int32_t *queue_tok;
  int32_t *queue_fin;
  int32_t *slot_seq;
  int32_t *slot_order;
  int32_t *slot_fin;
  int32_t *context_lens;
  int32_t *block_table;
  int32_t num_slots;
  int32_t num_pages;
  int32_t max_pages_per_seq;
  int32_t queue_cap;
} pa_sched_state_t;

int pa_schedule_step(const pa_sched_state_t *state, int32_t n_real, const int32_t *new_seq,
                     const int32_t *new_prompt, const int32_t *new_fin, int32_t n_new,
                     int32_t *query_start_loc, int32_t *finished_out, int32_t *info,
                     hipStream_t stream);

/* Static description of an error code (never NULL). */
const char *pa_strerror(int code);

#ifdef __cplusplus
}
#endif

#endif /* PAGEDATTN_H */
