/*
 * oracle.c -- plain, slow, obviously correct CPU definition of batched
 * paged-KV grouped-query attention (decode rows and causal chunked-prefill
 * rows).  TEST INFRASTRUCTURE ONLY: it exists to check the GPU library.  Only
 * the test suite, the smoke check and the benchmark's CPU-baseline leg may
 * load it; the product path never does.  It shares no code, header, helper or
 * table with the GPU library.
 *
 * What is computed (MoE-Lens, arXiv 2504.09345):
 *   - KV cache organised in fixed-size blocks of P token slots addressed
 *     through a per-sequence block table (Sec. 5.5, the paged-KV assumption of
 *     the Stage-2 model, after PagedAttention).
 *   - Grouped-query attention: a group of s = H_q / H_kv query heads shares one
 *     key/value head (Sec. 2, "Concepts in LLM Model Inference").  Reading:
 *     contiguous groups, kv head = h / s.
 *   - KV stored as bf16 and up-converted to fp32 for the arithmetic, whose
 *     primary operations are dot products (q.k) and scaled vector adds
 *     (saxpby over V) (Sec. 5.3, Eq. 6 and the text after it).  The oracle
 *     therefore computes in fp32 with no fused multiply-add (built with
 *     -ffp-contract=off), summing strictly in index order.
 *   - The new decode token's K/V are stored in the cache before decode
 *     attention runs (Sec. 6.4, compute-graph division: GPU task A yields
 *     "pre-attention" KV for decode tokens, the CPU task stores it and then
 *     attends).  So context_lens counts the current token and decode rows need
 *     no mask.
 *   - Chunked prefill (reading; the paper prefills whole prompts on the GPU,
 *     Sec. 6.4): a sequence with context C issuing a chunk of L query rows has
 *     the chunk's own K/V already in its pages; row j sits at absolute
 *     position C - L + j and attends causally to positions 0 .. C - L + j.
 *
 * Softmax is written in its three-pass textbook form (max, exponentials and
 * their sum, weighted sum of V divided once by the sum), not the online
 * (flash) form the paper's kernel uses: both give the same exact result, and
 * the two implementations share no algorithm.
 *
 * Layouts (row-major):
 *   q, out            [T_q][H_q][D]     (decode: T_q = B, one row per sequence)
 *   k_pages, v_pages  [num_pages][H_kv][P][D]
 *   block_table       [B][max_pages_per_seq]  int32
 *   context_lens      [B]  int32
 *   query_start_loc   [B+1] int32 (row offsets of each sequence's chunk)
 * dtype 0: bf16 bit patterns (uint16), dtype 1: fp32.  out is always fp32.
 * A row that sees no key (context 0) is defined as zeros.
 *
 * Return codes: 0 ok, -1 invalid argument (null pointer, inconsistent sizes,
 * block-table entry outside the pool, row offsets not monotone), -2 out of
 * memory.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

static int g_threads = 0; /* 0 = OpenMP default */

void oracle_set_threads(int n) { g_threads = n; }

int oracle_get_threads(void) {
#ifdef _OPENMP
  return g_threads > 0 ? g_threads : omp_get_max_threads();
#else
  return 1;
#endif
}

/* bf16 is the upper half of an IEEE fp32 word: widening is exact. */
static float bf16_bits_to_float(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  memcpy(&f, &u, sizeof f);
  return f;
}

static float load_elem(const void *base, int dtype, int64_t idx) {
  if (dtype == 0) return bf16_bits_to_float(((const uint16_t *)base)[idx]);
  return ((const float *)base)[idx];
}

typedef struct {
  const void *q, *k, *v;
  int dtype;
  const int32_t *block_table, *context_lens, *query_start_loc;
  int32_t B, H_q, H_kv, D, P, num_pages, max_pages_per_seq;
  float scale;
} problem_t;

/* Element index of dimension 0 of token t of sequence b in kv head g: the
 * block-table gather (page = table[b][t / P], slot = t % P). */
static int64_t kv_offset(const problem_t *p, int32_t b, int32_t t, int32_t g) {
  int32_t page = p->block_table[(int64_t)b * p->max_pages_per_seq + t / p->P];
  int32_t slot = t % p->P;
  return (((int64_t)page * p->H_kv + g) * p->P + slot) * p->D;
}

static int check_tables(const problem_t *p) {
  for (int32_t b = 0; b < p->B; ++b) {
    int32_t c = p->context_lens[b];
    if (c < 0) return -1;
    int32_t npg = (c + p->P - 1) / p->P;
    if (npg > p->max_pages_per_seq) return -1;
    for (int32_t i = 0; i < npg; ++i) {
      int32_t pg = p->block_table[(int64_t)b * p->max_pages_per_seq + i];
      if (pg < 0 || pg >= p->num_pages) return -1;
    }
    if (p->query_start_loc) {
      int32_t L = p->query_start_loc[b + 1] - p->query_start_loc[b];
      if (L < 0 || L > c) return -1;
    }
  }
  if (p->query_start_loc && p->query_start_loc[0] != 0) return -1;
  return 0;
}

/* One (sequence b, chunk row r of L, query head h): out_row[D] in fp32.
 * x is caller-provided scratch of at least context_lens[b] floats. */
static void attend_row(const problem_t *p, int32_t b, int32_t r, int32_t L,
                       int64_t qrow, int32_t h, float *x, float *out_row) {
  const int32_t s = p->H_q / p->H_kv;
  const int32_t g = h / s;
  const int32_t C = p->context_lens[b];
  const int32_t n_vis = C - L + r + 1; /* keys at positions 0 .. C-L+r */
  const int64_t q0 = (qrow * p->H_q + h) * p->D;
  int32_t t, d;

  for (d = 0; d < p->D; ++d) out_row[d] = 0.0f;
  if (C <= 0 || n_vis <= 0) return;

  /* pass 1: logits x_t = (q . k_t) * scale and their maximum */
  float m = -INFINITY;
  for (t = 0; t < n_vis; ++t) {
    const int64_t k0 = kv_offset(p, b, t, g);
    float acc = 0.0f;
    for (d = 0; d < p->D; ++d)
      acc += load_elem(p->q, p->dtype, q0 + d) * load_elem(p->k, p->dtype, k0 + d);
    x[t] = acc * p->scale;
    if (x[t] > m) m = x[t];
  }
  /* pass 2: unnormalised weights w_t = exp(x_t - m) and their sum l */
  float l = 0.0f;
  for (t = 0; t < n_vis; ++t) {
    x[t] = expf(x[t] - m);
    l += x[t];
  }
  /* pass 3: out = (sum_t w_t v_t) / l, one division per element */
  for (t = 0; t < n_vis; ++t) {
    const int64_t v0 = kv_offset(p, b, t, g);
    for (d = 0; d < p->D; ++d)
      out_row[d] += x[t] * load_elem(p->v, p->dtype, v0 + d);
  }
  for (d = 0; d < p->D; ++d) out_row[d] = out_row[d] / l;
}

static int run(const problem_t *p, int32_t total_rows, float *out) {
  /* Flatten (row, head) work items; rows are located by a linear scan. */
  int64_t *row_seq = (int64_t *)malloc(sizeof(int64_t) * (size_t)(total_rows > 0 ? total_rows : 1));
  if (!row_seq) return -2;
  for (int32_t b = 0; b < p->B; ++b) {
    int32_t r0 = p->query_start_loc ? p->query_start_loc[b] : b;
    int32_t r1 = p->query_start_loc ? p->query_start_loc[b + 1] : b + 1;
    for (int32_t r = r0; r < r1; ++r) row_seq[r] = b;
  }
  int32_t max_ctx = 1;
  for (int32_t b = 0; b < p->B; ++b)
    if (p->context_lens[b] > max_ctx) max_ctx = p->context_lens[b];

  const int64_t items = (int64_t)total_rows * p->H_q;
  int failed = 0;
#pragma omp parallel num_threads(oracle_get_threads())
  {
    float *x = (float *)malloc(sizeof(float) * (size_t)max_ctx);
    if (!x) {
#pragma omp atomic write
      failed = 1;
    } else {
#pragma omp for schedule(dynamic, 4)
      for (int64_t it = 0; it < items; ++it) {
        const int64_t row = it / p->H_q;
        const int32_t h = (int32_t)(it % p->H_q);
        const int32_t b = (int32_t)row_seq[row];
        int32_t r0 = p->query_start_loc ? p->query_start_loc[b] : b;
        int32_t L = p->query_start_loc ? p->query_start_loc[b + 1] - r0 : 1;
        attend_row(p, b, (int32_t)(row - r0), L, row, h, x, out + (row * p->H_q + h) * p->D);
      }
      free(x);
    }
  }
  free(row_seq);
  return failed ? -2 : 0;
}

static int fill_problem(problem_t *p, const void *q, const void *k, const void *v, int dtype,
                        const int32_t *block_table, int32_t max_pages_per_seq,
                        const int32_t *context_lens, const int32_t *query_start_loc, int32_t B,
                        int32_t H_q, int32_t H_kv, int32_t D, int32_t P, int32_t num_pages,
                        float scale) {
  if (!q || !k || !v || !block_table || !context_lens) return -1;
  if (dtype != 0 && dtype != 1) return -1;
  if (B < 0 || H_q <= 0 || H_kv <= 0 || D <= 0 || P <= 0 || num_pages < 0) return -1;
  if (H_q % H_kv != 0 || max_pages_per_seq < 0) return -1;
  p->q = q; p->k = k; p->v = v; p->dtype = dtype;
  p->block_table = block_table; p->context_lens = context_lens;
  p->query_start_loc = query_start_loc;
  p->B = B; p->H_q = H_q; p->H_kv = H_kv; p->D = D; p->P = P;
  p->num_pages = num_pages; p->max_pages_per_seq = max_pages_per_seq;
  p->scale = scale;
  return check_tables(p);
}

/* Decode: one query row per sequence (q, out: [B][H_q][D]). */
int oracle_paged_attn(const void *q, const void *k_pages, const void *v_pages, int dtype,
                      const int32_t *block_table, int32_t max_pages_per_seq,
                      const int32_t *context_lens, int32_t B, int32_t H_q, int32_t H_kv,
                      int32_t D, int32_t P, int32_t num_pages, float scale, float *out) {
  problem_t p;
  if (!out) return -1;
  int rc = fill_problem(&p, q, k_pages, v_pages, dtype, block_table, max_pages_per_seq,
                        context_lens, NULL, B, H_q, H_kv, D, P, num_pages, scale);
  if (rc) return rc;
  return run(&p, B, out);
}

/* Varlen: sequence b owns query rows query_start_loc[b] .. query_start_loc[b+1]-1
 * (a decode sequence has one row, a prefill chunk several), q/out [T_q][H_q][D]
 * with T_q = query_start_loc[B]. */
int oracle_paged_attn_varlen(const void *q, const void *k_pages, const void *v_pages, int dtype,
                             const int32_t *block_table, int32_t max_pages_per_seq,
                             const int32_t *context_lens, const int32_t *query_start_loc,
                             int32_t B, int32_t H_q, int32_t H_kv, int32_t D, int32_t P,
                             int32_t num_pages, float scale, float *out) {
  problem_t p;
  if (!out || !query_start_loc) return -1;
  for (int32_t b = 0; b < B; ++b)
    if (query_start_loc[b + 1] < query_start_loc[b]) return -1;
  int rc = fill_problem(&p, q, k_pages, v_pages, dtype, block_table, max_pages_per_seq,
                        context_lens, query_start_loc, B, H_q, H_kv, D, P, num_pages, scale);
  if (rc) return rc;
  return run(&p, B > 0 ? query_start_loc[B] : 0, out);
}

/* Flat pool row (page * P + slot) of every cached token, sequence-major:
 * rows_out has sum_b context_lens[b] entries. */
int oracle_gather_indices(const int32_t *block_table, int32_t max_pages_per_seq,
                          const int32_t *context_lens, int32_t B, int32_t P, int32_t num_pages,
                          int64_t *rows_out) {
  if (!block_table || !context_lens || !rows_out || B < 0 || P <= 0) return -1;
  int64_t n = 0;
  for (int32_t b = 0; b < B; ++b) {
    const int32_t C = context_lens[b];
    if (C < 0 || (C + P - 1) / P > max_pages_per_seq) return -1;
    for (int32_t t = 0; t < C; ++t) {
      const int32_t page = block_table[(int64_t)b * max_pages_per_seq + t / P];
      if (page < 0 || page >= num_pages) return -1;
      rows_out[n++] = (int64_t)page * P + t % P;
    }
  }
  return 0;
}

/* Normalised softmax weights w_t / l of one (sequence b, chunk row r, head h);
 * w_out receives n_vis = C - L + r + 1 values (L = chunk length, 1 for decode).
 * Returns n_vis, or a negative error code. */
int oracle_softmax_weights(const void *q, const void *k_pages, int dtype,
                           const int32_t *block_table, int32_t max_pages_per_seq,
                           const int32_t *context_lens, int32_t B, int32_t H_q, int32_t H_kv,
                           int32_t D, int32_t P, int32_t num_pages, float scale, int32_t b,
                           int32_t L, int32_t r, int64_t qrow, int32_t h, float *w_out) {
  problem_t p;
  if (!w_out || b < 0 || b >= B || h < 0 || h >= H_q || L < 1 || r < 0 || r >= L) return -1;
  int rc = fill_problem(&p, q, k_pages, k_pages, dtype, block_table, max_pages_per_seq,
                        context_lens, NULL, B, H_q, H_kv, D, P, num_pages, scale);
  if (rc) return rc;
  const int32_t s = H_q / H_kv, g = h / s, C = context_lens[b];
  const int32_t n_vis = C - L + r + 1;
  if (n_vis <= 0) return 0;
  const int64_t q0 = (qrow * H_q + h) * D;
  float m = -INFINITY, l = 0.0f;
  for (int32_t t = 0; t < n_vis; ++t) {
    const int64_t k0 = kv_offset(&p, b, t, g);
    float acc = 0.0f;
    for (int32_t d = 0; d < D; ++d)
      acc += load_elem(q, dtype, q0 + d) * load_elem(k_pages, dtype, k0 + d);
    w_out[t] = acc * scale;
    if (w_out[t] > m) m = w_out[t];
  }
  for (int32_t t = 0; t < n_vis; ++t) {
    w_out[t] = expf(w_out[t] - m);
    l += w_out[t];
  }
  for (int32_t t = 0; t < n_vis; ++t) w_out[t] = w_out[t] / l;
  return n_vis;
}

/* KV append: the step right before attention.  The new tokens' keys and values
 * are stored into the paged cache, and attention then runs over the cache
 * (Sec. 6.4: the task that receives a decode token's pre-attention K/V stores
 * it in the KV cache before it attends).
 *
 * Sequence b appends L_b tokens, which are the last L_b positions of its
 * context: with query_start_loc, row query_start_loc[b] + j (j < L_b) holds
 * position context_lens[b] - L_b + j; without it (decode), row b holds position
 * context_lens[b] - 1, and a sequence with context 0 appends nothing.  For each
 * such row and kv head g, the D elements k_new[row][g][.] and v_new[row][g][.]
 * are copied bit for bit into kv head g of slot (position % P) of page
 * block_table[b][position / P].  Nothing else in the pools changes.
 *   k_new, v_new      [T][H_kv][D], elements of elem_bytes bytes (2: bf16, 4: fp32)
 *   k_pages, v_pages  [num_pages][H_kv][P][D], updated in place
 * Returns 0, or -1 (null pointer, bad sizes, L_b > context_lens[b], row offsets
 * not monotone, or a written position whose page entry is outside the pool or
 * the table row); on -1 the pools are unchanged. */
int oracle_kv_append(const void *k_new, const void *v_new, int32_t elem_bytes,
                     const int32_t *block_table, int32_t max_pages_per_seq,
                     const int32_t *context_lens, const int32_t *query_start_loc, int32_t B,
                     int32_t H_kv, int32_t D, int32_t P, int32_t num_pages, void *k_pages,
                     void *v_pages) {
  if (!k_new || !v_new || !block_table || !context_lens || !k_pages || !v_pages) return -1;
  if (elem_bytes != 2 && elem_bytes != 4) return -1;
  if (B < 0 || H_kv <= 0 || D <= 0 || P <= 0 || num_pages < 0 || max_pages_per_seq < 0) return -1;
  if (query_start_loc && B > 0 && query_start_loc[0] != 0) return -1;
  /* validate everything first, so that a failure leaves the pools unchanged */
  for (int32_t b = 0; b < B; ++b) {
    const int32_t C = context_lens[b];
    int32_t L;
    if (query_start_loc) {
      L = query_start_loc[b + 1] - query_start_loc[b];
      if (L < 0) return -1;
    } else {
      L = C > 0 ? 1 : 0;
    }
    if (C < 0 || L > C) return -1;
    for (int32_t j = 0; j < L; ++j) {
      const int32_t pos = C - L + j;
      if (pos / P >= max_pages_per_seq) return -1;
      const int32_t page = block_table[(int64_t)b * max_pages_per_seq + pos / P];
      if (page < 0 || page >= num_pages) return -1;
    }
  }
  const size_t row_bytes = (size_t)D * (size_t)elem_bytes;
  for (int32_t b = 0; b < B; ++b) {
    const int32_t C = context_lens[b];
    const int32_t L = query_start_loc ? query_start_loc[b + 1] - query_start_loc[b] : (C > 0 ? 1 : 0);
    const int64_t row0 = query_start_loc ? query_start_loc[b] : b;
    for (int32_t j = 0; j < L; ++j) {
      const int32_t pos = C - L + j;
      const int32_t page = block_table[(int64_t)b * max_pages_per_seq + pos / P];
      const int32_t slot = pos % P;
      for (int32_t g = 0; g < H_kv; ++g) {
        const size_t src = ((size_t)(row0 + j) * H_kv + g) * row_bytes;
        const size_t dst = (((size_t)page * H_kv + g) * P + slot) * row_bytes;
        memcpy((char *)k_pages + dst, (const char *)k_new + src, row_bytes);
        memcpy((char *)v_pages + dst, (const char *)v_new + src, row_bytes);
      }
    }
  }
  return 0;
}

/* Scheduler step: the GPU-resident page allocator and block-table builder of
 * the paper's Resource-Aware Scheduler (Sec. 6: a prefill scheduler holding a
 * queue of waiting sequences and a decode scheduler that estimates the KV
 * blocks the next token needs, garbage-collects finished sequences and, when
 * blocks run short, preempts the newest decode sequences, which re-enter the
 * prefill queue ahead of new arrivals while admission pauses).
 *
 * State (updated in place): a stack of free pages free_pages[0 .. hdr[0]-1]
 * (top = last); hdr = {free count, next admission order, queue head, queue
 * length}; a circular queue of Q entries (logical id, tokens to prefill,
 * finish length); per slot: logical id (-1 = empty), admission order, finish
 * length, context length, block-table row of MP entries.  Pages hold 16
 * tokens.  One step:
 *   0. append the arrivals (valid: 1 <= prompt <= finish <= MP*16) at the
 *      queue tail while the queue keeps S entries free for preemption;
 *   1. free every slot whose context reached its finish length (its pages are
 *      pushed in slot order, page order), reporting its id;
 *   2. a decode slot needs a page iff its context is a multiple of 16;
 *   3. if more pages are needed than free, preempt the newest decode slots
 *      (largest admission order) until the rest fit: their pages are pushed
 *      (slot order) and they re-enter the queue front, lowest slot nearest the
 *      head, to prefill their whole context again; no admission this step;
 *   4. each remaining decode slot (slot order) pops its page if it needs one,
 *      and its context grows by one (this step's token);
 *   5. otherwise admit queue-head entries in order while their tokens stay
 *      within what the pass has left (n_real, the pipeline's token capacity
 *      per pass, minus the decode rows of step 4), their pages fit and empty
 *      slots remain: the i-th
 *      admitted takes the i-th lowest empty slot and pops its pages in order;
 *      its context is the prefilled length;
 *   6. rows: 1 per decode slot, the prefilled length per admitted slot, 0
 *      otherwise; query_start_loc[S+1] is their prefix sum.
 * info = {mode (1 = preemption), finished, preempted, admitted, decode slots,
 * accepted arrivals, free pages after, total rows}.  Returns 0, or -1 (and
 * changes nothing) on bad sizes or a state that is not one the step can
 * produce: a page index out of range, a context or finish length past the
 * table, a queued entry with no tokens or more tokens than its finish length,
 * more pages held and free than the pool has, or more sequences queued
 * and seated than the queue holds (steps 0 and 3 keep that sum within Q, so
 * preempted entries always fit). */
int oracle_schedule_step(int32_t *free_pages, int32_t *hdr, int32_t *queue_seq, int32_t *queue_tok,
                         int32_t *queue_fin, int32_t *slot_seq, int32_t *slot_order,
                         int32_t *slot_fin, int32_t *context_lens, int32_t *block_table,
                         int32_t S, int32_t P, int32_t MP, int32_t Q, int32_t n_real,
                         const int32_t *new_seq, const int32_t *new_prompt, const int32_t *new_fin,
                         int32_t n_new, int32_t *query_start_loc, int32_t *finished_out,
                         int32_t *info) {
  if (!free_pages || !hdr || !queue_seq || !queue_tok || !queue_fin || !slot_seq || !slot_order ||
      !slot_fin || !context_lens || !block_table || !query_start_loc || !finished_out || !info)
    return -1;
  if (S <= 0 || P < 0 || MP <= 0 || Q <= S || n_real < 0 || n_new < 0) return -1;
  if (n_new > 0 && (!new_seq || !new_prompt || !new_fin)) return -1;
  int32_t free_n = hdr[0], head = hdr[2], qlen = hdr[3];
  if (free_n < 0 || free_n > P || head < 0 || head >= Q || qlen < 0 || qlen > Q) return -1;
  int64_t held = 0, occupied = 0;
  for (int32_t s = 0; s < S; ++s) {
    if (slot_seq[s] < 0) continue;
    const int32_t c = context_lens[s];
    if (c < 1 || slot_fin[s] > MP * 16 || (c + 15) / 16 > MP) return -1;
    for (int32_t p = 0; p < (c + 15) / 16; ++p) {
      const int32_t pg = block_table[(int64_t)s * MP + p];
      if (pg < 0 || pg >= P) return -1;
    }
    held += (c + 15) / 16;
    ++occupied;
  }
  if (free_n + held > P || qlen + occupied > Q) return -1;
  for (int32_t k = 0; k < qlen; ++k) {
    const int32_t at = (int32_t)(((int64_t)head + k) % Q);
    if (queue_tok[at] < 1 || queue_fin[at] < queue_tok[at] || queue_fin[at] > MP * 16) return -1;
  }
  for (int i = 0; i < 8; ++i) info[i] = 0;
  int32_t *rows = (int32_t *)calloc((size_t)S, sizeof(int32_t));
  char *pre = (char *)calloc((size_t)S, 1);
  if (!rows || !pre) {
    free(rows);
    free(pre);
    return -2;
  }
  /* 0. arrivals */
  for (int32_t i = 0; i < n_new; ++i) {
    const int32_t pl = new_prompt[i], fin = new_fin[i];
    if (pl < 1 || fin < pl || fin > MP * 16 || qlen >= Q - S) continue;
    const int32_t at = (head + qlen) % Q;
    queue_seq[at] = new_seq[i];
    queue_tok[at] = pl;
    queue_fin[at] = fin;
    ++qlen;
    ++info[5];
  }
  /* 1. finished slots */
  for (int32_t s = 0; s < S; ++s) {
    if (slot_seq[s] < 0 || context_lens[s] < slot_fin[s]) continue;
    finished_out[info[1]++] = slot_seq[s];
    for (int32_t p = 0; p < (context_lens[s] + 15) / 16; ++p)
      free_pages[free_n++] = block_table[(int64_t)s * MP + p];
    slot_seq[s] = -1;
    context_lens[s] = 0;
  }
  /* 2. pages the decode slots need */
  int32_t need = 0;
  for (int32_t s = 0; s < S; ++s)
    if (slot_seq[s] >= 0 && context_lens[s] % 16 == 0) ++need;
  /* 3. preemption: newest first until the rest fit */
  if (need > free_n) {
    info[0] = 1;
    int32_t avail = free_n;
    while (need > avail) {
      int32_t newest = -1;
      for (int32_t s = 0; s < S; ++s)
        if (slot_seq[s] >= 0 && !pre[s] && (newest < 0 || slot_order[s] > slot_order[newest])) newest = s;
      pre[newest] = 1;
      avail += (context_lens[newest] + 15) / 16;
      if (context_lens[newest] % 16 == 0) --need;
    }
    int32_t n_pre = 0;
    for (int32_t s = 0; s < S; ++s) n_pre += pre[s];
    head = ((head - n_pre) % Q + Q) % Q;
    int32_t k = 0;
    for (int32_t s = 0; s < S; ++s) {
      if (!pre[s]) continue;
      for (int32_t p = 0; p < (context_lens[s] + 15) / 16; ++p)
        free_pages[free_n++] = block_table[(int64_t)s * MP + p];
      const int32_t at = (head + k++) % Q;
      queue_seq[at] = slot_seq[s];
      queue_tok[at] = context_lens[s];
      queue_fin[at] = slot_fin[s];
      slot_seq[s] = -1;
      context_lens[s] = 0;
    }
    qlen += n_pre;
    info[2] = n_pre;
  }
  /* 4. decode tokens */
  for (int32_t s = 0; s < S; ++s) {
    if (slot_seq[s] < 0) continue;
    if (context_lens[s] % 16 == 0) block_table[(int64_t)s * MP + context_lens[s] / 16] = free_pages[--free_n];
    context_lens[s] += 1;
    rows[s] = 1;
    ++info[4];
  }
  /* 5. admission */
  if (!info[0]) {
    const int32_t token_budget = n_real - info[4];
    int32_t tokens = 0;
    while (qlen > 0) {
      const int32_t len = queue_tok[head], pages = (len + 15) / 16;
      int32_t slot = -1;
      for (int32_t s = 0; s < S && slot < 0; ++s)
        if (slot_seq[s] < 0 && rows[s] == 0) slot = s;
      if (slot < 0 || tokens + len > token_budget || pages > free_n) break;
      for (int32_t j = 0; j < pages; ++j) block_table[(int64_t)slot * MP + j] = free_pages[--free_n];
      slot_seq[slot] = queue_seq[head];
      slot_order[slot] = hdr[1]++;
      slot_fin[slot] = queue_fin[head];
      context_lens[slot] = len;
      rows[slot] = len;
      tokens += len;
      head = (head + 1) % Q;
      --qlen;
      ++info[3];
    }
  }
  /* 6. rows */
  query_start_loc[0] = 0;
  for (int32_t s = 0; s < S; ++s) query_start_loc[s + 1] = query_start_loc[s] + rows[s];
  info[6] = free_n;
  info[7] = query_start_loc[S];
  hdr[0] = free_n;
  hdr[2] = head;
  hdr[3] = qlen;
  free(rows);
  free(pre);
  return 0;
}
