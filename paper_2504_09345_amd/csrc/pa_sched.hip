// One step of the GPU-resident scheduler that feeds the attention calls: the
// page allocator and block-table builder of the Resource-Aware Scheduler
// (MoE-Lens Sec. 6.2).  The paper keeps both schedulers' state in GPU memory
// and runs them on the GPU; here one step is one kernel launch, so a serving
// loop never waits on the host between passes.
//
// State (device memory, updated in place): a stack of free 16-token pages, a
// circular queue of sequences waiting to prefill (logical id, tokens to
// prefill, finish length), and per batch slot the logical id (-1 = empty),
// admission order, finish length, context length and block-table row.  One
// step:
//   0. queue the arrivals that are valid, while the queue keeps num_slots
//      entries free (room for every preemption);
//   1. garbage-collect the slots whose context reached its finish length;
//   2. count the decode slots whose next token opens a page;
//   3. if the free pages do not cover them, enter preemption mode: preempt the
//      newest slots (largest admission order) until the rest fit, push their
//      pages and re-queue them ahead of the queue head to prefill their whole
//      context again; admission pauses this step;
//   4. every remaining decode slot takes its page if it needs one and counts
//      this step's token;
//   5. in normal mode admit queue-head sequences in order while their tokens
//      fit the pass (n_real, the pipeline's tokens per pass, minus the decode
//      rows), their pages fit and empty slots remain;
//   6. write the rows of the pass: 1 per decode slot, the prefilled length per
//      admitted slot, as a prefix sum (the attention calls' query_start_loc).
// Every order ("slot order", "queue order", "page order") is fixed, so the
// result is a deterministic function of the state.
//
// Mapping: one workgroup of 1024 threads; thread t owns the K consecutive
// slots t*K .. t*K+K-1 in registers.  Each ordered step is a block-wide
// prefix sum over the threads (DPP lane scans + one LDS round), and the page
// moves of a step (a variable number of pages per sequence) are flattened:
// every thread takes page f, f + 1024, ... of the step's total and finds its
// sequence by binary search over the step's page prefix in LDS.  The
// preemption set "the newest slots until the rest fit" is the set of live
// slots with order >= t*, where t* is the largest order threshold whose slots
// free enough pages and page demands; the kernel finds t* by binary search
// over the orders with one block-wide sum per probe.
#include <climits>

#include "pa_device.h"
#include "pa_kernels.h"
#include "pa_sched.h"

namespace pa {

namespace {

constexpr int kSchedWaves = kSchedThreads / 64;

struct I4 {
  int x, y, z, w;
};

struct SchedSmem {
  int wave[2][kSchedWaves][4];  // per-wave totals, two rounds in flight
  int32_t seq[kSchedMaxSlots];  // slot of the j-th moved sequence of a step
  int32_t empty[kSchedMaxSlots];  // j-th empty slot (admission)
  int32_t pref[kSchedMaxSlots + 1];  // page prefix of the moved sequences
};

// Block-wide exclusive prefix sum of four counters; `round` alternates the
// LDS buffer so one barrier per call suffices (a buffer is rewritten two
// calls later, after every thread has passed the barrier of the call in
// between).  All threads must call it the same number of times.
struct Scanner {
  SchedSmem& sm;
  int round;
  __device__ I4 scan(I4 v, I4& total) {
    const I4 inc{wave_incl_scan(v.x), wave_incl_scan(v.y), wave_incl_scan(v.z), wave_incl_scan(v.w)};
    const int w = threadIdx.x >> 6;
    int(*buf)[4] = sm.wave[round & 1];
    ++round;
    if ((threadIdx.x & 63) == 63) {
      buf[w][0] = inc.x;
      buf[w][1] = inc.y;
      buf[w][2] = inc.z;
      buf[w][3] = inc.w;
    }
    __syncthreads();
    I4 before{0, 0, 0, 0};
    total = I4{0, 0, 0, 0};
#pragma unroll
    for (int i = 0; i < kSchedWaves; ++i) {
      const int a = buf[i][0], b = buf[i][1], c = buf[i][2], d = buf[i][3];
      if (i < w) {
        before.x += a;
        before.y += b;
        before.z += c;
        before.w += d;
      }
      total.x += a;
      total.y += b;
      total.z += c;
      total.w += d;
    }
    return I4{inc.x - v.x + before.x, inc.y - v.y + before.y, inc.z - v.z + before.z, inc.w - v.w + before.w};
  }
  __device__ int sum(int v) {
    I4 t;
    scan(I4{v, 0, 0, 0}, t);
    return t.x;
  }
  // min and max over the block (values of non-participants: INT_MAX / INT_MIN)
  __device__ void min_max(int lo, int hi, int& out_lo, int& out_hi) {
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      lo = min(lo, __shfl_xor(lo, off, 64));
      hi = max(hi, __shfl_xor(hi, off, 64));
    }
    const int w = threadIdx.x >> 6;
    int(*buf)[4] = sm.wave[round & 1];
    ++round;
    if ((threadIdx.x & 63) == 0) {
      buf[w][0] = lo;
      buf[w][1] = hi;
    }
    __syncthreads();
    out_lo = buf[0][0];
    out_hi = buf[0][1];
#pragma unroll
    for (int i = 1; i < kSchedWaves; ++i) {
      out_lo = min(out_lo, buf[i][0]);
      out_hi = max(out_hi, buf[i][1]);
    }
  }
};

__device__ __forceinline__ int pages_of(int tokens) { return (tokens + kPage - 1) / kPage; }

__device__ __forceinline__ int ring(int64_t i, int Q) { return (int)(((i % Q) + Q) % Q); }

// Page f of a step's flattened moves belongs to sequence j with
// pref[j] <= f < pref[j + 1] (n sequences, each holding >= 1 page).
__device__ __forceinline__ int find_seq(const int32_t* pref, int n, int f) {
  int lo = 0, hi = n;
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (pref[mid] <= f) lo = mid;
    else hi = mid;
  }
  return lo;
}

// Push the pages of the step's moved sequences (LDS seq/pref, n of them,
// `total` pages) onto the free stack above `base`, in sequence order and page
// order.
__device__ __forceinline__ void push_pages(const SchedArgs& a, const SchedSmem& sm, int n, int total, int base) {
  for (int f = threadIdx.x; f < total; f += kSchedThreads) {
    const int j = find_seq(sm.pref, n, f);
    const int s = sm.seq[j];
    a.free_pages[base + f] = a.block_table[(int64_t)s * a.MP + (f - sm.pref[j])];
  }
}

template <int K>
__global__ __launch_bounds__(kSchedThreads) void sched_kernel(SchedArgs a) {
  __shared__ SchedSmem sm;
  Scanner sc{sm, 0};
  const int tid = threadIdx.x;
  const int S = a.S, MP = a.MP, Q = a.Q;
  const int max_tokens = MP * kPage;

  int free_n = a.hdr[0], next_order = a.hdr[1], head = a.hdr[2], qlen = a.hdr[3];
  int seq[K], ord[K], fin[K], ctx[K], rows[K];
#pragma unroll
  for (int i = 0; i < K; ++i) {
    const int s = tid * K + i;
    const bool in = s < S;
    seq[i] = in ? a.slot_seq[s] : -1;
    ord[i] = in ? a.slot_order[s] : 0;
    fin[i] = in ? a.slot_fin[s] : 0;
    ctx[i] = in ? a.context_lens[s] : 0;
    rows[i] = 0;
  }
  // Loads that depend on nothing the step computes are issued now, beside the
  // state: the first chunk of arrivals, and the queue entries j = t*K .. t*K+K-1
  // (validation reads every queued entry; admission takes the head ones)
  const int qlen0 = qlen;
  const bool hdr_in = head >= 0 && head < Q && qlen >= 0 && qlen <= Q;
  int a_pl = 0, a_fl = 0, a_id = 0;
  if (tid < a.n_new) {
    a_pl = a.new_prompt[tid];
    a_fl = a.new_fin[tid];
    a_id = a.new_seq[tid];
  }
  // (up to two slots per thread: more would spill registers; larger grids
  // read the entries where they are used)
  constexpr bool kPre = K <= 2;
  int qtk[K], qfn[K], qid[K];
#pragma unroll
  for (int i = 0; i < K; ++i) {
    const int j = tid * K + i;
    qtk[i] = qfn[i] = qid[i] = 0;
    if (kPre && hdr_in && j < qlen) {
      const int q = ring((int64_t)head + j, Q);
      qtk[i] = a.queue_tok[q];
      qfn[i] = a.queue_fin[q];
      qid[i] = a.queue_seq[q];
    }
  }

  // --- the state must be one a step can produce --------------------------
  const bool hdr_bad = free_n < 0 || free_n > a.P || head < 0 || head >= Q || qlen < 0 || qlen > Q;
  {
    int bad = 0, held = 0, occ = 0;
#pragma unroll
    for (int i = 0; i < K; ++i) {
      if (seq[i] < 0) continue;
      if (ctx[i] < 1 || fin[i] > max_tokens || ctx[i] > max_tokens) bad = 1;
      held += bad ? 0 : pages_of(ctx[i]);
      ++occ;
    }
    if (!hdr_bad) {
      if constexpr (kPre) {
#pragma unroll
        for (int i = 0; i < K; ++i)
          if (tid * K + i < qlen && (qtk[i] < 1 || qfn[i] < qtk[i] || qfn[i] > max_tokens)) bad = 1;
      }
      for (int k = (kPre ? K * kSchedThreads : 0) + tid; k < qlen; k += kSchedThreads) {  // not prefetched
        const int q = ring((int64_t)head + k, Q);
        const int tk = a.queue_tok[q], fq = a.queue_fin[q];
        if (tk < 1 || fq < tk || fq > max_tokens) bad = 1;
      }
    }
    I4 t;
    sc.scan(I4{bad, held, occ, 0}, t);
    if (hdr_bad || t.x != 0 || (int64_t)free_n + t.y > a.P || (int64_t)qlen + t.z > Q) {
      if (tid == 0) {
        a.info[0] = -1;
        for (int i = 1; i < 8; ++i) a.info[i] = 0;
      }
      return;  // uniform: every thread took the same branch
    }
  }

  // --- 0. arrivals --------------------------------------------------------
  const int cap = max(0, Q - S - qlen);
  int valid_total = 0;
  for (int base = 0; base < a.n_new; base += kSchedThreads) {
    const int i = base + tid;
    int ok = 0, pl = 0, fl = 0, id = 0;
    if (i < a.n_new) {
      if (base == 0) {
        pl = a_pl;
        fl = a_fl;
        id = a_id;
      } else {
        pl = a.new_prompt[i];
        fl = a.new_fin[i];
        id = a.new_seq[i];
      }
      ok = pl >= 1 && fl >= pl && fl <= max_tokens;
    }
    I4 t;
    const int r = valid_total + sc.scan(I4{ok, 0, 0, 0}, t).x;
    if (ok && r < cap) {
      const int q = ring((int64_t)head + qlen + r, Q);
      a.queue_seq[q] = id;
      a.queue_tok[q] = pl;
      a.queue_fin[q] = fl;
    }
    valid_total += t.x;
  }
  const int accepted = min(valid_total, cap);
  qlen += accepted;

  // --- 1. finished slots, 2. page demand ----------------------------------
  int n_fin, need, live, need_before;  // need_before: needers in earlier threads
  {
    int nf = 0, pf = 0, nd = 0, nl = 0;
#pragma unroll
    for (int i = 0; i < K; ++i) {
      if (seq[i] < 0) continue;
      if (ctx[i] >= fin[i]) {
        ++nf;
        pf += pages_of(ctx[i]);
      } else {
        ++nl;
        nd += ctx[i] % kPage == 0;
      }
    }
    I4 t;
    const I4 ex = sc.scan(I4{nf, pf, nd, nl}, t);
    need_before = ex.z;
    int r = ex.x, pr = ex.y;
#pragma unroll
    for (int i = 0; i < K; ++i) {
      if (seq[i] < 0 || ctx[i] < fin[i]) continue;
      const int s = tid * K + i;
      a.finished_out[r] = seq[i];
      sm.seq[r] = s;
      sm.pref[r] = pr;
      ++r;
      pr += pages_of(ctx[i]);
      seq[i] = -1;
      ctx[i] = 0;
      a.slot_seq[s] = -1;
      a.context_lens[s] = 0;
    }
    if (tid == 0) sm.pref[t.x] = t.y;
    __syncthreads();
    push_pages(a, sm, t.x, t.y, free_n);
    free_n += t.y;
    n_fin = t.x;
    need = t.z;
    live = t.w;
    __syncthreads();  // pushed pages visible; LDS lists free again
  }

  // --- 3. preemption --------------------------------------------------------
  int mode = 0, n_pre = 0;
  if (need > free_n) {
    mode = 1;
    const int deficit = need - free_n;
    int lo_mine = INT_MAX, hi_mine = INT_MIN;
#pragma unroll
    for (int i = 0; i < K; ++i) {
      if (seq[i] < 0) continue;
      lo_mine = min(lo_mine, ord[i]);
      hi_mine = max(hi_mine, ord[i]);
    }
    int lo, hi;
    sc.min_max(lo_mine, hi_mine, lo, hi);
    // f(t) = sum over live slots with order >= t of (pages + opens-a-page);
    // f(lo) covers every live slot, so f(lo) >= need >= deficit; f(hi+1) = 0.
    int64_t hi_ex = (int64_t)hi + 1;
    while (hi_ex - lo > 1) {
      const int mid = (int)(lo + ((hi_ex - lo) >> 1));
      int f = 0;
#pragma unroll
      for (int i = 0; i < K; ++i)
        if (seq[i] >= 0 && ord[i] >= mid) f += pages_of(ctx[i]) + (ctx[i] % kPage == 0);
      if (sc.sum(f) >= deficit) lo = mid;
      else hi_ex = mid;
    }
    int pc = 0, pp = 0, pn = 0;
#pragma unroll
    for (int i = 0; i < K; ++i) {
      if (seq[i] < 0 || ord[i] < lo) continue;
      ++pc;
      pp += pages_of(ctx[i]);
      pn += ctx[i] % kPage == 0;
    }
    I4 t;
    const I4 ex = sc.scan(I4{pc, pp, pn, 0}, t);
    n_pre = t.x;
    const int new_head = ring((int64_t)head - n_pre, Q);
    int r = ex.x, pr = ex.y;
#pragma unroll
    for (int i = 0; i < K; ++i) {
      if (seq[i] < 0 || ord[i] < lo) continue;
      const int s = tid * K + i;
      const int q = ring((int64_t)new_head + r, Q);
      a.queue_seq[q] = seq[i];
      a.queue_tok[q] = ctx[i];
      a.queue_fin[q] = fin[i];
      sm.seq[r] = s;
      sm.pref[r] = pr;
      ++r;
      pr += pages_of(ctx[i]);
      seq[i] = -1;
      ctx[i] = 0;
      a.slot_seq[s] = -1;
      a.context_lens[s] = 0;
    }
    if (tid == 0) sm.pref[t.x] = t.y;
    __syncthreads();
    push_pages(a, sm, t.x, t.y, free_n);
    free_n += t.y;
    need -= t.z;
    live -= n_pre;
    head = new_head;
    qlen += n_pre;
    __syncthreads();
  }

  // --- 4. decode tokens -----------------------------------------------------
  {
    // ranks among the slots that open a page: the garbage-collection scan's,
    // unless preemption removed some of those slots
    int k = need_before, n_need = need;
    if (mode == 1) {  // workgroup-uniform
      int nd = 0;
#pragma unroll
      for (int i = 0; i < K; ++i) nd += seq[i] >= 0 && ctx[i] % kPage == 0;
      I4 t;
      k = sc.scan(I4{nd, 0, 0, 0}, t).x;
      n_need = t.x;
    }
#pragma unroll
    for (int i = 0; i < K; ++i) {
      if (seq[i] < 0) continue;
      const int s = tid * K + i;
      if (ctx[i] % kPage == 0) {
        a.block_table[(int64_t)s * MP + ctx[i] / kPage] = a.free_pages[free_n - 1 - k];
        ++k;
      }
      ctx[i] += 1;
      a.context_lens[s] = ctx[i];
      rows[i] = 1;
    }
    free_n -= n_need;
  }
  const int n_dec = live;

  // --- 5. admission -----------------------------------------------------------
  int n_adm = 0;
  if (mode == 0) {
    const int budget = a.n_real - n_dec;
    int ne = 0;
#pragma unroll
    for (int i = 0; i < K; ++i) ne += seq[i] < 0 && tid * K + i < S;
    I4 te;
    const int er = sc.scan(I4{ne, 0, 0, 0}, te).x;
    int erank[K];  // rank of each of this thread's empty slots (-1: not empty)
    {
      int r = er;
#pragma unroll
      for (int i = 0; i < K; ++i) {
        erank[i] = -1;
        if (seq[i] < 0 && tid * K + i < S) {
          erank[i] = r;
          sm.empty[r++] = tid * K + i;
        }
      }
    }
    const int m = min(qlen, te.x);
    // candidates j = tid*K + i < m, in queue order from the head
    // (entries not prefetched, such as this step's arrivals, written before
    // the garbage-collection barrier, are read here)
    int tk[K];
    int st = 0, sp = 0;
#pragma unroll
    for (int i = 0; i < K; ++i) {
      const int j = tid * K + i;
      if (j < m && (!kPre || j >= qlen0)) {
        const int q = ring((int64_t)head + j, Q);
        qtk[i] = a.queue_tok[q];
        if constexpr (kPre) {
          qfn[i] = a.queue_fin[q];
          qid[i] = a.queue_seq[q];
        }
      }
      tk[i] = j < m ? qtk[i] : 0;
      st += tk[i];
      sp += pages_of(tk[i]);
    }
    I4 tc;
    const I4 ex = sc.scan(I4{st, sp, 0, 0}, tc);
    int ct = ex.x, cp = ex.y, ok_n = 0;
#pragma unroll
    for (int i = 0; i < K; ++i) {
      const int j = tid * K + i;
      if (j >= m) continue;
      sm.pref[j] = cp;
      ct += tk[i];
      cp += pages_of(tk[i]);
      // cumulative tokens and pages only grow, so the admitted set is a prefix
      ok_n += ct <= budget && cp <= free_n;
      if (j == m - 1) sm.pref[m] = cp;
      sm.seq[j] = tk[i];  // (the moved-sequence list is free again)
    }
    n_adm = sc.sum(ok_n);  // its barrier also publishes sm.empty / sm.pref / sm.seq
    // the j-th admitted entry takes the j-th empty slot: its candidate thread
    // writes the slot, the slot's owner takes its rows
#pragma unroll
    for (int i = 0; i < K; ++i) {
      const int j = tid * K + i;
      if (j >= n_adm) continue;
      const int s = sm.empty[j];
      int id = qid[i], fn = qfn[i];
      if constexpr (!kPre) {
        const int q = ring((int64_t)head + j, Q);
        id = a.queue_seq[q];
        fn = a.queue_fin[q];
      }
      a.slot_seq[s] = id;
      a.slot_order[s] = next_order + j;
      a.slot_fin[s] = fn;
      a.context_lens[s] = sm.seq[j];
    }
#pragma unroll
    for (int i = 0; i < K; ++i) {
      const int r = erank[i];
      if (r >= 0 && r < n_adm) rows[i] = sm.seq[r];
    }
    // pages: the f-th page popped overall is free_pages[free_n - 1 - f]
    const int total = n_adm > 0 ? sm.pref[n_adm] : 0;
    for (int f = tid; f < total; f += kSchedThreads) {
      const int j = find_seq(sm.pref, n_adm, f);
      a.block_table[(int64_t)sm.empty[j] * MP + (f - sm.pref[j])] = a.free_pages[free_n - 1 - f];
    }
    free_n -= total;
    next_order += n_adm;
    head = ring((int64_t)head + n_adm, Q);
    qlen -= n_adm;
  }

  // --- 6. rows of the pass --------------------------------------------------
  {
    int rs = 0;
#pragma unroll
    for (int i = 0; i < K; ++i) rs += rows[i];
    I4 t;
    int run = sc.scan(I4{rs, 0, 0, 0}, t).x;
#pragma unroll
    for (int i = 0; i < K; ++i) {
      const int s = tid * K + i;
      if (s >= S) continue;
      run += rows[i];
      a.query_start_loc[s + 1] = run;
    }
    if (tid == 0) {
      a.query_start_loc[0] = 0;
      a.info[0] = mode;
      a.info[1] = n_fin;
      a.info[2] = n_pre;
      a.info[3] = n_adm;
      a.info[4] = n_dec;
      a.info[5] = accepted;
      a.info[6] = free_n;
      a.info[7] = t.x;
      a.hdr[0] = free_n;
      a.hdr[1] = next_order;
      a.hdr[2] = head;
      a.hdr[3] = qlen;
    }
  }
}

}  // namespace

int sched_slots_per_thread(int S) {
  for (int k : {1, 2, 4, 8})
    if (S <= k * kSchedThreads) return k;
  return 0;
}

hipError_t launch_sched(const SchedArgs& a, hipStream_t st) {
  const void* fn = nullptr;
  switch (sched_slots_per_thread(a.S)) {
    case 1: fn = reinterpret_cast<const void*>(&sched_kernel<1>); break;
    case 2: fn = reinterpret_cast<const void*>(&sched_kernel<2>); break;
    case 4: fn = reinterpret_cast<const void*>(&sched_kernel<4>); break;
    case 8: fn = reinterpret_cast<const void*>(&sched_kernel<8>); break;
    default: return hipErrorInvalidValue;
  }
  void* args[] = {const_cast<SchedArgs*>(&a)};
  hipError_t e = hipLaunchKernel(fn, dim3(1), dim3(kSchedThreads), args, 0, st);
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

}  // namespace pa
