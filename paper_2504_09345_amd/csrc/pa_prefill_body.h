// Body of the MFMA chunked-prefill workgroup, shared by the prefill kernel and
// the mixed prefill + decode kernel (design notes in pa_prefill.hip).
#pragma once

#include "pa_device.h"
#include "pa_kernels.h"
#include "pa_tile.h"

namespace pa {


using mfma::bf16x8_t;
using mfma::f32x4_t;
using mfma::lds_s16x4_t;
using mfma::s16x4_t;
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
template <bool V> struct PfBool { static constexpr bool value = V; };

constexpr int kPfWaves = 8;
constexpr int kPfThreads = 64 * kPfWaves;
constexpr int kPfBlocks = 2;                       // 16-row MFMA blocks per wave
constexpr int kPfRows = 16 * kPfBlocks * kPfWaves;  // 256 query rows per item
constexpr int kPfMaxPages = 2048;                  // block-table window in LDS (power of 2)
constexpr int kPfStep = 2;                         // pages per synchronised step
constexpr int kPfLdsSteps = 3;                     // steps staged in LDS at once
// Cache policy of the prefill K/V loads: the default (cached).  The items of
// one (sequence, KV head) re-read the same causal prefix of pages, so cached
// loads serve most re-reads from L2 / MALL; with non-temporal loads they went
// to HBM and slowed the decode workgroups running beside them by ~15%.
constexpr int kPfLoadPolicy = 0;

// LDS of one prefill workgroup (besides the per-sequence item prefix sums).
struct PrefillSmem {
  __attribute__((aligned(16))) uint8_t k[kPfLdsSteps][kPfStep * kPage * mfma::kD * 2];
  __attribute__((aligned(16))) uint8_t v[kPfLdsSteps][kPfStep * kPage * mfma::kD * 2];
  int32_t bt[kPfMaxPages];
  int32_t scan[kPfThreads];
  int32_t vwide;  // the item needs the bf16 pass (non-finite or tiny output rows after the fp16 pass)
};

// Prefill workgroup `bid` of a grid of G; s_cum holds B + 1 ints of LDS.
// TR: gather-trace instantiation (records every loaded token's pool row in
// a.trace besides computing the attention).
template <int D, int S, bool TR = false>
__device__ __forceinline__ void prefill_body(const PrefillArgs& a, PrefillSmem& sm, int32_t* s_cum, int bid,
                                             int G) {
  static_assert(D == mfma::kD, "prefill MFMA path is built for head_dim 128");
  constexpr int PB = kPfRows / S;       // chunk positions per item
  constexpr int KSTEPS = D / 32;        // QK MFMA steps over dims
  constexpr int MB = D / 16;            // PV MFMA blocks over dims
  constexpr int KT = kPage * D * 2;     // bytes of one tile
  constexpr int C16 = D / 8;            // 16-byte chunks per key
  static_assert(kPfStep * kPage * C16 == kPfThreads, "one 16-byte chunk of K and V per thread and step");

  static_assert(sizeof(sm.k[0]) == kPfStep * KT, "LDS step size");
  auto& s_k = sm.k;
  auto& s_v = sm.v;
  int32_t* s_bt = sm.bt;
  int32_t* s_scan = sm.scan;

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int B = a.B;

  // items per sequence: ceil(L / PB) * H_kv for chunks (L > 1), else 0;
  // s_cum[b] = items of sequences before b
  {
    const int per = (B + kPfThreads - 1) / kPfThreads;
    const int b0 = min(B, tid * per), b1 = min(B, b0 + per);
    int local = 0;
    for (int b = b0; b < b1; ++b) {
      const int L = a.query_start_loc[b + 1] - a.query_start_loc[b];
      s_cum[b] = local;
      local += L > 1 ? ((L + PB - 1) / PB) * a.H_kv : 0;
    }
    const int off = block_exclusive_scan<kPfThreads>(local, s_scan);
    for (int b = b0; b < b1; ++b) s_cum[b] += off;
    if (tid == kPfThreads - 1) s_cum[B] = off + local;
    __syncthreads();
  }
  const int n_items = s_cum[B];
  const BlockTable bt{a.block_table, a.bt_stride};
  const uint16_t* kp = reinterpret_cast<const uint16_t*>(a.k_pages);
  const uint16_t* vp = reinterpret_cast<const uint16_t*>(a.v_pages);
  const uint16_t* qg = reinterpret_cast<const uint16_t*>(a.q);
  uint16_t* og = reinterpret_cast<uint16_t*>(a.out);

  // staging role of this thread: 16-byte chunk st_c of key st_key of page
  // st_pg of a step (st_pg is wave-uniform)
  const int st_pg = w / (kPfWaves / kPfStep), st_j = tid % (kPage * C16);
  const int st_key = st_j / C16, st_c = st_j % C16;
  const int st_off = st_pg * KT + mfma::swz(st_key, st_c);
  const int st_off_v = st_pg * KT + mfma::swz_v(st_key, st_c);
  const int st_ld = st_j * 16;  // byte offset in the global tile
  const int n = lane & 15, Gq = lane >> 4;  // MFMA column (query row of a block) and lane group

  for (int round = 0;; ++round) {
    const int x = (round & 1) ? G - 1 - bid : bid;
    const int f = round * G + x;
    if (f >= n_items) break;
    // item f -> (b, g, block jb), order (b, g, jb)
    int lo = 0, hi = B - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (s_cum[mid] <= f) lo = mid; else hi = mid - 1;
    }
    const int b = lo;
    const int q0 = a.query_start_loc[b];
    const int L = a.query_start_loc[b + 1] - q0;
    const int C = a.context_lens[b];
    const int nblk = (L + PB - 1) / PB;
    const int rem = f - s_cum[b];
    const int g = rem / nblk, jb = rem - g * nblk;
    const int pos0 = jb * PB;                     // first chunk position of the block
    const int npos = min(PB, L - pos0);           // valid positions in the block
    const bool bad = C > a.max_context_len || L > C || (C + kPage - 1) / kPage > (int)a.bt_stride;

    __syncthreads();  // previous item's readers of s_k / s_v / s_bt are done
    if (bad) {  // contract violation: NaN rows, nothing read
      for (int idx = tid; idx < npos * S * D; idx += kPfThreads) {
        const int p = idx / (S * D), hd = idx % (S * D);
        og[((int64_t)(q0 + pos0 + p) * a.H_q + (int64_t)g * S) * D + hd] = 0x7fc0;
      }
      continue;
    }
    const int lim0 = C - L + pos0;                // last key of the block's first row
    const int npg = (lim0 + npos - 1) / kPage + 1;
    // block-table window: s_bt[p % kPfMaxPages] holds the entry of page p
    for (int i = tid; i < min(npg, kPfMaxPages); i += kPfThreads) s_bt[i] = bt.page(b, i);

    // this lane's rows: block rb, row m = (w * 2 + rb) * 16 + lane % 16
    u32x4 qt[kPfBlocks][KSTEPS];
    int lim[kPfBlocks];
    float mrow[kPfBlocks];
    f32x4_t acc[kPfBlocks][MB], acc_l[kPfBlocks];
#pragma unroll
    for (int rb = 0; rb < kPfBlocks; ++rb) {
      const int m = (w * kPfBlocks + rb) * 16 + n;
      const int p = m / S, h = m - p * S;
      const bool valid = p < npos;
      lim[rb] = valid ? lim0 + p : -1;
      const uint16_t* qrow = qg + ((int64_t)(q0 + pos0 + (valid ? p : 0)) * a.H_q + (int64_t)g * S + h) * D;
#pragma unroll
      for (int st = 0; st < KSTEPS; ++st)
        qt[rb][st] = valid ? *reinterpret_cast<const u32x4*>(qrow + st * 32 + Gq * 8) : u32x4{0, 0, 0, 0};
    }
    if (tid == 0) sm.vwide = 0;
    __syncthreads();  // s_bt is filled

    // Slots past the context (the tail of the last page) are staged as zeros:
    // their weights are 0, but the matrix product would still form 0 * V for
    // them, and those bytes may hold anything.
    // Loads, stores and the block-table read run unconditionally (no branch
    // the compiler's wait counting has to merge): a page at or past npg is a
    // null tile, staged as zeros and fully masked.
    const int nst = (npg + kPfStep - 1) / kPfStep;  // steps of kPfStep pages
    auto fetch = [&](int t, u32x4& kr, u32x4& vr) {
      const int pg = t * kPfStep + st_pg;
      // buffer loads past `valid` keys (all of them for pg >= npg) return 0
      const int valid = pg < npg ? min(kPage, C - pg * kPage) : 0;
      const int32_t entry = __builtin_amdgcn_readfirstlane(s_bt[pg & (kPfMaxPages - 1)]);
      const int32_t page = pg < npg ? entry : 0;
      const int64_t tile = ((int64_t)page * a.H_kv + g) * (int64_t)(kPage * D);
      if constexpr (TR) {
        if (st_c == 0 && st_key < valid)
          trace_put(a.trace, ((int64_t)g * B + b) * (a.bt_stride * kPage) + pg * kPage + st_key, tile / D + st_key);
      }
      const __amdgpu_buffer_rsrc_t rk = tile_rsrc<uint16_t, D>(kp + tile, valid);
      const __amdgpu_buffer_rsrc_t rv = tile_rsrc<uint16_t, D>(vp + tile, valid);
      kr = __builtin_amdgcn_raw_buffer_load_b128(rk, st_ld, 0, kPfLoadPolicy);
      vr = __builtin_amdgcn_raw_buffer_load_b128(rv, st_ld, 0, kPfLoadPolicy);
    };
    // With F16, V is staged as fp16: bf16 magnitudes in [2^-17, 2^16) and
    // zeros convert exactly, smaller ones to fp16 subnormals (absolute error
    // <= 2^-25), larger ones to infinity (the largest bf16 below 2^16, 65280,
    // is an fp16 value).  A value that is not finite in fp16 makes every row
    // of the item non-finite (a weight times infinity or NaN, and 0 times
    // either is NaN), which the check after the pass catches; the item then
    // runs again in bf16.
    auto stash = [&](auto f16, int t, const u32x4& kr, const u32x4& vr) {
      const int buf = t % kPfLdsSteps;
      *reinterpret_cast<u32x4*>(s_k[buf] + st_off) = kr;
      if constexpr (decltype(f16)::value) {
        u32x4 vh;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const f32x2_t f = f32x2_t{__uint_as_float(vr[i] << 16), __uint_as_float(vr[i] & 0xffff0000u)};
          vh[i] = __builtin_bit_cast(uint32_t, __builtin_convertvector(f, f16x2_t));
        }
        *reinterpret_cast<u32x4*>(s_v[buf] + st_off_v) = vh;
      } else {
        *reinterpret_cast<u32x4*>(s_v[buf] + st_off_v) = vr;
      }
    };
    // S^T = K . Q^T for the pages of step t (A: key lane%16, dims 32 st +
    // 8 (lane/16) .. +8), each K read shared by both row blocks
    // (the step's K operands are read from LDS first, all at once, so their
    // latency overlaps the staging work issued before the products)
    typedef u32x4 KOps[kPfStep][KSTEPS];
    auto k_read = [&](int t, KOps& kv) {
      const uint8_t* kt = s_k[t % kPfLdsSteps];
#pragma unroll
      for (int pp = 0; pp < kPfStep; ++pp)
#pragma unroll
        for (int st = 0; st < KSTEPS; ++st)
          kv[pp][st] = *reinterpret_cast<const u32x4*>(kt + pp * KT + mfma::swz(n, st * 4 + Gq));
    };
    auto qk = [&](const KOps& kv, f32x4_t (&sc)[kPfBlocks][kPfStep]) {
#pragma unroll
      for (int rb = 0; rb < kPfBlocks; ++rb)
#pragma unroll
        for (int pp = 0; pp < kPfStep; ++pp) sc[rb][pp] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int pp = 0; pp < kPfStep; ++pp)
#pragma unroll
        for (int st = 0; st < KSTEPS; ++st)
#pragma unroll
          for (int rb = 0; rb < kPfBlocks; ++rb)
            sc[rb][pp] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8_t, kv[pp][st]), __builtin_bit_cast(bf16x8_t, qt[rb][st]), sc[rb][pp], 0, 0, 0);
    };
    // online softmax of step t's scores and O^T += V^T . P^T.  Row sums come
    // from the matrix cores too: acc_l += ones . P^T (every entry of a lane's
    // acc_l holds its row's sum).
    const bf16x8_t ones = __builtin_bit_cast(
        bf16x8_t, u32x4{0x3f803f80u, 0x3f803f80u, 0x3f803f80u, 0x3f803f80u});
    const f16x8_t ones_h = __builtin_bit_cast(
        f16x8_t, u32x4{0x3c003c00u, 0x3c003c00u, 0x3c003c00u, 0x3c003c00u});
    auto softmax_pv = [&](auto f16, int t, const f32x4_t (&sc)[kPfBlocks][kPfStep]) {
      constexpr bool F16 = decltype(f16)::value;
      const uint8_t* vt = s_v[t % kPfLdsSteps];
      const int key0 = t * kPfStep * kPage;  // first key of the step
      // this lane holds keys key0 + 16 pp + 4 (lane/16) + i of its row; the
      // causal mask applies on the steps that cross the diagonal
      float xs[kPfBlocks][kPfStep * 4];
      if (key0 + kPfStep * kPage - 1 > lim0) {
#pragma unroll
        for (int rb = 0; rb < kPfBlocks; ++rb)
#pragma unroll
          for (int pp = 0; pp < kPfStep; ++pp)
#pragma unroll
            for (int i = 0; i < 4; ++i)
              xs[rb][pp * 4 + i] = key0 + pp * kPage + Gq * 4 + i <= lim[rb] ? sc[rb][pp][i] : -INFINITY;
      } else {
#pragma unroll
        for (int rb = 0; rb < kPfBlocks; ++rb)
#pragma unroll
          for (int pp = 0; pp < kPfStep; ++pp)
#pragma unroll
            for (int i = 0; i < 4; ++i) xs[rb][pp * 4 + i] = sc[rb][pp][i];
      }
      // weights against the current base; the base only moves when one of
      // them exceeds 2^kRescaleSlack (or is the first finite score of a row,
      // whose base is still kMInit: the weight is then +inf)
      float pw[kPfBlocks][kPfStep * 4];
      auto weights = [&]() {
        bool big = false;
#pragma unroll
        for (int rb = 0; rb < kPfBlocks; ++rb) {
          float pmax = 0.0f;
#pragma unroll
          for (int j = 0; j < kPfStep * 4; ++j) {
            pw[rb][j] = fast_exp2(fmaf(xs[rb][j], a.scale_log2, -mrow[rb]));
            pmax = fmaxf(pmax, pw[rb][j]);
          }
          big |= pmax > kRescaleLimit;
        }
        return big;
      };
      if (__builtin_amdgcn_ballot_w64(weights()) != 0) {  // rebase every row of the wave
#pragma unroll
        for (int rb = 0; rb < kPfBlocks; ++rb) {
          float mx = -INFINITY;
#pragma unroll
          for (int j = 0; j < kPfStep * 4; ++j) mx = fmaxf(mx, xs[rb][j]);
          // scale > 0, so the max commutes with it
          const float mc = fmaxf(mrow[rb], rows4_max(mx) * a.scale_log2);
          const float alpha = fast_exp2(mrow[rb] - mc);
          mrow[rb] = mc;
          acc_l[rb] *= alpha;
#pragma unroll
          for (int mb = 0; mb < MB; ++mb) acc[rb][mb] *= alpha;
        }
        weights();
      }
      // P operands: k slots 8 (lane/16) + 4 pp + i hold key 4 (lane/16) + i
      // of page pp, i.e. the lane's 8 weights in order.  V^T: lane p of group
      // Gq addresses key 4 Gq + p / 4, dims 16 mb + 4 (p % 4) of each page;
      // the two transposed reads form the A operand's k slots in the same
      // page-major order as P.
      const int vkey = 4 * Gq + (n >> 2);
      if constexpr (F16) {
        // fp16 P (nearest even, relative error <= 2^-11) and fp16 V: one product
        f16x8_t ph[kPfBlocks];
#pragma unroll
        for (int rb = 0; rb < kPfBlocks; ++rb) {
          u32x4 w4;
#pragma unroll
          for (int i = 0; i < 4; ++i)
            w4[i] = __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{pw[rb][2 * i], pw[rb][2 * i + 1]}), f16x2_t));
          ph[rb] = __builtin_bit_cast(f16x8_t, w4);
          acc_l[rb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(ones_h, ph[rb], acc_l[rb], 0, 0, 0);
        }
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const int d = mb * 16 + 4 * (n & 3);
          const int off = mfma::swz_v(vkey, d >> 3) + (d & 7) * 2;
          const s16x4_t v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(vt + off));
          const s16x4_t v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(vt + KT + off));
          const f16x8_t va = __builtin_bit_cast(f16x8_t, __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
          for (int rb = 0; rb < kPfBlocks; ++rb)
            acc[rb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(va, ph[rb], acc[rb][mb], 0, 0, 0);
        }
      } else {
        // bf16 V and P's bf16 high and low parts: two products
        bf16x8_t phi[kPfBlocks], plo[kPfBlocks];
#pragma unroll
        for (int rb = 0; rb < kPfBlocks; ++rb) {
          s16x4_t h[kPfStep], l[kPfStep];
#pragma unroll
          for (int pp = 0; pp < kPfStep; ++pp) {
            const float q4[4] = {pw[rb][pp * 4], pw[rb][pp * 4 + 1], pw[rb][pp * 4 + 2], pw[rb][pp * 4 + 3]};
            mfma::split_hi_lo(q4, h[pp], l[pp]);
          }
          phi[rb] = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(h[0], h[1], 0, 1, 2, 3, 4, 5, 6, 7));
          plo[rb] = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(l[0], l[1], 0, 1, 2, 3, 4, 5, 6, 7));
          acc_l[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, phi[rb], acc_l[rb], 0, 0, 0);
          acc_l[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ones, plo[rb], acc_l[rb], 0, 0, 0);
        }
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const int d = mb * 16 + 4 * (n & 3);
          const int off = mfma::swz_v(vkey, d >> 3) + (d & 7) * 2;
          const s16x4_t v0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(vt + off));
          const s16x4_t v1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(vt + KT + off));
          const bf16x8_t va = __builtin_bit_cast(bf16x8_t, __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7));
#pragma unroll
          for (int rb = 0; rb < kPfBlocks; ++rb) {
            acc[rb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, phi[rb], acc[rb][mb], 0, 0, 0);
            acc[rb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, plo[rb], acc[rb][mb], 0, 0, 0);
          }
        }
      }
    };

    // Pipeline.  Step t is staged through register set t & 1 and LDS buffer
    // t % 3.  Iteration t stores step t + 2 to LDS and refills its register
    // set with step t + 4 (steps t + 3 and t + 4 in flight), issues the QK
    // products of step t + 1 and then runs the softmax and PV of step t, so
    // the matrix cores work on QK(t + 1) while the VALU does softmax(t).
    auto step_barrier = [&](int t) {
      __syncthreads();  // steps t, t + 1 are in LDS; everyone is done with step t - 1
      const int pgf = (t + 4) * kPfStep;  // first page fetched next
      if ((pgf & (kPfMaxPages - 1)) == 0 && pgf < npg) {
        // slide the block-table window to pages pgf .. pgf + kPfMaxPages - 1
        for (int i = tid; i < min(npg - pgf, kPfMaxPages); i += kPfThreads) s_bt[i] = bt.page(b, pgf + i);
        __syncthreads();
      }
    };
    // One pass over the item's steps; acc, acc_l and mrow start afresh.
    auto pipeline = [&](auto f16) {
#pragma unroll
      for (int rb = 0; rb < kPfBlocks; ++rb) {
        mrow[rb] = kMInit;
        acc_l[rb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) acc[rb][mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      }
      u32x4 ka, va, kb, vb;
      // (scheduling barriers keep the issue order the loop's waits assume)
      fetch(0, ka, va);
      __builtin_amdgcn_sched_barrier(0);
      fetch(1, kb, vb);
      __builtin_amdgcn_sched_barrier(0);
      stash(f16, 0, ka, va);
      __builtin_amdgcn_sched_barrier(0);
      fetch(2, ka, va);
      __builtin_amdgcn_sched_barrier(0);
      stash(f16, 1, kb, vb);
      __builtin_amdgcn_sched_barrier(0);
      fetch(3, kb, vb);
      __builtin_amdgcn_sched_barrier(0);
      __syncthreads();  // steps 0 and 1 are in LDS
      f32x4_t sc[kPfBlocks][kPfStep], sn[kPfBlocks][kPfStep];
      KOps kv;
      k_read(0, kv);
      qk(kv, sc);
      // two steps per trip; with nst odd the last trip's second step is null
      for (int t = 0; t < nst; t += 2) {
        step_barrier(t);
        k_read(t + 1, kv);
        __builtin_amdgcn_sched_barrier(0);
        stash(f16, t + 2, ka, va);
        fetch(t + 4, ka, va);
        qk(kv, sn);
        softmax_pv(f16, t, sc);
        step_barrier(t + 1);
        k_read(t + 2, kv);
        __builtin_amdgcn_sched_barrier(0);
        stash(f16, t + 3, kb, vb);
        fetch(t + 5, kb, vb);
        qk(kv, sc);
        softmax_pv(f16, t + 1, sn);
      }
      if constexpr (decltype(f16)::value) {
        // fp16 V is exact for bf16 magnitudes in [2^-17, 2^16); smaller ones
        // carry an absolute error <= 2^-25, which stays below a tenth of the
        // relative tolerance only for rows whose output RMS is >= 2^-14;
        // larger ones (and infinities, NaNs) leave the rows non-finite.
        // Either marks the item for the bf16 pass (so does a NaN or infinite
        // K, whose rows are non-finite in both passes).
        bool redo = false;
#pragma unroll
        for (int rb = 0; rb < kPfBlocks; ++rb) {
          const float inv = 1.0f / acc_l[rb][0];
          float ss = 0.0f;
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int i = 0; i < 4; ++i) ss = fmaf(acc[rb][mb][i] * inv, acc[rb][mb][i] * inv, ss);
          // ss of the row's D dims
          const float row_ss = rows4_sum(ss);
          redo |= lim[rb] >= 0 && !(row_ss >= (float)D * 0x1p-28f && row_ss <= __FLT_MAX__);
        }
        if (__builtin_amdgcn_ballot_w64(redo) != 0 && lane == 0) sm.vwide = 1;
      }
    };
    // fp16 pass; an item whose V does not fit fp16 (or whose output rows are
    // too small for fp16's subnormal V) is recomputed in bf16
    pipeline(PfBool<true>{});
    __syncthreads();  // every wave's check of the pass has set or left the flag
    if (sm.vwide) {
      if (npg > kPfMaxPages) {  // the pass slid the block-table window: back to page 0
        for (int i = tid; i < kPfMaxPages; i += kPfThreads) s_bt[i] = bt.page(b, i);
        __syncthreads();
      }
      pipeline(PfBool<false>{});
    }

    // normalise and store straight from the accumulators: lane (n, Gq) holds
    // dims 16 mb + 4 Gq + i of row (w * 2 + rb) * 16 + n
#pragma unroll
    for (int rb = 0; rb < kPfBlocks; ++rb) {
      if (lim[rb] >= 0) {
        const float inv = 1.0f / acc_l[rb][0];
        const int m = (w * kPfBlocks + rb) * 16 + n;
        const int p = m / S, h = m - p * S;
        uint16_t* orow = og + ((int64_t)(q0 + pos0 + p) * a.H_q + (int64_t)g * S + h) * D;
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) {
          const uint32_t w0 = (uint32_t)f32_to_bf16(acc[rb][mb][0] * inv) | (uint32_t)f32_to_bf16(acc[rb][mb][1] * inv) << 16;
          const uint32_t w1 = (uint32_t)f32_to_bf16(acc[rb][mb][2] * inv) | (uint32_t)f32_to_bf16(acc[rb][mb][3] * inv) << 16;
          *reinterpret_cast<u32x2_t*>(orow + mb * 16 + 4 * Gq) = u32x2_t{w0, w1};
        }
      }
    }
  }
}

}  // namespace pa
