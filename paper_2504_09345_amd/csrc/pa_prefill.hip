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
// over 8 waves of one 16-row MFMA block each.  Per 16-key page:
//   S^T[key][row] = K . Q^T   (v_mfma_f32_16x16x32_bf16, K as the A operand)
//   online softmax per row (each lane owns one row and 4 of its keys)
//   O^T[dim][row] += V^T . P^T (v_mfma_f32_16x16x16_bf16, P in bf16)
// Computing the transposed products keeps "lane l % 16 = query row" in every
// accumulator, so the softmax statistics, the P operand and the O rescale all
// stay in the lane that owns the row: no register transposes.
// The page's K and V tiles are staged in LDS once per workgroup and read by
// all 8 waves: K with its 16-byte chunks XOR-swizzled by key (conflict-free
// operand reads), V transposed to [dim][key] so that each lane's PV operand
// (4 keys of one dim) is one 8-byte read.  Staging goes through registers,
// two pages ahead, so the global loads overlap a full page of work.
// A persistent grid walks the items in a snake order (item x and 2G-1-x per
// workgroup) so early and late causal blocks pair up.
#include "pa_device.h"
#include "pa_kernels.h"

namespace pa {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

namespace {

constexpr int kPfWaves = 8;
constexpr int kPfThreads = 64 * kPfWaves;
constexpr int kPfRows = 16 * kPfWaves;  // one 16-row MFMA block per wave

// Byte offset, inside a swizzled [16 keys][D] bf16 tile, of the 16-byte chunk
// c of key k: chunks of a key are permuted by XOR with the key.
template <int D>
__device__ __forceinline__ int swz_chunk(int k, int c) {
  return k * (D * 2) + ((c ^ (k & 15)) << 4);
}

// Split four fp32 softmax weights into bf16 high parts (round to nearest
// even) and bf16 low parts (the rounding residue, exact in fp32): hi + lo
// carries ~16 mantissa bits, so the PV product keeps fp32-level accuracy
// while both halves run on the bf16 matrix cores.
__device__ __forceinline__ void split_bf16x4(const float (&p)[4], s16x4_t& hi, s16x4_t& lo) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t u = __float_as_uint(p[i]);
    const uint32_t h = (u + 0x7fffu + ((u >> 16) & 1u)) & 0xffff0000u;
    const uint32_t ur = __float_as_uint(p[i] - __uint_as_float(h));
    hi[i] = (short)(h >> 16);
    lo[i] = (short)((ur + 0x7fffu + ((ur >> 16) & 1u)) >> 16);
  }
}

}  // namespace

template <int D, int S>
__global__ __launch_bounds__(kPfThreads) void prefill_kernel(PrefillArgs a) {
  static_assert(D == 128, "prefill MFMA path is built for head_dim 128");
  constexpr int PB = kPfRows / S;       // chunk positions per item
  constexpr int KSTEPS = D / 32;        // QK MFMA steps over dims
  constexpr int MB = D / 16;            // PV MFMA blocks over dims
  constexpr int KT = kPage * D * 2;     // bytes of one K tile
  constexpr int VT_STRIDE = kPage * 2 + 8;  // bytes per dim row of the V^T tile (padded)
  constexpr int VT = D * VT_STRIDE;
  constexpr int OUT_STRIDE = D * 2 + 16;
  constexpr int C8 = D / 4;             // 8-byte chunks per key

  __shared__ __attribute__((aligned(16))) uint8_t s_k[2][KT];
  __shared__ __attribute__((aligned(16))) uint8_t s_vt[2][VT];
  __shared__ __attribute__((aligned(16))) uint8_t s_out[kPfRows * OUT_STRIDE];
  __shared__ int32_t s_scan[kPfThreads];
  extern __shared__ int32_t s_cum[];  // [B + 1] prefix of items per sequence

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
  const int G = gridDim.x;
  const BlockTable bt{a.block_table, a.bt_stride};
  const uint16_t* kp = reinterpret_cast<const uint16_t*>(a.k_pages);
  const uint16_t* vp = reinterpret_cast<const uint16_t*>(a.v_pages);
  const uint16_t* qg = reinterpret_cast<const uint16_t*>(a.q);
  uint16_t* og = reinterpret_cast<uint16_t*>(a.out);

  // staging role of this thread: 8-byte chunk c8 of key st_key of a tile
  const int st_key = tid / C8, st_c8 = tid % C8;
  const int m = w * 16 + (lane & 15);  // this lane's query row in the block

  for (int round = 0;; ++round) {
    const int x = (round & 1) ? G - 1 - blockIdx.x : blockIdx.x;
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

    if (bad) {  // contract violation: NaN rows, nothing read
      __syncthreads();
      for (int idx = tid; idx < npos * S * D; idx += kPfThreads) {
        const int p = idx / (S * D), hd = idx % (S * D);
        og[((int64_t)(q0 + pos0 + p) * a.H_q + (int64_t)g * S) * D + hd] = 0x7fc0;
      }
      continue;
    }
    const int lim0 = C - L + pos0;                // last key of the block's first row
    const int npg = (lim0 + npos - 1) / kPage + 1;

    const int p = m / S, h = m - p * S;
    const bool valid = p < npos;
    const int lim = valid ? lim0 + p : -1;
    float mrow = kMInit, lrow = 0.0f;
    f32x4_t acc[MB];
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) acc[mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    u32x4 qt[KSTEPS];
    {
      const uint16_t* qrow = qg + ((int64_t)(q0 + pos0 + (valid ? p : 0)) * a.H_q + (int64_t)g * S + h) * D;
#pragma unroll
      for (int st = 0; st < KSTEPS; ++st)
        qt[st] = valid ? *reinterpret_cast<const u32x4*>(qrow + st * 32 + (lane >> 4) * 8) : u32x4{0, 0, 0, 0};
    }

    // Slots past the context (the tail of the last page) are staged as zeros:
    // their weights are 0, but the matrix product would still form 0 * V for
    // them, and those bytes may hold anything.
    auto fetch = [&](int pg, u32x2_t& kr, u32x2_t& vr) {
      if (pg < npg) {
        if (pg * kPage + st_key < C) {
          const int32_t page = bt.page(b, pg);
          const int64_t off = ((int64_t)page * a.H_kv + g) * (int64_t)(kPage * D) + st_key * D + st_c8 * 4;
          kr = __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(kp + off));
          vr = __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(vp + off));
        } else {
          kr = u32x2_t{0, 0};
          vr = u32x2_t{0, 0};
        }
      }
    };
    auto stash = [&](int pg, const u32x2_t& kr, const u32x2_t& vr) {
      if (pg < npg) {
        uint8_t* kt = s_k[pg & 1];
        *reinterpret_cast<u32x2_t*>(kt + swz_chunk<D>(st_key, st_c8 >> 1) + (st_c8 & 1) * 8) = kr;
        uint8_t* vt = s_vt[pg & 1] + st_key * 2;
        const int d0 = st_c8 * 4;
        *reinterpret_cast<uint16_t*>(vt + (d0 + 0) * VT_STRIDE) = (uint16_t)(vr.x & 0xffff);
        *reinterpret_cast<uint16_t*>(vt + (d0 + 1) * VT_STRIDE) = (uint16_t)(vr.x >> 16);
        *reinterpret_cast<uint16_t*>(vt + (d0 + 2) * VT_STRIDE) = (uint16_t)(vr.y & 0xffff);
        *reinterpret_cast<uint16_t*>(vt + (d0 + 3) * VT_STRIDE) = (uint16_t)(vr.y >> 16);
      }
    };
    auto consume = [&](int pg) {
      const uint8_t* kt = s_k[pg & 1];
      const uint8_t* vt = s_vt[pg & 1];
      // S^T = K . Q^T (A: key lane%16, dims 32 st + 8 (lane/16) .. +8)
      f32x4_t s = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < KSTEPS; ++st) {
        const u32x4 kv = *reinterpret_cast<const u32x4*>(kt + swz_chunk<D>(lane & 15, st * 4 + (lane >> 4)));
        s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, kv),
                                                    __builtin_bit_cast(bf16x8_t, qt[st]), s, 0, 0, 0);
      }
      // online softmax: this lane holds keys 4 (lane/16) + i of row m
      float xs[4];
      const bool need_mask = pg * kPage + kPage - 1 > lim0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        xs[i] = s[i] * a.scale_log2;
        if (need_mask) xs[i] = pg * kPage + (lane >> 4) * 4 + i <= lim ? xs[i] : -INFINITY;
      }
      float mx = fmaxf(fmaxf(xs[0], xs[1]), fmaxf(xs[2], xs[3]));
      mx = fmaxf(mx, xor_lanes<16>(mx));
      mx = fmaxf(mx, xor_lanes<32>(mx));
      const float mnew = fmaxf(mrow, mx);
      const float alpha = fast_exp2(mrow - mnew);
      mrow = mnew;
      float pw[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) pw[i] = fast_exp2(xs[i] - mnew);
      lrow = fmaf(lrow, alpha, (pw[0] + pw[1]) + (pw[2] + pw[3]));
      s16x4_t phi, plo;
      split_bf16x4(pw, phi, plo);
      // O^T += V^T . P^T (A: dim 16 mb + lane%16, keys 4 (lane/16) .. +4)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb) {
        const u32x2_t vv = *reinterpret_cast<const u32x2_t*>(vt + (mb * 16 + (lane & 15)) * VT_STRIDE + (lane >> 4) * 8);
        const s16x4_t va = __builtin_bit_cast(s16x4_t, vv);
        acc[mb] *= alpha;
        acc[mb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(va, phi, acc[mb], 0, 0, 0);
        acc[mb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(va, plo, acc[mb], 0, 0, 0);
      }
    };

    u32x2_t kr0 = {0, 0}, vr0 = {0, 0}, kr1 = {0, 0}, vr1 = {0, 0};
    __syncthreads();  // previous item's readers of s_k / s_vt / s_out are done
    fetch(0, kr0, vr0);
    fetch(1, kr1, vr1);
    stash(0, kr0, vr0);
    for (int pg = 0; pg < npg; pg += 2) {
      __syncthreads();  // page pg is in LDS; everyone is done with page pg-1
      stash(pg + 1, kr1, vr1);
      fetch(pg + 2, kr0, vr0);
      consume(pg);
      if (pg + 1 < npg) {
        __syncthreads();
        stash(pg + 2, kr0, vr0);
        fetch(pg + 3, kr1, vr1);
        consume(pg + 1);
      }
    }

    // normalise and stage the block's rows in LDS (row m: position m/S, head m%S)
    float l = lrow;
    l += xor_lanes<16>(l);
    l += xor_lanes<32>(l);
    const float inv = valid ? 1.0f / l : 0.0f;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int d = mb * 16 + (lane >> 4) * 4 + i;
        *reinterpret_cast<uint16_t*>(s_out + m * OUT_STRIDE + d * 2) = f32_to_bf16(acc[mb][i] * inv);
      }
    __syncthreads();
    // coalesced stores: 16 bytes per thread per step
    constexpr int CHUNKS = D / 8;
    for (int idx = tid; idx < npos * S * CHUNKS; idx += kPfThreads) {
      const int mm = idx / CHUNKS, c = idx % CHUNKS;
      const int pp = mm / S, hh = mm - pp * S;
      const u32x4 v = *reinterpret_cast<const u32x4*>(s_out + mm * OUT_STRIDE + c * 16);
      *reinterpret_cast<u32x4*>(og + ((int64_t)(q0 + pos0 + pp) * a.H_q + (int64_t)g * S + hh) * D + c * 8) = v;
    }
  }
}

static const void* prefill_fn(int s) {
  switch (s) {
    case 1: return reinterpret_cast<const void*>(&prefill_kernel<128, 1>);
    case 2: return reinterpret_cast<const void*>(&prefill_kernel<128, 2>);
    case 4: return reinterpret_cast<const void*>(&prefill_kernel<128, 4>);
    case 6: return reinterpret_cast<const void*>(&prefill_kernel<128, 6>);
    case 8: return reinterpret_cast<const void*>(&prefill_kernel<128, 8>);
  }
  return nullptr;
}

bool prefill_supported(int dtype, int D, int s) { return dtype == 0 && D == 128 && prefill_fn(s) != nullptr; }

int prefill_occupancy(int s, int B) {
  const void* fn = prefill_fn(s);
  if (fn == nullptr) return 0;
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, kPfThreads, (size_t)(B + 1) * sizeof(int32_t)) != hipSuccess)
    return 0;
  return n;
}

hipError_t launch_prefill(int s, const PrefillArgs& a, int G, hipStream_t st) {
  const void* fn = prefill_fn(s);
  if (fn == nullptr || G <= 0) return hipErrorInvalidValue;
  void* args[] = {const_cast<PrefillArgs*>(&a)};
  hipError_t e = hipLaunchKernel(fn, dim3(G), dim3(kPfThreads), args, (size_t)(a.B + 1) * sizeof(int32_t), st);
  if (e != hipSuccess) return e;
  return hipGetLastError();
}

}  // namespace pa
