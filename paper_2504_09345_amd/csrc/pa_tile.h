// Tile-level building blocks shared by the split-K and stream-K attention
// kernels: the lane layout of a (page, KV head) tile, the bf16 dot products,
// the buffer-descriptor loads, the online-softmax fold of one tile, the
// merge of a wave's lane rows, and the mapping from a query row to its
// sequence and visible keys.
#pragma once

#include "pa_device.h"

namespace pa {

template <typename T, int D, int S>
struct DecodeShape {
  static constexpr int VEC = 16 / (int)sizeof(T);  // elements per 16-byte lane load
  static constexpr int LPT = D / VEC;              // lanes per token row
  static constexpr int TPI = 64 / LPT;             // token rows per wave-wide load
  static constexpr int NI = kPage / TPI;           // loads per 16-token tile
  static_assert(LPT >= 2 && LPT <= 32 && 64 % LPT == 0 && kPage % TPI == 0, "unsupported shape");
};

// Partial dot product of the lane's VEC query elements with VEC key elements.
__device__ __forceinline__ float lane_dot(const u32x4& q, const u32x4& k, uint16_t) {
  float acc = 0.0f;
  acc = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(q.x), as_bf16x2(k.x), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(q.y), as_bf16x2(k.y), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(q.z), as_bf16x2(k.z), acc, false);
  acc = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(q.w), as_bf16x2(k.w), acc, false);
  return acc;
}
__device__ __forceinline__ float lane_dot(const u32x4& q, const u32x4& k, float) {
  float acc = __uint_as_float(q.x) * __uint_as_float(k.x);
  acc = fmaf(__uint_as_float(q.y), __uint_as_float(k.y), acc);
  acc = fmaf(__uint_as_float(q.z), __uint_as_float(k.z), acc);
  acc = fmaf(__uint_as_float(q.w), __uint_as_float(k.w), acc);
  return acc;
}

// Widen the lane's VEC value elements to fp32.
__device__ __forceinline__ void widen(const u32x4& v, float* f, uint16_t) {
  f[0] = bf16_lo(v.x); f[1] = bf16_hi(v.x);
  f[2] = bf16_lo(v.y); f[3] = bf16_hi(v.y);
  f[4] = bf16_lo(v.z); f[5] = bf16_hi(v.z);
  f[6] = bf16_lo(v.w); f[7] = bf16_hi(v.w);
}
__device__ __forceinline__ void widen(const u32x4& v, float* f, float) {
  f[0] = __uint_as_float(v.x); f[1] = __uint_as_float(v.y);
  f[2] = __uint_as_float(v.z); f[3] = __uint_as_float(v.w);
}

template <typename T, int D, int S>
struct DecodeState {
  using Sh = DecodeShape<T, D, S>;
  u32x4 q[S];                  // lane's slice of the s query vectors (raw)
  float o[S][Sh::VEC];         // unnormalised output slice per head
  float m[S], l[S];            // running max (log2 units) and sum per head
};

// Buffer descriptor (raw, untyped) of one (page, g) tile of `valid` tokens:
// loads at byte offsets >= valid * D * sizeof(T) return zeros without a
// memory access, so slots past the context (and whole null tiles, valid = 0)
// never reach the arithmetic as anything but 0.
template <typename T, int D>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const T* base, int valid) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<T*>(base), (short)0, valid * D * (int)sizeof(T),
                                           0x00020000);
}

// Cache policy of the K/V tile loads: non-temporal (each byte is read once
// per call).  On MI355X this streams randomly placed 32 KiB pages at ~7.0
// TB/s against ~6.2 TB/s with the default policy.
constexpr int kKvLoadPolicy = 2;  // nt

// Issue the NI K and NI V 16-byte-per-lane loads of one tile.  Lane l reads
// bytes [16 l, 16 l + 16) of each 1 KiB slice: fully coalesced.
template <int NI>
__device__ __forceinline__ void issue_tile(__amdgpu_buffer_rsrc_t rk, __amdgpu_buffer_rsrc_t rv, int lane_off,
                                           u32x4 (&k)[NI], u32x4 (&v)[NI]) {
#pragma unroll
  for (int i = 0; i < NI; ++i) k[i] = __builtin_amdgcn_raw_buffer_load_b128(rk, lane_off, i * 1024, kKvLoadPolicy);
#pragma unroll
  for (int i = 0; i < NI; ++i) v[i] = __builtin_amdgcn_raw_buffer_load_b128(rv, lane_off, i * 1024, kKvLoadPolicy);
}

// Loads issued as inline assembly, for the stream kernel's split-KV loop:
// the compiler's wait-count insertion does not see them, so its own waits
// never drain them, and the caller waits for them with vm_wait.  rs is a
// buffer descriptor in scalar registers (loads past num_records return
// zeros); lane_off the lane's byte offset; load i reads STRIDE bytes
// further on (a 1 KiB slice of a tile, or the next 32 dims of a query row).
__device__ __forceinline__ u32x4 scalar_rsrc(const void* base, int num_bytes) {
  const uint64_t p = (uint64_t)base;
  return u32x4{(uint32_t)p, (uint32_t)(p >> 32) & 0xffffu, (uint32_t)num_bytes, 0x00020000u};
}
template <int NI, int STRIDE = 1024>
__device__ __forceinline__ void asm_issue(const u32x4& rs, int lane_off, u32x4 (&x)[NI]) {
  static_assert((NI - 1) * STRIDE < 4096, "immediate offset range");
#pragma unroll
  for (int i = 0; i < NI; ++i)
    asm volatile("buffer_load_dwordx4 %0, %1, %2, 0 offen offset:%3 nt"
                 : "=v"(x[i])
                 : "v"(lane_off), "s"(rs), "i"(i * STRIDE)
                 : "memory");
}
// One 8-byte load at p (the same address in every lane) with device scope,
// as a relaxed device-scope atomic load is compiled, issued as inline
// assembly like asm_issue's loads and waited for with vm_wait.
__device__ __forceinline__ void asm_load_dev(const void* p, u32x2_t& x) {
  asm volatile("global_load_dwordx2 %0, %1, off sc1" : "=v"(x) : "v"(p) : "memory");
}
// Wait until at most N vector-memory operations are outstanding, then hand
// x to the code after the wait (the empty statements keep every use of x
// below it).
template <int N, int NI>
__device__ __forceinline__ void vm_wait(u32x4 (&x)[NI]) {
  asm volatile("s_waitcnt vmcnt(%0)" : : "i"(N) : "memory");
#pragma unroll
  for (int i = 0; i < NI; ++i) asm volatile("" : "+v"(x[i]));
}
template <int N>
__device__ __forceinline__ void vm_wait(u32x2_t& x) {
  asm volatile("s_waitcnt vmcnt(%0)" : : "i"(N) : "memory");
  asm volatile("" : "+v"(x));
}

// Fold one tile into the running state.  `valid` (wave-uniform) is the number
// of live tokens in the tile; tokens at or past it get logit -inf (their V
// was already read as 0 by the buffer range check), so whatever bytes the
// unused slots hold (even NaN) cannot reach the result.
template <typename T, int D, int S>
__device__ __forceinline__ void fold_tile(DecodeState<T, D, S>& st, const u32x4 (&k)[DecodeShape<T, D, S>::NI],
                                          const u32x4 (&v)[DecodeShape<T, D, S>::NI], int row, int valid,
                                          float scale_log2) {
  using Sh = DecodeShape<T, D, S>;
  float x[S][Sh::NI];
#pragma unroll
  for (int i = 0; i < Sh::NI; ++i)
#pragma unroll
    for (int j = 0; j < S; ++j) x[j][i] = lane_dot(st.q[j], k[i], T());
#pragma unroll
  for (int i = 0; i < Sh::NI; ++i)
#pragma unroll
    for (int j = 0; j < S; ++j) x[j][i] = group_sum<Sh::LPT>(x[j][i]) * scale_log2;
  if (valid < kPage) {  // wave-uniform: only a sequence's last page
#pragma unroll
    for (int i = 0; i < Sh::NI; ++i) {
      const bool dead = row + Sh::TPI * i >= valid;
#pragma unroll
      for (int j = 0; j < S; ++j) x[j][i] = dead ? -INFINITY : x[j][i];
    }
  }
  float vf[Sh::NI][Sh::VEC];
#pragma unroll
  for (int i = 0; i < Sh::NI; ++i) widen(v[i], vf[i], T());
#pragma unroll
  for (int j = 0; j < S; ++j) {
    float mx = x[j][0];
#pragma unroll
    for (int i = 1; i < Sh::NI; ++i) mx = fmaxf(mx, x[j][i]);
    const float mnew = fmaxf(st.m[j], mx);
    const float alpha = fast_exp2(st.m[j] - mnew);
    st.m[j] = mnew;
    float p[Sh::NI];
    float psum = 0.0f;
#pragma unroll
    for (int i = 0; i < Sh::NI; ++i) {
      p[i] = fast_exp2(x[j][i] - mnew);
      psum += p[i];
    }
    st.l[j] = fmaf(st.l[j], alpha, psum);
#pragma unroll
    for (int e = 0; e < Sh::VEC; ++e) {
      float acc = st.o[j][e] * alpha;
#pragma unroll
      for (int i = 0; i < Sh::NI; ++i) acc = fmaf(p[i], vf[i][e], acc);
      st.o[j][e] = acc;
    }
  }
}

// Sequence b and visible-key count n_vis of query row `row`.  Decode: row = b
// and all ctx keys are visible.  Varlen: b is the largest sequence with
// query_start_loc[b] <= row, and row r of a chunk of length L sees keys
// 0 .. ctx - L + r.  Returns false when the row breaks the call's contract
// (negative length, a context above max_context_len, a chunk longer than its
// context); such rows are written as NaN by the attention kernel and left
// alone by the reduction.
__device__ __forceinline__ bool row_context(const int32_t* __restrict__ qsl,
                                            const int32_t* __restrict__ context_lens, int B,
                                            int max_context_len, int row, int& b, int& n_vis) {
  if (qsl == nullptr) {
    b = row;
    n_vis = context_lens[row];
    return n_vis >= 0 && n_vis <= max_context_len;
  }
  int lo = 0, hi = B - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (qsl[mid] <= row) lo = mid; else hi = mid - 1;
  }
  b = lo;
  const int ctx = context_lens[b];
  const int L = qsl[b + 1] - qsl[b];
  n_vis = ctx - L + (row - qsl[b]) + 1;
  return ctx >= 0 && ctx <= max_context_len && n_vis >= 1;
}

// Decode row of sequence b for the stream kernel.  Returns 1 (attend: q/out
// row `row`, all nv cached keys visible), 0 (nothing to do here: a varlen
// sequence with no row, or a prefill chunk of several rows, which the
// per-row kernel takes), -1 (contract violation: NaN output).
__device__ __forceinline__ int seq_decode_row(const int32_t* __restrict__ qsl, const int32_t* __restrict__ context_lens,
                                              int max_context_len, int b, int& row, int& nv) {
  nv = context_lens[b];
  if (qsl == nullptr) {
    row = b;
    return (nv < 0 || nv > max_context_len) ? -1 : 1;
  }
  row = qsl[b];
  if (qsl[b + 1] - row != 1) return 0;
  return (nv < 1 || nv > max_context_len) ? -1 : 1;
}

// Log-sum-exp merge of the TPI lane rows of a wave for every head: on return
// every lane holds, for head j, the wave's max M[j], sum L[j] and the
// unnormalised output slice O[j][e] of its dims dl * VEC + e.
template <typename T, int D, int S>
__device__ __forceinline__ void merge_rows(const DecodeState<T, D, S>& st, float (&M)[S], float (&L)[S],
                                           float (&O)[S][DecodeShape<T, D, S>::VEC]) {
  using Sh = DecodeShape<T, D, S>;
#pragma unroll
  for (int j = 0; j < S; ++j) {
    M[j] = across_groups_max<Sh::LPT>(st.m[j]);
    const float w = fast_exp2(st.m[j] - M[j]);
    L[j] = across_groups_sum<Sh::LPT>(st.l[j] * w);
#pragma unroll
    for (int e = 0; e < Sh::VEC; ++e) O[j][e] = across_groups_sum<Sh::LPT>(st.o[j][e] * w);
  }
}

// Store the VEC consecutive outputs of one lane as one 16-byte vector store.
__device__ __forceinline__ void store_vec(uint16_t* p, const float* v) {
  u32x4 w;
  w.x = (uint32_t)f32_to_bf16(v[0]) | (uint32_t)f32_to_bf16(v[1]) << 16;
  w.y = (uint32_t)f32_to_bf16(v[2]) | (uint32_t)f32_to_bf16(v[3]) << 16;
  w.z = (uint32_t)f32_to_bf16(v[4]) | (uint32_t)f32_to_bf16(v[5]) << 16;
  w.w = (uint32_t)f32_to_bf16(v[6]) | (uint32_t)f32_to_bf16(v[7]) << 16;
  *reinterpret_cast<u32x4*>(p) = w;
}
__device__ __forceinline__ void store_vec(float* p, const float* v) {
  u32x4 w;
  w.x = __float_as_uint(v[0]);
  w.y = __float_as_uint(v[1]);
  w.z = __float_as_uint(v[2]);
  w.w = __float_as_uint(v[3]);
  *reinterpret_cast<u32x4*>(p) = w;
}

// Finish one (row, KV head) item in place: out[j][d] = O[j][d] / L[j] for the
// s heads, written by the lanes of row 0 (out points at head j = 0).
template <typename T, int D, int S>
__device__ __forceinline__ void finish_rows(const DecodeState<T, D, S>& st, int row, int dl, T* out) {
  using Sh = DecodeShape<T, D, S>;
  float M[S], L[S], O[S][Sh::VEC];
  merge_rows<T, D, S>(st, M, L, O);
  if (row == 0) {
#pragma unroll
    for (int j = 0; j < S; ++j) {
      float v[Sh::VEC];
#pragma unroll
      for (int e = 0; e < Sh::VEC; ++e) v[e] = O[j][e] / L[j];
      store_vec(out + j * D + dl * Sh::VEC, v);
    }
  }
}

// Partial record of one item: unnormalised O [S][D], then (M, L) per head.
template <typename T, int D, int S>
__device__ __forceinline__ void partial_rows(const DecodeState<T, D, S>& st, int row, int dl, int lane, float* o,
                                             float* ml) {
  using Sh = DecodeShape<T, D, S>;
  float M[S], L[S], O[S][Sh::VEC];
  merge_rows<T, D, S>(st, M, L, O);
  if (row == 0) {
#pragma unroll
    for (int j = 0; j < S; ++j) {
#pragma unroll
      for (int e = 0; e < Sh::VEC; e += 2) store_dev(o + j * D + dl * Sh::VEC + e, O[j][e], O[j][e + 1]);
    }
  }
  if (lane == 0) {
#pragma unroll
    for (int j = 0; j < S; ++j) store_dev(ml + j * 2, M[j], L[j]);
  }
}


// ---------------------------------------------------------------------------
// Matrix-core variant of the decode fold (bf16, head_dim 128).
//
// The s query heads of a group are the columns of a 16-wide MFMA tile (padded
// with zero queries), the 16 tokens of a page its rows:
//   S^T[token][head] = K . Q^T   4 x v_mfma_f32_16x16x32_bf16 (K as the A operand)
//   O^T[dim][head]  += V^T . P^T 8 x v_mfma_f32_16x16x32_bf16 (P split into bf16
//                                high and low parts for fp32-level accuracy;
//                                the k dimension holds 4 tokens x {hi, lo})
// Lane l owns head column l % 16 and tokens 4 (l / 16) .. +3 of every tile, so
// the softmax state and the rescale stay in the lane.  The wave stages each
// tile through its own 8 KiB of LDS, K and V with 16-byte chunks XOR-swizzled
// by token (conflict-free operand reads), V read back as the
// transposed PV operand with ds_read_b64_tr_b16 (lane j of a 16-lane group
// receives element j % 4 of the 8-byte blocks addressed by lanes j / 4 + 4 i).
namespace mfma {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef short s16x8_t __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

constexpr int kD = 128;
constexpr int kTile = kPage * kD * 2;  // 4 KiB

// Byte offset of 16-byte chunk `chunk` of key `key` in a staged [16][kD] bf16
// tile.  K: chunks XOR-ed with the key, so the 16 lanes of a QK operand read
// (16 keys, one chunk each) hit 16 distinct bank groups.  V: chunks XOR-ed
// with 2 (key mod 8), so a transposed PV read (per half wave: 8 keys x 2
// adjacent chunks) also hits 16 distinct 16-byte bank groups.
__device__ __forceinline__ int swz(int key, int chunk) { return key * (kD * 2) + ((chunk ^ (key & 15)) << 4); }
__device__ __forceinline__ int swz_v(int key, int chunk) { return key * (kD * 2) + ((chunk ^ ((key & 7) << 1)) << 4); }

template <int S>
struct State {
  u32x4 qt[kD / 32];   // Q^T operand: head lane%16 (zero when >= s), dims 32 st + 8 (lane/16) .. +8
  f32x4_t acc[kD / 16];  // O^T: head lane%16, dims 16 mb + 4 (lane/16) + i
  float m, l;          // softmax base (log2 units, shared by the 4 lanes of a head) and partial sum
};

// An item's queries (the Q^T operand), and its fresh softmax state.
template <int S>
__device__ __forceinline__ void load_q(State<S>& st, const uint16_t* q_group, int lane) {
  const int n = lane & 15, G = lane >> 4;
#pragma unroll
  for (int s = 0; s < kD / 32; ++s)
    st.qt[s] = n < S ? *reinterpret_cast<const u32x4*>(q_group + n * kD + s * 32 + G * 8) : u32x4{0, 0, 0, 0};
}
template <int S>
__device__ __forceinline__ void reset(State<S>& st) {
#pragma unroll
  for (int mb = 0; mb < kD / 16; ++mb) st.acc[mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  st.m = kMInit;
  st.l = 0.0f;
}
template <int S>
__device__ __forceinline__ void begin_item(State<S>& st, const uint16_t* q_group, int lane) {
  load_q<S>(st, q_group, lane);
  reset<S>(st);
}

// Split four fp32 softmax weights into bf16 high parts (round to nearest
// even) and bf16 low parts (the rounding residue, exact in fp32): hi + lo
// carries ~16 mantissa bits, so the PV product keeps fp32-level accuracy
// while both halves run on the bf16 matrix cores.  Conversions are gfx950's
// v_cvt_pk_bf16_f32 (two values per instruction, nearest even).
__device__ __forceinline__ void split_hi_lo(const float (&p)[4], s16x4_t& hi, s16x4_t& lo) {
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  typedef __bf16 bf16x2v_t __attribute__((ext_vector_type(2)));
  const f32x2_t p01 = f32x2_t{p[0], p[1]}, p23 = f32x2_t{p[2], p[3]};
  const bf16x2v_t h01 = __builtin_convertvector(p01, bf16x2v_t);
  const bf16x2v_t h23 = __builtin_convertvector(p23, bf16x2v_t);
  const bf16x2v_t l01 = __builtin_convertvector(p01 - __builtin_convertvector(h01, f32x2_t), bf16x2v_t);
  const bf16x2v_t l23 = __builtin_convertvector(p23 - __builtin_convertvector(h23, f32x2_t), bf16x2v_t);
  // whole-vector bit casts only (a bit cast of one vector element misreads)
  hi = __builtin_bit_cast(s16x4_t, u32x2_t{__builtin_bit_cast(uint32_t, h01), __builtin_bit_cast(uint32_t, h23)});
  lo = __builtin_bit_cast(s16x4_t, u32x2_t{__builtin_bit_cast(uint32_t, l01), __builtin_bit_cast(uint32_t, l23)});
}

// acc += V^T . (P_hi + P_lo)^T in one 16x16x32 product: the lane's k slots
// 8 G .. 8 G + 7 carry its 4 tokens twice in A (va = V^T of tokens 4 G + i)
// and P's high then low parts in B, so the sum over k adds both products.
__device__ __forceinline__ f32x4_t pv_mfma(const s16x4_t& va, const s16x4_t& phi, const s16x4_t& plo, f32x4_t acc) {
  const s16x8_t a = __builtin_shufflevector(va, va, 0, 1, 2, 3, 0, 1, 2, 3);
  const s16x8_t b = __builtin_shufflevector(phi, plo, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a), __builtin_bit_cast(bf16x8_t, b), acc,
                                                 0, 0, 0);
}

// The fold of one tile in two halves, so that a tile's V loads can be waited
// for after its K half is done.  k / v: the tile as loaded (lane l: token
// l/16 + 4 i, 16-byte chunk l%16); lds: this wave's 8 KiB (K then V); valid:
// live tokens of the tile.
//
// fold_qk: K to LDS, S^T = K . Q^T, online softmax; the P^T operands (bf16
// high and low parts of the lane's 4 weights) come back in phi / plo.
template <int S>
__device__ __forceinline__ void fold_qk(State<S>& st, const u32x4 (&k)[4], uint8_t* lds, int lane, int valid,
                                        float scale_log2, s16x4_t& phi, s16x4_t& plo) {
  const int G = lane >> 4, p = lane & 15;
#pragma unroll
  for (int i = 0; i < 4; ++i) *reinterpret_cast<u32x4*>(lds + swz(G + 4 * i, p)) = k[i];
  // S^T = K . Q^T
  f32x4_t s = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int step = 0; step < kD / 32; ++step) {
    const u32x4 ka = *reinterpret_cast<const u32x4*>(lds + swz(p, step * 4 + G));
    s = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, ka), __builtin_bit_cast(bf16x8_t, st.qt[step]),
                                                s, 0, 0, 0);
  }
  // online softmax over this lane's 4 tokens, max shared by the head's 4
  // lanes; the base moves only past the slack (the branch is wave-uniform)
  float x[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    x[i] = s[i];
    if (valid < kPage) x[i] = 4 * G + i < valid ? x[i] : -INFINITY;
  }
  // scale > 0, so the max commutes with it
  const float mx = rows4_max(fmaxf(fmaxf(x[0], x[1]), fmaxf(x[2], x[3]))) * scale_log2;
  const float mc = fmaxf(st.m, mx);
  if (__builtin_amdgcn_ballot_w64(mc > st.m + kRescaleSlack) != 0) {
    const float alpha = fast_exp2(st.m - mc);
    st.m = mc;
    st.l *= alpha;
#pragma unroll
    for (int mb = 0; mb < kD / 16; ++mb) st.acc[mb] *= alpha;
  }
  float pw[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) pw[i] = fast_exp2(fmaf(x[i], scale_log2, -st.m));
  st.l += (pw[0] + pw[1]) + (pw[2] + pw[3]);
  split_hi_lo(pw, phi, plo);
}

// fold_pv: V to LDS, O^T += V^T . P^T; lane p of group G addresses token
// 4 G + p / 4, dims 16 mb + 4 (p % 4).
template <int S>
__device__ __forceinline__ void fold_pv(State<S>& st, const u32x4 (&v)[4], uint8_t* lds, int lane,
                                        const s16x4_t& phi, const s16x4_t& plo) {
  const int G = lane >> 4, p = lane & 15;
#pragma unroll
  for (int i = 0; i < 4; ++i) *reinterpret_cast<u32x4*>(lds + kTile + swz_v(G + 4 * i, p)) = v[i];
  const int vtok = 4 * G + (p >> 2);
#pragma unroll
  for (int mb = 0; mb < kD / 16; ++mb) {
    const int d = mb * 16 + 4 * (p & 3);
    const lds_s16x4_t* src = (const lds_s16x4_t*)(lds + kTile + swz_v(vtok, d >> 3) + (d & 7) * 2);
    const s16x4_t va = __builtin_amdgcn_ds_read_tr16_b64_v4i16(const_cast<lds_s16x4_t*>(src));
    st.acc[mb] = pv_mfma(va, phi, plo, st.acc[mb]);
  }
}

// Both halves of one tile.
template <int S>
__device__ __forceinline__ void fold(State<S>& st, const u32x4 (&k)[4], const u32x4 (&v)[4], uint8_t* lds, int lane,
                                     int valid, float scale_log2) {
  s16x4_t phi, plo;
  fold_qk<S>(st, k, lds, lane, valid, scale_log2, phi, plo);
  fold_pv<S>(st, v, lds, lane, phi, plo);
}

// Totals of the head column of this lane: L summed over the 4 lane groups.
template <int S>
__device__ __forceinline__ float total_l(const State<S>& st) {
  return rows4_sum(st.l);
}

// Finish an item in place: out points at head 0 of the group ([s][D]).
template <int S, typename T>
__device__ __forceinline__ void finish(const State<S>& st, int lane, T* out) {
  const float L = total_l(st);
  const int n = lane & 15, G = lane >> 4;
  if (n < S) {
    const float inv = 1.0f / L;
#pragma unroll
    for (int mb = 0; mb < kD / 16; ++mb) {
      const int d = mb * 16 + 4 * G;
      const uint32_t lo = (uint32_t)f32_to_bf16(st.acc[mb][0] * inv) | (uint32_t)f32_to_bf16(st.acc[mb][1] * inv) << 16;
      const uint32_t hi = (uint32_t)f32_to_bf16(st.acc[mb][2] * inv) | (uint32_t)f32_to_bf16(st.acc[mb][3] * inv) << 16;
      *reinterpret_cast<uint2*>(out + n * kD + d) = make_uint2(lo, hi);
    }
  }
}

// Partial record: unnormalised O [s][D] and (M, L) per head (device-coherent
// stores: the record is read by another workgroup of the same launch).
template <int S>
__device__ __forceinline__ void partial(const State<S>& st, int lane, float* o, float* ml) {
  const float L = total_l(st);
  const int n = lane & 15, G = lane >> 4;
  if (n < S) {
#pragma unroll
    for (int mb = 0; mb < kD / 16; ++mb) {
      const int d = mb * 16 + 4 * G;
      store_dev(o + n * kD + d, st.acc[mb][0], st.acc[mb][1]);
      store_dev(o + n * kD + d + 2, st.acc[mb][2], st.acc[mb][3]);
    }
    if (G == 0) store_dev(ml + n * 2, st.m, L);
  }
}

}  // namespace mfma
}  // namespace pa
