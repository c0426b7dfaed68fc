// Device-side helpers shared by the gfx950 attention kernels: bf16 packing,
// wave64 lane reductions (DPP inside a 16-lane row, swizzle/bpermute across
// rows) and the block-table address function every kernel uses.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pa {

constexpr int kPage = 16;  // token slots per KV page

// Running-max start value.  Finite, so that exp2(m_old - m_new) is 1 and not
// NaN while a row has seen only masked keys; far below any real logit.
constexpr float kMInit = -1.0e30f;

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));  // one 16-byte lane load
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

// Reinterpret one packed pair.  Takes the word by value: bit-casting an
// ext-vector element lvalue directly (v.y) has been seen to read element 0.
__device__ __forceinline__ bf16x2_t as_bf16x2(uint32_t w) { return __builtin_bit_cast(bf16x2_t, w); }

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// fp32 -> bf16 bit pattern, round to nearest even; NaN -> quiet NaN.
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;
  return (uint16_t)((u + 0x7fffu + ((u >> 16) & 1u)) >> 16);
}

template <typename T> __device__ __forceinline__ void store_out(T* p, float v);
template <> __device__ __forceinline__ void store_out<uint16_t>(uint16_t* p, float v) { *p = f32_to_bf16(v); }
template <> __device__ __forceinline__ void store_out<float>(float* p, float v) { *p = v; }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// --- lane exchanges -------------------------------------------------------
// DPP controls: quad_perm [1,0,3,2] (xor 1), [2,3,0,1] (xor 2), row_half_mirror
// (lane i <-> 7-i inside 8), row_mirror (i <-> 15-i inside 16).  Once all
// lanes of a group of 4 (resp. 8) hold equal values, the mirrors pair each
// group with its neighbour, so the four steps form a full butterfly over 16.
__device__ __forceinline__ float dpp_xor1(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));
}
__device__ __forceinline__ float dpp_xor2(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));
}
__device__ __forceinline__ float dpp_half_mirror(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x141, 0xF, 0xF, false));
}
__device__ __forceinline__ float dpp_mirror(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x140, 0xF, 0xF, false));
}
// xor 16 inside each 32-lane half (ds_swizzle bit mode: and 0x1f, xor 0x10)
__device__ __forceinline__ float swz_xor16(float v) {
  return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x401F));
}
__device__ __forceinline__ float xor32(float v) {
  return __int_as_float(__builtin_amdgcn_ds_bpermute((int)((__lane_id() ^ 32) << 2), __float_as_int(v)));
}

// Sum over aligned groups of N lanes (N = 1, 2, 4, 8, 16, 32, 64); every lane
// of a group ends with the group total.
template <int N> __device__ __forceinline__ float group_sum(float v) {
  if constexpr (N >= 2) v += dpp_xor1(v);
  if constexpr (N >= 4) v += dpp_xor2(v);
  if constexpr (N >= 8) v += dpp_half_mirror(v);
  if constexpr (N >= 16) v += dpp_mirror(v);
  if constexpr (N >= 32) v += swz_xor16(v);
  if constexpr (N >= 64) v += xor32(v);
  return v;
}

// Exchange with lane l ^ OFF (OFF a power of two below 64).
template <int OFF> __device__ __forceinline__ float xor_lanes(float v) {
  static_assert(OFF >= 1 && OFF <= 32 && (OFF & (OFF - 1)) == 0, "power of two");
  if constexpr (OFF == 1) return dpp_xor1(v);
  else if constexpr (OFF == 2) return dpp_xor2(v);
  else if constexpr (OFF == 32) return xor32(v);
  else return __int_as_float(__builtin_amdgcn_ds_swizzle(__float_as_int(v), 0x1F | (OFF << 10)));
}

// Partial records of the stream-K kernel are exchanged between workgroups of
// one launch that may sit on different XCDs, whose L2 caches are not coherent
// with each other.  They are written and read with device-scope relaxed
// atomics (coherent at the device level, no L2 writeback or invalidate of the
// whole cache), 8 bytes at a time.
__device__ __forceinline__ void store_dev(float* p, float a, float b) {
  const unsigned long long v = (unsigned long long)__float_as_uint(a) | (unsigned long long)__float_as_uint(b) << 32;
  __hip_atomic_store(reinterpret_cast<unsigned long long*>(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void load_dev2(const float* p, float& a, float& b) {
  const unsigned long long v =
      __hip_atomic_load(reinterpret_cast<const unsigned long long*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  a = __uint_as_float((uint32_t)v);
  b = __uint_as_float((uint32_t)(v >> 32));
}
__device__ __forceinline__ float load_dev(const float* p) {
  return __uint_as_float(__hip_atomic_load(reinterpret_cast<const unsigned int*>(p), __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT));
}

// Lazy rebasing of the online softmax (matrix-core paths): a row's running
// max m is moved only when a new score exceeds it by more than this many log2
// units; until then weights exp2(x - m) stay below 2^kRescaleSlack and the
// output accumulators need no rescale.  Any base gives the same normalised
// result, since numerator and denominator share it.
constexpr float kRescaleSlack = 8.0f;
constexpr float kRescaleLimit = 256.0f;  // 2^kRescaleSlack

// Max / sum of v over the four 16-lane rows of the wave (lanes l, l ^ 16,
// l ^ 32, l ^ 48), all lanes ending with the result.  gfx950's row-swap
// permutes (v_permlane16_swap / v_permlane32_swap) run on the VALU: with the
// same register as both operands, the swap returns rows (0, 0, 2, 2) and
// (1, 1, 3, 3) (resp. halves (0, 0) and (1, 1)), so one max of the pair folds
// the rows pairwise.
__device__ __forceinline__ float rows4_max(float v) {
  const uint32_t u = __float_as_uint(v);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const float m = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  const uint32_t um = __float_as_uint(m);
  const auto b = __builtin_amdgcn_permlane32_swap(um, um, false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float rows4_sum(float v) {
  const uint32_t u = __float_as_uint(v);
  const auto a = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  const float t = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  const uint32_t ut = __float_as_uint(t);
  const auto b = __builtin_amdgcn_permlane32_swap(ut, ut, false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Max / sum across the aligned lane groups of size G that tile a wave: lane
// l combines with l ^ G, l ^ 2G, ..., l ^ 32; every lane ends with the result.
template <int G> __device__ __forceinline__ float across_groups_max(float v) {
  if constexpr (G < 64) {
    v = fmaxf(v, xor_lanes<G>(v));
    return across_groups_max<G * 2>(v);
  } else {
    return v;
  }
}
template <int G> __device__ __forceinline__ float across_groups_sum(float v) {
  if constexpr (G < 64) {
    v += xor_lanes<G>(v);
    return across_groups_sum<G * 2>(v);
  } else {
    return v;
  }
}

// Inclusive prefix sum over the 64 lanes of a wave, on the VALU's DPP
// lane paths: shifts by 1, 2, 4, 8 inside each 16-lane row (lanes shifted in
// from outside the row read 0), then lane 15 of rows 0 and 2 added into rows
// 1 and 3 (row_bcast:15), then lane 31 into rows 2 and 3 (row_bcast:31).
__device__ __forceinline__ int wave_incl_scan(int x) {
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, true);   // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, true);   // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, true);   // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, true);   // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false);  // row_bcast:15
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false);  // row_bcast:31
  return x;
}

// Exclusive prefix sum of one value per thread over a workgroup of NT
// threads: an inclusive scan inside each wave, one LDS round for the wave
// totals (s_tmp holds NT / 64 ints), two barriers.
template <int NT>
__device__ __forceinline__ int block_exclusive_scan(int v, int* s_tmp) {
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int x = wave_incl_scan(v);
  if constexpr (NT <= 64) {
    return x - v;
  } else {
    if (lane == 63) s_tmp[wv] = x;
    __syncthreads();
    int before = 0;
#pragma unroll
    for (int i = 0; i < NT / 64; ++i) before += i < wv ? s_tmp[i] : 0;
    __syncthreads();  // s_tmp may be rewritten by the caller next
    return before + x - v;
  }
}

// Gather trace (instantiations with a trace array only): record the pool row
// that a kernel loaded for token t of sequence b under KV head g at
// trace[(g * B + b) * stride_tokens + t].  Entries start at -1; a second load
// of the same token with a different row marks the entry -2.
__device__ __forceinline__ void trace_put(int64_t* trace, int64_t idx, int64_t row) {
  unsigned long long* p = reinterpret_cast<unsigned long long*>(trace + idx);
  const unsigned long long old = atomicCAS(p, ~0ull, (unsigned long long)row);
  if (old != ~0ull && old != (unsigned long long)row) atomicExch(p, (unsigned long long)-2ll);
}

// Block-table address function.  Token t of sequence b sits in slot t % 16 of
// page block_table[b][t / 16]; the pool row of that token is page * 16 + slot
// and, for KV head g of a [page][H_kv][16][D] pool, its first element is
// ((page * H_kv + g) * 16 + slot) * D.  Every attention kernel goes through
// BlockTable::page and tile_offset (or, in the prefill kernel, the same
// offset formula over its LDS window of the table).
struct BlockTable {
  const int32_t* table;
  int64_t stride;  // max_pages_per_seq
  __device__ __forceinline__ int32_t page(int b, int p) const { return table[(int64_t)b * stride + p]; }
};

__device__ __forceinline__ int64_t tile_offset(int32_t page, int g, int H_kv, int D) {
  return ((int64_t)page * H_kv + g) * (int64_t)(kPage * D);
}

}  // namespace pa
