// HBM read-stream probe: the decode kernels' load pattern with no arithmetic
// (declared in pa_probe.h).  Each wave reads 4 KiB slices with four 16-byte
// raw buffer loads per lane (one 1 KiB row of 64 lanes per load, fully
// coalesced).  With DEPTH 2 it keeps the next slice's loads in flight while
// it folds the current one, as the attention kernels' two-tile ring does;
// with DEPTH 1 it waits for each slice before loading the next.  Every load
// is issued unconditionally (a slice past the range gets an empty buffer
// descriptor, which loads zeros without touching memory) and each stage is
// a scheduling region of its own, so the compiler's wait counts keep exactly
// DEPTH slices in flight.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pa_probe.h"

namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kSlice = 4096;

template <int POLICY>
__device__ __forceinline__ void load_slice(const uint8_t* p, bool in_range, int lane, u32x4 (&r)[4]) {
  const __amdgpu_buffer_rsrc_t rs =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(p), (short)0, in_range ? kSlice : 0, 0x00020000);
#pragma unroll
  for (int i = 0; i < 4; ++i) r[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, lane * 16, i * 1024, POLICY);
}

template <int POLICY, int kWaves, int DEPTH>
__global__ __launch_bounds__(64 * kWaves) void read_probe_kernel(const uint8_t* buf, const int64_t* offs,
                                                                 int spc_log2, int64_t n_slices, uint32_t* sink) {
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int64_t G = gridDim.x, x = blockIdx.x;
  const int64_t s0 = n_slices * x / G, s1 = n_slices * (x + 1) / G;
  uint32_t acc = 0;
  if (s0 < s1) {
    // slice j of the range; a j past it reads the range's last slice's
    // address with an empty descriptor (zeros, no memory access)
    auto load = [&](int64_t j, u32x4 (&r)[4]) {
      const int64_t jj = j < s1 ? j : s1 - 1;
      const int64_t c = jj >> spc_log2, sub = jj & ((1 << spc_log2) - 1);
      const int64_t base = offs != nullptr ? offs[c] : (c << spc_log2) * kSlice;
      load_slice<POLICY>(buf + base + sub * kSlice, j < s1, lane, r);
    };
    u32x4 r[DEPTH][4];
    const int64_t j0 = s0 + w;
#pragma unroll
    for (int d = 0; d + 1 < DEPTH; ++d) load(j0 + d * kWaves, r[d]);
    for (int64_t j = j0; j < s1; j += DEPTH * kWaves) {
#pragma unroll
      for (int d = 0; d < DEPTH; ++d) {
        // issue the slice DEPTH - 1 stages ahead, then fold this stage's
        load(j + (d + DEPTH - 1) * kWaves, r[(d + DEPTH - 1) % DEPTH]);
#pragma unroll
        for (int i = 0; i < 4; ++i) acc ^= r[d][i].x ^ r[d][i].y ^ r[d][i].z ^ r[d][i].w;
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  sink[x * 64 * kWaves + threadIdx.x] = acc;
}

template <int POLICY>
const void* read_fn(int waves, int depth) {
  if (waves == 8) return depth == 2 ? reinterpret_cast<const void*>(&read_probe_kernel<POLICY, 8, 2>)
                                    : reinterpret_cast<const void*>(&read_probe_kernel<POLICY, 8, 1>);
  return depth == 2 ? reinterpret_cast<const void*>(&read_probe_kernel<POLICY, 4, 2>)
                    : reinterpret_cast<const void*>(&read_probe_kernel<POLICY, 4, 1>);
}

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// Issue-overlap probe: four independent matrix products per iteration (four
// accumulator chains) and NV vector instructions per product (independent
// FMAs, or exponentials, over 16 registers).  MODE 0 runs both in every wave,
// each product followed by its NV vector instructions (the order is pinned
// with scheduling-group barriers); MODE 1 only the products; MODE 2 only the
// vector work; MODE 3 splits the workgroup: its first half of waves runs the
// products, the second half (on the same SIMDs) the vector work.  Lane 0 of
// every wave records the shader-clock cycles its loop took.
template <bool BIG, int NV, bool EXP, int MODE>
__global__ __launch_bounds__(512) void issue_probe_kernel(float* sink, uint64_t* cycles, int iters, float c) {
  bf16x8_t a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(threadIdx.x * 0.001f + i);
    b[i] = (__bf16)(i * 0.5f);
  }
  float v[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) v[i] = threadIdx.x * 0.01f + i;
  f32x4_t acc4[4];
  f32x16_t acc16[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    acc4[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < 16; ++j) acc16[i][j] = 0.f;
  }
  auto product = [&](int m) {
    if constexpr (BIG) acc16[m] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc16[m], 0, 0, 0);
    else acc4[m] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc4[m], 0, 0, 0);
  };
  auto valu = [&](int m) {
#pragma unroll
    for (int f = 0; f < NV; ++f) {
      float& x = v[(m * NV + f) & 15];
      if constexpr (EXP) x = __builtin_amdgcn_exp2f(x);
      else x = fmaf(x, c, 0.5f);
    }
  };
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const bool products = MODE == 0 || MODE == 1 || (MODE == 3 && wave < (int)(blockDim.x >> 7));
  const bool vector = MODE == 0 || MODE == 2 || (MODE == 3 && !products);
  const uint64_t t0 = __builtin_amdgcn_s_memtime();
  if (products && vector) {
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        product(m);
        valu(m);
      }
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // one matrix product
        // then its vector work (exponentials form their own group, transcendental)
        if constexpr (NV > 0) __builtin_amdgcn_sched_group_barrier(EXP ? 0x400 : 0x002, NV, 0);
      }
    }
  } else if (products) {
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int m = 0; m < 4; ++m) product(m);
    }
  } else if (vector) {
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int m = 0; m < 4; ++m) valu(m);
    }
  }
  const uint64_t t1 = __builtin_amdgcn_s_memtime();
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
#pragma unroll
    for (int j = 0; j < 4; ++j) s += acc4[i][j];
#pragma unroll
    for (int j = 0; j < 16; ++j) s += acc16[i][j];
  }
#pragma unroll
  for (int i = 0; i < 16; ++i) s += v[i];
  sink[(int64_t)blockIdx.x * blockDim.x + threadIdx.x] = s;
  if (cycles != nullptr && (threadIdx.x & 63) == 0) cycles[(int64_t)blockIdx.x * (blockDim.x >> 6) + wave] = t1 - t0;
}

template <bool BIG, bool EXP, int MODE>
const void* issue_fn(int nv) {
  switch (nv) {
    case 0: return reinterpret_cast<const void*>(&issue_probe_kernel<BIG, 0, EXP, MODE>);
    case 1: return reinterpret_cast<const void*>(&issue_probe_kernel<BIG, 1, EXP, MODE>);
    case 2: return reinterpret_cast<const void*>(&issue_probe_kernel<BIG, 2, EXP, MODE>);
    case 3: return reinterpret_cast<const void*>(&issue_probe_kernel<BIG, 3, EXP, MODE>);
    case 4: return reinterpret_cast<const void*>(&issue_probe_kernel<BIG, 4, EXP, MODE>);
    case 6: return reinterpret_cast<const void*>(&issue_probe_kernel<BIG, 6, EXP, MODE>);
    case 8: return reinterpret_cast<const void*>(&issue_probe_kernel<BIG, 8, EXP, MODE>);
    case 16: return reinterpret_cast<const void*>(&issue_probe_kernel<BIG, 16, EXP, MODE>);
  }
  return nullptr;
}

template <bool BIG, bool EXP>
const void* issue_fn_mode(int mode, int nv) {
  switch (mode) {
    case 0: return issue_fn<BIG, EXP, 0>(nv);
    case 1: return issue_fn<BIG, EXP, 1>(nv);
    case 2: return issue_fn<BIG, EXP, 2>(nv);
    case 3: return issue_fn<BIG, EXP, 3>(nv);
  }
  return nullptr;
}

}  // namespace

extern "C" int pa_issue_probe(int32_t grid, int32_t waves, int32_t iters, int32_t big_mfma, int32_t valu_per_mfma,
                              int32_t exp2, int32_t mode, float* sink, uint64_t* cycles, hipStream_t stream) {
  if (sink == nullptr || !(waves == 1 || waves == 2 || waves == 4 || waves == 8) || iters < 1 || grid < 1 ||
      grid > 65535 || mode < 0 || mode > 3 || (mode == 3 && waves < 2))
    return -1;
  const void* fn = big_mfma ? (exp2 ? issue_fn_mode<true, true>(mode, valu_per_mfma)
                                    : issue_fn_mode<true, false>(mode, valu_per_mfma))
                            : (exp2 ? issue_fn_mode<false, true>(mode, valu_per_mfma)
                                    : issue_fn_mode<false, false>(mode, valu_per_mfma));
  if (fn == nullptr) return -1;  // a count the probe is not built for
  float c = 0.999f;
  void* args[] = {&sink, &cycles, &iters, &c};
  if (hipLaunchKernel(fn, dim3(grid), dim3(64 * waves), args, 0, stream) != hipSuccess) return -4;
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

extern "C" int pa_read_probe(const void* buf, int64_t chunk_bytes, const int64_t* chunk_offsets,
                             int64_t n_chunks, int32_t grid, int32_t waves, int32_t depth, int32_t non_temporal,
                             uint32_t* sink, hipStream_t stream) {
  if (buf == nullptr || sink == nullptr || chunk_bytes <= 0 || chunk_bytes % kSlice != 0 || n_chunks < 0 ||
      grid < 1 || grid > 65535 || !(waves == 4 || waves == 8) || !(depth == 1 || depth == 2))
    return -1;
  const int64_t spc = chunk_bytes / kSlice;
  if ((spc & (spc - 1)) != 0 || spc > (1 << 20)) return -1;  // a power of two slices per chunk
  int spc_log2 = 0;
  while ((int64_t(1) << spc_log2) < spc) ++spc_log2;
  int64_t n_slices = spc * n_chunks;
  const uint8_t* p = static_cast<const uint8_t*>(buf);
  void* args[] = {&p, &chunk_offsets, &spc_log2, &n_slices, &sink};
  const void* fn = non_temporal ? read_fn<2>(waves, depth) : read_fn<0>(waves, depth);
  if (hipLaunchKernel(fn, dim3(grid), dim3(64 * waves), args, 0, stream) != hipSuccess) return -4;
  return hipGetLastError() == hipSuccess ? 0 : -4;
}
