// Host-side calculator of the MoE-Lens performance model (Sec. 5, Eqs. 1-14).
// A pure function of its input: no device, no allocation.
#include <math.h>

#include <algorithm>

#include "pa_perf_model.h"

namespace {

// sum_{n=0}^{N} floor(n / b) for N >= -1: with N + 1 = k b + r (0 <= r < b)
// the full groups contribute b (0 + 1 + ... + k-1) and the last r terms k each.
long double floor_prefix(int64_t N, int64_t b) {
  if (N < 0) return 0.0L;
  const int64_t k = (N + 1) / b, r = (N + 1) % b;
  return (long double)b * (long double)k * (long double)(k - 1) / 2.0L + (long double)r * (long double)k;
}

// sum_{i=0}^{g} ceil((p + i) / b) = sum_{m=p+b-1}^{p+g+b-1} floor(m / b)
double lifetime_blocks(int64_t p, int64_t g, int64_t b) {
  return (double)(floor_prefix(p + g + b - 1, b) - floor_prefix(p + b - 2, b));
}

}  // namespace

extern "C" int pa_perf_model(const pa_pm_input_t* in, pa_pm_output_t* out) {
  if (in == nullptr || out == nullptr) return -1;
  const pa_pm_input_t& x = *in;
  if (!(x.num_experts > 0 && x.top_k > 0 && x.top_k <= x.num_experts && x.model_dim > 0 && x.expert_dim > 0 &&
        x.gqa_group > 0 && x.model_bytes > 0 && x.kv_bytes_per_token > 0 && x.gemm_flops > 0 && x.io_bw > 0 &&
        x.kv_capacity_bytes > 0 && x.batch > 0 && x.attn_bw >= 0 && x.attn_intensity >= 0))
    return -1;
  if (x.prompt < 1 || x.gen < 1 || x.block < 1) return -1;
  const double p = x.prompt, g = x.gen;
  const double M = x.kv_capacity_bytes / x.kv_bytes_per_token;
  const double N = floor(M / x.block);
  if (!(N >= 1)) return -1;

  pa_pm_output_t o;
  // Eq. 1: per token, the active parameters' FLOPs over all weight bytes
  const double h2 = x.model_dim * x.model_dim;
  const double proj = 4.0 * h2 * (1.0 + 1.0 / x.gqa_group);
  o.intensity_per_token = (6.0 * x.top_k * x.model_dim * x.expert_dim + proj) /
                          (6.0 * x.num_experts * x.model_dim * x.expert_dim + proj);
  // Eq. 2 with the sparsity approximation of Eq. 1
  const double n_sat = x.gemm_flops * x.num_experts / (x.io_bw * x.top_k);
  o.tokens_to_saturate = n_sat;
  o.pme = 2.0 * (p + g) / ((2.0 * p + g) * g);  // Eq. 3
  o.delta = x.model_bytes / x.io_bw;
  o.kv_tokens = M;
  o.t_gpu = n_sat / o.delta;
  o.t_max = std::min(o.pme * M / o.delta, o.t_gpu);  // Eq. 4
  o.kv_bw = x.kv_capacity_bytes / o.delta;
  o.mem_bw = o.kv_bw + x.io_bw;                        // Eq. 5: B_KV + B_IO
  o.attn_flops = 2.0 * x.gqa_group * x.attn_intensity * o.kv_bw;  // Eq. 6
  o.kv_effective = x.kv_capacity_bytes * (p + g) / (p + 0.5 * g);  // Eq. 7
  o.kv_blocks = N;
  o.q = N / lifetime_blocks(x.prompt, x.gen, x.block);  // Eq. 8
  o.decode_seqs = g * o.q;                              // Eq. 9
  const double K = x.batch;
  o.t1 = K / (K + o.decode_seqs) * (o.decode_seqs / o.delta);  // Eq. 10
  // Eqs. 11-13 count tokens per iteration: the GPU's limit is n_sat
  o.t_prefill = n_sat * p / (p + g);
  const double prologue = 0.5 * (o.t_prefill + n_sat) * g;
  o.iterations = 2.0 * g + (K * p - prologue) / o.t_prefill;
  o.t2 = K * g / (o.iterations * o.delta);
  o.t = std::min(o.t1, o.t2);  // Eq. 14
  if (x.attn_bw > 0) {
    o.attn_headroom = x.attn_bw / o.kv_bw;
    o.delta_eff = std::max(o.delta, x.kv_capacity_bytes / x.attn_bw);
  } else {
    o.attn_headroom = 0.0;
    o.delta_eff = o.delta;
  }
  o.t_attn_bound = o.t * (o.delta / o.delta_eff);
  *out = o;
  return 0;
}
