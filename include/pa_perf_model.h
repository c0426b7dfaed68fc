/*
 * pa_perf_model.h -- the MoE-Lens performance model (arXiv 2504.09345,
 * Sec. 5, Eqs. 1-14) as a host-side calculator in libpagedattn.so.
 *
 * The paper models offloaded MoE inference: weights stream to the GPU at
 * B_IO once per iteration (delta = model bytes / B_IO), the KV cache sits in
 * a memory of fixed capacity and is read once per iteration by the attention,
 * and the GPU computes the GEMMs for every token in flight.  Stage 1 bounds
 * the throughput by the GPU and by the KV capacity through the
 * parallelism-memory efficiency PME (Eqs. 2-4); Sec. 5.3 gives the memory
 * bandwidth and attention compute the KV side must sustain (Eqs. 5-6);
 * Sec. 5.4 the capacity gain of overlapping prefill and decode (Eq. 7); and
 * Stage 2 adds the paged cache of N blocks of b tokens, a request batch of K
 * sequences and the pipeline's prologue and epilogue (Eqs. 8-14).
 *
 * Units are SI: FLOP/s, bytes, bytes/s, seconds, tokens.  The calculator is a
 * pure function of its input; it touches no device and allocates nothing.
 */
#ifndef PA_PERF_MODEL_H
#define PA_PERF_MODEL_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  /* model (Sec. 5.1 notation) */
  double num_experts;        /* N_e */
  double top_k;              /* N_k, 1 <= N_k <= N_e */
  double model_dim;          /* h */
  double expert_dim;         /* h_i */
  double gqa_group;          /* s */
  double model_bytes;        /* weights moved per iteration */
  double kv_bytes_per_token; /* K and V of one token over all layers */
  /* hardware */
  double gemm_flops;         /* C_GPU, FLOP/s */
  double io_bw;              /* B_IO, bytes/s */
  double kv_capacity_bytes;  /* memory holding the KV cache */
  double attn_bw;            /* measured attention read bandwidth, bytes/s;
                                0 = not given */
  double attn_intensity;     /* I_attn of Eq. 6, FLOP per KV byte read */
  /* workload */
  double batch;              /* K, sequences in the request batch (> 0) */
  int32_t prompt;            /* p >= 1 */
  int32_t gen;               /* g >= 1 */
  int32_t block;             /* b, tokens per KV block >= 1 */
} pa_pm_input_t;

typedef struct {
  double intensity_per_token; /* Eq. 1 without n: GEMM FLOP per weight byte per token */
  double tokens_to_saturate;  /* Eq. 2: C_GPU / B_IO * N_e / N_k (tokens per iteration) */
  double pme;                 /* Eq. 3: 2 (p + g) / ((2p + g) g) */
  double delta;               /* model_bytes / B_IO, seconds per iteration */
  double kv_tokens;           /* M: KV capacity in tokens */
  double t_gpu;               /* T_GPU = tokens_to_saturate / delta, tokens/s */
  double t_max;               /* Eq. 4: min(PME * M / delta, T_GPU), tokens/s */
  double mem_bw;              /* Eq. 5: (weights + KV) / weights * B_IO */
  double kv_bw;               /* B_KV = kv_capacity_bytes / delta */
  double attn_flops;          /* Eq. 6: 2 s I_attn B_KV */
  double kv_effective;        /* Eq. 7: (p + g) / (p + g/2) * capacity, bytes */
  double kv_blocks;           /* N = floor(M / b) */
  double q;                   /* Eq. 8: N / sum_{i=0}^{g} ceil((p + i) / b) */
  double decode_seqs;         /* Eq. 9: g q */
  double t1;                  /* Eq. 10: K g / ((K / q + g) delta), tokens/s */
  double t_prefill;           /* Eq. 11: T_GPU p / (p + g), tokens per iteration */
  double iterations;          /* Eq. 12 */
  double t2;                  /* Eq. 13: K g / (It delta), tokens/s */
  double t;                   /* Eq. 14: min(T1, T2), tokens/s */
  /* Sec. 5.3's requirement with a measured attention bandwidth: attention
   * reads the whole KV cache once per iteration, so an attention slower than
   * B_KV stretches the iteration to capacity / attn_bw.  With attn_bw = 0:
   * headroom 0, delta_eff = delta, t_attn_bound = t. */
  double attn_headroom;       /* attn_bw / B_KV */
  double delta_eff;           /* max(delta, capacity / attn_bw) */
  double t_attn_bound;        /* t * delta / delta_eff */
} pa_pm_output_t;

/* Evaluate every quantity of Sec. 5 for one configuration.
 * Returns 0, or -1 (PA_EINVAL) for a null pointer or a size out of range
 * (non-positive N_e, N_k, h, h_i, s, model bytes, bytes per token, C_GPU,
 * B_IO, capacity or K; N_k > N_e; negative attn_bw or I_attn; p, g or b
 * below 1; a capacity holding less than one block).  `out` is written only
 * on success. */
int pa_perf_model(const pa_pm_input_t *in, pa_pm_output_t *out);

#ifdef __cplusplus
}
#endif

#endif /* PA_PERF_MODEL_H */
