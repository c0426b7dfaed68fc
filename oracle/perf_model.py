"""Oracle of the MoE-Lens performance model (arXiv 2504.09345, Sec. 5).

TEST INFRASTRUCTURE ONLY: plain float64 Python, one function per equation,
written from the paper's definitions; only the test suite and the
benchmark's CPU-baseline leg use it.  The library's calculator is separate
code and is compared with this one.

Units are SI (FLOP/s, bytes, bytes/s, seconds, tokens).  The paper's worked
numbers use binary prefixes for TFLOPS and GB/s in Eq. 2 (150 TFLOPS over
32 GB/s gives its 19,200 tokens only as 150 * 2^40 / (32 * 2^30) * 4); the
tests pass the paper's inputs in whatever unit reproduces its printed value.
"""
from __future__ import annotations

import math


def gemm_intensity_per_token(N_e, N_k, h, h_i, s):
    """Eq. 1 without the factor n: GEMM FLOPs per weight byte per token,
    (6 N_k h h_i + 4 h^2 + 4 h^2 / s) / (6 N_e h h_i + 4 h^2 + 4 h^2 / s)."""
    att = 4.0 * h * h + 4.0 * h * h / s
    return (6.0 * N_k * h * h_i + att) / (6.0 * N_e * h * h_i + att)


def tokens_to_saturate(C_gpu, B_io, N_e, N_k):
    """Eq. 2: the tokens in flight that make the GEMMs compute-bound,
    n >= C_GPU / B * N_e / N_k (the sparsity approximation of Eq. 1)."""
    return C_gpu / B_io * N_e / N_k


def pme(p, g):
    """Eq. 3: parallelism-memory efficiency 2 (p + g) / ((2p + g) g)."""
    return 2.0 * (p + g) / ((2.0 * p + g) * g)


def delta(model_bytes, B_io):
    """Time to move the weights once: model size / B_IO (Sec. 5.2)."""
    return model_bytes / B_io


def t_max(p, g, M_tokens, dlt, T_gpu):
    """Eq. 4: min(PME * M / delta, T_GPU), tokens per second."""
    return min(pme(p, g) * M_tokens / dlt, T_gpu)


def mem_bandwidth(M_total_bytes, M_weight_bytes, B_io):
    """Eq. 5: B_Mem = B_KV + B_IO = M / M_weight * B_IO, with M the memory
    holding weights and KV cache together."""
    return M_total_bytes / M_weight_bytes * B_io


def attn_flops_required(s, I_attn, B_kv):
    """Eq. 6: T_CPU = 2 s I_attn B_KV."""
    return 2.0 * s * I_attn * B_kv


def kv_effective(p, g, C_kv):
    """Eq. 7: (p + g) / (p + g/2) * C_KV."""
    return (p + g) / (p + g / 2.0) * C_kv


def blocks_per_lifetime(p, g, b):
    """Denominator of Eq. 8: sum over i = 0 .. g of ceil((p + i) / b)."""
    return sum(-(-(p + i) // b) for i in range(g + 1))


def prefill_per_iteration(N_blocks, p, g, b):
    """Eq. 8: q = N / sum_{i=0}^{g} ceil((p + i) / b)."""
    return N_blocks / blocks_per_lifetime(p, g, b)


def t1(K, g, q, dlt):
    """Eq. 10: K g / ((K / q + g) delta), generated tokens per second when
    the KV capacity bounds the pipeline."""
    return K * g / ((K / q + g) * dlt)


def t_prefill(T_gpu_iter, p, g):
    """Eq. 11: prefill tokens per iteration in the pipeline's main stages,
    T_GPU p / (p + g)."""
    return T_gpu_iter * p / (p + g)


def iterations(K, p, g, T_gpu_iter):
    """Eq. 12: 2 g + (K p - (T_prefill + T_GPU) / 2 * g) / T_prefill."""
    tp = t_prefill(T_gpu_iter, p, g)
    return 2.0 * g + (K * p - (tp + T_gpu_iter) / 2.0 * g) / tp


def t2(K, p, g, T_gpu_iter, dlt):
    """Eq. 13: K g / (It delta) when GPU compute bounds the pipeline."""
    return K * g / (iterations(K, p, g, T_gpu_iter) * dlt)


def stage2(K, p, g, b, N_blocks, T_gpu_iter, dlt):
    """Eqs. 8-14: (q, g q, T1, T2, T = min(T1, T2))."""
    q = prefill_per_iteration(N_blocks, p, g, b)
    a = t1(K, g, q, dlt)
    c = t2(K, p, g, T_gpu_iter, dlt)
    return q, g * q, a, c, min(a, c)


def evaluate(inp: dict) -> dict:
    """Every quantity of Sec. 5 for one configuration (the calculator's
    contract).  Keys of `inp`: N_e, N_k, h, h_i, s, model_bytes,
    kv_bytes_per_token, C_gpu, B_io, kv_capacity_bytes, attn_bw (0: not
    given), p, g, K, b, I_attn."""
    n_sat = tokens_to_saturate(inp["C_gpu"], inp["B_io"], inp["N_e"], inp["N_k"])
    dlt = delta(inp["model_bytes"], inp["B_io"])
    M_tok = inp["kv_capacity_bytes"] / inp["kv_bytes_per_token"]
    T_gpu = n_sat / dlt
    p, g, b = int(inp["p"]), int(inp["g"]), int(inp["b"])
    N_blocks = math.floor(M_tok / b)
    q, gq, a1, a2, t = stage2(inp["K"], p, g, b, N_blocks, n_sat, dlt)
    B_kv = inp["kv_capacity_bytes"] / dlt
    out = dict(
        intensity_per_token=gemm_intensity_per_token(inp["N_e"], inp["N_k"], inp["h"], inp["h_i"], inp["s"]),
        tokens_to_saturate=n_sat, pme=pme(p, g), delta=dlt, kv_tokens=M_tok, t_gpu=T_gpu,
        t_max=t_max(p, g, M_tok, dlt, T_gpu),
        mem_bw=mem_bandwidth(inp["model_bytes"] + inp["kv_capacity_bytes"], inp["model_bytes"], inp["B_io"]),
        kv_bw=B_kv, attn_flops=attn_flops_required(inp["s"], inp["I_attn"], B_kv),
        kv_effective=kv_effective(p, g, inp["kv_capacity_bytes"]), kv_blocks=N_blocks,
        q=q, decode_seqs=gq, t1=a1, t_prefill=t_prefill(n_sat, p, g),
        iterations=iterations(inp["K"], p, g, n_sat), t2=a2, t=t)
    # Sec. 5.3's condition made explicit: attention must read the whole KV
    # cache once per iteration (B_KV); a measured attention bandwidth below it
    # stretches the iteration from delta to capacity / attn_bw.
    if inp.get("attn_bw", 0) > 0:
        d_eff = max(dlt, inp["kv_capacity_bytes"] / inp["attn_bw"])
        out["attn_headroom"] = inp["attn_bw"] / B_kv
        out["delta_eff"] = d_eff
        out["t_attn_bound"] = t * dlt / d_eff
    return out
