"""Pins of the performance-model oracle (oracle/perf_model.py) to what the
paper prints and to what its definitions imply (MoE-Lens Sec. 5):

* Sec. 5.1: 19,200 tokens saturate an A40 on Mixtral-8x7B (Eq. 2), and the
  three GPUs of Table 2;
* Sec. 5.2: with a 100 GB KV cache (763k tokens) on that A40, p = 100 and
  g = 32 reach the GPU limit while g = 64 reaches about 77 % of it (Eq. 4);
* Sec. 5.3: a KV cache twice the weights needs three times the PCIe
  bandwidth, 60 GB/s (Eq. 5);
* Eq. 3's closed form against its own sum definition, Eq. 1's exact ratio for
  the Mixtral shapes, Eq. 8 by brute force, Eq. 10's two printed forms,
  Eq. 9's comparison, Stage 2 approaching Stage 1, and a hand-worked Eq. 12-13
  example."""
import importlib.util
import math
import os

import pytest

# PERF_MODEL_ORACLE points the pins at another copy of the oracle; the mutant
# test uses it to check that mistakes planted in a copy fail these pins.
if os.environ.get("PERF_MODEL_ORACLE"):
    _spec = importlib.util.spec_from_file_location("perf_model_copy", os.environ["PERF_MODEL_ORACLE"])
    pm = importlib.util.module_from_spec(_spec)
    _spec.loader.exec_module(pm)
else:
    from oracle import perf_model as pm

T, G = 2.0 ** 40, 2.0 ** 30  # the paper's prefixes in Eq. 2
MIXTRAL = dict(N_e=8, N_k=2, h=4096, h_i=14336, s=4)
KV_PER_TOKEN = 131072  # 128 KiB over 32 layers (8 KV heads x 128 x 2 B x 2)


def test_eq2_a40_example_and_table2_tokens():
    assert pm.tokens_to_saturate(150 * T, 32 * G, 8, 2) == 19200
    for tflops, printed_k in ((150, 19.2), (181, 23.2), (312, 40.0)):
        n = pm.tokens_to_saturate(tflops * T, 32 * G, 8, 2)
        assert round(n / 1000, 1) == printed_k or abs(n / 1000 - printed_k) < 0.07


def test_eq4_sec52_example_saturates_then_77_percent():
    """100 GB KV cache = 763k tokens (decimal GB); A40, B = 32 GB/s, model
    size any (it cancels in T_max / T_GPU)."""
    M = 100e9 / KV_PER_TOKEN
    assert round(M / 1000) == 763
    n_sat = pm.tokens_to_saturate(150 * T, 32 * G, 8, 2)
    dlt = pm.delta(94e9, 32 * G)
    T_gpu = n_sat / dlt
    assert pm.t_max(100, 32, M, dlt, T_gpu) == T_gpu  # GPU-bound
    util = pm.t_max(100, 64, M, dlt, T_gpu) / T_gpu
    assert round(util, 2) == 0.77


def test_eq5_kv_twice_weights_needs_three_times_io():
    w = 94e9
    assert pm.mem_bandwidth(w + 2 * w, w, 20e9) == pytest.approx(60e9, rel=1e-12)


def test_eq3_closed_form_is_the_mean_of_its_two_sums():
    """The lifetime KV footprint sum_{j} (p + j) over g steps lies between the
    left sum (j = 0 .. g-1) and the right sum (j = 1 .. g); the closed form's
    (2p + g) g / 2 is exactly their mean, and (p + g) over it is PME."""
    for p, g in ((98, 32), (926, 128), (128, 512), (1, 1), (450, 7)):
        left = sum(p + j for j in range(g))
        right = sum(p + j for j in range(1, g + 1))
        assert (p + g) / ((left + right) / 2) == pytest.approx(pm.pme(p, g), rel=1e-15)
        assert (p + g) / right < pm.pme(p, g) < (p + g) / left


def test_eq1_exact_ratio_for_mixtral_and_the_sparsity_limit():
    r = pm.gemm_intensity_per_token(**MIXTRAL)
    # (6*2*4096*14336 + 4*4096^2 + 4096^2) / (6*8*4096*14336 + 4*4096^2 + 4096^2)
    assert r == pytest.approx(788529152 / 2902458368, rel=1e-15)
    # experts dominate: the ratio tends to N_k / N_e as h_i grows
    big = pm.gemm_intensity_per_token(8, 2, 4096, 4096 * 10 ** 6, 4)
    assert big == pytest.approx(0.25, rel=1e-6)


def test_eq8_blocks_by_brute_force():
    for p, g, b in ((98, 128, 16), (100, 32, 16), (7, 3, 4), (926, 128, 1)):
        blocks = 0
        for i in range(g + 1):
            n = p + i
            blocks += n // b + (1 if n % b else 0)
        assert pm.blocks_per_lifetime(p, g, b) == blocks
    # b = 1: the sum is (g + 1)(2p + g) / 2
    assert pm.blocks_per_lifetime(100, 32, 1) == 33 * 232 // 2


def test_eq10_two_forms_agree():
    for K, g, q, d in ((20000, 32, 350.5, 4.7), (10 ** 6, 256, 12.25, 3.0), (50, 1, 0.5, 1.0)):
        assert pm.t1(K, g, q, d) == pytest.approx(K / (K + g * q) * (g * q / d), rel=1e-12)


def test_eq9_overlap_decodes_more_sequences_in_the_papers_settings():
    """g q > N / (p + g) holds when g (g - 1) > 2p at b = 1 (expanding the
    ceiling-free sum); it holds for every setting the paper evaluates."""
    N = 10 ** 6
    for p, g in ((98, 32), (98, 64), (98, 128), (98, 256), (926, 128), (128, 512), (100, 128)):
        q = pm.prefill_per_iteration(N, p, g, 1)
        assert g * q > N / (p + g)
    q = pm.prefill_per_iteration(N, 450, 16, 1)  # g (g - 1) = 240 < 900
    assert 16 * q < N / (450 + 16)


def test_stage2_approaches_stage1():
    """As K grows and b = 1, the memory-bound token rate q (p + g) / delta
    approaches Stage 1's PME * M / delta, up to the sum's g + 1 terms."""
    p, g, M, d = 100, 128, 10 ** 6, 2.0
    q = pm.prefill_per_iteration(M, p, g, 1)
    assert q * (p + g) / d == pytest.approx(pm.pme(p, g) * M / d * g / (g + 1), rel=1e-12)
    K = 10 ** 12
    assert pm.t1(K, g, q, d) == pytest.approx(g * q / d, rel=1e-6)


def test_eq12_13_hand_worked_example():
    """T_GPU = 1200 tokens per iteration, p = 100, g = 20, K = 1220,
    delta = 0.5 s: T_prefill = 1200 * 100/120 = 1000; the prologue's g = 20
    iterations prefill (1000 + 1200)/2 * 20 = 22,000 of the K p = 122,000
    tokens; the remaining 100,000 take 100 iterations; It = 2*20 + 100 = 140;
    T2 = 1220 * 20 / (140 * 0.5) = 24,400 / 70 tokens/s."""
    assert pm.t_prefill(1200, 100, 20) == 1000
    assert pm.iterations(1220, 100, 20, 1200) == 140
    assert pm.t2(1220, 100, 20, 1200, 0.5) == pytest.approx(24400 / 70, rel=1e-15)


def test_eq7_effective_capacity():
    # p = g: (2p) / (1.5 p) = 4/3
    assert pm.kv_effective(64, 64, 70e9) == pytest.approx(70e9 * 4 / 3, rel=1e-15)
    assert pm.kv_effective(10 ** 9, 1, 1.0) == pytest.approx(1.0, rel=1e-9)


def test_evaluate_is_consistent():
    inp = dict(MIXTRAL, model_bytes=94e9, kv_bytes_per_token=KV_PER_TOKEN, C_gpu=150 * T,
               B_io=19.5e9, kv_capacity_bytes=70e9, attn_bw=0, p=98, g=128, K=20000, b=16,
               I_attn=1.0)
    o = pm.evaluate(inp)
    assert o["tokens_to_saturate"] == pytest.approx(150 * T / 19.5e9 * 4)
    assert o["t"] == min(o["t1"], o["t2"])
    assert o["t_max"] <= o["t_gpu"]
    assert o["mem_bw"] == pytest.approx(o["kv_bw"] + 19.5e9, rel=1e-12)
    assert "attn_headroom" not in o
    o2 = pm.evaluate(dict(inp, attn_bw=o["kv_bw"] / 2))
    assert o2["attn_headroom"] == pytest.approx(0.5) and o2["t_attn_bound"] == pytest.approx(o["t"] / 2)
    assert math.isfinite(o["iterations"])


def _counted_decode_attention(n_tokens, s, D, seed=0):
    """A small decode attention written out as the paper's CPU kernel does it
    (Sec. 5.3: a dot product of the query with each key, then a saxpby of the
    weighted value into the output), over bf16 K/V widened to fp32, counting
    every floating-point multiply and add of those two operations and every
    byte the kernel reads from the cache (the bf16 bytes) and computes on (the
    widened fp32 bytes).  The exp of the softmax is a per-token scalar and not
    part of the paper's intensity (dot products and saxpby only)."""
    import random
    rnd = random.Random(seed)
    K = [[rnd.uniform(-1, 1) for _ in range(D)] for _ in range(n_tokens)]
    V = [[rnd.uniform(-1, 1) for _ in range(D)] for _ in range(n_tokens)]
    flops = 0
    for _h in range(s):  # the s query heads of one GQA group share this KV head
        q = [rnd.uniform(-1, 1) for _ in range(D)]
        m, l, o = -math.inf, 0.0, [0.0] * D
        for t in range(n_tokens):
            x = 0.0
            for d in range(D):  # dot product: one multiply, one add per element
                x += q[d] * K[t][d]
                flops += 2
            m_new = max(m, x)
            a, w = math.exp(m - m_new) if m > -math.inf else 0.0, math.exp(x - m_new)
            for d in range(D):  # saxpby o = a o + w v: rescale folded into the add
                o[d] = a * o[d] + w * V[t][d]
                flops += 2
            l, m = a * l + w, m_new
    bf16_bytes = n_tokens * 2 * D * 2  # K and V, read once for the whole group
    fp32_bytes_per_query = n_tokens * 2 * D * 4  # what one query computes on
    return flops, bf16_bytes, fp32_bytes_per_query


def test_eq6_equals_the_counted_flops_of_a_decode_attention():
    """Eq. 6 (T_CPU = 2 s I B_KV) against an operation count: one query
    attending to a KV head performs 4 D FLOPs per token (dot product and
    saxpby) on 2 D fp32 values (8 D bytes once bf16 is up-converted), so
    I_cpu_attn = 1/2; the s heads of a group share the KV bytes, of which the
    cache holds 4 D bf16 bytes per token.  The FLOP rate needed to consume
    B_KV bf16 bytes per second is then the counted FLOPs per bf16 byte times
    B_KV, and Eq. 6 must give the same number."""
    for n, s, D in ((5, 4, 8), (3, 6, 16), (7, 1, 4), (2, 8, 12)):
        flops, kv_bytes, fp32_bytes = _counted_decode_attention(n, s, D)
        I_attn = (flops / s) / fp32_bytes  # one query's FLOPs per fp32 byte
        assert I_attn == 0.5
        B_kv = 40e9
        assert pm.attn_flops_required(s, I_attn, B_kv) == pytest.approx(flops / kv_bytes * B_kv, rel=1e-15)
        # s FLOPs per cached bf16 byte
        assert flops / kv_bytes == s


def test_eq6_sec53_example_is_hundreds_of_gflops():
    """Sec. 5.3: a KV cache twice the weights needs B_Mem = 3 B_IO = 60 GB/s,
    of which B_KV = 40 GB/s streams the cache; at Mixtral's s = 4 and the
    flash-attention intensity of 1/2 FLOP per fp32 byte, Eq. 6 asks for
    160 GFLOP/s, 'on the order of hundreds of GFLOPs'."""
    w, B_io = 94e9, 20e9
    B_kv = pm.mem_bandwidth(3 * w, w, B_io) - B_io
    assert B_kv == pytest.approx(40e9, rel=1e-12)
    T_cpu = pm.attn_flops_required(4, 0.5, B_kv)
    assert T_cpu == pytest.approx(160e9, rel=1e-12)
    assert 100e9 <= T_cpu < 1000e9


def test_evaluate_hand_worked_compositions():
    """evaluate() composes the equations: C_GPU = 100 TFLOP/s over
    B_IO = 25 GB/s at N_e / N_k = 4 saturates at n = 16,000 tokens (Eq. 2);
    50 GB of weights take delta = 2 s to move, so T_GPU = n / delta =
    8,000 tokens/s; a 100 GB cache read once per iteration is
    B_KV = 100 GB / 2 s = 50 GB/s, and Eq. 6 at s = 4, I = 1/2 asks for
    200 GFLOP/s; 100 GB of 128 KiB tokens are 762,939.45 tokens."""
    inp = dict(N_e=8, N_k=2, h=4096, h_i=14336, s=4, model_bytes=50e9, kv_bytes_per_token=131072,
               C_gpu=100e12, B_io=25e9, kv_capacity_bytes=100e9, attn_bw=0, p=100, g=32, K=10000,
               b=16, I_attn=0.5)
    o = pm.evaluate(inp)
    assert o["tokens_to_saturate"] == pytest.approx(16000, rel=1e-15)
    assert o["delta"] == pytest.approx(2.0, rel=1e-15)
    assert o["t_gpu"] == pytest.approx(8000, rel=1e-15)
    assert o["kv_bw"] == pytest.approx(50e9, rel=1e-15)
    assert o["attn_flops"] == pytest.approx(200e9, rel=1e-15)
    assert o["kv_tokens"] == pytest.approx(100e9 / 131072, rel=1e-15)
    assert o["kv_blocks"] == math.floor(100e9 / 131072 / 16)
    # an attention reading 25 GB/s (half of B_KV) stretches each iteration
    # to 100 GB / 25 GB/s = 4 s, halving the token rate
    o2 = pm.evaluate(dict(inp, attn_bw=25e9))
    assert o2["delta_eff"] == pytest.approx(4.0, rel=1e-15)
    assert o2["attn_headroom"] == pytest.approx(0.5, rel=1e-15)
