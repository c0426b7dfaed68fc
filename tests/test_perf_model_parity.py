"""The library's performance-model calculator (pa_perf_model, host code behind
the C ABI) against the oracle (oracle/perf_model.py): every output on the
paper's own configurations and on random ones, to 1e-12 relative (both are
float64; the calculator sums Eq. 8's ceilings in closed form, the oracle
term by term, and the integer sums must agree exactly), and its input
validation."""
import math

import numpy as np
import pytest

from oracle import perf_model as pm
from paper_2504_09345_amd import binding as pb

T, G = 2.0 ** 40, 2.0 ** 30
KV_PER_TOKEN = 131072


def _oracle(x):
    return pm.evaluate(dict(
        N_e=x["num_experts"], N_k=x["top_k"], h=x["model_dim"], h_i=x["expert_dim"], s=x["gqa_group"],
        model_bytes=x["model_bytes"], kv_bytes_per_token=x["kv_bytes_per_token"], C_gpu=x["gemm_flops"],
        B_io=x["io_bw"], kv_capacity_bytes=x["kv_capacity_bytes"], attn_bw=x.get("attn_bw", 0.0),
        p=x["prompt"], g=x["gen"], K=x["batch"], b=x["block"], I_attn=x["attn_intensity"]))


def _check(x):
    got = pb.pa_perf_model(**x)
    ref = _oracle(x)
    for k, v in ref.items():
        assert got[k] == pytest.approx(v, rel=1e-12, abs=0), (k, got[k], v, x)
    if "attn_headroom" not in ref:
        assert got["attn_headroom"] == 0 and got["delta_eff"] == got["delta"]
        assert got["t_attn_bound"] == got["t"]
    # Eq. 8's denominator is an integer: the two sums agree exactly
    assert round(got["kv_blocks"] / got["q"]) == pm.blocks_per_lifetime(x["prompt"], x["gen"], x["block"])
    return got


def _mixtral(**kw):
    x = dict(num_experts=8, top_k=2, model_dim=4096, expert_dim=14336, gqa_group=4, model_bytes=94e9,
             kv_bytes_per_token=KV_PER_TOKEN, gemm_flops=150 * T, io_bw=19.5e9, kv_capacity_bytes=70e9,
             attn_bw=0.0, attn_intensity=1.0, batch=20000, prompt=98, gen=32, block=16)
    x.update(kw)
    return x


@pytest.mark.parametrize("gen,cap", [(32, 70e9), (64, 70e9), (128, 70e9), (256, 70e9), (128, 210e9)])
def test_paper_configurations(gen, cap):
    """MTBench on Mixtral-8x7B with the paper's 70 GB and 210 GB KV caches and
    its measured B_IO of 19.5 GB/s (Sec. 7)."""
    _check(_mixtral(gen=gen, kv_capacity_bytes=cap))


def test_paper_printed_examples_through_the_abi():
    o = pb.pa_perf_model(**_mixtral(io_bw=32 * G, kv_capacity_bytes=100e9, prompt=100, gen=64))
    assert o["tokens_to_saturate"] == 19200
    assert round(o["t_max"] / o["t_gpu"], 2) == 0.77
    o = pb.pa_perf_model(**_mixtral(io_bw=20e9, kv_capacity_bytes=2 * 94e9))
    assert o["mem_bw"] == pytest.approx(60e9, rel=1e-12)


def test_random_configurations():
    rng = np.random.default_rng(4)
    for _ in range(300):
        N_e = int(rng.integers(1, 129))
        x = dict(num_experts=N_e, top_k=int(rng.integers(1, N_e + 1)),
                 model_dim=float(rng.integers(256, 16385)), expert_dim=float(rng.integers(256, 65537)),
                 gqa_group=float(rng.choice([1, 2, 4, 6, 8])), model_bytes=float(rng.uniform(1e9, 1e12)),
                 kv_bytes_per_token=float(rng.integers(1024, 1 << 20)),
                 gemm_flops=float(rng.uniform(1e13, 1e16)), io_bw=float(rng.uniform(1e9, 1e13)),
                 kv_capacity_bytes=float(rng.uniform(1e10, 1e12)),
                 attn_bw=float(rng.choice([0.0, rng.uniform(1e10, 1e13)])),
                 attn_intensity=float(rng.uniform(0, 4)), batch=float(rng.integers(1, 10 ** 6)),
                 prompt=int(rng.integers(1, 4096)), gen=int(rng.integers(1, 1024)),
                 block=int(rng.choice([1, 2, 16, 32, 256])))
        if x["kv_capacity_bytes"] / x["kv_bytes_per_token"] < x["block"]:
            continue
        _check(x)


def test_large_sums_stay_exact():
    """Eq. 8's closed form against the term-by-term sum at long lifetimes."""
    for p, g, b in ((1, 1, 1), (15, 1, 16), (16, 16, 16), (4095, 1023, 7), (100000, 50000, 16)):
        o = pb.pa_perf_model(**_mixtral(prompt=p, gen=g, block=b, kv_capacity_bytes=1e12))
        assert o["kv_blocks"] / o["q"] == pytest.approx(pm.blocks_per_lifetime(p, g, b), rel=1e-15)


@pytest.mark.parametrize("field,val", [("num_experts", 0), ("top_k", 9), ("top_k", 0), ("model_dim", -1),
                                       ("gqa_group", 0), ("model_bytes", 0), ("io_bw", 0), ("batch", 0),
                                       ("attn_bw", -1), ("attn_intensity", -1), ("prompt", 0), ("gen", 0),
                                       ("block", 0), ("kv_capacity_bytes", 1000.0),
                                       ("gemm_flops", math.nan)])
def test_rejects_out_of_range_inputs(field, val):
    with pytest.raises(pb.PagedAttnError):
        pb.pa_perf_model(**_mixtral(**{field: val}))


def test_null_pointers_rejected():
    lib = pb.load()
    assert lib.pa_perf_model(None, None) == pb.PA_EINVAL
