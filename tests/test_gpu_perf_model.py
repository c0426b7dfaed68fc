"""The performance-model calculator fed with numbers measured on the GPU
(bench.py --perf-model): the pinned host-to-device rate, the attention's own
KV read rate and the HBM capacity.  Every output of every case must equal
the oracle's (oracle/perf_model.evaluate) on the same measured inputs to
1e-12 relative (Sec. 5, Eqs. 1-14)."""
import pytest

import bench
from oracle import perf_model as pm

from parity_util import announce

pytestmark = pytest.mark.gpu


def _oracle(x):
    return pm.evaluate(dict(
        N_e=x["num_experts"], N_k=x["top_k"], h=x["model_dim"], h_i=x["expert_dim"], s=x["gqa_group"],
        model_bytes=x["model_bytes"], kv_bytes_per_token=x["kv_bytes_per_token"], C_gpu=x["gemm_flops"],
        B_io=x["io_bw"], kv_capacity_bytes=x["kv_capacity_bytes"], attn_bw=x["attn_bw"],
        p=x["prompt"], g=x["gen"], K=x["batch"], b=x["block"], I_attn=x["attn_intensity"]))


def test_perf_model_leg_matches_the_oracle_on_measured_inputs():
    import torch
    announce("perf-model leg with measured inputs")
    attn_bw = 6.4e12  # a measured attention read rate (bytes/s) of the decode kernel
    out = bench._perf_model_leg(torch, attn_bw, keep_raw=True)
    assert out["io_bw_measured_gb_s"] > 1.0
    assert len(out["raw"]) == 2
    for inp, got in out["raw"]:
        assert inp["attn_bw"] == attn_bw and inp["io_bw"] > 1e9
        ref = _oracle(inp)
        for key, val in ref.items():
            assert got[key] == pytest.approx(val, rel=1e-12, abs=0), (key, got[key], val)
        # the attention reads its cache far faster than the weight stream
        # needs it: the measured rate does not stretch the iteration
        assert got["attn_headroom"] > 1 and got["delta_eff"] == got["delta"]
