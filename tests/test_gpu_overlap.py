"""Attention of one partition overlapped with the other partition's layer
GEMMs on a second stream (the pipelined engine of Sec. 6.4, on one GPU):
attention's output is bit-identical with and without the concurrent GEMMs,
and the overlapped output matches the oracle on partition alpha."""
import numpy as np
import pytest

import bench
from paper_2504_09345_amd import workloads as W

from parity_util import announce, assert_parity, run_oracle, sub_batch

pytestmark = pytest.mark.gpu


def test_attention_under_concurrent_gemms_matches_the_oracle():
    import torch
    announce("attention / GEMM overlap")
    b = W.generate("mixtral-256", seed=4, overrides=dict(B=48, ctx=("uniform", 64, 900)))
    to = lambda a: bench.to_device(a, torch)
    q, bt, cl, k, v = to(b.q), to(b.block_table), to(b.context_lens), to(b.k_pages), to(b.v_pages)
    res = bench._overlap_gemm(torch, b, q, k, v, bt, cl, b.scale, 3, "mixtral-256", keep_output=True)
    assert res["attn_bit_identical_under_overlap"]
    assert res["partition_alpha_seqs"] == 24
    for key in ("attn_alone_us", "gemm_alone_us", "phase_overlapped_us"):
        assert res[key] > 0
    # partition alpha = the first half of the sequences, decode attention
    sb, rows = sub_batch(b, np.arange(24))
    assert_parity(res["out_alpha"], run_oracle(sb), strict=True, what="overlapped partition alpha")
