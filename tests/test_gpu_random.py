"""Seeded random sweep of the attention calls against the oracle: each case
draws a shape (KV heads, group size, head dim, dtype), a context mix (empty,
one-token, page-boundary and long contexts), a launch path (stream-K or an
explicit split granule) and, for varlen cases, chunk lengths, and runs the
whole batch through the library and the oracle; a second set draws larger
batches.  The draws are fixed by the case number, so a failing case names a
reproducible batch."""
import numpy as np
import pytest

from paper_2504_09345_amd import workloads as W

from parity_util import announce, assert_parity, run_gpu, run_oracle

pytestmark = pytest.mark.gpu

EDGE_CTX = [0, 1, 2, 15, 16, 17, 31, 32, 33, 255, 256, 257]


def _draw(case):
    rng = np.random.default_rng(1000 + case)
    H_kv = int(rng.choice([1, 2, 4, 8]))
    s = int(rng.choice([1, 2, 4, 6, 8]))
    D = int(rng.choice([64, 128]))
    dtype = "bf16" if rng.random() < 0.75 else "fp32"
    B = int(rng.integers(1, 40))
    ctx = [int(rng.choice(EDGE_CTX)) if rng.random() < 0.4 else int(rng.integers(1, 3000)) for _ in range(B)]
    pps = int(rng.choice([0, 0, 0, 1, 7]))
    varlen = rng.random() < 0.35
    return H_kv, s, D, dtype, ctx, pps, varlen, rng


@pytest.mark.parametrize("case", range(24))
def test_random_batch(case):
    H_kv, s, D, dtype, ctx, pps, varlen, rng = _draw(case)
    announce(f"random case {case}: H_kv={H_kv} s={s} D={D} {dtype} B={len(ctx)} pps={pps} varlen={varlen}")
    if not varlen:
        b = W.generate("tiny", seed=2000 + case, dtype=dtype,
                       overrides=dict(H_q=s * H_kv, H_kv=H_kv, D=D, ctx=("list", ctx), pool=("factor", 1.3)))
    else:
        n_pre = int(rng.integers(1, 4))
        chunk = int(rng.integers(2, 300))
        b = W.generate("mixed", seed=2000 + case, dtype=dtype,
                       overrides=dict(H_q=s * H_kv, H_kv=H_kv, D=D, prefill=(n_pre, chunk, 0, 700),
                                      decode=(int(rng.integers(0, 20)), 1, 2500), pool=("factor", 1.3)))
    got = run_gpu(b, pages_per_split=pps)
    # varlen rows of fp32 or D = 64 chunks take the per-row kernel; the MFMA
    # prefill rows round P and V to fp16 (the strict floor is for decode only)
    assert_parity(got, run_oracle(b), strict=not varlen, what=f"case {case}")


def _draw_large(case):
    rng = np.random.default_rng(5000 + case)
    H_kv = int(rng.choice([1, 2, 8]))
    s = int(rng.choice([1, 4, 6, 8]))
    varlen = rng.random() < 0.5
    pps = int(rng.choice([0, 0, 0, 16]))
    return H_kv, s, varlen, pps, rng


@pytest.mark.parametrize("case", range(16))
def test_random_large_batch(case):
    """Larger seeded shapes (bf16, head_dim 128): up to 120 sequences with a
    fifth of the contexts up to 20k tokens, or up to 4 chunks of up to 1,500
    rows on up to 3,000 cached tokens beside up to 60 decode rows, so items
    cut across many stream ranges and chunks span several prefill items."""
    H_kv, s, varlen, pps, rng = _draw_large(case)
    if not varlen:
        B = int(rng.integers(1, 120))
        ctx = [int(rng.integers(1, 20000)) if rng.random() < 0.2 else int(rng.integers(1, 3000)) for _ in range(B)]
        b = W.generate("tiny", seed=6000 + case, overrides=dict(H_q=s * H_kv, H_kv=H_kv, D=128,
                                                               ctx=("list", ctx), pool=("factor", 1.2)))
    else:
        n_pre, chunk = int(rng.integers(1, 5)), int(rng.integers(2, 1500))
        b = W.generate("mixed", seed=6000 + case,
                       overrides=dict(H_q=s * H_kv, H_kv=H_kv, D=128, prefill=(n_pre, chunk, 0, 3000),
                                      decode=(int(rng.integers(0, 60)), 1, 6000), pool=("factor", 1.2)))
    announce(f"large random case {case}: H_kv={H_kv} s={s} B={b.num_seqs} rows={b.num_q_rows} pps={pps}")
    assert_parity(run_gpu(b, pages_per_split=pps), run_oracle(b), strict=not varlen, what=f"large case {case}")
