"""Scores that grow along the context, so the kernels' lazy softmax rebase
(the running base moves only when a score exceeds it by more than 8 log2
units, Sec. 5.3's flash-attention fold) fires in the middle of an item and
more than once: K of the later pages of every sequence is scaled by 2^2 and
then 2^4 (exact in bf16), which makes the later logits 4x and 16x larger.
Decode rows (stream-K matrix-core fold, the VALU fold for fp32 and head_dim
64, split-K) and chunked-prefill rows (MFMA prefill kernel, alone and in the
mixed launch) are compared with the oracle."""
import numpy as np
import pytest

from paper_2504_09345_amd import workloads as W

from parity_util import announce, assert_parity, run_gpu, run_oracle

pytestmark = pytest.mark.gpu


def _ramp_k(b, shift_pages=None):
    """K pages of each sequence: the second third x4, the last third x16."""
    if b.dtype == "bf16":
        k = W.bf16_bits_to_f32(b.k_pages).copy()
    else:
        k = b.k_pages.copy()
    for j in range(b.num_seqs):
        n = (int(b.context_lens[j]) + 15) // 16
        if n < 3:
            continue
        pages = b.block_table[j, :n]
        k[pages[n // 3: 2 * n // 3]] *= np.float32(4.0)
        k[pages[2 * n // 3:]] *= np.float32(16.0)
    kk = W.f32_to_bf16_bits(k) if b.dtype == "bf16" else k
    return W.Batch(**{**b.__dict__, "k_pages": kk})


@pytest.mark.parametrize("dtype,D,pps", [("bf16", 128, 0), ("bf16", 128, 5), ("fp32", 64, 0), ("bf16", 64, 0)])
def test_decode_scores_growing_along_the_context(dtype, D, pps):
    announce(f"rebase decode dtype={dtype} D={D} pps={pps}")
    ctx = [3, 48, 200, 777, 1500, 2048, 16, 33, 1000, 4000]
    b = W.generate("mixtral-256", seed=61, dtype=dtype,
                   overrides=dict(D=D, ctx=("list", ctx), pool=("factor", 1.3)))
    b = _ramp_k(b)
    assert_parity(run_gpu(b, pages_per_split=pps), run_oracle(b), what=f"rebase decode {dtype} D={D} pps={pps}")


@pytest.mark.parametrize("H_kv", [2, 8])
def test_prefill_scores_growing_along_the_context(H_kv):
    """H_kv = 2: the prefill kernel alone; H_kv = 8 with enough decode rows:
    the mixed launch."""
    announce(f"rebase prefill H_kv={H_kv}")
    from test_gpu_parity import _chunk_batch
    chunks = [(96, 40), (200, 900), (64, 0), (130, 1500)]
    decode_ctx = [16, 300, 2000] + ([700] * 60 if H_kv == 8 else [])
    b = _chunk_batch(4, 62, chunks, decode_ctx=decode_ctx, H_kv=H_kv)
    b = _ramp_k(b)
    assert_parity(run_gpu(b), run_oracle(b), strict=False, what=f"rebase prefill H_kv={H_kv}")
