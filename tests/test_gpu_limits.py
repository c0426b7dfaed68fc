"""GPU parity at the edges of the launch plans: every waves-per-workgroup
choice (H_kv = 1, 2, 4, 8 and 16, i.e. W = 1, 2, 4, 8 and two head blocks),
a batch whose per-workgroup ranges reach the LDS unit-table limit (the grid
grows past three quarters of the CUs), and a batch one sequence past the
stream tables (split-K path), and batches with ranges of one unit or none.
Sizes keep the oracle to sampled sequences where they are large."""
import numpy as np
import pytest

from paper_2504_09345_amd import binding as pb
from paper_2504_09345_amd import workloads as W

from parity_util import announce, assert_parity, run_gpu, run_oracle, sub_batch

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("H_kv", [1, 2, 4, 8, 16])
def test_waves_per_workgroup_variants(H_kv):
    """W = largest power of two <= 8 dividing H_kv; H_kv = 16 makes two head
    blocks per page.  Contexts cut across ranges and single-page ones."""
    announce(f"H_kv={H_kv} variants")
    ctx = [1, 16, 17, 300, 1000, 33, 2048, 5, 700, 64] * 2
    b = W.generate("tiny", seed=40 + H_kv, overrides=dict(H_q=4 * H_kv, H_kv=H_kv, D=128,
                                                          ctx=("list", ctx), pool=("factor", 1.3)))
    ref = run_oracle(b)
    assert_parity(run_gpu(b), ref, what=f"stream H_kv={H_kv}")
    assert_parity(run_gpu(b, pages_per_split=8), ref, what=f"split H_kv={H_kv}")


@pytest.mark.slow
def test_stream_ranges_at_the_unit_table_limit():
    """8192 sequences of 800-1000 tokens with one KV head: about 460k units,
    so the grid grows to ceil(max units / 2048) workgroups and each range
    holds close to the 2048-unit table.  Sampled sequences against the
    oracle."""
    announce("unit-table limit: generate B=8192")
    b = W.generate("mixtral-256", seed=31, overrides=dict(B=8192, H_q=4, H_kv=1, D=128,
                                                          ctx=("uniform", 800, 1000)))
    units = int(((b.context_lens + 15) // 16).sum())
    u_max = 8192 * ((int(b.context_lens.max()) + 15) // 16)
    assert units > 192 * 2048 * 0.9 and u_max > 192 * 2048  # past the 3/4-CU grid
    announce(f"unit-table limit: gpu run units={units}")
    got = run_gpu(b)
    seqs = [0, 1, 2, 1000, 2047, 2048, 4095, 4096, 6000, 8000, 8190, 8191]
    sb, rows = sub_batch(b, seqs)
    assert_parity(got[rows], run_oracle(sb), what="unit-table limit")


def test_batch_past_the_stream_tables_takes_split_k():
    """8193 sequences exceed the stream-K row tables: the split-K kernel runs
    every row (pa_workspace_size plans it) and matches the oracle."""
    announce("B=8193 split-K")
    b = W.generate("mixtral-256", seed=32, overrides=dict(B=8193, H_q=8, H_kv=2, D=64,
                                                          ctx=("uniform", 1, 40)))
    dims = pb.PaDims(num_seqs=8193, num_q_heads=8, num_kv_heads=2, head_dim=64, page_size=16,
                     num_pages=int(b.k_pages.shape[0]), max_pages_per_seq=b.block_table.shape[1],
                     max_context_len=int(b.context_lens.max()), pages_per_split=0,
                     dtype=pb.PA_BF16, num_q_rows=0, max_q_len=0)
    dims_small = pb.PaDims(**{f: getattr(dims, f) for f, _ in pb.PaDims._fields_})
    dims_small.num_seqs = 8192
    # split-K planning: per-row partials, not the stream records
    assert pb.pa_workspace_size(dims) != pb.pa_workspace_size(dims_small)
    got = run_gpu(b)
    seqs = list(range(0, 8193, 431)) + [8192]
    sb, rows = sub_batch(b, seqs)
    assert_parity(got[rows], run_oracle(sb), what="B=8193")


@pytest.mark.parametrize("B,lo,hi", [(104, 33, 48), (70, 17, 32), (150, 17, 48)])
def test_ranges_of_one_unit_or_none(B, lo, hi):
    """Batches with fewer units than twice the grid (Mixtral shape, two or
    three pages per sequence): ranges of one unit, empty ranges, and items
    of two or three units cut at every range boundary, so a range's only
    unit can be the first part of a two-part item (its counter read before
    the loop) and a cut item can skip an empty range.  Every row against the
    oracle, and the same bits on a second launch."""
    announce(f"one-unit ranges B={B} ctx {lo}..{hi}")
    b = W.generate("mixtral-256", seed=B, overrides=dict(B=B, ctx=("uniform", lo, hi)))
    units = int(((b.context_lens + 15) // 16).sum())
    assert units < 2 * 208
    got = run_gpu(b)
    assert_parity(got, run_oracle(b), what=f"one-unit ranges B={B}")
    assert np.array_equal(got.view(np.uint32), run_gpu(b).view(np.uint32))
