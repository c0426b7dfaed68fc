"""Bit-exact block-table gather of the attention kernels themselves.

pa_gather_trace runs an attention call through instantiations of the same
kernels that also record, for every token they load, the pool row the tile
load's element offset points at.  That record is compared, entry by entry,
with the oracle's gather (oracle_gather_indices: token t of sequence b sits
in slot t % 16 of page block_table[b][t / 16], MoE-Lens Sec. 5.5 paging)
expanded over the KV heads (GQA, Sec. 2): for KV head g the row of the
[num_pages][H_kv][16] pool is (page * H_kv + g) * 16 + slot.  Every path is
covered: the stream-K decode kernel (unit table), the MFMA prefill kernel
(its block-table window, including a slide past 2,048 pages), the mixed
launch, and the split-K kernel (explicit split granules, fp32 chunk rows).
The traced call's output must equal the plain call's bit for bit (the same
kernels) and match the oracle."""
import functools

import numpy as np
import pytest

import oracle
from paper_2504_09345_amd import binding as pb
from paper_2504_09345_amd import workloads as W
from parity_util import announce, assert_parity, run_gpu, run_oracle, sub_batch, upload

pytestmark = pytest.mark.gpu


def expected_rows(b):
    """[H_kv][B][max_pages_per_seq * 16] int64 from the oracle's gather."""
    H, B, mp = b.num_kv_heads, b.num_seqs, b.max_pages_per_seq
    flat = oracle.gather_indices(b.block_table, b.context_lens, 16, b.num_pages)
    exp = np.full((H, B, mp * 16), -1, np.int64)
    start = 0
    for s in range(B):
        c = int(b.context_lens[s])
        rows = flat[start:start + c]
        start += c
        page, slot = rows // 16, rows % 16
        for g in range(H):
            exp[g, s, :c] = (page * H + g) * 16 + slot
    return exp


def run_trace(b, pages_per_split=0, max_context_len=None):
    import torch
    dev = upload(b)
    mcl = int(b.context_lens.max()) if max_context_len is None else max_context_len
    out = torch.empty_like(dev["q"])
    rows = torch.empty((b.num_kv_heads, b.num_seqs, b.max_pages_per_seq * 16), dtype=torch.int64,
                       device="cuda")
    if b.query_start_loc is None:
        dims = pb.make_dims(dev["q"], dev["k"], dev["bt"], mcl, pages_per_split)
        pb.pa_gather_trace(dev["q"], dev["k"], dev["v"], dev["bt"], dev["cl"], b.scale, out, dims, rows)
    else:
        dims = pb.make_dims(dev["q"], dev["k"], dev["bt"], mcl, pages_per_split,
                            num_q_rows=b.num_q_rows, max_q_len=int(b.q_lens.max()))
        pb.pa_gather_trace(dev["q"], dev["k"], dev["v"], dev["bt"], dev["cl"], b.scale, out, dims, rows,
                           query_start_loc=dev["qsl"])
    torch.cuda.synchronize()
    plain = run_gpu(b, dev=dev, pages_per_split=pages_per_split, max_context_len=mcl)
    return out.float().cpu().numpy(), rows.cpu().numpy(), plain


def check(b, what, pages_per_split=0, max_context_len=None, sample=None, strict=True):
    announce(f"gather trace {what}: B={b.num_seqs} rows={b.num_q_rows}")
    got, rows, plain = run_trace(b, pages_per_split, max_context_len)
    exp = expected_rows(b)
    bad = rows != exp
    assert not bad.any(), (what, int(bad.sum()), np.argwhere(bad)[:5].tolist())
    assert np.array_equal(got.view(np.uint32), plain.view(np.uint32)), what
    if sample is None:
        assert_parity(got, run_oracle(b), strict=strict, what=what)
    else:
        sb, r = sub_batch(b, sample)
        assert_parity(got[r], run_oracle(sb), strict=strict, what=what)


@functools.lru_cache(maxsize=1)
def _full(name, seed):
    return W.generate(name, seed=seed)


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("pps", [0, 2])
def test_trace_tiny(dtype, pps):
    check(W.generate("tiny", seed=0, dtype=dtype), f"tiny {dtype} pps={pps}", pages_per_split=pps)


@pytest.mark.parametrize("H_kv", [1, 2, 4, 8, 16])
def test_trace_every_waves_per_workgroup(H_kv):
    ctx = [1, 16, 17, 300, 1000, 33, 2048, 5, 700, 64]
    b = W.generate("tiny", seed=50 + H_kv, overrides=dict(H_q=4 * H_kv, H_kv=H_kv, D=128,
                                                          ctx=("list", ctx), pool=("factor", 1.3)))
    check(b, f"H_kv={H_kv}")


@pytest.mark.slow
@pytest.mark.parametrize("name,seed", [("mixtral-256", 1), ("long-ctx-64", 2), ("dbrx-512", 3)])
def test_trace_full_size_decode(name, seed):
    b = _full(name, seed)
    lens = b.context_lens
    sample = sorted({0, b.num_seqs - 1, int(np.argmax(lens)), int(np.argmin(lens))} |
                    set(range(1, b.num_seqs, max(1, b.num_seqs // 12))))
    check(b, name, sample=sample)


@pytest.mark.slow
def test_trace_full_size_mixed():
    b = _full("mixed", 4)
    sample = list(range(8)) + list(range(8, 520, 32))
    check(b, "mixed", sample=sample, strict=False)


def _chunks(s, seed, chunks, decode_ctx, H_kv, dtype="bf16"):
    from test_gpu_parity import _chunk_batch
    return _chunk_batch(s, seed, chunks, decode_ctx=decode_ctx, H_kv=H_kv, dtype=dtype)


@pytest.mark.parametrize("H_kv", [2, 8])
def test_trace_chunk_past_the_block_table_window(H_kv):
    """A chunk on 40,000 cached tokens: its items slide the prefill kernel's
    2,048-entry block-table window (H_kv = 2: the prefill kernel alone;
    H_kv = 8: the mixed launch)."""
    decode_ctx = [3, 500] + ([16, 900, 33, 64, 200, 1000, 7, 300] if H_kv == 8 else [])
    b = _chunks(4, 95, [(64, 40000), (40, 100)], decode_ctx, H_kv)
    check(b, f"40k chunk H_kv={H_kv}", strict=False)


def test_trace_fp32_chunks_take_split_k():
    b = _chunks(4, 96, [(40, 300), (17, 0)], [5, 700], H_kv=2, dtype="fp32")
    check(b, "fp32 chunks", strict=False)


@pytest.mark.slow
@pytest.mark.parametrize("D", [128, 64])
def test_grid_beyond_resident_workgroups(D):
    """A batch whose declared context bound needs more stream-K ranges than
    the GPU holds at once (2,048 sequences declared up to 8,192 tokens: 512
    ranges of at most 2,048 units, against one resident workgroup per CU for
    the matrix-core kernel; D = 64 declares 16,384 tokens for 1,024 ranges
    against two per CU).  Cut items are merged by whichever part finishes
    last, so the launch completes whatever the residency; trace and output
    are checked."""
    rng = np.random.default_rng(97)
    ctx = rng.integers(1, 200, 2048)
    ctx[::97] = rng.integers(1500, 2500, ctx[::97].shape[0])
    b = W.generate("mixtral-256", seed=97, overrides=dict(B=2048, D=D, ctx=("list", ctx.tolist())))
    declared = 8192 if D == 128 else 16384
    mp = declared // 16
    bt = np.full((b.num_seqs, mp), b.meta["spare_page"], np.int32)
    bt[:, :b.max_pages_per_seq] = b.block_table
    b = W.Batch(**{**b.__dict__, "block_table": bt})
    units_max = b.num_seqs * mp  # one head block of 8 KV heads
    assert -(-units_max // 2048) > 256 * (1 if D == 128 else 2)
    sample = list(range(0, 2048, 97)) + [1, 2, 3, 2047]
    check(b, f"grid beyond residency D={D}", max_context_len=declared, sample=sorted(set(sample)))
