"""GPU parity: the HIP path through the C ABI against the CPU oracle on the
same seeded inputs, element by element, plus the structural checks (bit-exact
block-table gather, split-size invariance, determinism, poisoned pools, edge
cases).  Full-size workloads are checked on sampled sequences in the launch
configuration the benchmark times.  The kernels' own block-table gather is
checked bit for bit in test_gpu_gather.py."""
import functools

import numpy as np
import pytest

import oracle
from paper_2504_09345_amd import binding as pb
from paper_2504_09345_amd import workloads as W
from parity_util import (announce, assert_parity, parity_stats, run_gpu, run_oracle, sub_batch,
                         upload)

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    return torch


# --- tiny and small shapes -------------------------------------------------

@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("pps", [0, 1, 3])
def test_tiny_decode(dtype, pps):
    announce(f"tiny decode dtype={dtype} pages_per_split={pps}")
    b = W.generate("tiny", seed=0, dtype=dtype)
    got = run_gpu(b, pages_per_split=pps)
    assert_parity(got, run_oracle(b), what=f"tiny {dtype} pps={pps}")


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_tiny_poisoned_pool(dtype):
    announce(f"tiny poison dtype={dtype}")
    b = W.generate("tiny", seed=1, dtype=dtype, poison=True)
    for pps in (0, 2):
        got = run_gpu(b, pages_per_split=pps)
        assert_parity(got, run_oracle(b), what=f"poison pps={pps}")


def test_fp32_inputs_match_tightly():
    # with fp32 inputs and output only accumulation order differs
    announce("tiny fp32 tight")
    b = W.generate("tiny", seed=2, dtype="fp32")
    st = parity_stats(run_gpu(b), run_oracle(b))
    assert st["max_rel_global"] < 2e-5, st


@pytest.mark.parametrize("s", [1, 2, 4, 6, 8])
@pytest.mark.parametrize("D", [64, 128])
def test_group_sizes_and_head_dims(s, D):
    announce(f"edge contexts s={s} D={D}")
    ctx = [1, 2, 15, 16, 17, 31, 32, 33, 100, 255, 256, 257, 511, 512, 513, 1000]
    b = W.generate("tiny", seed=3 + s, overrides=dict(H_q=2 * s, H_kv=2, D=D,
                                                      ctx=("list", ctx), pool=("factor", 1.5)))
    ref = run_oracle(b)
    for pps in (0, 1, 5):
        assert_parity(run_gpu(b, pages_per_split=pps), ref, what=f"s={s} D={D} pps={pps}")


def test_split_size_invariance():
    announce("split invariance fp32 long contexts")
    b = W.generate("tiny", seed=7, dtype="fp32",
                   overrides=dict(ctx=("list", [3000, 777, 4096, 1, 2049]), pool=("factor", 1.3)))
    outs = {pps: run_gpu(b, pages_per_split=pps) for pps in (1, 3, 32, 256)}
    base = outs[256]
    scale = np.abs(base).max()
    for pps, o in outs.items():
        assert np.abs(o - base).max() <= 1e-5 * scale, pps
    assert_parity(base, run_oracle(b))


def test_one_token_context_returns_v_exactly():
    torch = _torch()
    for dtype in ("bf16", "fp32"):
        announce(f"ctx=1 exact dtype={dtype}")
        b = W.generate("tiny", seed=8, dtype=dtype)
        b.context_lens[:] = 1
        got = run_gpu(b, max_context_len=200)
        s = b.num_q_heads // b.num_kv_heads
        for i in range(b.num_seqs):
            page = b.block_table[i, 0]
            for h in range(b.num_q_heads):
                v0 = b.v_pages[page, h // s, 0]
                v0 = W.bf16_bits_to_f32(v0) if dtype == "bf16" else v0
                assert np.array_equal(got[i, h], v0)


def test_empty_context_gives_zeros_and_determinism():
    announce("ctx=0 zeros, determinism")
    b = W.generate("tiny", seed=9)
    b.context_lens[2] = 0
    a1 = run_gpu(b, pages_per_split=2, max_context_len=200)
    a2 = run_gpu(b, pages_per_split=2, max_context_len=200)
    assert np.all(a1[2] == 0)
    assert np.array_equal(a1.view(np.uint32), a2.view(np.uint32))
    assert_parity(a1, run_oracle(b))


def test_batch_independence():
    announce("batch independence")
    b = W.generate("tiny", seed=10, overrides=dict(ctx=("list", [50, 300, 7, 1024])))
    full = run_gpu(b, max_context_len=1024)
    for i in range(b.num_seqs):
        sb, _ = sub_batch(b, [i])
        alone = run_gpu(sb, max_context_len=1024)
        assert np.array_equal(alone[0].view(np.uint32), full[i].view(np.uint32))


def test_context_beyond_declared_bound_is_flagged():
    # a context longer than max_context_len breaks the contract: the library
    # reports NaN for that sequence instead of reading past the block-table row
    announce("contract violation -> NaN")
    b = W.generate("tiny", seed=11)
    got = run_gpu(b, max_context_len=150)  # ctx 200 > 150 (table row holds 13 pages)
    assert np.isnan(got[3]).all()
    assert_parity(got[:3], run_oracle(b)[:3])


# --- varlen: causal prefill chunks sharing the launch with decode rows ------

@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_varlen_small(dtype):
    announce(f"varlen small dtype={dtype}")
    b = W.generate("mixed", seed=3, dtype=dtype,
                   overrides=dict(prefill=(3, 40, 0, 70), decode=(6, 1, 300), pool=("factor", 1.5)))
    ref = run_oracle(b)
    for pps in (0, 1, 4):
        assert_parity(run_gpu(b, pages_per_split=pps), ref, strict=False, what=f"pps={pps}")


def test_varlen_single_rows_equal_decode():
    announce("varlen L=1 equals decode")
    b = W.generate("tiny", seed=12, overrides=dict(ctx=("list", [33, 100, 1, 640])))
    dec = run_gpu(b)
    vb = W.Batch(**{**b.__dict__, "query_start_loc": np.arange(b.num_seqs + 1, dtype=np.int32)})
    var = run_gpu(vb)
    assert np.array_equal(dec.view(np.uint32), var.view(np.uint32))


# --- full-size workloads ---------------------------------------------------

@functools.lru_cache(maxsize=1)
def _full(name, seed):
    return W.generate(name, seed=seed)


@pytest.mark.slow
@pytest.mark.parametrize("name,seed", [("mixtral-256", 1), ("long-ctx-64", 2), ("dbrx-512", 3)])
def test_full_size_decode(name, seed):
    """The benchmark's decode batches at full size, every sequence against the
    oracle (the oracle streams these batches in well under a second)."""
    announce(f"full {name} seed={seed}: generate")
    b = _full(name, seed)
    announce(f"full {name}: gpu run B={b.num_seqs} max_ctx={int(b.context_lens.max())}")
    got = run_gpu(b)
    assert_parity(got, run_oracle(b), what=name)


@pytest.mark.slow
def test_full_size_mixed():
    """The mixed launch at full size: all 8 prefill chunks (4,096 rows) and all
    512 decode rows against the oracle."""
    announce("full mixed seed=4: generate")
    b = _full("mixed", 4)
    announce(f"full mixed: gpu run rows={b.num_q_rows}")
    got = run_gpu(b)
    assert_parity(got, run_oracle(b), strict=False, what="mixed")


@pytest.mark.slow
def test_full_size_prefill_alone():
    """The 8 chunks of the mixed workload without decode rows, as the
    benchmark's prefill workload times them: the chunked-prefill kernel alone
    on every CU.  All 4,096 rows are compared."""
    announce("full prefill-8x512 seed=1: generate")
    b = _full("prefill-8x512", 1)
    assert b.num_seqs == 8 and int(b.q_lens.min()) > 1  # no decode row: the prefill kernel alone
    announce(f"full prefill-8x512: gpu run rows={b.num_q_rows}")
    got = run_gpu(b)
    ref = run_oracle(b)
    assert_parity(got, ref, strict=False, what="prefill-8x512")


@pytest.mark.slow
def test_full_size_prefill_heavy_sampled():
    """16 chunks of 2,048 rows on 2,048-4,096 tokens, as the benchmark's
    prefill-heavy workload times them (the chunked-prefill kernel alone, 16
    items per workgroup): the shortest, the longest and two more
    sequences, every row of each (8,192 rows), against the oracle."""
    announce("full prefill-16x2048 seed=1: generate")
    b = _full("prefill-16x2048", 1)
    assert b.num_seqs == 16 and int(b.q_lens.min()) == 2048
    announce(f"full prefill-16x2048: gpu run rows={b.num_q_rows}")
    got = run_gpu(b)
    lens = b.context_lens
    seqs = sorted({int(np.argmin(lens)), int(np.argmax(lens)), 0, 9})
    sb, rows = sub_batch(b, seqs)
    assert_parity(got[rows], run_oracle(sb), strict=False, what="prefill-16x2048")


@pytest.mark.slow
@pytest.mark.parametrize("name,seed", [("mixtral-256", 1), ("dbrx-512", 3)])
def test_full_size_decode_repeats_bit_identically(name, seed):
    """An item cut by a range boundary is merged by whichever of its parts
    finishes last: the range's end part from its registers when the other
    part has already counted, otherwise the last part to count, from the
    stored records, with the same operations in the same order.  Which part
    merges depends on timing, so repeated launches of the full batch must
    give the same bits."""
    announce(f"full {name} seed={seed}: repeated launches")
    b = _full(name, seed)
    dev = upload(b)
    first = run_gpu(b, dev=dev)
    for i in range(16):
        again = run_gpu(b, dev=dev)
        assert np.array_equal(first.view(np.uint32), again.view(np.uint32)), (name, i)


# --- stream-K vs split-K ----------------------------------------------------

@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("s", [4, 6])
def test_stream_and_split_paths_agree(dtype, s):
    announce(f"stream vs split dtype={dtype} s={s}")
    b = W.generate("dbrx-512", seed=21, dtype=dtype,
                   overrides=dict(B=48, H_q=8 * s, ctx=("lognormal", 300, 1.2, 1, 3000)))
    stream = run_gpu(b)                       # library choice: stream-K
    split = run_gpu(b, pages_per_split=16)    # per-row split-K
    scale = np.abs(split).max()
    if dtype == "fp32":
        assert np.abs(stream - split).max() <= 1e-5 * scale
    sb, rows = sub_batch(b, list(range(0, 48, 3)))
    ref = run_oracle(sb)
    assert_parity(stream[rows], ref, what="stream")
    assert_parity(split[rows], ref, what="split")


def test_stream_handles_more_workgroups_than_pages():
    # a few one-page sequences: most persistent workgroups get no units and
    # items are cut into single units spread over many ranges
    announce("stream tiny batch")
    b = W.generate("tiny", seed=22, overrides=dict(H_q=32, H_kv=8, D=128,
                                                   ctx=("list", [1, 5, 16, 17, 40, 3])))
    assert_parity(run_gpu(b), run_oracle(b))


# --- MFMA chunked prefill ---------------------------------------------------

def _chunk_batch(s, seed, chunks, decode_ctx, dtype="bf16", poison=False, H_kv=2):
    """Sequences with (chunk length L, prior cached tokens) plus decode rows,
    interleaved, identity-free random page placement."""
    rng = np.random.default_rng(seed)
    seqs = [(L, prior) for L, prior in chunks] + [(1, c - 1) for c in decode_ctx]
    order = rng.permutation(len(seqs))
    seqs = [seqs[i] for i in order]
    ctx = [L + prior for L, prior in seqs]
    qlen = [L for L, _ in seqs]
    b = W.generate("tiny", seed=seed, dtype=dtype, poison=poison,
                   overrides=dict(H_q=H_kv * s, H_kv=H_kv, D=128, ctx=("list", ctx), pool=("factor", 1.4)))
    # re-draw q with one row per query position
    T = int(sum(qlen))
    q = W._fill_normal((T, H_kv * s, 128), seed + 1, "q", 1.0, dtype, 1)
    qsl = np.zeros(len(seqs) + 1, np.int32)
    qsl[1:] = np.cumsum(qlen)
    return W.Batch(**{**b.__dict__, "q": q, "query_start_loc": qsl})


@pytest.mark.parametrize("s", [1, 2, 4, 6, 8])
def test_prefill_chunks_mfma(s):
    announce(f"prefill chunks s={s}")
    chunks = [(2, 0), (17, 5), (32, 0), (33, 100), (100, 0), (64, 1000), (200, 37), (130, 700)]
    b = _chunk_batch(s, 30 + s, chunks, decode_ctx=[1, 16, 300, 2000])
    got = run_gpu(b)
    ref = run_oracle(b)
    assert_parity(got, ref, strict=False, what=f"prefill s={s}")


@pytest.mark.parametrize("s", [1, 2, 4, 6, 8])
def test_mixed_batch_one_launch(s):
    """8 KV heads and enough decode rows: decode rows and prefill chunks run as
    the two halves of one mixed launch (decode and prefill workgroups side by
    side; chunk rows x s <= 40 x sequences)."""
    announce(f"mixed one launch s={s}")
    chunks = [(17, 5), (100, 0), (64, 600), (130, 300), (2, 40)]
    rng = np.random.default_rng(70 + s)
    decode_ctx = [1, 16, 300, 2000, 777, 64] + rng.integers(1, 1500, 58).tolist()
    assert (sum(L for L, _ in chunks) - len(chunks)) * s <= 40 * (len(chunks) + len(decode_ctx))
    b = _chunk_batch(s, 60 + s, chunks, decode_ctx=decode_ctx, H_kv=8)
    got = run_gpu(b)
    assert_parity(got, run_oracle(b), strict=False, what=f"mixed s={s}")
    assert np.array_equal(got.view(np.uint32), run_gpu(b).view(np.uint32))


def test_prefill_heavy_batch_runs_kernels_in_turn():
    """Chunk rows outweigh the decode rows: stream-K then prefill on all CUs."""
    announce("prefill-heavy batch")
    chunks = [(300, 100), (250, 0), (400, 20)]
    b = _chunk_batch(4, 80, chunks, decode_ctx=[5, 900], H_kv=8)
    assert (sum(L for L, _ in chunks) - len(chunks)) * 4 > 40 * (len(chunks) + 2)
    assert_parity(run_gpu(b), run_oracle(b), strict=False, what="prefill-heavy")


@pytest.mark.parametrize("lens", [(64, 64, 64, 64, 64), (64, 40, 64, 2, 64)])
def test_prefill_only_batches(lens):
    """Chunks and no decode row.  Equal chunk lengths (the rows add up to
    num_seqs x max_q_len) let the host skip the stream-K launch; unequal ones
    launch it and it finds no work.  Both match the oracle."""
    announce(f"prefill-only batch {lens}")
    priors = [0, 700, 33, 1500, 16]
    b = _chunk_batch(4, 85, list(zip(lens, priors)), decode_ctx=[], H_kv=8)
    assert (b.q_lens > 1).all()
    assert_parity(run_gpu(b), run_oracle(b), strict=False, what=f"prefill-only {lens}")


def test_prefill_poisoned_pool():
    announce("prefill poison")
    b = _chunk_batch(4, 40, [(48, 7), (96, 300), (31, 0)], decode_ctx=[33, 500], poison=True)
    got = run_gpu(b)
    assert np.isfinite(got).all()
    assert_parity(got, run_oracle(b), strict=False)


def _scale_v(b, seqs, factor):
    """V pages of sequences `seqs` times a power of two (exact in bf16)."""
    v = W.bf16_bits_to_f32(b.v_pages).copy()
    for j in seqs:
        v[b.block_table[j, :(int(b.context_lens[j]) + 15) // 16]] *= np.float32(factor)
    return W.Batch(**{**b.__dict__, "v_pages": W.f32_to_bf16_bits(v)})


@pytest.mark.parametrize("H_kv", [2, 8])
@pytest.mark.parametrize("log2_factor", [17, 40, -6, -12, -24, -60])
def test_prefill_value_range(H_kv, log2_factor):
    """Chunk rows whose V is far from unit scale.  Magnitudes of 2^16 and up
    do not fit fp16, and V below 2^-17 is not exact in it; either way the
    chunk must still match the oracle in relative terms (the absolute bound
    is meaningless for scaled values), and the other rows of the batch must
    stay within the full tolerance.  H_kv = 8 runs the chunks in the mixed
    decode + prefill launch."""
    announce(f"prefill V range 2^{log2_factor} H_kv={H_kv}")
    chunks = [(96, 40), (130, 300), (64, 0), (33, 700)]
    decode_ctx = [1, 16, 300, 2000] + ([700] * 60 if H_kv == 8 else [])
    b = _chunk_batch(4, 90 + log2_factor % 17, chunks, decode_ctx=decode_ctx, H_kv=H_kv)
    chunk_seqs = [j for j in range(b.num_seqs) if b.q_lens[j] > 1]
    scaled = chunk_seqs[::2]  # every other chunk sequence
    b = _scale_v(b, scaled, 2.0 ** log2_factor)
    _assert_scaled_parity(b, scaled, f"2^{log2_factor}")


@pytest.mark.parametrize("value", ["nan", "inf"])
def test_prefill_nonfinite_v(value):
    """A NaN or infinity in one V element that chunk rows attend to: the item
    takes the bf16 pass; the rows that see that key are non-finite exactly
    where the oracle's are, and every row outside the key's work item
    matches the oracle.  Rows of that item before the key are left open:
    their zero weight meets the value inside the matrix product (0 x inf is
    NaN), where the oracle never visits a masked key."""
    announce(f"prefill V {value}")
    b = _chunk_batch(4, 88, [(96, 40), (130, 300), (64, 0)], decode_ctx=[16, 300], H_kv=8)
    seqs = [j for j in range(b.num_seqs) if b.q_lens[j] > 1]
    j = seqs[1]
    C, L = int(b.context_lens[j]), int(b.q_lens[j])
    r_key = 20
    t = C - L + r_key  # key of chunk row 20: rows 20.. see it
    v = b.v_pages.copy()
    v[b.block_table[j, t // 16], 1, t % 16, 5] = W.BF16_NAN if value == "nan" else np.uint16(0x7F80)
    b = W.Batch(**{**b.__dict__, "v_pages": v})
    got, ref = run_gpu(b), run_oracle(b)
    q0 = int(b.query_start_loc[j])
    # rows before the key in its work item (64 positions at s = 4), which
    # runs the key's step for all of its rows
    open_rows = np.zeros(got.shape[0], bool)
    open_rows[q0:q0 + r_key] = True
    sees = np.zeros(got.shape[0], bool)
    sees[q0 + r_key:q0 + L] = True
    assert (~np.isfinite(ref[sees])).any()
    assert np.array_equal(~np.isfinite(got[sees]), ~np.isfinite(ref[sees]))
    fin = np.isfinite(ref[sees])
    st = parity_stats(np.where(fin, got[sees], 0), np.where(fin, ref[sees], 0))
    assert st["max_abs"] <= 1e-2 and st["max_rel"] <= 5e-3, st
    rest = ~(sees | open_rows)
    assert_parity(got[rest], ref[rest], strict=False, what=f"rows away from the {value}")


@pytest.mark.parametrize("H_kv", [2, 8])
@pytest.mark.parametrize("log2_factor", [0, 17])
def test_prefill_past_the_block_table_window(log2_factor, H_kv):
    """A chunk on 40,000 cached tokens (2,505 pages): the workgroup's window of
    2,048 block-table entries slides during the item; with V past the fp16
    range the item's bf16 pass starts again from the first window.  H_kv = 8
    with ten decode rows runs the chunks in the mixed launch."""
    announce(f"prefill 40k context, V x 2^{log2_factor}, H_kv={H_kv}")
    decode_ctx = [3, 500] + ([16, 900, 33, 64, 200, 1000, 7, 300] if H_kv == 8 else [])
    b = _chunk_batch(4, 95, [(64, 40000), (40, 100)], decode_ctx=decode_ctx, H_kv=H_kv)
    long_seq = [j for j in range(b.num_seqs) if b.context_lens[j] > 40000]
    assert len(long_seq) == 1 and (int(b.context_lens[long_seq[0]]) + 15) // 16 > 2048
    scaled = long_seq if log2_factor else []
    if scaled:
        b = _scale_v(b, scaled, 2.0 ** log2_factor)
    _assert_scaled_parity(b, scaled, f"40k context, 2^{log2_factor}")


def _assert_scaled_parity(b, scaled, what):
    """Rows of the `scaled` sequences: relative bound only; the rest: the
    full tolerance."""
    got, ref = run_gpu(b), run_oracle(b)
    qsl = b.query_start_loc
    rows = np.zeros(got.shape[0], bool)
    for j in scaled:
        rows[qsl[j]:qsl[j + 1]] = True
    if rows.any():
        st = parity_stats(got[rows], ref[rows])
        assert st["finite"] and st["max_rel"] <= 5e-3, (what, st)
    assert_parity(got[~rows], ref[~rows], strict=False, what=f"unscaled rows, {what}")


def test_prefill_determinism_and_single_rows_match_decode():
    announce("prefill determinism")
    b = _chunk_batch(4, 41, [(64, 200), (7, 3)], decode_ctx=[100, 900])
    a1, a2 = run_gpu(b), run_gpu(b)
    assert np.array_equal(a1.view(np.uint32), a2.view(np.uint32))
