"""Seeded input generator: determinism, bf16 rounding, layout invariants."""
import numpy as np
import pytest
import torch

from paper_2504_09345_amd import workloads as W


def test_bf16_rounding_matches_torch():
    # torch's float32 -> bfloat16 cast rounds to nearest even: a library pin
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32) * 10.0 ** rng.integers(-6, 6, 100000),
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 3.4e38, -1e-40], np.float32)])
    ours = W.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    back = W.bf16_bits_to_f32(ours)
    assert np.array_equal(back, torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_same_seed_same_bytes_any_thread_count():
    a = W.generate("tiny", seed=5, threads=1)
    b = W.generate("tiny", seed=5, threads=4)
    for f in ("q", "k_pages", "v_pages", "block_table", "context_lens"):
        assert np.array_equal(getattr(a, f), getattr(b, f))
    c = W.generate("tiny", seed=6)
    assert not np.array_equal(a.k_pages, c.k_pages)


def test_tiny_matches_its_description():
    b = W.generate("tiny", seed=0)
    assert list(b.context_lens) == [17, 64, 129, 200]
    assert b.num_pages == 64 and b.num_q_heads == 8 and b.num_kv_heads == 2 and b.head_dim == 64
    assert b.scale == 1.0 / 8.0
    used = np.concatenate([b.block_table[i, : (c + 15) // 16] for i, c in enumerate(b.context_lens)])
    assert len(np.unique(used)) == len(used) == 28  # disjoint pages
    assert used.min() >= 0 and used.max() < 64


@pytest.mark.parametrize("name", ["mixtral-256", "long-ctx-64", "dbrx-512", "mixed", "prefill-8x512",
                                  "prefill-16x2048"])
def test_length_mixes(name):
    # only the small draws: lengths and the page permutation (patch the bulk draw)
    orig = W._fill_normal
    W._fill_normal = lambda shape, *a, **k: np.zeros((1,) + tuple(shape[1:]), np.uint16)
    try:
        b = W.generate(name, seed=1)
    finally:
        W._fill_normal = orig
    ctx = b.context_lens
    cfg = W.CONFIGS[name]
    if name == "mixtral-256":
        assert len(ctx) == 256 and ctx.min() >= 512 and ctx.max() <= 2048
    if name == "long-ctx-64":
        assert len(ctx) == 64 and ctx.min() >= 8192 and ctx.max() <= 32768
    if name == "dbrx-512":
        assert len(ctx) == 512 and ctx.min() >= 128 and ctx.max() <= 8192
        assert 800 < np.median(ctx) < 1300
    if name == "mixed":
        ql = b.q_lens
        assert (ql[:8] == 512).all() and (ql[8:] == 1).all() and len(ql) == 520
        assert (ctx[:8] >= 512).all() and (ctx[:8] <= 2048).all()
        assert (ctx[8:] >= 256).all() and (ctx[8:] <= 4096).all()
    if name == "prefill-8x512":
        assert (b.q_lens == 512).all() and len(ctx) == 8
        assert (ctx >= 512).all() and (ctx <= 2048).all()
    if name == "prefill-16x2048":
        assert (b.q_lens == 2048).all() and len(ctx) == 16
        assert (ctx >= 2048).all() and (ctx <= 4096).all()
    need = int(((ctx + 15) // 16).sum())
    assert b.meta["pages_used"] == need
    # pool sized 1.25x the need, pages disjoint
    used = np.concatenate([b.block_table[i, : (c + 15) // 16] for i, c in enumerate(ctx)])
    assert len(np.unique(used)) == need


def test_poison_marks_only_unread_bytes():
    b = W.generate("tiny", seed=2, poison=True)
    clean = W.generate("tiny", seed=2)
    for i, c in enumerate(b.context_lens):
        for t in range(c):
            pg = b.block_table[i, t // 16]
            assert np.array_equal(b.k_pages[pg, :, t % 16], clean.k_pages[pg, :, t % 16])
    assert (b.k_pages[b.meta["spare_page"]] == W.BF16_NAN).all()
    last = b.block_table[0, 1]  # ctx 17: slot 1.. of page 1 are past the context
    assert (b.v_pages[last, :, 1:] == W.BF16_NAN).all()


def test_permute_pages_keeps_logical_content():
    b = W.generate("tiny", seed=3)
    p = W.permute_pages(b, seed=9)
    for i, c in enumerate(b.context_lens):
        for t in (0, c // 2, c - 1):
            assert np.array_equal(b.k_pages[b.block_table[i, t // 16], :, t % 16],
                                  p.k_pages[p.block_table[i, t // 16], :, t % 16])
