"""Seeded synthetic inputs for paged-KV GQA attention.

This module only draws inputs: it holds none of the attention arithmetic, and
both the GPU path and the CPU oracle take its arrays.  The paper measures
end-to-end serving on MTBench, RAG and AIME prompts (Sec. 7, Table 3) with
Mixtral-8x7B, Mixtral-8x22B and DBRX; none of those datasets or weights is used
here.  Synthetic batches with the models' attention shapes and the stated
context-length mixes stand in for them.

Draw order for one batch (one ``numpy`` generator seeded with ``seed`` for the
small draws): context lengths, then the page permutation.  The bulk arrays q,
K and V come from independent PCG64 streams keyed (seed, array id, chunk) so
that they can be filled by several threads with a result independent of the
thread count.  Values are N(0, 1) * std, rounded to bf16 with
round-to-nearest-even on the integer bit pattern.

Pool: a random permutation of ``num_pages`` pages; sequence b takes the next
ceil(ctx_b / 16) entries of that permutation as its block-table row.  Unused
block-table entries point at a page no sequence uses.  With ``poison=True``
every byte the attention must not read (unused pool pages, the slots past the
context in each sequence's last page, the page that unused block-table entries
point at) holds NaN, so any stray read shows up in the output.
"""
from __future__ import annotations

import math
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field

import numpy as np

PAGE_SIZE = 16
BF16_NAN = np.uint16(0x7FC0)

# Named workloads.  Shapes are the attention shapes of the paper's models
# (Sec. 7): Mixtral-8x7B has 32 query heads over 8 KV heads, DBRX and
# Mixtral-8x22B 48 over 8, all with head dim 128.
CONFIGS = {
    # correctness-sized decode step
    "tiny": dict(kind="decode", B=4, H_q=8, H_kv=2, D=64, ctx=("list", [17, 64, 129, 200]),
                 pool=("fixed", 64), std=1.0),
    # Mixtral-8x7B-shaped decode step, batch 256
    "mixtral-256": dict(kind="decode", B=256, H_q=32, H_kv=8, D=128, ctx=("uniform", 512, 2048),
                        pool=("factor", 1.25), std=0.5),
    # long contexts: split-K over page ranges is required
    "long-ctx-64": dict(kind="decode", B=64, H_q=32, H_kv=8, D=128,
                        ctx=("uniform", 8192, 32768), pool=("factor", 1.25), std=0.5),
    # DBRX / Mixtral-8x22B-shaped decode step, GQA group 6
    "dbrx-512": dict(kind="decode", B=512, H_q=48, H_kv=8, D=128,
                     ctx=("lognormal", 1024, 1.0, 128, 8192), pool=("factor", 1.25), std=0.5),
    # 8 causal prefill chunks of 512 rows over 0..1536 cached tokens, plus 512
    # decode sequences, in one launch
    "mixed": dict(kind="varlen", H_q=32, H_kv=8, D=128, prefill=(8, 512, 0, 1536),
                  decode=(512, 256, 4096), pool=("factor", 1.25), std=0.5),
    # the same 8 prefill chunks on their own (the chunked-prefill kernel alone)
    "prefill-8x512": dict(kind="varlen", H_q=32, H_kv=8, D=128, prefill=(8, 512, 0, 1536),
                          decode=(0, 256, 4096), pool=("factor", 1.25), std=0.5),
    # a prefill-heavy step: 16 causal chunks of 2048 rows over 0..2048 cached
    # tokens, the chunked-prefill kernel alone
    "prefill-16x2048": dict(kind="varlen", H_q=32, H_kv=8, D=128, prefill=(16, 2048, 0, 2048),
                            decode=(0, 256, 4096), pool=("factor", 1.25), std=0.5),
}


@dataclass
class Batch:
    """One synthetic batch.  Arrays are host NumPy arrays; bf16 data is held as
    uint16 bit patterns."""
    name: str
    dtype: str                    # "bf16" or "fp32"
    q: np.ndarray                 # [T_q][H_q][D]
    k_pages: np.ndarray           # [num_pages][H_kv][16][D]
    v_pages: np.ndarray           # [num_pages][H_kv][16][D]
    block_table: np.ndarray       # int32 [B][max_pages_per_seq]
    context_lens: np.ndarray      # int32 [B]
    query_start_loc: np.ndarray | None  # int32 [B+1] for varlen, else None
    scale: float
    seed: int
    poison: bool = False
    meta: dict = field(default_factory=dict)

    @property
    def num_seqs(self) -> int:
        return int(self.context_lens.shape[0])

    @property
    def num_q_heads(self) -> int:
        return int(self.q.shape[1])

    @property
    def num_kv_heads(self) -> int:
        return int(self.k_pages.shape[1])

    @property
    def head_dim(self) -> int:
        return int(self.q.shape[2])

    @property
    def num_pages(self) -> int:
        return int(self.k_pages.shape[0])

    @property
    def max_pages_per_seq(self) -> int:
        return int(self.block_table.shape[1])

    @property
    def num_q_rows(self) -> int:
        return int(self.q.shape[0])

    @property
    def q_lens(self) -> np.ndarray:
        if self.query_start_loc is None:
            return np.ones(self.num_seqs, np.int32)
        return np.diff(self.query_start_loc).astype(np.int32)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (nearest, ties to even) and return the bit patterns.
    NaN stays a quiet NaN."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = ((u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))) >> np.uint32(16))
    r = r.astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        r[nan] = BF16_NAN
    return r


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 (exact)."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


_CHUNK = 1 << 20
_ARRAY_IDS = {"q": 1, "k": 2, "v": 3}


def _fill_normal(shape, seed: int, array: str, std: float, dtype: str, threads: int | None):
    """N(0,1)*std in the requested storage type, chunk c drawn from
    PCG64(SeedSequence([seed, array id, c]))."""
    n = int(np.prod(shape))
    out = np.empty(n, np.uint16 if dtype == "bf16" else np.float32)
    nchunks = (n + _CHUNK - 1) // _CHUNK
    aid = _ARRAY_IDS[array]

    def work(c):
        lo, hi = c * _CHUNK, min(n, (c + 1) * _CHUNK)
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, aid, c])))
        x = g.standard_normal(hi - lo, dtype=np.float32)
        if std != 1.0:
            x *= np.float32(std)
        out[lo:hi] = f32_to_bf16_bits(x) if dtype == "bf16" else x

    if threads is None:
        threads = min(16, os.cpu_count() or 1)
    if nchunks <= 1 or threads <= 1:
        for c in range(nchunks):
            work(c)
    else:
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(work, range(nchunks)))
    return out.reshape(shape)


def _draw_lengths(spec, n, rng):
    kind = spec[0]
    if kind == "list":
        return np.array(spec[1], np.int64)
    if kind == "uniform":  # integers, both ends inclusive
        return rng.integers(spec[1], spec[2], size=n, endpoint=True)
    if kind == "lognormal":  # round(median * exp(sigma Z)), clipped
        med, sigma, lo, hi = spec[1:]
        z = rng.standard_normal(n)
        return np.clip(np.rint(med * np.exp(sigma * z)), lo, hi).astype(np.int64)
    raise ValueError(spec)


def generate(name: str, seed: int = 0, dtype: str = "bf16", poison: bool = False,
             threads: int | None = None, overrides: dict | None = None) -> Batch:
    """Draw the named workload.  ``overrides`` replaces config keys (used by
    tests to shrink a workload while keeping its structure)."""
    cfg = dict(CONFIGS[name])
    if overrides:
        cfg.update(overrides)
    if dtype not in ("bf16", "fp32"):
        raise ValueError(dtype)
    rng = np.random.default_rng(seed)
    H_q, H_kv, D = cfg["H_q"], cfg["H_kv"], cfg["D"]

    # 1. context lengths (and chunk lengths for varlen)
    if cfg["kind"] == "decode":
        B = cfg["B"] if cfg["ctx"][0] != "list" else len(cfg["ctx"][1])
        ctx = _draw_lengths(cfg["ctx"], B, rng)
        qlen = np.ones(B, np.int64)
    else:
        n_pre, chunk, prior_lo, prior_hi = cfg["prefill"]
        n_dec, dlo, dhi = cfg["decode"]
        prior = rng.integers(prior_lo, prior_hi, size=n_pre, endpoint=True)
        dctx = rng.integers(dlo, dhi, size=n_dec, endpoint=True)
        ctx = np.concatenate([prior + chunk, dctx])
        qlen = np.concatenate([np.full(n_pre, chunk), np.ones(n_dec, np.int64)])
        B = n_pre + n_dec
    ctx = ctx.astype(np.int64)
    npages = (ctx + PAGE_SIZE - 1) // PAGE_SIZE
    need = int(npages.sum())

    # 2. pool and page permutation
    pk = cfg["pool"]
    num_pages = pk[1] if pk[0] == "fixed" else int(math.ceil(pk[1] * need))
    num_pages = max(num_pages, need + 1)  # at least one spare page
    perm = rng.permutation(num_pages).astype(np.int32)
    mp = max(1, int(npages.max()) if B else 1)
    spare = int(perm[need])  # first page no sequence uses
    block_table = np.full((B, mp), spare, np.int32)
    off = 0
    for b in range(B):
        block_table[b, : npages[b]] = perm[off: off + npages[b]]
        off += npages[b]

    # 3..5. q, K, V
    T = int(qlen.sum())
    std = float(cfg["std"])
    q = _fill_normal((T, H_q, D), seed, "q", std, dtype, threads)
    k = _fill_normal((num_pages, H_kv, PAGE_SIZE, D), seed, "k", std, dtype, threads)
    v = _fill_normal((num_pages, H_kv, PAGE_SIZE, D), seed, "v", std, dtype, threads)

    if poison:
        nanv = BF16_NAN if dtype == "bf16" else np.float32(np.nan)
        used = np.zeros(num_pages, bool)
        used[perm[:need]] = True
        k[~used] = nanv
        v[~used] = nanv
        for b in range(B):
            c = int(ctx[b])
            if c % PAGE_SIZE:
                last = block_table[b, npages[b] - 1]
                k[last, :, c % PAGE_SIZE:, :] = nanv
                v[last, :, c % PAGE_SIZE:, :] = nanv

    qsl = None
    if cfg["kind"] == "varlen":
        qsl = np.zeros(B + 1, np.int32)
        qsl[1:] = np.cumsum(qlen)
    return Batch(name=name, dtype=dtype, q=q, k_pages=k, v_pages=v, block_table=block_table,
                 context_lens=ctx.astype(np.int32), query_start_loc=qsl,
                 scale=1.0 / math.sqrt(D), seed=seed, poison=poison,
                 meta=dict(cfg=cfg, spare_page=spare, pages_used=need))


def identity_layout(B: int, ctx, H_q: int, H_kv: int, D: int, seed: int, dtype: str = "bf16",
                    std: float = 1.0, qlen=None) -> Batch:
    """Sequence b owns pages [b*mp, (b+1)*mp) in order (identity block table), so
    the pool reshapes to dense per-sequence K/V without any gather."""
    ctx = np.asarray(ctx, np.int64)
    mp = max(1, int(((ctx + PAGE_SIZE - 1) // PAGE_SIZE).max()))
    num_pages = B * mp
    block_table = np.arange(num_pages, dtype=np.int32).reshape(B, mp)
    qlen = np.ones(B, np.int64) if qlen is None else np.asarray(qlen, np.int64)
    T = int(qlen.sum())
    q = _fill_normal((T, H_q, D), seed, "q", std, dtype, 1)
    k = _fill_normal((num_pages, H_kv, PAGE_SIZE, D), seed, "k", std, dtype, 1)
    v = _fill_normal((num_pages, H_kv, PAGE_SIZE, D), seed, "v", std, dtype, 1)
    qsl = None
    if not np.all(qlen == 1):
        qsl = np.zeros(B + 1, np.int32)
        qsl[1:] = np.cumsum(qlen)
    return Batch(name="identity", dtype=dtype, q=q, k_pages=k, v_pages=v, block_table=block_table,
                 context_lens=ctx.astype(np.int32), query_start_loc=qsl,
                 scale=1.0 / math.sqrt(D), seed=seed)


def permute_pages(batch: Batch, seed: int) -> Batch:
    """Move every page to a new random place in the pool and rewrite the block
    table to match: the logical content of every sequence is unchanged."""
    rng = np.random.default_rng(seed)
    N = batch.num_pages
    new_of_old = rng.permutation(N).astype(np.int32)
    k = np.empty_like(batch.k_pages)
    v = np.empty_like(batch.v_pages)
    k[new_of_old] = batch.k_pages
    v[new_of_old] = batch.v_pages
    bt = new_of_old[batch.block_table]
    return Batch(name=batch.name + "+perm", dtype=batch.dtype, q=batch.q, k_pages=k, v_pages=v,
                 block_table=bt.astype(np.int32), context_lens=batch.context_lens,
                 query_start_loc=batch.query_start_loc, scale=batch.scale, seed=batch.seed,
                 poison=batch.poison, meta=dict(batch.meta))


# --- request arrival streams (scheduler inputs) -----------------------------
# Prompt and generation lengths of the paper's evaluation workloads (Table 4):
# (average prompt, maximum prompt, maximum generation).  Prompts are drawn
# lognormal with sigma 0.8 around a median chosen so the unclipped mean is the
# average, then clipped to [1, maximum]; generation lengths are uniform in
# [1, maximum generation].  Synthetic stand-ins: no benchmark item is used.
ARRIVAL_MIXES = {
    "mtbench-g32": (98, 450, 32),
    "mtbench-g128": (98, 450, 128),
    "mtbench-g256": (98, 450, 256),
    "rag": (926, 1843, 128),
    "aime": (128, 410, 512),
    "tiny": (20, 60, 40),  # small pools for tests that need preemption often
}


def arrival_stream(mix: str, steps: int, per_step: float, seed: int, first_id: int = 0):
    """Arrivals for `steps` scheduler steps: a Poisson(per_step) count per step,
    each arrival (logical id, prompt tokens, finish length = prompt +
    generation).  Returns a list of (ids, prompts, finishes) int32 arrays."""
    avg, pmax, gmax = ARRIVAL_MIXES[mix]
    rng = np.random.default_rng(seed)
    sigma = 0.8
    med = avg / math.exp(sigma * sigma / 2)
    out, nid = [], first_id
    for _ in range(steps):
        n = int(rng.poisson(per_step))
        p = _draw_lengths(("lognormal", med, sigma, 1, pmax), n, rng)
        g = rng.integers(1, gmax, size=n, endpoint=True)
        ids = np.arange(nid, nid + n, dtype=np.int32)
        nid += n
        out.append((ids, p.astype(np.int32), (p + g).astype(np.int32)))
    return out
