"""Shared helpers of the GPU parity tests: upload a seeded batch, run the
library through its C ABI, run the oracle on the same host arrays, cut
sub-batches for sampled checks, and the tolerance rule.

Tolerance (bf16 inputs, fp32 accumulation): max abs error 1e-2 and max rel
error 5e-3.  Relative error is taken against max(|ref|, rho) with rho the
RMS of that (row, head) reference vector, so that entries near zero do not
divide by ~0.  The absolute bound applies to entries with |ref| < 4: from 4
on, bf16 values are 2^-5 apart, so even the correctly rounded output can be
1.6e-2 away, and there the relative bound (5e-3 |ref| >= 2e-2) governs.  The decode tests also check the fixed floor max(|ref|, 1e-3)
(decode keeps P in fp32, or as bf16 high + low parts of ~16 significant bits
on the matrix cores).  A bf16 output alone contributes up to 2^-8 = 3.9e-3
relative error (8 significant bits, round to nearest), so that floor leaves
little room for entries near 1e-3 and is a check of the committed cases
rather than a bound.
"""
from __future__ import annotations

import sys

import numpy as np

from paper_2504_09345_amd import binding as pb
from paper_2504_09345_amd import workloads as W

MAX_ABS = 1e-2
MAX_REL = 5e-3
ABS_RANGE = 4.0  # entries checked against MAX_ABS: |ref| below this


def announce(msg: str) -> None:
    """Name the case on the real stdout before a GPU step (pytest captures
    sys.stdout; a run that dies on the GPU still shows what it was doing)."""
    sys.__stdout__.write(f"[gpu] {msg}\n")
    sys.__stdout__.flush()


def upload(batch: W.Batch, device="cuda"):
    import torch

    def t(a):
        if a.dtype == np.uint16:
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(device)
        return torch.from_numpy(np.ascontiguousarray(a)).to(device)

    d = dict(q=t(batch.q), k=t(batch.k_pages), v=t(batch.v_pages), bt=t(batch.block_table),
             cl=t(batch.context_lens))
    if batch.query_start_loc is not None:
        d["qsl"] = t(batch.query_start_loc)
    return d


def run_gpu(batch: W.Batch, dev=None, pages_per_split=0, max_context_len=None, out=None):
    """Run paged_attn (decode) or paged_attn_varlen on the GPU; returns the
    output as float32 numpy."""
    import torch
    dev = dev or upload(batch)
    mcl = int(batch.context_lens.max()) if max_context_len is None else max_context_len
    if out is None:
        out = torch.empty_like(dev["q"])
    if batch.query_start_loc is None:
        dims = pb.make_dims(dev["q"], dev["k"], dev["bt"], mcl, pages_per_split)
        pb.paged_attn(dev["q"], dev["k"], dev["v"], dev["bt"], dev["cl"], batch.scale, out, dims)
    else:
        dims = pb.make_dims(dev["q"], dev["k"], dev["bt"], mcl, pages_per_split,
                            num_q_rows=batch.num_q_rows, max_q_len=int(batch.q_lens.max()))
        pb.paged_attn_varlen(dev["q"], dev["k"], dev["v"], dev["bt"], dev["cl"], dev["qsl"],
                             batch.scale, out, dims)
    torch.cuda.synchronize()
    return out.float().cpu().numpy()


def run_oracle(batch: W.Batch):
    import oracle
    if batch.query_start_loc is None:
        return oracle.paged_attn(batch.q, batch.k_pages, batch.v_pages, batch.block_table,
                                 batch.context_lens, batch.scale)
    return oracle.paged_attn_varlen(batch.q, batch.k_pages, batch.v_pages, batch.block_table,
                                    batch.context_lens, batch.query_start_loc, batch.scale)


def sub_batch(batch: W.Batch, seqs) -> W.Batch:
    """The batch restricted to the given sequences (same page pools).  Returns
    the sub-batch and the rows of the full output that correspond to it."""
    seqs = np.asarray(seqs)
    if batch.query_start_loc is None:
        rows = seqs
        qsl = None
    else:
        qsl_full = batch.query_start_loc
        rows = np.concatenate([np.arange(qsl_full[b], qsl_full[b + 1]) for b in seqs])
        qlen = qsl_full[seqs + 1] - qsl_full[seqs]
        qsl = np.zeros(len(seqs) + 1, np.int32)
        qsl[1:] = np.cumsum(qlen)
    sb = W.Batch(name=batch.name + "[sub]", dtype=batch.dtype, q=batch.q[rows],
                 k_pages=batch.k_pages, v_pages=batch.v_pages,
                 block_table=batch.block_table[seqs], context_lens=batch.context_lens[seqs],
                 query_start_loc=qsl, scale=batch.scale, seed=batch.seed)
    return sb, rows


def parity_stats(gpu: np.ndarray, ref: np.ndarray) -> dict:
    g = gpu.astype(np.float64)
    r = ref.astype(np.float64)
    err = np.abs(g - r)
    rho = np.sqrt((r * r).mean(axis=-1, keepdims=True))
    # the absolute bound is checked where a bf16 output can meet it: below
    # |ref| = 4 the bf16 grid is at most 2^-7 from any value, from 4 on its
    # half-spacing is 2^-6 > 1e-2 and the relative bound (then >= 2e-2) governs
    small = np.abs(r) < ABS_RANGE
    return dict(
        finite=bool(np.isfinite(g).all()),
        max_abs=float(err[small].max(initial=0.0)),
        max_abs_all=float(err.max(initial=0.0)),
        max_rel=float((err / np.maximum(np.abs(r), np.maximum(rho, 1e-30))).max(initial=0.0)),
        max_rel_floor=float((err / np.maximum(np.abs(r), 1e-3)).max(initial=0.0)),
        max_rel_global=float(err.max(initial=0.0) / max(np.abs(r).max(initial=0.0), 1e-30)),
    )


def assert_parity(gpu, ref, strict=True, what=""):
    st = parity_stats(gpu, ref)
    assert st["finite"], f"{what}: non-finite output"
    assert st["max_abs"] <= MAX_ABS, f"{what}: {st}"
    assert st["max_rel"] <= MAX_REL, f"{what}: {st}"
    if strict:
        assert st["max_rel_floor"] <= MAX_REL, f"{what}: {st}"
    return st
