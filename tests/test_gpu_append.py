"""GPU parity of the KV-append kernel (pa_kv_append) against the oracle's
plain scatter: bit-exact pools after the append, for the varlen and decode
layouts, both dtypes, contract violations, and the append followed by
attention on the same stream."""
import numpy as np
import pytest
import torch

import oracle
from paper_2504_09345_amd import binding as pb
from paper_2504_09345_amd import workloads as W

from parity_util import announce, assert_parity, run_oracle, upload

pytestmark = pytest.mark.gpu


def _new_rows(T, H_kv, D, dtype, seed):
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((T, H_kv, D)).astype(np.float32)
    return W.f32_to_bf16_bits(x) if dtype == "bf16" else x


def _dev(a):
    if a.dtype == np.uint16:
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _host(t, dtype):
    t = t.cpu()
    return t.view(torch.int16).numpy().view(np.uint16) if dtype == "bf16" else t.numpy()


def _append_gpu(batch, kn, vn, dev, varlen, max_context_len=None):
    mcl = int(batch.context_lens.max()) if max_context_len is None else max_context_len
    rows = batch.num_q_rows if varlen else 0
    dims = pb.make_dims(dev["q"], dev["k"], dev["bt"], mcl, num_q_rows=rows)
    pb.pa_kv_append(_dev(kn), _dev(vn), dev["bt"], dev["cl"], dev["k"], dev["v"], dims,
                    query_start_loc=dev["qsl"] if varlen else None)
    torch.cuda.synchronize()


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_append_varlen_bit_exact(dtype):
    announce(f"kv append varlen dtype={dtype}")
    b = W.generate("mixed", seed=12, dtype=dtype, overrides=dict(
        prefill=(3, 70, 0, 90), decode=(9, 1, 300), H_q=8, H_kv=2, D=128))
    T = int(b.query_start_loc[-1])
    kn = _new_rows(T, b.num_kv_heads, b.head_dim, dtype, 1)
    vn = _new_rows(T, b.num_kv_heads, b.head_dim, dtype, 2)
    ek, ev = oracle.kv_append(kn, vn, b.block_table, b.context_lens, b.k_pages, b.v_pages,
                              query_start_loc=b.query_start_loc)
    dev = upload(b)
    _append_gpu(b, kn, vn, dev, varlen=True)
    assert np.array_equal(_host(dev["k"], dtype), ek)
    assert np.array_equal(_host(dev["v"], dtype), ev)


def test_append_varlen_many_sequences_bit_exact():
    """16,400 sequences in a varlen call: past the 16,383 whose
    query_start_loc the kernel stages in LDS, the rows find their sequence in
    global memory instead (two chunks among single-row sequences)."""
    announce("kv append varlen 16400 sequences")
    b = W.generate("mixed", seed=13, overrides=dict(
        prefill=(2, 40, 0, 60), decode=(16398, 1, 40), H_q=4, H_kv=1, D=64))
    assert b.num_seqs == 16400
    T = int(b.query_start_loc[-1])
    kn = _new_rows(T, b.num_kv_heads, b.head_dim, "bf16", 3)
    vn = _new_rows(T, b.num_kv_heads, b.head_dim, "bf16", 4)
    ek, ev = oracle.kv_append(kn, vn, b.block_table, b.context_lens, b.k_pages, b.v_pages,
                              query_start_loc=b.query_start_loc)
    dev = upload(b)
    _append_gpu(b, kn, vn, dev, varlen=True)
    assert np.array_equal(_host(dev["k"], "bf16"), ek)
    assert np.array_equal(_host(dev["v"], "bf16"), ev)


@pytest.mark.parametrize("D", [64, 128])
def test_append_decode_layout_bit_exact(D):
    announce(f"kv append decode D={D}")
    b = W.generate("tiny", seed=13, overrides=dict(D=D, ctx=("list", [17, 0, 129, 16, 1, 200])))
    kn = _new_rows(b.num_seqs, b.num_kv_heads, D, "bf16", 3)
    vn = _new_rows(b.num_seqs, b.num_kv_heads, D, "bf16", 4)
    ek, ev = oracle.kv_append(kn, vn, b.block_table, b.context_lens, b.k_pages, b.v_pages)
    dev = upload(b)
    _append_gpu(b, kn, vn, dev, varlen=False)
    assert np.array_equal(_host(dev["k"], "bf16"), ek)
    assert np.array_equal(_host(dev["v"], "bf16"), ev)


def test_append_skips_contract_violations():
    """A page entry outside the pool and a context above max_context_len: those
    sequences write nothing; the others are written as the oracle writes them."""
    announce("kv append violations")
    b = W.generate("tiny", seed=14, overrides=dict(ctx=("list", [40, 33, 150, 64])))
    kn = _new_rows(b.num_seqs, b.num_kv_heads, b.head_dim, "bf16", 5)
    vn = _new_rows(b.num_seqs, b.num_kv_heads, b.head_dim, "bf16", 6)
    bt = b.block_table.copy()
    bt[1, (int(b.context_lens[1]) - 1) // 16] = b.num_pages + 5   # outside the pool
    ok = b.context_lens.copy()
    ok[1] = ok[2] = 0                                            # expected: nothing for seqs 1, 2
    ek, ev = oracle.kv_append(kn, vn, b.block_table, ok, b.k_pages, b.v_pages)
    dev = upload(b)
    dev["bt"] = _dev(bt)
    _append_gpu(b, kn, vn, dev, varlen=False, max_context_len=149)  # seq 2 (ctx 150) is above it
    assert np.array_equal(_host(dev["k"], "bf16"), ek)
    assert np.array_equal(_host(dev["v"], "bf16"), ev)


def test_append_then_attention_restores_the_cache():
    """Poison every sequence's last cached token, append its K/V, attend on the
    same stream: the output equals attention on the untouched pool, bit for
    bit, and matches the oracle."""
    announce("kv append then attention")
    b = W.generate("mixed", seed=15, overrides=dict(prefill=(2, 40, 10, 60), decode=(6, 20, 400),
                                                    H_q=16, H_kv=4, D=128))
    qsl, ctx = b.query_start_loc, b.context_lens
    rows = oracle.gather_indices(b.block_table, ctx, 16, b.num_pages)
    starts = np.concatenate([[0], np.cumsum(ctx)])
    new = []
    for s in range(b.num_seqs):
        L = int(qsl[s + 1] - qsl[s])
        new += [rows[starts[s] + ctx[s] - L + j] for j in range(L)]
    new = np.array(new)
    kn = b.k_pages[new // 16, :, new % 16, :].copy()   # [T][H_kv][D]
    vn = b.v_pages[new // 16, :, new % 16, :].copy()
    dev = upload(b)
    out_ref = torch.empty_like(dev["q"])
    dims = pb.make_dims(dev["q"], dev["k"], dev["bt"], int(ctx.max()), num_q_rows=b.num_q_rows,
                        max_q_len=int(b.q_lens.max()))
    pb.paged_attn_varlen(dev["q"], dev["k"], dev["v"], dev["bt"], dev["cl"], dev["qsl"], b.scale,
                         out_ref, dims)
    idx_p, idx_s = torch.from_numpy(new // 16).cuda(), torch.from_numpy(new % 16).cuda()
    dev["k"][idx_p, :, idx_s, :] = float("nan")
    dev["v"][idx_p, :, idx_s, :] = float("nan")
    pb.pa_kv_append(_dev(kn), _dev(vn), dev["bt"], dev["cl"], dev["k"], dev["v"], dims,
                    query_start_loc=dev["qsl"])
    out = torch.empty_like(dev["q"])
    pb.paged_attn_varlen(dev["q"], dev["k"], dev["v"], dev["bt"], dev["cl"], dev["qsl"], b.scale,
                         out, dims)
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), out_ref.view(torch.int16))
    assert_parity(out.float().cpu().numpy(), run_oracle(b), strict=False, what="append+attention")


@pytest.mark.slow
def test_append_full_size_mixed():
    """The mixed batch's 8 x 512 chunk rows and 512 decode rows: written
    vectors bit-exact; every other pool byte unchanged (compared on the
    device against a copy)."""
    announce("kv append full-size mixed")
    b = W.generate("mixed", seed=1)
    qsl, ctx = b.query_start_loc, b.context_lens
    T = int(qsl[-1])
    kn = _new_rows(T, b.num_kv_heads, b.head_dim, "bf16", 7)
    vn = _new_rows(T, b.num_kv_heads, b.head_dim, "bf16", 8)
    dev = upload(b)
    k0, v0 = dev["k"].clone(), dev["v"].clone()
    _append_gpu(b, kn, vn, dev, varlen=True)
    rows = oracle.gather_indices(b.block_table, ctx, 16, b.num_pages)
    starts = np.concatenate([[0], np.cumsum(ctx)])
    new = np.concatenate([rows[starts[s] + ctx[s] - (qsl[s + 1] - qsl[s]) + np.arange(qsl[s + 1] - qsl[s])]
                          for s in range(b.num_seqs)])
    ip, isl = torch.from_numpy(new // 16).cuda(), torch.from_numpy(new % 16).cuda()
    got_k = dev["k"][ip, :, isl, :].view(torch.int16).cpu().numpy().view(np.uint16)
    got_v = dev["v"][ip, :, isl, :].view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(got_k, kn) and np.array_equal(got_v, vn)
    # restore the written vectors from the copy: the pools must then equal the copy
    dev["k"][ip, :, isl, :] = k0[ip, :, isl, :]
    dev["v"][ip, :, isl, :] = v0[ip, :, isl, :]
    assert torch.equal(dev["k"].view(torch.int16), k0.view(torch.int16))
    assert torch.equal(dev["v"].view(torch.int16), v0.view(torch.int16))
