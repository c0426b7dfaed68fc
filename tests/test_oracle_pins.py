"""Pins of the CPU oracle against facts fixed by the mathematics, independent
of the oracle's own code: a library routine on a dense layout, invariances,
closed forms, brute force on tiny inputs and a hand-derived gather fixture.

The attention being defined is the paged GQA decode attention of MoE-Lens
(arXiv 2504.09345): paged KV blocks (Sec. 5.5), grouped-query heads (Sec. 2),
bf16 storage with fp32 arithmetic (Sec. 5.3, Eq. 6), causal prefill chunks
(the library's reading of Sec. 6.4).  The paper prints no worked attention
example, so no pin comes from printed attention values.
"""
import math
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2504_09345_amd import workloads as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _f32(a):
    return W.bf16_bits_to_f32(a) if a.dtype == np.uint16 else a.astype(np.float32)


def _dense_sdpa_f64(batch):
    """torch SDPA (float64, CPU) on the identity-layout pool reshaped to dense
    per-sequence K/V: no block-table gather is involved."""
    B, H_q, H_kv, D = batch.num_seqs, batch.num_q_heads, batch.num_kv_heads, batch.head_dim
    mp, P = batch.max_pages_per_seq, W.PAGE_SIZE
    s = H_q // H_kv
    k = torch.from_numpy(_f32(batch.k_pages)).double()
    v = torch.from_numpy(_f32(batch.v_pages)).double()
    # [B*mp][H_kv][P][D] -> [B][H_kv][mp*P][D]
    k = k.reshape(B, mp, H_kv, P, D).permute(0, 2, 1, 3, 4).reshape(B, H_kv, mp * P, D)
    v = v.reshape(B, mp, H_kv, P, D).permute(0, 2, 1, 3, 4).reshape(B, H_kv, mp * P, D)
    q_all = torch.from_numpy(_f32(batch.q)).double()
    qsl = batch.query_start_loc if batch.query_start_loc is not None else np.arange(B + 1)
    out = torch.zeros_like(q_all)
    for b in range(B):
        C = int(batch.context_lens[b])
        r0, r1 = int(qsl[b]), int(qsl[b + 1])
        L = r1 - r0
        if C == 0 or L == 0:
            continue
        qb = q_all[r0:r1].permute(1, 0, 2).unsqueeze(0)            # [1][H_q][L][D]
        kb = k[b, :, :C].repeat_interleave(s, dim=0).unsqueeze(0)  # [1][H_q][C][D]
        vb = v[b, :, :C].repeat_interleave(s, dim=0).unsqueeze(0)
        pos = torch.arange(C - L, C).unsqueeze(1)                  # absolute query positions
        mask = torch.arange(C).unsqueeze(0) <= pos                 # [L][C]
        ob = torch.nn.functional.scaled_dot_product_attention(qb, kb, vb, attn_mask=mask,
                                                              scale=batch.scale)
        out[r0:r1] = ob[0].permute(1, 0, 2)
    return out.numpy()


def _run_oracle(batch):
    if batch.query_start_loc is None:
        return oracle.paged_attn(batch.q, batch.k_pages, batch.v_pages, batch.block_table,
                                 batch.context_lens, batch.scale)
    return oracle.paged_attn_varlen(batch.q, batch.k_pages, batch.v_pages, batch.block_table,
                                    batch.context_lens, batch.query_start_loc, batch.scale)


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("H_q,H_kv,D", [(8, 2, 64), (6, 6, 64), (12, 2, 128), (4, 1, 32)])
def test_decode_equals_dense_sdpa(dtype, H_q, H_kv, D):
    ctx = [1, 16, 17, 37, 100]
    batch = W.identity_layout(len(ctx), ctx, H_q, H_kv, D, seed=11, dtype=dtype)
    got = _run_oracle(batch)
    ref = _dense_sdpa_f64(batch)
    np.testing.assert_allclose(got, ref, rtol=2e-5, atol=2e-6)


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_prefill_chunks_equal_dense_causal_sdpa(dtype):
    # chunk lengths with prior context 0 (plain causal), partial and decode rows
    ctx = [40, 70, 33, 9, 64]
    qlen = [40, 21, 1, 9, 17]
    batch = W.identity_layout(len(ctx), ctx, 8, 2, 64, seed=5, dtype=dtype, qlen=qlen)
    got = _run_oracle(batch)
    ref = _dense_sdpa_f64(batch)
    np.testing.assert_allclose(got, ref, rtol=2e-5, atol=2e-6)


def test_prefill_prior_zero_is_plain_causal():
    # with no prior context the chunk is ordinary causal self-attention: SDPA's
    # own is_causal path (top-left aligned) must agree
    ctx, L = [48], [48]
    batch = W.identity_layout(1, ctx, 4, 2, 64, seed=8, dtype="fp32", qlen=L)
    got = _run_oracle(batch)
    k = torch.from_numpy(batch.k_pages).double().reshape(3, 2, 16, 64).permute(1, 0, 2, 3)
    k = k.reshape(2, 48, 64).repeat_interleave(2, dim=0)[None]
    v = torch.from_numpy(batch.v_pages).double().reshape(3, 2, 16, 64).permute(1, 0, 2, 3)
    v = v.reshape(2, 48, 64).repeat_interleave(2, dim=0)[None]
    q = torch.from_numpy(batch.q).double().permute(1, 0, 2)[None]
    ref = torch.nn.functional.scaled_dot_product_attention(q, k, v, is_causal=True,
                                                           scale=batch.scale)
    np.testing.assert_allclose(got, ref[0].permute(1, 0, 2).numpy(), rtol=2e-5, atol=2e-6)


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_page_permutation_invariance_bit_exact(dtype):
    batch = W.generate("tiny", seed=3, dtype=dtype)
    a = _run_oracle(batch)
    for s in (1, 2):
        b = _run_oracle(W.permute_pages(batch, seed=100 + s))
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_one_token_context_returns_v_exactly(dtype):
    batch = W.generate("tiny", seed=4, dtype=dtype)
    batch.context_lens[:] = 1
    out = _run_oracle(batch)
    s = batch.num_q_heads // batch.num_kv_heads
    for b in range(batch.num_seqs):
        page = batch.block_table[b, 0]
        for h in range(batch.num_q_heads):
            v0 = _f32(batch.v_pages[page, h // s, 0])
            assert np.array_equal(out[b, h].view(np.uint32), v0.view(np.uint32))


def _brute_weights(batch, b, h, L=1, r=0, qrow=None):
    """float64 softmax weights with math.exp, pure Python loops (tiny only)."""
    s = batch.num_q_heads // batch.num_kv_heads
    g = h // s
    C = int(batch.context_lens[b])
    qrow = b if qrow is None else qrow
    qv = [float(x) for x in _f32(batch.q[qrow, h])]
    xs = []
    for t in range(C - L + r + 1):
        page = int(batch.block_table[b, t // 16])
        kv = _f32(batch.k_pages[page, g, t % 16])
        xs.append(sum(qv[d] * float(kv[d]) for d in range(len(qv))) * batch.scale)
    m = max(xs)
    e = [math.exp(x - m) for x in xs]
    tot = sum(e)
    return [x / tot for x in e]


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_softmax_weights_sum_to_one_and_match_brute_force(dtype):
    batch = W.generate("tiny", seed=6, dtype=dtype)
    for b in range(batch.num_seqs):
        for h in (0, 3, 5, 7):
            w = oracle.softmax_weights(batch.q, batch.k_pages, batch.block_table,
                                       batch.context_lens, batch.scale, b, h)
            assert w.shape[0] == batch.context_lens[b]
            assert abs(float(np.sum(w, dtype=np.float64)) - 1.0) < 1e-6
            ref = np.array(_brute_weights(batch, b, h))
            np.testing.assert_allclose(w, ref, rtol=1e-6, atol=1e-9)


def test_softmax_weights_prefill_row_brute_force():
    batch = W.identity_layout(1, [50], 4, 2, 64, seed=2, dtype="bf16", qlen=[20])
    for r in (0, 7, 19):
        w = oracle.softmax_weights(batch.q, batch.k_pages, batch.block_table,
                                   batch.context_lens, batch.scale, 0, 3, L=20, r=r, qrow=r)
        assert w.shape[0] == 50 - 20 + r + 1
        np.testing.assert_allclose(w, _brute_weights(batch, 0, 3, L=20, r=r, qrow=r),
                                   rtol=1e-6, atol=1e-9)


def test_constant_v_returns_that_vector():
    batch = W.generate("tiny", seed=7, dtype="fp32")
    # every token of (page, kv head) g gets the same V row, per kv head
    rows = np.random.default_rng(1).standard_normal((batch.num_kv_heads, batch.head_dim))
    batch.v_pages[:] = rows.astype(np.float32)[None, :, None, :]
    out = _run_oracle(batch)
    s = batch.num_q_heads // batch.num_kv_heads
    for h in range(batch.num_q_heads):
        np.testing.assert_allclose(out[:, h], np.broadcast_to(rows[h // s], out[:, h].shape),
                                   rtol=2e-6, atol=1e-7)


@pytest.mark.parametrize("zero", ["q", "scale"])
def test_zero_logits_give_mean_of_visible_v(zero):
    batch = W.generate("tiny", seed=9, dtype="fp32")
    if zero == "q":
        batch.q[:] = 0
    else:
        batch.scale = 0.0
    out = _run_oracle(batch)
    s = batch.num_q_heads // batch.num_kv_heads
    for b in range(batch.num_seqs):
        C = int(batch.context_lens[b])
        pages = batch.block_table[b, : (C + 15) // 16]
        vv = batch.v_pages[pages].astype(np.float64)             # [np][H_kv][16][D]
        vv = vv.transpose(1, 0, 2, 3).reshape(batch.num_kv_heads, -1, batch.head_dim)[:, :C]
        mean = vv.mean(axis=1)
        for h in range(batch.num_q_heads):
            np.testing.assert_allclose(out[b, h], mean[h // s], rtol=1e-5, atol=1e-6)


def test_large_scale_selects_argmax_value_row():
    batch = W.generate("tiny", seed=10, dtype="fp32")
    batch.scale = 1.0e4
    out = _run_oracle(batch)
    s = batch.num_q_heads // batch.num_kv_heads
    checked = 0
    for b in range(batch.num_seqs):
        C = int(batch.context_lens[b])
        for h in range(batch.num_q_heads):
            g = h // s
            logits, vals = [], []
            for t in range(C):
                page = batch.block_table[b, t // 16]
                logits.append(float(np.dot(batch.q[b, h].astype(np.float64),
                                           batch.k_pages[page, g, t % 16].astype(np.float64))))
                vals.append(batch.v_pages[page, g, t % 16])
            order = np.argsort(logits)
            if logits[order[-1]] - logits[order[-2]] < 0.05:  # need a clear winner
                continue
            np.testing.assert_array_equal(out[b, h], vals[order[-1]])
            checked += 1
    assert checked > 16


def test_single_row_chunks_equal_decode_and_last_chunk_row_equals_decode():
    batch = W.identity_layout(3, [30, 64, 81], 8, 2, 64, seed=12, dtype="bf16", qlen=[12, 1, 30])
    full = _run_oracle(batch)
    qsl = batch.query_start_loc
    # decode at the same context with the chunk's last query row
    last_rows = batch.q[qsl[1:] - 1]
    dec = oracle.paged_attn(last_rows, batch.k_pages, batch.v_pages, batch.block_table,
                            batch.context_lens, batch.scale)
    assert np.array_equal(full[qsl[1:] - 1].view(np.uint32), dec.view(np.uint32))
    # a chunk row j equals decode over a context cut at its own position
    ctx_cut = batch.context_lens.copy()
    ctx_cut[2] = 81 - 30 + 5 + 1
    dec5 = oracle.paged_attn(batch.q[qsl[:-1] + np.array([0, 0, 5])], batch.k_pages,
                             batch.v_pages, batch.block_table, ctx_cut, batch.scale)
    assert np.array_equal(full[qsl[2] + 5].view(np.uint32), dec5[2].view(np.uint32))


def test_empty_context_gives_zeros():
    batch = W.generate("tiny", seed=13, dtype="bf16")
    batch.context_lens[1] = 0
    out = _run_oracle(batch)
    assert np.all(out[1] == 0)
    assert np.all(np.isfinite(out))


def test_poisoned_pool_does_not_leak():
    a = _run_oracle(W.generate("tiny", seed=14, dtype="bf16"))
    b = _run_oracle(W.generate("tiny", seed=14, dtype="bf16", poison=True))
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def _read_gather_fixture(path):
    """Sections of integer rows from a hand-derived fixture under tests/golden."""
    sec, data = None, {}
    with open(path) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            if line.endswith(":"):
                sec = line[:-1]
                data[sec] = []
            else:
                data[sec].append([int(x) for x in line.split()])
    return data


def test_gather_indices_hand_fixture():
    fx = _read_gather_fixture(os.path.join(GOLDEN, "gather_tiny.txt"))
    bt = np.array(fx["block_table"], np.int32)
    ctx = np.array(fx["context_lens"][0], np.int32)
    rows = oracle.gather_indices(bt, ctx, 16, int(fx["num_pages"][0][0]))
    expect = np.array([x for r in fx["rows"] for x in r], np.int64)
    assert np.array_equal(rows, expect)


def test_gather_indices_identity_and_permuted():
    batch = W.identity_layout(3, [5, 16, 40], 2, 1, 8, seed=0)
    rows = oracle.gather_indices(batch.block_table, batch.context_lens, 16, batch.num_pages)
    mp = batch.max_pages_per_seq
    expect = np.concatenate([b * mp * 16 + np.arange(c) for b, c in enumerate([5, 16, 40])])
    assert np.array_equal(rows, expect)
    perm = W.permute_pages(batch, seed=3)
    prow = oracle.gather_indices(perm.block_table, perm.context_lens, 16, perm.num_pages)
    # permuted rows hold the same token data as the identity rows
    flat_id = batch.k_pages.transpose(0, 2, 1, 3).reshape(-1, batch.num_kv_heads * batch.head_dim)
    flat_pm = perm.k_pages.transpose(0, 2, 1, 3).reshape(-1, perm.num_kv_heads * perm.head_dim)
    assert np.array_equal(flat_id[rows], flat_pm[prow])
    assert len(np.unique(prow)) == len(prow)


def test_oracle_rejects_out_of_pool_page():
    batch = W.generate("tiny", seed=1)
    batch.block_table[0, 0] = batch.num_pages
    with pytest.raises(ValueError):
        _run_oracle(batch)


def test_oracle_thread_count_does_not_change_result():
    batch = W.generate("tiny", seed=15, dtype="bf16")
    oracle.set_threads(1)
    a = _run_oracle(batch)
    oracle.set_threads(4)
    b = _run_oracle(batch)
    oracle.set_threads(0)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


# --- KV append: the cache write before attention -----------------------------

def _kv_rows(T, H_kv, D, dtype=np.uint16):
    """Row r, kv head g holds (100 r + 10 g + 1, 100 r + 10 g + 2, ...)."""
    r = np.arange(T)[:, None, None]
    g = np.arange(H_kv)[None, :, None]
    d = np.arange(D)[None, None, :]
    k = (100 * r + 10 * g + 1 + d).astype(dtype)
    return k, (k + 1000).astype(dtype)


@pytest.mark.parametrize("layout", ["varlen", "decode"])
def test_kv_append_hand_fixture(layout):
    fx = _read_gather_fixture(os.path.join(GOLDEN, "kv_append_tiny.txt"))
    bt = np.array(fx["block_table"], np.int32)
    ctx = np.array(fx["context_lens"][0], np.int32)
    N, H_kv, P, D = int(fx["num_pages"][0][0]), 2, 4, 2
    qsl = np.array(fx["query_start_loc"][0], np.int32) if layout == "varlen" else None
    T = int(qsl[-1]) if layout == "varlen" else len(ctx)
    kn, vn = _kv_rows(T, H_kv, D)
    kp = np.full((N, H_kv, P, D), 7, np.uint16)
    vp = np.full((N, H_kv, P, D), 9, np.uint16)
    k2, v2 = oracle.kv_append(kn, vn, bt, ctx, kp, vp, query_start_loc=qsl)
    ek, ev = kp.copy(), vp.copy()
    for row, page, slot in fx[f"{layout}_writes"]:
        ek[page, :, slot, :] = kn[row]
        ev[page, :, slot, :] = vn[row]
    assert np.array_equal(k2, ek) and np.array_equal(v2, ev)
    assert np.array_equal(kp, np.full_like(kp, 7))  # inputs untouched


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_kv_append_lands_where_the_gather_reads(dtype):
    """After the append, the gather (an independent oracle function) finds the
    new rows at each sequence's last positions; every other pool row is
    unchanged."""
    b = W.generate("mixed", seed=5, dtype=dtype, overrides=dict(
        prefill=(3, 40, 0, 70), decode=(5, 1, 90), H_q=8, H_kv=2, D=64))
    qsl, ctx = b.query_start_loc, b.context_lens
    T, H_kv, D = int(qsl[-1]), b.num_kv_heads, b.head_dim
    rng = np.random.default_rng(11)
    mk = (lambda shape: rng.integers(0, 1 << 16, shape, dtype=np.uint16)) if dtype == "bf16" else \
        (lambda shape: rng.standard_normal(shape).astype(np.float32))
    kn, vn = mk((T, H_kv, D)), mk((T, H_kv, D))
    k2, v2 = oracle.kv_append(kn, vn, b.block_table, ctx, b.k_pages, b.v_pages, query_start_loc=qsl)
    rows = oracle.gather_indices(b.block_table, ctx, 16, b.num_pages)
    starts = np.concatenate([[0], np.cumsum(ctx)])
    flat = lambda a: a.transpose(0, 2, 1, 3).reshape(-1, H_kv, D)
    new_rows = []
    for s in range(b.num_seqs):
        L = int(qsl[s + 1] - qsl[s])
        for j in range(L):
            fr = rows[starts[s] + ctx[s] - L + j]
            new_rows.append(fr)
            assert np.array_equal(flat(k2)[fr], kn[qsl[s] + j])
            assert np.array_equal(flat(v2)[fr], vn[qsl[s] + j])
    keep = np.setdiff1d(np.arange(flat(k2).shape[0]), new_rows)
    assert np.array_equal(flat(k2)[keep], flat(b.k_pages)[keep])
    assert np.array_equal(flat(v2)[keep], flat(b.v_pages)[keep])


def test_kv_append_restores_the_cache_attention_reads():
    """Poison each sequence's last cached token, append its original K/V as
    the decode token: the pool is restored bit for bit, and so is attention."""
    b = W.generate("tiny", seed=6)
    rows = oracle.gather_indices(b.block_table, b.context_lens, 16, b.num_pages)
    starts = np.concatenate([[0], np.cumsum(b.context_lens)])
    last = rows[starts[1:] - 1]
    H_kv, D = b.num_kv_heads, b.head_dim
    flat = lambda a: a.transpose(0, 2, 1, 3).reshape(-1, H_kv, D)
    kn, vn = flat(b.k_pages)[last].copy(), flat(b.v_pages)[last].copy()
    kp, vp = b.k_pages.copy(), b.v_pages.copy()
    kp[last // 16, :, last % 16, :] = 0x7FC0  # NaN
    vp[last // 16, :, last % 16, :] = 0x7FC0
    assert np.isnan(W.bf16_bits_to_f32(kp)).any()
    k2, v2 = oracle.kv_append(kn, vn, b.block_table, b.context_lens, kp, vp)
    assert np.array_equal(k2, b.k_pages) and np.array_equal(v2, b.v_pages)
    ref = oracle.paged_attn(b.q, b.k_pages, b.v_pages, b.block_table, b.context_lens, b.scale)
    got = oracle.paged_attn(b.q, k2, v2, b.block_table, b.context_lens, b.scale)
    assert np.array_equal(ref, got)


def test_kv_append_rejects_bad_inputs_and_leaves_pools_unchanged():
    b = W.generate("tiny", seed=7)
    kn = np.zeros((b.num_seqs, b.num_kv_heads, b.head_dim), np.uint16)
    bt = b.block_table.copy()
    c = int(b.context_lens[0]) - 1
    bt[0, c // 16] = b.num_pages  # the page of seq 0's new token is outside the pool
    with pytest.raises(ValueError):
        oracle.kv_append(kn, kn, bt, b.context_lens, b.k_pages, b.v_pages)
    qsl = np.array([0, 1, 1 + int(b.context_lens[1]) + 1, 0, 0], np.int32)  # L > ctx for seq 1
    qsl[3:] = qsl[2]
    kq = np.zeros((int(qsl[-1]), b.num_kv_heads, b.head_dim), np.uint16)
    with pytest.raises(ValueError):
        oracle.kv_append(kq, kq, b.block_table, b.context_lens, b.k_pages, b.v_pages, query_start_loc=qsl)


# --- scheduler step: page allocator and block-table builder -----------------

def _read_schedule_fixture():
    scen, cur = [], None
    with open(os.path.join(GOLDEN, "schedule_tiny.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].split()
            if not line:
                continue
            key, vals = line[0], [int(x) for x in line[1:] if x.lstrip("-").isdigit()]
            if key == "scenario":
                cur = dict(dims=vals, steps=[])
                scen.append(cur)
            elif key == "step":
                cur["steps"].append({})
            else:
                cur["steps"][-1][key] = vals
    return scen


def test_schedule_hand_fixture():
    for sc in _read_schedule_fixture():
        S, P, MP, Q, n_real = sc["dims"]
        st = oracle.sched_init(S, P, MP, Q)
        for stp in sc["steps"]:
            a = np.array(stp["arrivals"], np.int32).reshape(-1, 3)
            st, qsl, fin, info = oracle.schedule_step(st, n_real, a[:, 0], a[:, 1], a[:, 2])
            assert info.tolist() == stp["info"]
            assert qsl.tolist() == stp["qsl"]
            assert st["hdr"].tolist() == stp["hdr"]
            sl = np.array(stp["slots"]).reshape(-1, 2)
            assert st["slot_seq"].tolist() == sl[:, 0].tolist()
            assert st["context_lens"].tolist() == sl[:, 1].tolist()
            # block-table entries in use, slot-major
            used = [int(st["block_table"][s, p]) for s in range(S) if st["slot_seq"][s] >= 0
                    for p in range(-(-int(st["context_lens"][s]) // 16))]
            assert used == stp["bt"]


def _pages_in_use(st):
    return [(s, int(st["block_table"][s, p])) for s in range(len(st["slot_seq"]))
            if st["slot_seq"][s] >= 0 for p in range(-(-int(st["context_lens"][s]) // 16))]


def test_schedule_invariants_on_random_streams():
    """Properties every step must keep, checked on random arrival streams with
    tight page pools (so preemption happens): pages are conserved and never
    shared, every surviving decode slot gains exactly its token, preemption
    happens only when pages run short and takes the newest slots, admission
    follows the queue order, and the rows describe the step."""
    rng = np.random.default_rng(2)
    preempted_total = admitted_total = 0
    for trial in range(10):
        S, MP, Q = int(rng.integers(3, 9)), 12, 40
        P = int(rng.integers(S + 2, 4 * S + 4))
        n_real = int(rng.integers(40, 200))
        st = oracle.sched_init(S, P, MP, Q)
        next_id = 100
        expect_queue = []  # logical ids in queue order (model of the queue)
        for step in range(60):
            n = int(rng.integers(0, 3))
            ids = list(range(next_id, next_id + n)); next_id += n
            pr = rng.integers(1, 40, n)
            fin = np.minimum(pr + rng.integers(0, 60, n), MP * 16)
            prev = {k: v.copy() for k, v in st.items()}
            st, qsl, finished, info = oracle.schedule_step(st, n_real, ids, pr, fin)
            mode, n_fin, n_pre, n_adm, n_dec, n_acc = (int(x) for x in info[:6])
            expect_queue += ids[:n_acc]
            # pages: a permutation of 0..P-1 split between free stack and slots
            used = [p for _, p in _pages_in_use(st)]
            free = st["free_pages"][:st["hdr"][0]].tolist()
            assert sorted(used + free) == list(range(P))
            # finished: exactly the slots that had reached their length
            was = [s for s in range(S) if prev["slot_seq"][s] >= 0
                   and prev["context_lens"][s] >= prev["slot_fin"][s]]
            assert sorted(finished.tolist()) == sorted(int(prev["slot_seq"][s]) for s in was)
            # survivors gained one token each and kept their earlier pages
            live = [s for s in range(S) if prev["slot_seq"][s] >= 0 and s not in was]
            survivors = [s for s in live if st["slot_seq"][s] == prev["slot_seq"][s]
                         and st["slot_order"][s] == prev["slot_order"][s]]
            gone = [s for s in live if s not in survivors]
            assert len(gone) == n_pre and n_dec == len(survivors)
            for s in survivors:
                c = int(prev["context_lens"][s])
                assert st["context_lens"][s] == c + 1
                assert (st["block_table"][s, :-(-c // 16)] == prev["block_table"][s, :-(-c // 16)]).all()
                assert qsl[s + 1] - qsl[s] == 1
            if n_pre:
                assert mode == 1 and n_adm == 0
                free_before = int(prev["hdr"][0]) + sum(-(-int(prev["context_lens"][s]) // 16) for s in was)
                need = sum(1 for s in live if prev["context_lens"][s] % 16 == 0)
                assert need > free_before
                # the newest slots went, and without the youngest of them it would not fit
                assert min(prev["slot_order"][s] for s in gone) > max([prev["slot_order"][s] for s in survivors] or [-1])
                preempted_total += n_pre
                expect_queue = [int(prev["slot_seq"][s]) for s in sorted(gone)] + expect_queue
            # admitted: the queue head, in order, into the lowest empty slots
            adm = [s for s in range(S) if st["slot_seq"][s] >= 0 and s not in survivors]
            assert len(adm) == n_adm
            adm_ids = [int(st["slot_seq"][s]) for s in sorted(adm, key=lambda s: st["slot_order"][s])]
            assert adm_ids == expect_queue[:n_adm]
            expect_queue = expect_queue[n_adm:]
            admitted_total += n_adm
            assert int(st["hdr"][3]) == len(expect_queue)
            assert sum(int(st["context_lens"][s]) for s in adm) <= n_real - n_dec
            if not n_pre and st["hdr"][3] > 0:
                # admission stopped for a reason: the next entry does not fit
                nxt = int(st["queue_tok"][st["hdr"][2]])
                empty = sum(1 for s in range(S) if st["slot_seq"][s] < 0)
                adm_tok = sum(int(st["context_lens"][s]) for s in adm)
                assert (empty == 0 or adm_tok + nxt > n_real - n_dec
                        or -(-nxt // 16) > st["hdr"][0])
            for s in adm:
                assert qsl[s + 1] - qsl[s] == st["context_lens"][s]
            assert qsl[-1] == info[7] and int(st["hdr"][0]) == info[6]
    assert preempted_total > 20 and admitted_total > 100, (preempted_total, admitted_total)


def test_schedule_rejects_states_it_cannot_produce():
    S, P, MP, Q = 2, 4, 2, 5
    st = oracle.sched_init(S, P, MP, Q)
    st, *_ = oracle.schedule_step(st, 40, [10, 11, 12], [16, 5, 3], [18, 7, 4])
    assert st["hdr"].tolist() == [2, 2, 2, 1]  # id 12 waits at queue entry 2
    bad = []
    for field, idx, val in [("block_table", (0, 0), 4), ("block_table", (1, 0), -1),
                            ("context_lens", 0, 33), ("context_lens", 1, 0), ("slot_fin", 0, 33),
                            ("hdr", 0, 3), ("hdr", 2, 5), ("hdr", 3, 4), ("queue_tok", 2, 0),
                            ("queue_fin", 2, 2), ("queue_fin", 2, 33)]:
        t = {k: v.copy() for k, v in st.items()}
        t[field][idx] = val
        before = {k: v.copy() for k, v in t.items()}
        with pytest.raises(ValueError):
            oracle.schedule_step(t, 40)
        bad.append(all((before[k] == t[k]).all() for k in t))
    assert all(bad)
