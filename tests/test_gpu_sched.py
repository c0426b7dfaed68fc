"""GPU parity of the scheduler step (pa_schedule_step) against the oracle's
step: the two run in lockstep on the same seeded arrival streams and every
array of the state, the rows (query_start_loc), the finished ids and the step
summary must be bit-identical after every step.  Covers the hand-derived
fixture, every slots-per-thread variant of the kernel, preemption-heavy pools,
the paper's three length mixes, rejected states, and the scheduler feeding the
KV append and the attention of the pass."""
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2504_09345_amd import binding as pb
from paper_2504_09345_amd import workloads as W

from parity_util import announce, assert_parity

pytestmark = pytest.mark.gpu

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


class GpuSched:
    """Device copy of a scheduler state plus the step's output buffers."""

    def __init__(self, st):
        self.arrays = {k: torch.from_numpy(np.ascontiguousarray(st[k])).cuda() for k in oracle.SCHED_FIELDS}
        self.c = pb.make_sched_state(self.arrays)
        S = st["block_table"].shape[0]
        self.qsl = torch.zeros(S + 1, dtype=torch.int32, device="cuda")
        self.fin = torch.zeros(S, dtype=torch.int32, device="cuda")
        self.info = torch.zeros(8, dtype=torch.int32, device="cuda")

    def step(self, n_real, ids=(), prompts=(), fins=()):
        n = len(ids)
        dev = [torch.from_numpy(np.ascontiguousarray(x, np.int32)).cuda() if n else None
               for x in (ids, prompts, fins)]
        pb.pa_schedule_step(self.c, n_real, *dev, n, self.qsl, self.fin, self.info)
        torch.cuda.synchronize()
        info = self.info.cpu().numpy()
        return self.qsl.cpu().numpy(), self.fin.cpu().numpy()[:max(info[1], 0)], info

    def host(self):
        return {k: v.cpu().numpy() for k, v in self.arrays.items()}


def _same_state(gpu_st, ref_st, what):
    for k in oracle.SCHED_FIELDS:
        assert np.array_equal(gpu_st[k], ref_st[k]), f"{what}: {k} differs"


def _lockstep(S, P, MP, Q, n_real, mix, steps, per_step, seed, check_every=1):
    announce(f"scheduler lockstep S={S} P={P} MP={MP} Q={Q} n_real={n_real} mix={mix} seed={seed}")
    st = oracle.sched_init(S, P, MP, Q)
    g = GpuSched(st)
    totals = np.zeros(8, np.int64)
    for i, (ids, pr, fn) in enumerate(W.arrival_stream(mix, steps, per_step, seed)):
        fn = np.minimum(fn, MP * 16)
        st, eq, ef, ei = oracle.schedule_step(st, n_real, ids, pr, fn)
        q, f, info = g.step(n_real, ids, pr, fn)
        what = f"step {i}"
        assert info.tolist() == ei.tolist(), f"{what}: info {info} != {ei}"
        assert np.array_equal(q, eq), f"{what}: query_start_loc"
        assert np.array_equal(f, ef), f"{what}: finished ids"
        if i % check_every == 0 or i == steps - 1:
            _same_state(g.host(), st, what)
        totals += ei
    return totals


def test_hand_fixture_on_gpu():
    from test_oracle_pins import _read_schedule_fixture
    for sc in _read_schedule_fixture():
        S, P, MP, Q, n_real = sc["dims"]
        announce(f"scheduler fixture S={S} P={P}")
        st = oracle.sched_init(S, P, MP, Q)
        g = GpuSched(st)
        for stp in sc["steps"]:
            a = np.array(stp["arrivals"], np.int32).reshape(-1, 3)
            st, eq, ef, ei = oracle.schedule_step(st, n_real, a[:, 0], a[:, 1], a[:, 2])
            q, f, info = g.step(n_real, a[:, 0], a[:, 1], a[:, 2])
            assert info.tolist() == stp["info"]
            assert q.tolist() == stp["qsl"]
            hs = g.host()
            assert hs["hdr"].tolist() == stp["hdr"]
            _same_state(hs, st, "fixture")


@pytest.mark.parametrize("S,P,MP,Q,n_real,mix,steps,rate", [
    (8, 20, 8, 24, 120, "tiny", 80, 0.8),              # tiny pool: frequent preemption
    (256, 900, 45, 600, 2048, "mtbench-g256", 160, 12),  # one slot per thread
    (1500, 6000, 45, 3200, 8192, "mtbench-g128", 60, 80),  # two per thread
    (3000, 9000, 45, 6500, 16384, "mtbench-g32", 50, 160),  # four per thread
    (8192, 30000, 45, 17000, 32768, "mtbench-g32", 40, 500),  # eight per thread
    (64, 2500, 125, 200, 4096, "rag", 80, 2),            # long prompts
    (128, 2200, 60, 300, 2048, "aime", 150, 3),          # long generations
])
def test_lockstep_parity(S, P, MP, Q, n_real, mix, steps, rate):
    t = _lockstep(S, P, MP, Q, n_real, mix, steps, rate, seed=S + steps)
    # every scenario exercises admission, decode and garbage collection
    assert t[3] > 0 and t[4] > 0 and t[1] > 0, t


def test_preemption_paths_are_exercised():
    """A pool far too small for the decode set: many preemption steps, each
    bit-identical to the oracle's (the re-queued entries, their order, the
    pages pushed and popped)."""
    t = _lockstep(48, 60, 20, 120, 600, "tiny", 200, 1.5, seed=5)
    assert t[2] >= 10, t


def test_no_arrivals_and_full_queue():
    """Steps without arrivals, and arrivals refused because the queue keeps
    room for preemption."""
    S, P, MP, Q = 4, 12, 4, 7
    st = oracle.sched_init(S, P, MP, Q)
    g = GpuSched(st)
    rng = np.random.default_rng(3)
    for i in range(30):
        n = int(rng.integers(0, 5)) if i % 3 else 0
        ids = np.arange(100 * i, 100 * i + n, dtype=np.int32)
        pr = rng.integers(1, 30, n).astype(np.int32)
        fn = np.minimum(pr + rng.integers(0, 20, n), MP * 16).astype(np.int32)
        if n:
            pr[0] = 0  # an invalid arrival is dropped by both
        st, eq, ef, ei = oracle.schedule_step(st, 50, ids, pr, fn)
        q, f, info = g.step(50, ids, pr, fn)
        assert info.tolist() == ei.tolist() and np.array_equal(q, eq) and np.array_equal(f, ef)
        _same_state(g.host(), st, f"step {i}")


def test_rejected_states_change_nothing():
    S, P, MP, Q = 2, 4, 2, 5
    st = oracle.sched_init(S, P, MP, Q)
    st, *_ = oracle.schedule_step(st, 40, [10, 11, 12], [16, 5, 3], [18, 7, 4])
    for field, idx, val in [("context_lens", 0, 33), ("context_lens", 1, 0), ("slot_fin", 0, 33),
                            ("hdr", 0, 3), ("hdr", 0, -1), ("hdr", 2, 5), ("hdr", 3, 4),
                            ("queue_tok", 2, 0), ("queue_fin", 2, 2), ("queue_fin", 2, 33)]:
        announce(f"scheduler rejects {field}[{idx}]={val}")
        bad = {k: v.copy() for k, v in st.items()}
        bad[field][idx] = val
        with pytest.raises(ValueError):
            oracle.schedule_step(bad, 40)
        g = GpuSched(bad)
        _, _, info = g.step(40, [20], [3], [5])
        assert info.tolist() == [-1, 0, 0, 0, 0, 0, 0, 0]
        _same_state(g.host(), bad, f"{field} rejected")


def test_scheduler_feeds_append_and_attention():
    """The pass the scheduler builds runs through the KV append and the
    varlen attention: pools bit-identical to the oracle's append, attention
    within tolerance of the oracle's, for every step of a stream with
    admissions, decodes, finishes and preemptions."""
    S, P, MP, Q, n_real = 12, 24, 8, 40, 160
    H_q, H_kv, D = 8, 2, 128
    st = oracle.sched_init(S, P, MP, Q)
    g = GpuSched(st)
    rng = np.random.default_rng(21)
    k_pool = W.f32_to_bf16_bits(rng.standard_normal((P, H_kv, 16, D)).astype(np.float32))
    v_pool = W.f32_to_bf16_bits(rng.standard_normal((P, H_kv, 16, D)).astype(np.float32))

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()

    dk, dv = bf(k_pool), bf(v_pool)
    preempted = 0
    for i, (ids, pr, fn) in enumerate(W.arrival_stream("tiny", 60, 1.0, 8)):
        fn = np.minimum(fn, MP * 16)
        st, eq, ef, ei = oracle.schedule_step(st, n_real, ids, pr, fn)
        q_loc, f, info = g.step(n_real, ids, pr, fn)
        assert info.tolist() == ei.tolist() and np.array_equal(q_loc, eq)
        preempted += int(ei[2])
        T = int(eq[-1])
        if T == 0:
            continue
        announce(f"scheduler pass {i}: rows={T} info={ei.tolist()}")
        kn = W.f32_to_bf16_bits(rng.standard_normal((T, H_kv, D)).astype(np.float32))
        vn = W.f32_to_bf16_bits(rng.standard_normal((T, H_kv, D)).astype(np.float32))
        q = W.f32_to_bf16_bits(rng.standard_normal((T, H_q, D)).astype(np.float32))
        k_pool, v_pool = oracle.kv_append(kn, vn, st["block_table"], st["context_lens"], k_pool, v_pool,
                                          query_start_loc=eq)
        ref = oracle.paged_attn_varlen(q, k_pool, v_pool, st["block_table"], st["context_lens"], eq,
                                       1.0 / np.sqrt(D))
        bt, cl = g.arrays["block_table"], g.arrays["context_lens"]
        dq = bf(q)
        dims = pb.make_dims(dq, dk, bt, MP * 16, num_q_rows=T, max_q_len=int(np.diff(eq).max()))
        pb.pa_kv_append(bf(kn), bf(vn), bt, cl, dk, dv, dims, query_start_loc=g.qsl)
        out = torch.empty_like(dq)
        pb.paged_attn_varlen(dq, dk, dv, bt, cl, g.qsl, 1.0 / np.sqrt(D), out, dims)
        torch.cuda.synchronize()
        assert np.array_equal(dk.cpu().view(torch.int16).numpy().view(np.uint16), k_pool)
        assert np.array_equal(dv.cpu().view(torch.int16).numpy().view(np.uint16), v_pool)
        # decode rows to the strict floor; chunk rows (fp16 P and V on the
        # matrix cores) to the relative bound, like every chunk test
        got, qlen = out.float().cpu().numpy(), np.diff(eq)
        dec = np.repeat(qlen == 1, qlen)
        assert_parity(got[dec], ref[dec], what=f"pass {i}, decode rows")
        assert_parity(got[~dec], ref[~dec], strict=False, what=f"pass {i}, chunk rows")
    assert preempted > 0
