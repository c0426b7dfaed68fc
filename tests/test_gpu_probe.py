"""The read-stream probe (pa_read_probe) reads exactly the bytes it is given:
its fold of the buffer equals the XOR of every 32-bit word each lane reads,
computed on the host, for sequential and permuted chunks.  (The probe times
the access pattern of the decode kernels; its result only keeps the loads
alive, but checking it shows every slice was read once.)"""
import numpy as np
import pytest

from paper_2504_09345_amd import binding as pb

from parity_util import announce

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("chunk,permute,grid,waves,depth", [
    (32768, False, 3, 8, 2), (32768, True, 5, 8, 2), (4096, True, 7, 8, 2), (32768, True, 5, 4, 2),
    (4096, False, 3, 4, 1), (32768, True, 6, 8, 1)])
def test_probe_reads_every_slice(chunk, permute, grid, waves, depth):
    import torch
    announce(f"read probe chunk={chunk} permute={permute} grid={grid} waves={waves} depth={depth}")
    n_chunks = 24
    rng = np.random.default_rng(5)
    data = rng.integers(0, 2 ** 32, size=n_chunks * chunk // 4, dtype=np.uint64).astype(np.uint32)
    buf = torch.from_numpy(data.view(np.int32)).cuda()
    offs_np = (rng.permutation(n_chunks) * chunk).astype(np.int64) if permute else None
    offs = torch.from_numpy(offs_np).cuda() if permute else None
    sink = torch.zeros(grid * 64 * waves, dtype=torch.int32, device="cuda")
    pb.pa_read_probe(buf, chunk, offs, n_chunks, grid, waves, depth, 1, sink)
    torch.cuda.synchronize()
    got = sink.cpu().numpy().view(np.uint32)
    # host model: slice j -> chunk, wave w of workgroup x takes slices
    # s0 + w, s0 + w + waves, ...; lane l reads 16 bytes at 16 l + 1024 i, i < 4
    spc = chunk // 4096
    S = spc * n_chunks
    words = data.reshape(-1)
    exp = np.zeros(grid * 64 * waves, np.uint32)
    for x in range(grid):
        s0, s1 = S * x // grid, S * (x + 1) // grid
        for w in range(waves):
            for j in range(s0 + w, s1, waves):
                c, sub = divmod(j, spc)
                base = (offs_np[c] if permute else c * chunk) + sub * 4096
                for lane in range(64):
                    acc = 0
                    for i in range(4):
                        o = (base + 16 * lane + 1024 * i) // 4
                        acc ^= int(np.bitwise_xor.reduce(words[o:o + 4]))
                    exp[(x * waves + w) * 64 + lane] ^= np.uint32(acc)
    assert np.array_equal(got, exp)


def _bf16(x):
    """Round float32 values to bfloat16 (nearest, ties to even), as float64."""
    u = np.asarray(x, np.float32).view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


@pytest.mark.parametrize("big", [0, 1])
@pytest.mark.parametrize("mode,waves", [(0, 4), (1, 4), (2, 4), (3, 8)])
def test_issue_probe_runs_the_work_it_times(big, mode, waves):
    """pa_issue_probe does the work it claims: per wave, the sum of the sink
    over its lanes equals iters x 4 products' worth of the sum of every output
    element (sum over k of A's column sum times B's row sum, with A and B the
    per-lane bf16 fills: each k is held by one lane group at one vector
    index), plus the 16 vector registers, which the FMA recurrence
    v <- 0.999 v + 0.5 moves once per iteration (4 FMAs per product), in
    closed form."""
    import torch
    announce(f"issue probe big={big} mode={mode} waves={waves}")
    grid, iters, nv, n = 3, 50, 4, 16 if big == 0 else 32
    sink = torch.full((grid * 64 * waves,), -12345.0, dtype=torch.float32, device="cuda")
    cyc = torch.zeros(grid * waves, dtype=torch.int64, device="cuda")
    pb.pa_issue_probe(grid, waves, iters, big, nv, 0, mode, sink, cyc)
    torch.cuda.synchronize()
    assert (cyc.cpu().numpy() > 0).all()  # every wave's loop timed
    got = sink.cpu().numpy().astype(np.float64).reshape(grid, waves, 64)
    t = np.arange(64 * waves, dtype=np.float64).reshape(waves, 64)
    i = np.arange(8)
    a = _bf16((t[..., None] * np.float32(0.001)).astype(np.float32) + i.astype(np.float32))  # [waves, 64, 8]
    b = _bf16((i * 0.5).astype(np.float32))
    products = iters * 4 * n * (a * b).sum(axis=(1, 2))  # per wave
    v0 = (t[..., None] * np.float32(0.01)).astype(np.float32) + np.arange(16, dtype=np.float32)  # [waves, 64, 16]
    c = float(np.float32(0.999))
    v_moved = (c ** iters * v0 + 0.5 * (1 - c ** iters) / (1 - c)).sum(axis=(1, 2))
    v_still = v0.astype(np.float64).sum(axis=(1, 2))
    w = np.arange(waves)
    has_p = {0: w >= 0, 1: w >= 0, 2: w < 0, 3: w < waves // 2}[mode]
    has_v = {0: w >= 0, 1: w < 0, 2: w >= 0, 3: w >= waves // 2}[mode]
    exp = np.where(has_p, products, 0.0) + np.where(has_v, v_moved, v_still)
    np.testing.assert_allclose(got.sum(axis=2), np.broadcast_to(exp, (grid, waves)), rtol=1e-4)


def test_issue_probe_exp_cases_run():
    import torch
    announce("issue probe exponentials")
    sink = torch.full((2 * 512,), -12345.0, dtype=torch.float32, device="cuda")
    for big, nv, mode, waves in ((0, 4, 0, 4), (1, 2, 2, 4), (1, 4, 3, 8)):
        pb.pa_issue_probe(2, waves, 20, big, nv, 1, mode, sink)
    torch.cuda.synchronize()
    assert not (sink[:2 * 64 * 8].cpu().numpy() == -12345.0).any()
