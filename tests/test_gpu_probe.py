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


@pytest.mark.parametrize("chunk,permute,grid", [(32768, False, 3), (32768, True, 5), (4096, True, 7)])
def test_probe_reads_every_slice(chunk, permute, grid):
    import torch
    announce(f"read probe chunk={chunk} permute={permute} grid={grid}")
    n_chunks = 24
    rng = np.random.default_rng(5)
    data = rng.integers(0, 2 ** 32, size=n_chunks * chunk // 4, dtype=np.uint64).astype(np.uint32)
    buf = torch.from_numpy(data.view(np.int32)).cuda()
    offs_np = (rng.permutation(n_chunks) * chunk).astype(np.int64) if permute else None
    offs = torch.from_numpy(offs_np).cuda() if permute else None
    sink = torch.zeros(grid * 512, dtype=torch.int32, device="cuda")
    pb.pa_read_probe(buf, chunk, offs, n_chunks, grid, 1, sink)
    torch.cuda.synchronize()
    got = sink.cpu().numpy().view(np.uint32)
    # host model: slice j -> chunk, wave w of workgroup x takes slices
    # s0 + w, s0 + w + 8, ...; lane l reads 16 bytes at 16 l + 1024 i, i < 4
    spc = chunk // 4096
    S = spc * n_chunks
    words = data.reshape(-1)
    exp = np.zeros(grid * 512, np.uint32)
    for x in range(grid):
        s0, s1 = S * x // grid, S * (x + 1) // grid
        for w in range(8):
            for j in range(s0 + w, s1, 8):
                c, sub = divmod(j, spc)
                base = (offs_np[c] if permute else c * chunk) + sub * 4096
                for lane in range(64):
                    acc = 0
                    for i in range(4):
                        o = (base + 16 * lane + 1024 * i) // 4
                        acc ^= int(np.bitwise_xor.reduce(words[o:o + 4]))
                    exp[x * 512 + w * 64 + lane] ^= np.uint32(acc)
    assert np.array_equal(got, exp)
