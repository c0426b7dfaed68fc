"""paged_attn_varlen_noalloc (the no-allocation entry point, for callers that
cannot allocate: graph capture, tight serving loops) against
paged_attn_varlen with a caller-owned workspace, through the C ABI: two
calls in a row, the second on a smaller batch, each bit-identical to the
workspace entry (the same kernels, the same arithmetic) and within the
oracle's tolerance; a decode batch through query_start_loc = 0..B; and a call
that needs more than the fixed scratch is rejected with nothing written."""
import ctypes

import numpy as np
import pytest

from paper_2504_09345_amd import binding as pb
from paper_2504_09345_amd import workloads as W

from parity_util import announce, assert_parity, run_oracle, upload

pytestmark = pytest.mark.gpu


def _dims(b, dev):
    return pb.make_dims(dev["q"], dev["k"], dev["bt"], int(b.context_lens.max()),
                        num_q_rows=b.num_q_rows, max_q_len=int(b.q_lens.max()))


def _both(b):
    """(no-allocation output, workspace-entry output) as float32 arrays."""
    import torch
    dev = upload(b)
    if "qsl" not in dev:
        dev["qsl"] = torch.arange(b.num_seqs + 1, dtype=torch.int32, device="cuda")
    dims = _dims(b, dev)
    if b.query_start_loc is None:
        dims.num_q_rows, dims.max_q_len = b.num_seqs, 1
    out_n = torch.full_like(dev["q"], float("nan"))
    out_w = torch.full_like(dev["q"], float("nan"))
    lib = pb.load()
    rc = lib.paged_attn_varlen_noalloc(dev["q"].data_ptr(), dev["k"].data_ptr(), dev["v"].data_ptr(),
                                       dev["bt"].data_ptr(), dev["cl"].data_ptr(), dev["qsl"].data_ptr(),
                                       ctypes.c_float(b.scale), out_n.data_ptr(), ctypes.byref(dims),
                                       None, None)
    assert rc == pb.PA_OK, pb.pa_strerror(rc)
    pb.paged_attn_varlen(dev["q"], dev["k"], dev["v"], dev["bt"], dev["cl"], dev["qsl"], b.scale, out_w,
                         dims)
    torch.cuda.synchronize()
    return out_n.float().cpu().numpy(), out_w.float().cpu().numpy()


def test_noalloc_matches_the_workspace_entry_twice_then_smaller():
    big = W.generate("mixed", seed=5, overrides=dict(prefill=(3, 200, 0, 900), decode=(300, 200, 3000)))
    small = W.generate("mixed", seed=6, overrides=dict(prefill=(1, 40, 0, 100), decode=(12, 1, 400)))
    for name, b in (("first, larger", big), ("second, smaller", small)):
        announce(f"no-alloc entry: {name} batch rows={b.num_q_rows}")
        got, ref_ws = _both(b)
        assert np.array_equal(got.view(np.uint32), ref_ws.view(np.uint32)), name
        assert_parity(got, run_oracle(b), strict=False, what=f"no-alloc {name}")


def test_noalloc_decode_batch():
    announce("no-alloc entry: decode batch via query_start_loc = 0..B")
    b = W.generate("mixtral-256", seed=7, overrides=dict(B=64, ctx=("uniform", 1, 3000)))
    got, ref_ws = _both(b)
    assert np.array_equal(got.view(np.uint32), ref_ws.view(np.uint32))
    assert_parity(got, run_oracle(b), what="no-alloc decode")


def test_noalloc_rejects_calls_beyond_the_scratch():
    """fp32 chunk rows take the split-K kernel, whose partials here need
    2,048 rows x 32 heads x 2 splits x 130 floats = 68 MB > 32 MiB: rejected,
    nothing enqueued, the output untouched."""
    import torch
    announce("no-alloc entry: rejection beyond the scratch")
    chunks = [(512, 1800)] * 4
    ctx = [L + p for L, p in chunks]
    b = W.generate("tiny", seed=8, dtype="fp32", overrides=dict(H_q=32, H_kv=8, D=128, ctx=("list", ctx),
                                                                pool=("factor", 1.2)))
    q = W._fill_normal((2048, 32, 128), 8, "q", 1.0, "fp32", 1)
    qsl = np.array([0, 512, 1024, 1536, 2048], np.int32)
    b = W.Batch(**{**b.__dict__, "q": q, "query_start_loc": qsl})
    dev = upload(b)
    dims = _dims(b, dev)
    assert pb.pa_workspace_size(dims) > (32 << 20)
    out = torch.full_like(dev["q"], 7.0)
    rc = pb.load().paged_attn_varlen_noalloc(dev["q"].data_ptr(), dev["k"].data_ptr(), dev["v"].data_ptr(),
                                             dev["bt"].data_ptr(), dev["cl"].data_ptr(), dev["qsl"].data_ptr(),
                                             ctypes.c_float(b.scale), out.data_ptr(), ctypes.byref(dims),
                                             None, None)
    torch.cuda.synchronize()
    assert rc == pb.PA_ENOSPC
    assert bool((out == 7.0).all())
