"""C ABI of libpagedattn.so on the host: the library loads, exports every entry
point the header declares, and its host-side validation and workspace
planning return the documented codes.  Validation runs before any HIP call,
so the rejected calls below enqueue nothing; they use placeholder addresses
and therefore run only where no GPU is visible (on a GPU the parity tests
exercise the same paths with real buffers)."""
import os
import re
import subprocess

import pytest

from paper_2504_09345_amd import binding as pb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pagedattn.h")
HEADERS = [os.path.join(ROOT, "include", f) for f in sorted(os.listdir(os.path.join(ROOT, "include")))
           if f.endswith(".h")]


def _gpu_visible():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:
        return False


host_only = pytest.mark.skipif(_gpu_visible(), reason="placeholder addresses: host-only check")


def _declared():
    text = "\n".join(open(h).read() for h in HEADERS)
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:int|const char \*)\s*(\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_entry_points():
    assert _declared() == sorted(pb.EXPORTED)


def test_library_exports_every_declared_symbol():
    lib = pb.load()
    for name in _declared():
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", pb.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    syms = {l.split()[-1] for l in out.splitlines() if l.strip()}
    for name in _declared():
        assert name in syms, name


def test_library_is_gfx950_only():
    # the offload bundle of our own build names its code-object targets
    blob = open(pb.LIB_PATH, "rb").read()
    targets = set(re.findall(rb"amdgcn-amd-amdhsa-+(gfx[0-9a-z]+)", blob))
    assert targets == {b"gfx950"}


def test_strerror():
    for code in (0, -1, -2, -3, -4):
        assert len(pb.pa_strerror(code)) > 5
    assert pb.pa_strerror(-99) == "unknown error code"
    assert "workspace" in pb.pa_strerror(pb.PA_ENOSPC)


def dims(**kw):
    base = dict(num_seqs=256, num_q_heads=32, num_kv_heads=8, head_dim=128, page_size=16,
                num_pages=25600, max_pages_per_seq=128, max_context_len=2048, pages_per_split=0,
                dtype=pb.PA_BF16, num_q_rows=0, max_q_len=0)
    base.update(kw)
    return pb.PaDims(**base)


def _align(x):
    return (x + 255) // 256 * 256


def _stream_ws(B, H_q, D, W=8):
    recs = 1024 * 2 * H_q  # (workgroup, slot) x (waves x group) = all query heads of a head block
    # records, (m, l), arrival counters per (first range, wave)
    return _align(recs * D * 4) + _align(recs * 2 * 4) + _align(1024 * W * 8)


def _split_ws(rows, H_q, D, max_ctx, pps):
    slots = -(-(-(-max_ctx // 16)) // pps)
    if slots <= 1:
        return 0
    items = rows * H_q * slots
    return _align(items * D * 4) + _align(items * 2 * 4)


def test_workspace_size_formula():
    # library choice: the persistent stream-K path, partial records + prefix sums
    assert pb.pa_workspace_size(dims()) == _stream_ws(256, 32, 128)
    # explicit granule: the per-row split-K path (2048 tokens = 128 pages = 4 splits of 32)
    assert pb.pa_workspace_size(dims(pages_per_split=32)) == _split_ws(256, 32, 128, 2048, 32)
    assert pb.pa_workspace_size(dims(max_context_len=512, pages_per_split=32)) == 0
    assert pb.pa_workspace_size(dims(max_context_len=512, pages_per_split=8)) > 0
    # varlen bf16: stream records for the decode rows; the MFMA prefill kernel
    # needs no workspace
    vl = dict(num_q_rows=4608, max_q_len=512, num_seqs=520, max_context_len=4096,
              max_pages_per_seq=256)
    assert pb.pa_workspace_size(dims(**vl)) == _stream_ws(520, 32, 128)
    # varlen fp32: chunk rows take the per-row split-K kernel
    assert pb.pa_workspace_size(dims(dtype=pb.PA_FP32, **vl)) == (
        _stream_ws(520, 32, 128) + _split_ws(4608, 32, 128, 4096, 128))
    # too many sequences for the stream path's tables: split-K
    big = dims(num_seqs=9000)
    assert pb.pa_workspace_size(big) == _split_ws(9000, 32, 128, 2048, 128)
    assert pb.pa_workspace_size(dims(num_seqs=0)) >= 0


@pytest.mark.parametrize("kw,code", [
    (dict(num_q_heads=30), pb.PA_EINVAL),           # H_q not a multiple of H_kv
    (dict(num_seqs=-1), pb.PA_EINVAL),
    (dict(num_kv_heads=0), pb.PA_EINVAL),
    (dict(head_dim=96), pb.PA_ENOTSUP),
    (dict(page_size=32), pb.PA_ENOTSUP),
    (dict(dtype=7), pb.PA_ENOTSUP),
    (dict(num_q_heads=24, num_kv_heads=8), pb.PA_ENOTSUP),  # group of 3
    (dict(max_pages_per_seq=100), pb.PA_EINVAL),    # row too short for max_context_len
    (dict(max_context_len=-5), pb.PA_EINVAL),
    (dict(pages_per_split=10000), pb.PA_EINVAL),
    (dict(pages_per_split=-1), pb.PA_EINVAL),
])
def test_workspace_size_rejects(kw, code):
    with pytest.raises(pb.PagedAttnError) as e:
        pb.pa_workspace_size(dims(**kw))
    assert e.value.code == code


FAKE = 0x1000  # never dereferenced: every call below fails validation first


@host_only
@pytest.mark.parametrize("case", ["null_q", "null_out", "bad_group", "small_ws", "no_ws",
                                  "nan_scale", "zero_scale", "neg_scale", "decode_rows",
                                  "decode_qlen", "hd"])
def test_paged_attn_validation(case):
    d = dims()
    args = dict(q=FAKE, k=FAKE, v=FAKE, bt=FAKE, cl=FAKE, scale=0.088, out=FAKE, ws=FAKE,
                ws_bytes=pb.pa_workspace_size(d))
    expect = pb.PA_EINVAL
    if case == "null_q":
        args["q"] = None
    elif case == "null_out":
        args["out"] = None
    elif case == "bad_group":
        d.num_q_heads = 20
    elif case == "small_ws":
        args["ws_bytes"] -= 1
        expect = pb.PA_ENOSPC
    elif case == "no_ws":
        args["ws"] = None
        expect = pb.PA_ENOSPC
    elif case == "nan_scale":
        args["scale"] = float("nan")
    elif case == "zero_scale":
        args["scale"] = 0.0
    elif case == "neg_scale":
        args["scale"] = -0.088
    elif case == "decode_rows":
        d.num_q_rows = 7
    elif case == "decode_qlen":
        d.max_q_len = 3
    elif case == "hd":
        d.head_dim = 256
        expect = pb.PA_ENOTSUP
    lib = pb.load()
    import ctypes
    rc = lib.paged_attn(args["q"], args["k"], args["v"], args["bt"], args["cl"], args["scale"],
                        args["out"], ctypes.byref(d), args["ws"], args["ws_bytes"], None, None)
    assert rc == expect


@host_only
@pytest.mark.parametrize("case", ["null_qsl", "rows_without_qlen", "qlen_over_ctx", "small_ws"])
def test_paged_attn_varlen_validation(case):
    import ctypes
    d = dims(num_seqs=520, num_q_rows=4608, max_q_len=512, max_context_len=4096,
             max_pages_per_seq=256)
    qsl, ws_bytes, expect = FAKE, pb.pa_workspace_size(d), pb.PA_EINVAL
    if case == "null_qsl":
        qsl = None
    elif case == "rows_without_qlen":
        d.max_q_len = 0
        ws_bytes = 1 << 40
    elif case == "qlen_over_ctx":
        d.max_q_len = 5000
        ws_bytes = 1 << 40
    elif case == "small_ws":
        ws_bytes -= 256
        expect = pb.PA_ENOSPC
    rc = pb.load().paged_attn_varlen(FAKE, FAKE, FAKE, FAKE, FAKE, qsl, 0.088, FAKE,
                                     ctypes.byref(d), FAKE, ws_bytes, None, None)
    assert rc == expect


@host_only
def test_gather_trace_validation():
    import ctypes
    lib = pb.load()

    def call(d, q=FAKE, qsl=None, rows=FAKE, ws_bytes=None, scale=0.088):
        ws_bytes = pb.pa_workspace_size(d) if ws_bytes is None else ws_bytes
        return lib.pa_gather_trace(q, FAKE, FAKE, FAKE, FAKE, qsl, scale, FAKE, ctypes.byref(d), FAKE,
                                   ws_bytes, rows, None)
    assert call(dims(), q=None) == pb.PA_EINVAL
    assert call(dims(), rows=None) == pb.PA_EINVAL
    assert call(dims(), scale=0.0) == pb.PA_EINVAL
    assert call(dims(), ws_bytes=100) == pb.PA_ENOSPC
    assert call(dims(page_size=8), ws_bytes=0) == pb.PA_ENOTSUP
    assert call(dims(max_pages_per_seq=3), ws_bytes=0) == pb.PA_EINVAL
    assert lib.pa_gather_trace(FAKE, FAKE, FAKE, FAKE, FAKE, None, 0.088, FAKE, None, FAKE, 0, FAKE,
                               None) == pb.PA_EINVAL
    # varlen trace: the varlen call's validation
    vd = dims(num_seqs=520, num_q_rows=4608, max_q_len=0, max_context_len=4096, max_pages_per_seq=256)
    assert call(vd, qsl=FAKE, ws_bytes=1 << 40) == pb.PA_EINVAL
    # nothing to trace: success without touching the pointers
    d4 = dims(num_seqs=0)
    assert lib.pa_gather_trace(None, None, None, None, None, None, 0.088, None, ctypes.byref(d4), None, 0,
                               None, None) == pb.PA_OK


@host_only
@pytest.mark.parametrize("dtype,D", [(pb.PA_FP32, 128), (pb.PA_BF16, 64), (pb.PA_FP32, 64)])
def test_varlen_all_single_rows_fit_the_sized_workspace(dtype, D):
    """A varlen call whose rows are all decode rows (every L_b = 1) is planned
    like the decode call: the stream kernel takes every row, so no split-K
    partials are reserved, also where the chunk kernel does not apply (fp32,
    head_dim 64) and contexts exceed one split granule.  Validation must pass
    with exactly pa_workspace_size() bytes (it then reaches the first HIP call,
    which fails where no GPU is visible)."""
    import ctypes
    d = dims(dtype=dtype, head_dim=D, num_seqs=64, num_q_rows=64, max_q_len=1, max_context_len=4096,
             max_pages_per_seq=256)
    need = pb.pa_workspace_size(d)
    dec = dims(dtype=dtype, head_dim=D, num_seqs=64, max_context_len=4096, max_pages_per_seq=256)
    assert need == pb.pa_workspace_size(dec)
    rc = pb.load().paged_attn_varlen(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 0.088, FAKE, ctypes.byref(d),
                                     FAKE, need, None, None)
    assert rc == pb.PA_EHIP
    # the same call with chunk rows reserves split-K partials (fp32 / D 64
    # chunk rows take the per-row kernel)
    d.num_q_rows, d.max_q_len = 128, 2
    assert pb.pa_workspace_size(d) > need


@host_only
@pytest.mark.parametrize("case", ["null_q", "null_qsl", "nan_scale", "bad_group", "rows_without_qlen"])
def test_noalloc_validation(case):
    """The no-allocation entry validates like paged_attn_varlen on the host,
    before it touches a device."""
    import ctypes
    d = dims(num_seqs=520, num_q_rows=4608, max_q_len=512, max_context_len=4096, max_pages_per_seq=256)
    q, qsl, scale = FAKE, FAKE, 0.088
    if case == "null_q":
        q = None
    elif case == "null_qsl":
        qsl = None
    elif case == "nan_scale":
        scale = float("nan")
    elif case == "bad_group":
        d.num_q_heads = 20
    elif case == "rows_without_qlen":
        d.max_q_len = 0
    rc = pb.load().paged_attn_varlen_noalloc(q, FAKE, FAKE, FAKE, FAKE, qsl, scale, FAKE, ctypes.byref(d),
                                             None, None)
    assert rc == pb.PA_EINVAL


@host_only
def test_read_probe_validation():
    lib = pb.load()
    assert lib.pa_read_probe(None, 4096, None, 1, 1, 8, 2, 1, FAKE, None) == pb.PA_EINVAL
    assert lib.pa_read_probe(FAKE, 4096, None, 1, 1, 8, 2, 1, None, None) == pb.PA_EINVAL
    assert lib.pa_read_probe(FAKE, 1000, None, 1, 1, 8, 2, 1, FAKE, None) == pb.PA_EINVAL
    assert lib.pa_read_probe(FAKE, 0, None, 1, 1, 8, 2, 1, FAKE, None) == pb.PA_EINVAL
    assert lib.pa_read_probe(FAKE, 4096, None, -1, 1, 8, 2, 1, FAKE, None) == pb.PA_EINVAL
    assert lib.pa_read_probe(FAKE, 4096, None, 1, 0, 8, 2, 1, FAKE, None) == pb.PA_EINVAL
    assert lib.pa_read_probe(FAKE, 4096, None, 1, 70000, 8, 2, 1, FAKE, None) == pb.PA_EINVAL
    for waves in (0, 2, 6, 16):
        assert lib.pa_read_probe(FAKE, 4096, None, 1, 1, waves, 2, 1, FAKE, None) == pb.PA_EINVAL
    assert lib.pa_read_probe(FAKE, 3 * 4096, None, 1, 1, 8, 2, 1, FAKE, None) == pb.PA_EINVAL
    for depth in (0, 3, -1):
        assert lib.pa_read_probe(FAKE, 4096, None, 1, 1, 8, depth, 1, FAKE, None) == pb.PA_EINVAL


@host_only
def test_empty_batch_is_a_no_op():
    import ctypes
    d = dims(num_seqs=0, max_context_len=0)
    assert pb.load().paged_attn(None, None, None, None, None, 1.0, None, ctypes.byref(d), None, 0,
                                None, None) == pb.PA_OK


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(pb, "_lib", None)
    monkeypatch.setattr(pb, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(RuntimeError, match="no fallback"):
        pb.load()


@host_only
@pytest.mark.parametrize("case", ["null_dims", "null_knew", "null_pool", "fp16", "hd", "page",
                                  "table_short", "decode_rows", "neg_rows", "rows_no_seqs"])
def test_kv_append_validation(case):
    import ctypes
    d = dims()
    args = dict(kn=FAKE, vn=FAKE, bt=FAKE, cl=FAKE, qsl=None, kp=FAKE, vp=FAKE)
    expect = pb.PA_EINVAL
    if case == "null_knew":
        args["kn"] = None
    elif case == "null_pool":
        args["vp"] = None
    elif case == "fp16":
        d.dtype = 7
        expect = pb.PA_ENOTSUP
    elif case == "hd":
        d.head_dim = 96
        expect = pb.PA_ENOTSUP
    elif case == "page":
        d.page_size = 32
        expect = pb.PA_ENOTSUP
    elif case == "table_short":
        d.max_pages_per_seq = 100
    elif case == "decode_rows":
        d.num_q_rows = 7
    elif case == "neg_rows":
        args["qsl"] = FAKE
        d.num_q_rows = -1
    elif case == "rows_no_seqs":
        args["qsl"] = FAKE
        d.num_seqs, d.num_q_rows = 0, 5
    lib = pb.load()
    rc = lib.pa_kv_append(args["kn"], args["vn"], args["bt"], args["cl"], args["qsl"], args["kp"],
                          args["vp"], None if case == "null_dims" else ctypes.byref(d), None)
    assert rc == expect


@host_only
def test_kv_append_without_rows_touches_nothing():
    import ctypes
    lib = pb.load()
    d = dims(num_seqs=0)
    assert lib.pa_kv_append(None, None, None, None, None, None, None, ctypes.byref(d), None) == pb.PA_OK
    d = dims(num_q_rows=0)
    assert lib.pa_kv_append(None, None, None, None, FAKE, None, None, ctypes.byref(d), None) == pb.PA_OK


def _sched_state(S=4, P=8, MP=2, Q=8):
    st = pb.PaSchedState(**{n: FAKE for n in pb.SCHED_ARRAYS})
    st.num_slots, st.num_pages, st.max_pages_per_seq, st.queue_cap = S, P, MP, Q
    return st


@host_only
@pytest.mark.parametrize("case", ["null_state", "null_hdr", "null_info", "no_slots", "queue_small",
                                  "neg_pages", "no_table", "neg_budget", "neg_arrivals",
                                  "null_arrivals", "too_many_slots", "int32_range"])
def test_schedule_step_validation(case):
    import ctypes
    st = _sched_state()
    args = dict(n_real=64, ns=FAKE, npr=FAKE, nf=FAKE, n_new=2, qsl=FAKE, fin=FAKE, info=FAKE)
    expect = pb.PA_EINVAL
    if case == "null_hdr":
        st.hdr = None
    elif case == "null_info":
        args["info"] = None
    elif case == "no_slots":
        st.num_slots = 0
    elif case == "queue_small":
        st.queue_cap = st.num_slots
    elif case == "neg_pages":
        st.num_pages = -1
    elif case == "no_table":
        st.max_pages_per_seq = 0
    elif case == "neg_budget":
        args["n_real"] = -1
    elif case == "neg_arrivals":
        args["n_new"] = -1
    elif case == "null_arrivals":
        args["npr"] = None
    elif case == "too_many_slots":
        st.num_slots, st.queue_cap = 8193, 9000
        expect = pb.PA_ENOTSUP
    elif case == "int32_range":
        st.num_slots, st.queue_cap, st.max_pages_per_seq = 4096, 5000, 1 << 16
    lib = pb.load()
    rc = lib.pa_schedule_step(None if case == "null_state" else ctypes.byref(st), args["n_real"],
                              args["ns"], args["npr"], args["nf"], args["n_new"], args["qsl"],
                              args["fin"], args["info"], None)
    assert rc == expect


def test_issue_probe_validation():
    lib = pb.load()
    ok = dict(grid=1, waves=4, iters=1, big=0, nv=2, exp2=0, mode=0, sink=FAKE)

    def call(**kw):
        a = {**ok, **kw}
        return lib.pa_issue_probe(a["grid"], a["waves"], a["iters"], a["big"], a["nv"], a["exp2"], a["mode"],
                                  a["sink"], None, None)

    for bad in (dict(sink=None), dict(waves=3), dict(waves=16), dict(iters=0), dict(grid=0), dict(grid=70000),
                dict(mode=4), dict(mode=-1), dict(mode=3, waves=1), dict(nv=5), dict(nv=17), dict(nv=-1)):
        assert call(**bad) == pb.PA_EINVAL, bad
