"""ctypes binding of libpagedattn.so, the C ABI declared in include/pagedattn.h.

Argument marshalling only: every step of the attention runs in the library's
HIP kernels.  Device buffers are passed as torch tensors (torch provides
device memory and streams here) or as raw integer device addresses.  The
library is loaded on first use; if it has not been built the call raises
instead of falling back to anything else.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
# PAGEDATTN_LIB selects another build of the same library (e.g. one compiled
# with different tuning macros); default: the in-tree build.
LIB_PATH = os.environ.get("PAGEDATTN_LIB") or os.path.join(HERE, "_lib", "libpagedattn.so")

PA_OK, PA_EINVAL, PA_ENOTSUP, PA_ENOSPC, PA_EHIP = 0, -1, -2, -3, -4
PA_BF16, PA_FP32 = 0, 1
PAGE_SIZE = 16

EXPORTED = ("pa_workspace_size", "paged_attn", "paged_attn_varlen", "paged_attn_varlen_noalloc",
            "pa_gather_trace",
            "pa_kv_append", "pa_schedule_step", "pa_perf_model", "pa_read_probe", "pa_issue_probe",
            "pa_strerror")


class PaDims(ctypes.Structure):
    """pa_dims_t"""
    _fields_ = [(n, ctypes.c_int32) for n in (
        "num_seqs", "num_q_heads", "num_kv_heads", "head_dim", "page_size", "num_pages",
        "max_pages_per_seq", "max_context_len", "pages_per_split", "dtype", "num_q_rows",
        "max_q_len")]


class PaTiming(ctypes.Structure):
    """pa_timing_t: three hipEvent_t handles (NULL = not recorded)."""
    _fields_ = [("attn_begin", ctypes.c_void_p), ("attn_end", ctypes.c_void_p),
                ("reduce_end", ctypes.c_void_p)]


SCHED_ARRAYS = ("free_pages", "hdr", "queue_seq", "queue_tok", "queue_fin", "slot_seq",
                "slot_order", "slot_fin", "context_lens", "block_table")


class PaSchedState(ctypes.Structure):
    """pa_sched_state_t: ten device array pointers, then four sizes."""
    _fields_ = [(n, ctypes.c_void_p) for n in SCHED_ARRAYS] + [
        (n, ctypes.c_int32) for n in ("num_slots", "num_pages", "max_pages_per_seq", "queue_cap")]


def make_sched_state(arrays) -> PaSchedState:
    """pa_sched_state_t from a mapping of the ten int32 device arrays (torch
    tensors or addresses); the sizes come from their shapes."""
    bt = arrays["block_table"]
    st = PaSchedState(**{n: _addr(arrays[n]) for n in SCHED_ARRAYS})
    st.num_slots, st.max_pages_per_seq = int(bt.shape[0]), int(bt.shape[1])
    st.num_pages = int(arrays["free_pages"].shape[0])
    st.queue_cap = int(arrays["queue_seq"].shape[0])
    return st


PM_INPUT_DOUBLES = ("num_experts", "top_k", "model_dim", "expert_dim", "gqa_group", "model_bytes",
                    "kv_bytes_per_token", "gemm_flops", "io_bw", "kv_capacity_bytes", "attn_bw",
                    "attn_intensity", "batch")
PM_INPUT_INTS = ("prompt", "gen", "block")
PM_OUTPUTS = ("intensity_per_token", "tokens_to_saturate", "pme", "delta", "kv_tokens", "t_gpu",
              "t_max", "mem_bw", "kv_bw", "attn_flops", "kv_effective", "kv_blocks", "q",
              "decode_seqs", "t1", "t_prefill", "iterations", "t2", "t", "attn_headroom",
              "delta_eff", "t_attn_bound")


class PaPmInput(ctypes.Structure):
    """pa_pm_input_t (include/pa_perf_model.h)"""
    _fields_ = [(n, ctypes.c_double) for n in PM_INPUT_DOUBLES] + [(n, ctypes.c_int32) for n in PM_INPUT_INTS]


class PaPmOutput(ctypes.Structure):
    """pa_pm_output_t"""
    _fields_ = [(n, ctypes.c_double) for n in PM_OUTPUTS]


class PagedAttnError(RuntimeError):
    def __init__(self, fn, code):
        super().__init__(f"{fn} returned {code}: {pa_strerror(code)}")
        self.code = code


_lib = None


def load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() "
                           "(there is no fallback path)")
    lib = ctypes.CDLL(LIB_PATH)
    P, SZ = ctypes.c_void_p, ctypes.c_size_t
    DP, TP = ctypes.POINTER(PaDims), ctypes.POINTER(PaTiming)
    lib.pa_workspace_size.argtypes = [DP, ctypes.POINTER(SZ)]
    lib.pa_workspace_size.restype = ctypes.c_int
    lib.paged_attn.argtypes = [P, P, P, P, P, ctypes.c_float, P, DP, P, SZ, P, TP]
    lib.paged_attn.restype = ctypes.c_int
    lib.paged_attn_varlen.argtypes = [P, P, P, P, P, P, ctypes.c_float, P, DP, P, SZ, P, TP]
    lib.paged_attn_varlen.restype = ctypes.c_int
    lib.paged_attn_varlen_noalloc.argtypes = [P, P, P, P, P, P, ctypes.c_float, P, DP, P, TP]
    lib.paged_attn_varlen_noalloc.restype = ctypes.c_int
    lib.pa_gather_trace.argtypes = [P, P, P, P, P, P, ctypes.c_float, P, DP, P, SZ, P, P]
    lib.pa_gather_trace.restype = ctypes.c_int
    lib.pa_kv_append.argtypes = [P, P, P, P, P, P, P, DP, P]
    lib.pa_kv_append.restype = ctypes.c_int
    lib.pa_schedule_step.argtypes = [ctypes.POINTER(PaSchedState), ctypes.c_int32, P, P, P,
                                     ctypes.c_int32, P, P, P, P]
    lib.pa_schedule_step.restype = ctypes.c_int
    lib.pa_perf_model.argtypes = [ctypes.POINTER(PaPmInput), ctypes.POINTER(PaPmOutput)]
    lib.pa_perf_model.restype = ctypes.c_int
    lib.pa_read_probe.argtypes = [P, ctypes.c_int64, P, ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32,
                                  ctypes.c_int32, P, P]
    lib.pa_read_probe.restype = ctypes.c_int
    lib.pa_issue_probe.argtypes = [ctypes.c_int32] * 7 + [P, P, P]
    lib.pa_issue_probe.restype = ctypes.c_int
    lib.pa_strerror.argtypes = [ctypes.c_int]
    lib.pa_strerror.restype = ctypes.c_char_p
    _lib = lib
    return lib


def _addr(x):
    """Device address of a torch tensor, an int address, or None (NULL)."""
    if x is None:
        return None
    if isinstance(x, int):
        return x or None
    return x.data_ptr() or None


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream or None
    if isinstance(stream, int):
        return stream or None
    return stream.cuda_stream or None


def _dtype_code(t):
    import torch
    if t.dtype == torch.bfloat16:
        return PA_BF16
    if t.dtype == torch.float32:
        return PA_FP32
    raise TypeError(f"unsupported dtype {t.dtype}")


def make_dims(q, k_pages, block_table, max_context_len, pages_per_split=0, num_q_rows=0,
              max_q_len=0, num_seqs=None) -> PaDims:
    """pa_dims_t from tensor shapes: q [rows][H_q][D], k_pages [N][H_kv][16][D],
    block_table [B][max_pages_per_seq]."""
    rows, H_q, D = q.shape
    N, H_kv, P, D2 = k_pages.shape
    B = block_table.shape[0] if num_seqs is None else num_seqs
    return PaDims(num_seqs=B, num_q_heads=H_q, num_kv_heads=H_kv, head_dim=D, page_size=P,
                  num_pages=N, max_pages_per_seq=block_table.shape[1],
                  max_context_len=int(max_context_len), pages_per_split=int(pages_per_split),
                  dtype=_dtype_code(q), num_q_rows=int(num_q_rows), max_q_len=int(max_q_len))


def pa_workspace_size(dims: PaDims) -> int:
    n = ctypes.c_size_t(0)
    rc = load().pa_workspace_size(ctypes.byref(dims), ctypes.byref(n))
    if rc != PA_OK:
        raise PagedAttnError("pa_workspace_size", rc)
    return int(n.value)


def pa_strerror(code: int) -> str:
    return load().pa_strerror(int(code)).decode()


def _workspace(dims, workspace, device, stream=None):
    """The caller's workspace, or a temporary one of pa_workspace_size()
    bytes.  A temporary is allocated on torch's current stream; when the call
    runs on another stream, the allocation is also recorded on that stream, so
    torch's caching allocator does not hand the memory to other work before
    the call's kernels have finished with it."""
    need = pa_workspace_size(dims)
    if workspace is None and need > 0:
        import torch
        if isinstance(stream, int) and stream:
            # torch cannot track work on a raw stream handle
            raise ValueError("pass a workspace (or a torch stream) when calling on a raw stream handle")
        workspace = torch.empty(need, dtype=torch.uint8, device=device)
        if stream is not None and stream != torch.cuda.current_stream(workspace.device):
            workspace.record_stream(stream)
    size = 0 if workspace is None else (workspace.numel() * workspace.element_size()
                                        if hasattr(workspace, "numel") else need)
    return workspace, size


def paged_attn(q, k_pages, v_pages, block_table, context_lens, scale, out, dims: PaDims,
               workspace=None, stream=None, timing: PaTiming | None = None, check=True) -> int:
    """int paged_attn(...): decode attention; out is written in place."""
    ws, ws_bytes = _workspace(dims, workspace, getattr(q, "device", None), stream)
    rc = load().paged_attn(_addr(q), _addr(k_pages), _addr(v_pages), _addr(block_table),
                           _addr(context_lens), float(scale), _addr(out), ctypes.byref(dims),
                           _addr(ws), ws_bytes, _stream(stream),
                           ctypes.byref(timing) if timing is not None else None)
    if check and rc != PA_OK:
        raise PagedAttnError("paged_attn", rc)
    return rc


def paged_attn_varlen(q, k_pages, v_pages, block_table, context_lens, query_start_loc, scale, out,
                      dims: PaDims, workspace=None, stream=None, timing: PaTiming | None = None,
                      check=True) -> int:
    """int paged_attn_varlen(...): causal prefill chunks plus decode rows."""
    ws, ws_bytes = _workspace(dims, workspace, getattr(q, "device", None), stream)
    rc = load().paged_attn_varlen(_addr(q), _addr(k_pages), _addr(v_pages), _addr(block_table),
                                  _addr(context_lens), _addr(query_start_loc), float(scale),
                                  _addr(out), ctypes.byref(dims), _addr(ws), ws_bytes,
                                  _stream(stream),
                                  ctypes.byref(timing) if timing is not None else None)
    if check and rc != PA_OK:
        raise PagedAttnError("paged_attn_varlen", rc)
    return rc


def paged_attn_varlen_noalloc(q, k_pages, v_pages, block_table, context_lens, query_start_loc, scale, out,
                              dims: PaDims, stream=None, timing: PaTiming | None = None, check=True) -> int:
    """int paged_attn_varlen_noalloc(...): paged_attn_varlen with the library's
    fixed device scratch in place of a workspace (allocates nothing)."""
    rc = load().paged_attn_varlen_noalloc(_addr(q), _addr(k_pages), _addr(v_pages), _addr(block_table),
                                          _addr(context_lens), _addr(query_start_loc), float(scale),
                                          _addr(out), ctypes.byref(dims), _stream(stream),
                                          ctypes.byref(timing) if timing is not None else None)
    if check and rc != PA_OK:
        raise PagedAttnError("paged_attn_varlen_noalloc", rc)
    return rc


def pa_gather_trace(q, k_pages, v_pages, block_table, context_lens, scale, out, dims: PaDims,
                    rows_out, query_start_loc=None, workspace=None, stream=None, check=True) -> int:
    """int pa_gather_trace(...): the attention call (decode, or varlen when
    query_start_loc is given) through the kernels' trace instantiations;
    rows_out [H_kv][B][max_pages_per_seq * 16] int64 receives the pool row of
    every loaded token."""
    ws, ws_bytes = _workspace(dims, workspace, getattr(q, "device", None), stream)
    rc = load().pa_gather_trace(_addr(q), _addr(k_pages), _addr(v_pages), _addr(block_table),
                                _addr(context_lens), _addr(query_start_loc), float(scale),
                                _addr(out), ctypes.byref(dims), _addr(ws), ws_bytes,
                                _addr(rows_out), _stream(stream))
    if check and rc != PA_OK:
        raise PagedAttnError("pa_gather_trace", rc)
    return rc


def pa_kv_append(k_new, v_new, block_table, context_lens, k_pages, v_pages, dims: PaDims,
                 query_start_loc=None, stream=None, check=True) -> int:
    """int pa_kv_append(...): store the new tokens' K/V into the paged pools."""
    rc = load().pa_kv_append(_addr(k_new), _addr(v_new), _addr(block_table), _addr(context_lens),
                             _addr(query_start_loc), _addr(k_pages), _addr(v_pages),
                             ctypes.byref(dims), _stream(stream))
    if check and rc != PA_OK:
        raise PagedAttnError("pa_kv_append", rc)
    return rc


def pa_schedule_step(state: PaSchedState, n_real, new_seq, new_prompt, new_fin, n_new,
                     query_start_loc, finished_out, info, stream=None, check=True) -> int:
    """int pa_schedule_step(...): one scheduler step on the device-resident state."""
    rc = load().pa_schedule_step(ctypes.byref(state), int(n_real), _addr(new_seq),
                                 _addr(new_prompt), _addr(new_fin), int(n_new),
                                 _addr(query_start_loc), _addr(finished_out), _addr(info),
                                 _stream(stream))
    if check and rc != PA_OK:
        raise PagedAttnError("pa_schedule_step", rc)
    return rc


def pa_read_probe(buf, chunk_bytes, chunk_offsets, n_chunks, grid, waves, depth, non_temporal, sink, stream=None,
                  check=True) -> int:
    """int pa_read_probe(...): read n_chunks chunks of buf with the decode
    kernels' load pattern (include/pa_probe.h)."""
    rc = load().pa_read_probe(_addr(buf), int(chunk_bytes), _addr(chunk_offsets), int(n_chunks), int(grid),
                              int(waves), int(depth), int(non_temporal), _addr(sink), _stream(stream))
    if check and rc != PA_OK:
        raise PagedAttnError("pa_read_probe", rc)
    return rc


def pa_issue_probe(grid, waves, iters, big_mfma, valu_per_mfma, exp2, mode, sink, cycles=None, stream=None,
                   check=True) -> int:
    """int pa_issue_probe(...): matrix products beside vector work
    (include/pa_probe.h); the caller times the launch."""
    rc = load().pa_issue_probe(int(grid), int(waves), int(iters), int(big_mfma), int(valu_per_mfma), int(exp2),
                               int(mode), _addr(sink), _addr(cycles), _stream(stream))
    if check and rc != PA_OK:
        raise PagedAttnError("pa_issue_probe", rc)
    return rc


def pa_perf_model(**inputs) -> dict:
    """int pa_perf_model(...): the Sec. 5 performance model for one
    configuration; keyword names are the pa_pm_input_t fields (missing ones
    are 0).  Returns the pa_pm_output_t fields as a dict."""
    unknown = set(inputs) - set(PM_INPUT_DOUBLES) - set(PM_INPUT_INTS)
    if unknown:
        raise TypeError(f"unknown inputs {sorted(unknown)}")
    x = PaPmInput(**inputs)
    o = PaPmOutput()
    rc = load().pa_perf_model(ctypes.byref(x), ctypes.byref(o))
    if rc != PA_OK:
        raise PagedAttnError("pa_perf_model", rc)
    return {n: getattr(o, n) for n in PM_OUTPUTS}
