"""CPU oracle for batched paged-KV grouped-query attention.

TEST INFRASTRUCTURE ONLY.  This package is a plain, slow fp32 definition of
what the GPU library computes, used to check it.  Only the test suite, the
smoke check and the benchmark's CPU-baseline leg may import it; the product
path (the GPU library and its Python binding) never does, and the two share no
code.  The arithmetic lives in ``oracle.c``; this module only marshals NumPy
arrays through ctypes.

Definition (MoE-Lens, arXiv 2504.09345): paged KV blocks addressed through a
block table (Sec. 5.5), grouped-query heads sharing one KV head (Sec. 2),
bf16 storage with fp32 arithmetic built from dot products and scaled vector
adds (Sec. 5.3, Eq. 6), decode KV stored before attention (Sec. 6.4).
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# ORACLE_LIB points the binding at another build of oracle.c; the test suite
# uses it to check that mistakes planted in a copy of the source fail the pins.
_LIB_PATH = os.environ.get("ORACLE_LIB") or os.path.join(_HERE, "liboracle.so")
_lib = None

BF16, FP32 = 0, 1


def _load():
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        from . import build as _b  # the checker is built on demand
        _b.build()
    _lib = _bind(ctypes.CDLL(_LIB_PATH))
    return _lib


def _bind(lib):
    P = ctypes.c_void_p
    I32 = ctypes.c_int32
    lib.oracle_paged_attn.argtypes = [P, P, P, ctypes.c_int, P, I32, P, I32, I32, I32, I32, I32,
                                      I32, ctypes.c_float, P]
    lib.oracle_paged_attn.restype = ctypes.c_int
    lib.oracle_paged_attn_varlen.argtypes = [P, P, P, ctypes.c_int, P, I32, P, P, I32, I32, I32,
                                             I32, I32, I32, ctypes.c_float, P]
    lib.oracle_paged_attn_varlen.restype = ctypes.c_int
    lib.oracle_gather_indices.argtypes = [P, I32, P, I32, I32, I32, P]
    lib.oracle_gather_indices.restype = ctypes.c_int
    lib.oracle_softmax_weights.argtypes = [P, P, ctypes.c_int, P, I32, P, I32, I32, I32, I32, I32,
                                           I32, ctypes.c_float, I32, I32, I32, ctypes.c_int64,
                                           I32, P]
    lib.oracle_softmax_weights.restype = ctypes.c_int
    lib.oracle_kv_append.argtypes = [P, P, I32, P, I32, P, P, I32, I32, I32, I32, I32, P, P]
    lib.oracle_kv_append.restype = ctypes.c_int
    lib.oracle_schedule_step.argtypes = [P] * 10 + [I32] * 5 + [P, P, P, I32, P, P, P]
    lib.oracle_schedule_step.restype = ctypes.c_int
    lib.oracle_set_threads.argtypes = [ctypes.c_int]
    lib.oracle_set_threads.restype = None
    lib.oracle_get_threads.argtypes = []
    lib.oracle_get_threads.restype = ctypes.c_int
    return lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _dtype_code(a: np.ndarray) -> int:
    if a.dtype == np.uint16:
        return BF16
    if a.dtype == np.float32:
        return FP32
    raise TypeError(f"oracle takes bf16 bit patterns (uint16) or float32, got {a.dtype}")


def _c(a, dt=None):
    return np.ascontiguousarray(a if dt is None else np.asarray(a, dtype=dt))


def set_threads(n: int) -> None:
    _load().oracle_set_threads(int(n))


def get_threads() -> int:
    return int(_load().oracle_get_threads())


def paged_attn(q, k_pages, v_pages, block_table, context_lens, scale):
    """Decode attention, one query row per sequence.

    q [B][H_q][D]; k_pages, v_pages [num_pages][H_kv][P][D] (uint16 bf16 bits or
    float32, all the same dtype); block_table [B][max_pages_per_seq] int32;
    context_lens [B] int32.  Returns float32 [B][H_q][D].
    """
    q, k_pages, v_pages = _c(q), _c(k_pages), _c(v_pages)
    bt, cl = _c(block_table, np.int32), _c(context_lens, np.int32)
    dt = _dtype_code(q)
    assert _dtype_code(k_pages) == dt and _dtype_code(v_pages) == dt
    B, H_q, D = q.shape
    N, H_kv, P, D2 = k_pages.shape
    assert D2 == D and v_pages.shape == k_pages.shape and bt.shape[0] == B and cl.shape == (B,)
    out = np.zeros((B, H_q, D), np.float32)
    rc = _load().oracle_paged_attn(_ptr(q), _ptr(k_pages), _ptr(v_pages), dt, _ptr(bt),
                                   bt.shape[1], _ptr(cl), B, H_q, H_kv, D, P, N, float(scale),
                                   _ptr(out))
    if rc != 0:
        raise ValueError(f"oracle_paged_attn failed with code {rc}")
    return out


def paged_attn_varlen(q, k_pages, v_pages, block_table, context_lens, query_start_loc, scale):
    """Mixed decode / causal chunked-prefill attention.

    q [T_q][H_q][D] with sequence b owning rows query_start_loc[b] ..
    query_start_loc[b+1]-1; row j of a chunk of length L in a sequence of
    context C attends to positions 0 .. C-L+j.  Returns float32 [T_q][H_q][D].
    """
    q, k_pages, v_pages = _c(q), _c(k_pages), _c(v_pages)
    bt, cl = _c(block_table, np.int32), _c(context_lens, np.int32)
    qsl = _c(query_start_loc, np.int32)
    dt = _dtype_code(q)
    T, H_q, D = q.shape
    N, H_kv, P, _ = k_pages.shape
    B = cl.shape[0]
    assert qsl.shape == (B + 1,) and int(qsl[-1]) == T
    out = np.zeros((T, H_q, D), np.float32)
    rc = _load().oracle_paged_attn_varlen(_ptr(q), _ptr(k_pages), _ptr(v_pages), dt, _ptr(bt),
                                          bt.shape[1], _ptr(cl), _ptr(qsl), B, H_q, H_kv, D, P,
                                          N, float(scale), _ptr(out))
    if rc != 0:
        raise ValueError(f"oracle_paged_attn_varlen failed with code {rc}")
    return out


def gather_indices(block_table, context_lens, page_size, num_pages):
    """Flat pool row page*P + slot of every cached token, sequence-major (int64)."""
    bt, cl = _c(block_table, np.int32), _c(context_lens, np.int32)
    rows = np.zeros(int(cl.sum()), np.int64)
    rc = _load().oracle_gather_indices(_ptr(bt), bt.shape[1], _ptr(cl), cl.shape[0],
                                       int(page_size), int(num_pages), _ptr(rows))
    if rc != 0:
        raise ValueError(f"oracle_gather_indices failed with code {rc}")
    return rows


def softmax_weights(q, k_pages, block_table, context_lens, scale, b, h, L=1, r=0, qrow=None):
    """Normalised attention weights of (sequence b, chunk row r of L, head h).

    qrow is the row of q holding that query (defaults to b, the decode layout).
    Returns float32 [n_vis] with n_vis = C - L + r + 1.
    """
    q, k_pages = _c(q), _c(k_pages)
    bt, cl = _c(block_table, np.int32), _c(context_lens, np.int32)
    dt = _dtype_code(q)
    T, H_q, D = q.shape
    N, H_kv, P, _ = k_pages.shape
    n_max = max(int(cl[b]) - L + r + 1, 0)
    w = np.zeros(max(n_max, 1), np.float32)
    rc = _load().oracle_softmax_weights(_ptr(q), _ptr(k_pages), dt, _ptr(bt), bt.shape[1],
                                        _ptr(cl), cl.shape[0], H_q, H_kv, D, P, N, float(scale),
                                        int(b), int(L), int(r), int(b if qrow is None else qrow),
                                        int(h), _ptr(w))
    if rc < 0:
        raise ValueError(f"oracle_softmax_weights failed with code {rc}")
    return w[:rc]


def kv_append(k_new, v_new, block_table, context_lens, k_pages, v_pages, query_start_loc=None):
    """New pools after storing the new tokens' K/V (rows of k_new / v_new,
    [T][H_kv][D]) at the last positions of each sequence's context.

    query_start_loc=None is the decode layout (row b, position context_lens[b]-1).
    The input pools are not modified; updated copies are returned.
    """
    k_new, v_new = _c(k_new), _c(v_new)
    if k_new.dtype != v_new.dtype or k_new.shape != v_new.shape:
        raise ValueError("k_new and v_new must match")
    kp, vp = np.array(k_pages, copy=True, order="C"), np.array(v_pages, copy=True, order="C")
    if kp.dtype != k_new.dtype or vp.dtype != k_new.dtype:
        raise ValueError("pool and new rows must share the element type")
    bt, cl = _c(block_table, np.int32), _c(context_lens, np.int32)
    qsl = None if query_start_loc is None else _c(query_start_loc, np.int32)
    N, H_kv, P, D = kp.shape
    rc = _load().oracle_kv_append(_ptr(k_new), _ptr(v_new), k_new.dtype.itemsize, _ptr(bt),
                                  bt.shape[1], _ptr(cl), None if qsl is None else _ptr(qsl),
                                  cl.shape[0], H_kv, D, P, N, _ptr(kp), _ptr(vp))
    if rc != 0:
        raise ValueError(f"oracle_kv_append failed with code {rc}")
    return kp, vp


SCHED_FIELDS = ("free_pages", "hdr", "queue_seq", "queue_tok", "queue_fin", "slot_seq", "slot_order",
                "slot_fin", "context_lens", "block_table")


def sched_init(S, P, MP, Q):
    """Empty scheduler state: all P pages free (stack top = page P-1), empty
    queue of Q entries, S empty slots of MP block-table entries."""
    return dict(free_pages=np.arange(P, dtype=np.int32), hdr=np.array([P, 0, 0, 0], np.int32),
                queue_seq=np.zeros(Q, np.int32), queue_tok=np.zeros(Q, np.int32),
                queue_fin=np.zeros(Q, np.int32), slot_seq=np.full(S, -1, np.int32),
                slot_order=np.zeros(S, np.int32), slot_fin=np.zeros(S, np.int32),
                context_lens=np.zeros(S, np.int32), block_table=np.zeros((S, MP), np.int32))


def schedule_step(state, n_real, new_seq=(), new_prompt=(), new_fin=()):
    """One scheduler step on a copy of `state` (see oracle_schedule_step);
    n_real is the pass's token capacity (decode rows plus prefill tokens).
    Returns (new state, query_start_loc [S+1], finished ids, info [8])."""
    st = {k: np.array(state[k], dtype=np.int32, copy=True, order="C") for k in SCHED_FIELDS}
    S, MP = st["block_table"].shape
    P, Q = st["free_pages"].shape[0], st["queue_seq"].shape[0]
    ns = np.ascontiguousarray(new_seq, np.int32)
    npr = np.ascontiguousarray(new_prompt, np.int32)
    nf = np.ascontiguousarray(new_fin, np.int32)
    qsl = np.zeros(S + 1, np.int32)
    fin_out = np.zeros(S, np.int32)
    info = np.zeros(8, np.int32)
    rc = _load().oracle_schedule_step(*[_ptr(st[k]) for k in SCHED_FIELDS], S, P, MP, Q,
                                      int(n_real), _ptr(ns) if ns.size else None,
                                      _ptr(npr) if npr.size else None, _ptr(nf) if nf.size else None,
                                      int(ns.size), _ptr(qsl), _ptr(fin_out), _ptr(info))
    if rc != 0:
        raise ValueError(f"oracle_schedule_step failed with code {rc}")
    return st, qsl, fin_out[:info[1]].copy(), info
