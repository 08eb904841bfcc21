"""CPU oracle for the RegVGGT per-frame hot path -- TEST INFRASTRUCTURE ONLY.

A plain fp64 implementation of what the paper defines (Sec. 3.1 Eq. 2-3; Sec. 3.3
Eq. 6, the head-specific retention rule, the LSE equation and the A_ij equation),
used to prove the HIP library right.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the benchmark's ``cpu_baseline`` leg may import it; the product path never does.  It
shares no code with the HIP library: numbers meet only through the seeded input
generator, which holds none of the method's arithmetic.

Arrays are numpy.  bf16 tensors are carried as their raw 16-bit patterns
(``numpy.uint16``) and widened exactly to fp64 inside the C code.
Layouts: current frame Q, K, V ``[n_tokens, n_heads, head_dim]``; memory
``[n_heads, head_stride, head_dim]``; per-head vectors ``[n_heads, n]``.
"""
import ctypes
import os

import numpy as np

from . import build as _build

_lib = None


def _load():
    global _lib
    if _lib is None:
        path = _build.LIB
        if not os.path.exists(path):
            _build.build()
        lib = ctypes.CDLL(path)
        i32, i64, vp = ctypes.c_int, ctypes.c_int64, ctypes.c_void_p
        lib.rvo_qsub_index.argtypes = [i32, i32, i32, i32, vp, i32]
        lib.rvo_attend.argtypes = [vp, vp, vp, i32, i32, i32, vp, vp, i64, i64, vp, i32, vp, vp]
        lib.rvo_column_mass.argtypes = [vp, i32, i32, i32, vp, i32, vp, vp, i32, i64, i64, vp]
        lib.rvo_topk.argtypes = [vp, i32, i32, i32, vp]
        lib.rvo_append.argtypes = [vp, vp, i64, i64, vp, vp, i32, i32, i32, vp, i32]
        for f in (lib.rvo_qsub_index, lib.rvo_attend, lib.rvo_column_mass, lib.rvo_topk,
                  lib.rvo_append, lib.rvo_num_threads):
            f.restype = ctypes.c_int
        _lib = lib
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _check(rc, what):
    if rc != 0:
        raise ValueError(f"oracle {what} rejected its arguments (code {rc})")


def _u16(a):
    a = np.ascontiguousarray(a)
    if a.dtype != np.uint16:
        raise TypeError("bf16 tensors are passed as uint16 bit patterns")
    return a


def num_threads() -> int:
    return _load().rvo_num_threads()


def qsub_index(grid_h: int, grid_w: int, n_special: int, stride: int) -> np.ndarray:
    """Sampled query positions Q~ (Sec. 3.3, head-specific retention)."""
    lib = _load()
    n = lib.rvo_qsub_index(grid_h, grid_w, n_special, stride, None, 0)
    _check(0 if n >= 0 else n, "qsub_index")
    out = np.zeros(max(n, 1), dtype=np.int32)
    lib.rvo_qsub_index(grid_h, grid_w, n_special, stride, _ptr(out), n)
    return out[:n]


def attend(Q, K, V, memK=None, memV=None, mem_len=0, rows=None):
    """Attention of the frame over memory + frame, with per-query LSE (Sec. 3.1 Eq. 3).

    Returns (out [n_rows, H, d] fp64, lse [H, n_rows] fp64)."""
    Q, K, V = _u16(Q), _u16(K), _u16(V)
    n, H, d = Q.shape
    if mem_len > 0:
        memK, memV = _u16(memK), _u16(memV)
        head_stride = memK.shape[1]
    else:
        memK = memV = None
        head_stride = 0
    if rows is not None:
        rows = np.ascontiguousarray(rows, dtype=np.int32)
        n_rows = len(rows)
    else:
        n_rows = n
    out = np.zeros((n_rows, H, d), dtype=np.float64)
    lse = np.zeros((H, n_rows), dtype=np.float64)
    rc = _load().rvo_attend(_ptr(Q), _ptr(K), _ptr(V), n, H, d, _ptr(memK), _ptr(memV),
                            int(mem_len), int(head_stride), _ptr(rows), n_rows,
                            _ptr(out), _ptr(lse))
    _check(rc, "attend")
    return out, lse


def column_mass(Q, qidx, lse_q, keys, key_layout="frame"):
    """Attention mass each key column receives from the sampled queries.

    ``keys`` is the current frame's K ``[n, H, d]`` (key_layout="frame": the paper's
    saliency S_j) or a memory block ``[H, rows, d]`` (key_layout="memory").
    ``lse_q`` is ``[H, n_q]``: the LSE of the sampled queries.  Returns ``[H, n_keys]``."""
    Q = _u16(Q)
    keys = _u16(keys)
    n, H, d = Q.shape
    qidx = np.ascontiguousarray(qidx, dtype=np.int32)
    lse_q = np.ascontiguousarray(lse_q, dtype=np.float64)
    if key_layout == "frame":
        n_keys, tok_stride, head_stride = keys.shape[0], H * d, d
    elif key_layout == "memory":
        n_keys, tok_stride, head_stride = keys.shape[1], d, keys.shape[1] * d
    else:
        raise ValueError(key_layout)
    S = np.zeros((H, n_keys), dtype=np.float64)
    rc = _load().rvo_column_mass(_ptr(Q), n, H, d, _ptr(qidx), len(qidx), _ptr(lse_q),
                                 _ptr(keys), n_keys, tok_stride, head_stride, _ptr(S))
    _check(rc, "column_mass")
    return S


def saliency(Q, K, lse, qidx):
    """S_j for every current-frame key (Sec. 3.3); ``lse`` is ``[H, n]`` for all queries."""
    qidx = np.asarray(qidx, dtype=np.int32)
    return column_mass(Q, qidx, np.asarray(lse)[:, qidx], K, "frame")


def topk(sal, budget):
    """Per-head top-``budget`` token indices, ties to the lower index, ascending."""
    sal = np.ascontiguousarray(sal, dtype=np.float64)
    H, n = sal.shape
    idx = np.zeros((H, max(budget, 0)), dtype=np.int32)
    rc = _load().rvo_topk(_ptr(sal), n, H, int(budget), _ptr(idx))
    _check(rc, "topk")
    return idx


def topk_head_average(sal, budget):
    """One top-``budget`` per layer on the saliency averaged over heads (the arm without
    head-specific retention in the ablation of Sec. 4.5, Table 4): the mean over the
    head axis in fp64, then the same ranking as ``topk`` (ties to the lower index)."""
    mean = np.asarray(sal, dtype=np.float64).mean(axis=0, keepdims=True)
    return topk(mean, budget)[0]


class Memory:
    """The oracle's own KV memory: ``[H, capacity, d]`` bf16 patterns + length."""

    def __init__(self, n_heads, head_dim, capacity):
        self.K = np.zeros((n_heads, capacity, head_dim), dtype=np.uint16)
        self.V = np.zeros((n_heads, capacity, head_dim), dtype=np.uint16)
        self.len = 0

    def append(self, K, V, idx):
        K, V = _u16(K), _u16(V)
        idx = np.ascontiguousarray(idx, dtype=np.int32)
        H, budget = idx.shape
        n, _, d = K.shape
        rc = _load().rvo_append(_ptr(self.K), _ptr(self.V), self.len, self.K.shape[1],
                                _ptr(K), _ptr(V), n, H, d, _ptr(idx), budget)
        _check(rc, "append")
        self.len += budget


def step(mem: Memory, Q, K, V, qidx, budget):
    """One frame of the paper's per-layer streaming step (Sec. 3.3):
    attend over memory + frame, LSE-saliency over the sampled queries, per-head top-k,
    append.  Returns dict(out, lse, sal, idx)."""
    out, lse = attend(Q, K, V, mem.K, mem.V, mem.len)
    sal = saliency(Q, K, lse, qidx)
    idx = topk(sal, budget)
    mem.append(K, V, idx)
    return {"out": out, "lse": lse, "sal": sal, "idx": idx}
