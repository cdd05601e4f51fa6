"""fp64 CPU oracle for link-stage attention (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg import
this package. The product path (the HIP library and its binding) never does.

``link_attn`` computes, from the same input bytes the GPU path reads, the
joint softmax attention of each query row over its request's linked chunk
caches concatenated in link order (unmasked, Sec. 4.2 Eq. 7) followed by the
request's own KV under the causal mask (Sec. 4.1 Eq. 2), in double precision.
The arithmetic lives in ``link_oracle.c``; this module only marshals numpy
arrays and builds the shared object with gcc.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "link_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

F32, BF16 = 0, 1


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (portable flags: the result runs on other x86-64 hosts)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O3", "-fopenmp", "-fPIC", "-shared", "-std=c99",
                               "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        lib = ctypes.CDLL(_LIB)
        vp = ctypes.c_void_p
        lib.oracle_link_attn.restype = ctypes.c_int
        lib.oracle_link_attn.argtypes = [ctypes.c_int] * 7 + [vp] * 4 + [vp] * 2 + [vp] * 3 + \
            [ctypes.c_double, vp, vp, vp, vp]
        lib.oracle_num_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def link_attn(*, dtype: int, mla: bool, n_q_heads: int, d_v: int,
              links: Sequence[Sequence[tuple]], q: np.ndarray, q_offsets: np.ndarray,
              k_self: Optional[np.ndarray] = None, v_self: Optional[np.ndarray] = None,
              self_offsets: Optional[np.ndarray] = None, tau: float,
              q_doc_limits: Optional[np.ndarray] = None,
              row_select: Optional[np.ndarray] = None):
    """Reference output and log-sum-exp.

    links[r] is the ordered list of (k, v) chunk tensors request r links:
    k token-major [len, H_kv, d_k], v [len, H_kv, d_v] (None for MLA).
    q is [Tq, H_q, d_k]; own KV is [Ts, H_kv, d_*] with self_offsets, or absent.
    q_doc_limits[t], if given, is the number of leading document rows of its
    request that query token t sees (the rest of the documents are masked).
    bf16 tensors are passed as uint16 bit patterns, fp32 ones as float32.
    Returns (out float64 [Tq, H_q, d_v], lse float64 [Tq, H_q]).
    """
    lib = _load()
    edt = np.uint16 if dtype == BF16 else np.float32
    batch = len(links)
    q = np.ascontiguousarray(q, dtype=edt)
    tq, hq, d_k = q.shape
    assert hq == n_q_heads
    flat_k, flat_v, lens = [], [], []
    offs = np.zeros(batch + 1, np.int32)
    n_kv = None
    for r, req in enumerate(links):
        for (k, v) in req:
            k = np.ascontiguousarray(k, dtype=edt)
            assert k.ndim == 3 and k.shape[2] == d_k
            n_kv = k.shape[1] if n_kv is None else n_kv
            assert k.shape[1] == n_kv
            flat_k.append(k)
            if mla:
                flat_v.append(None)
            else:
                v = np.ascontiguousarray(v, dtype=edt)
                assert v.shape == (k.shape[0], n_kv, d_v)
                flat_v.append(v)
            lens.append(k.shape[0])
        offs[r + 1] = len(lens)
    if k_self is not None:
        k_self = np.ascontiguousarray(k_self, dtype=edt)
        n_kv = k_self.shape[1] if n_kv is None else n_kv
        if not mla:
            v_self = np.ascontiguousarray(v_self, dtype=edt)
    if n_kv is None:
        n_kv = 1 if mla else n_q_heads
    n = len(lens)
    karr = (ctypes.c_void_p * max(n, 1))(*[a.ctypes.data for a in flat_k])
    varr = (ctypes.c_void_p * max(n, 1))(*[(a.ctypes.data if a is not None else 0) for a in flat_v])
    larr = np.asarray(lens if lens else [0], dtype=np.int64)
    q_offsets = np.ascontiguousarray(q_offsets, dtype=np.int32)
    so = None if self_offsets is None else np.ascontiguousarray(self_offsets, dtype=np.int32)
    out = np.zeros((tq, hq, d_v), np.float64)
    lse = np.zeros((tq, hq), np.float64)
    lims = None if q_doc_limits is None else np.ascontiguousarray(q_doc_limits, dtype=np.int32)
    if lims is not None:
        assert lims.shape == (tq,)
    sel = None if row_select is None else np.ascontiguousarray(row_select, dtype=np.uint8)
    if sel is not None:
        assert sel.size == tq * hq
    rc = lib.oracle_link_attn(int(dtype), int(bool(mla)), batch, n_q_heads, int(n_kv), d_k, d_v,
                              _ptr(offs), ctypes.cast(karr, ctypes.c_void_p),
                              ctypes.cast(varr, ctypes.c_void_p), _ptr(larr), _ptr(q_offsets),
                              _ptr(so), _ptr(q), _ptr(k_self), _ptr(v_self if not mla else None),
                              float(tau), _ptr(lims), _ptr(sel), _ptr(out), _ptr(lse))
    if rc != 0:
        raise ValueError("oracle rejected its arguments")
    return out, lse


def workload_links(wl, chunks) -> list:
    """Per-request ordered (k, v) lists for a Workload, given a store-index -> (k, v) mapping."""
    plan = wl.plan
    res = []
    for r in range(plan.batch):
        idx = plan.chunk_index[plan.chunk_offsets[r]:plan.chunk_offsets[r + 1]]
        res.append([chunks[int(c)] for c in idx])
    return res


def run_workload(wl, chunks, row_select=None):
    """Oracle over a whole Workload (see paper_2602_01519_amd.workloads)."""
    cfg = wl.cfg
    return link_attn(dtype=cfg.dtype, mla=cfg.kind == 1, n_q_heads=cfg.n_q_heads, d_v=cfg.d_v,
                     links=workload_links(wl, chunks), q=wl.q, q_offsets=wl.plan.q_offsets,
                     k_self=wl.k_self, v_self=wl.v_self, self_offsets=wl.plan.self_offsets,
                     tau=float(np.float32(cfg.scale)), row_select=row_select)


from .mla_proj import mla_absorb_q, mla_up_v  # noqa: E402  (dense MLA projections, fp64)
