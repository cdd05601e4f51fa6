"""Python binding of the link-attention C ABI (include/pic.h), by ctypes.

Argument marshalling only: every step of the path runs in the HIP library.
Tensors are passed as raw device pointers (torch tensors are accepted and
their ``data_ptr()`` is taken); host arrays are numpy arrays. Streams are
``hipStream_t`` handles as integers (``torch.cuda.current_stream().cuda_stream``)
or None for the null stream. Every non-OK status raises PicError.

The library must have been built (paper_2602_01519_amd/build.py); importing
a function of this module without it raises PicError -- there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import Optional

import numpy as np

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libpic.so")
_HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "pic.h")
_lib = None

OK, ERR_INVALID, ERR_NOT_FOUND, ERR_EXISTS, ERR_OOM, ERR_HIP, ERR_UNSUPPORTED = 0, -1, -2, -3, -4, -5, -6
F32, BF16 = 0, 1
GQA, MLA = 0, 1
PREFILL, DECODE = 0, 1


class PicError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{status_name(status)}: {message}")
        self.status = status


_NAMES = {0: "PIC_OK", -1: "PIC_ERR_INVALID", -2: "PIC_ERR_NOT_FOUND", -3: "PIC_ERR_EXISTS",
          -4: "PIC_ERR_OOM", -5: "PIC_ERR_HIP", -6: "PIC_ERR_UNSUPPORTED"}


def status_name(st: int) -> str:
    return _NAMES.get(st, f"status {st}")


class StoreDesc(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int32), ("dtype", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("d_k", ctypes.c_int32), ("d_v", ctypes.c_int32), ("n_layers", ctypes.c_int32),
                ("capacity_tokens", ctypes.c_int64)]


class LinkReq(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int32), ("layer", ctypes.c_int32),
                ("chunk_offsets", ctypes.c_void_p), ("chunk_ids", ctypes.c_void_p),
                ("q_offsets", ctypes.c_void_p), ("self_offsets", ctypes.c_void_p),
                ("chunk_starts", ctypes.c_void_p), ("q_doc_limits", ctypes.c_void_p)]


def lib_path() -> str:
    return _LIB_PATH


def lib():
    """The loaded libpic.so; raises PicError if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise PicError(ERR_UNSUPPORTED, f"{_LIB_PATH} is not built; run paper_2602_01519_amd/build.py")
        L = ctypes.CDLL(_LIB_PATH)
        vp, i32, i64, u64, f32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64, ctypes.c_float
        sig = {
            "pic_store_create": [vp, vp],
            "pic_store_destroy": [vp],
            "pic_store_put": [vp, u64, i64, vp, vp, vp],
            "pic_store_lookup": [vp, u64, vp],
            "pic_store_remove": [vp, u64, vp],
            "pic_store_derive": [vp, u64, u64, i32, vp, vp],
            "pic_store_write_rows": [vp, u64, i32, i32, vp, vp, vp, vp],
            "pic_store_usage": [vp, vp, vp, vp],
            "pic_store_export": [vp, vp, ctypes.c_size_t, vp],
            "pic_store_import": [vp, ctypes.c_size_t, vp],
            "pic_link_attn": [vp, vp, i32, vp, vp, vp, f32, vp, vp, vp],
            "pic_link_decode": [vp, vp, i32, vp, vp, vp, f32, i32, vp, vp, vp],
            "pic_link_decode_noalloc": [vp, vp, i32, vp, vp, vp, f32, i32, vp, vp, vp],
            "pic_debug_gather": [vp, vp, i32, i32, vp, vp, vp],
            "pic_debug_request_order": [vp, vp, vp, i32, i32, i32, i32, i32, vp, vp],
            "pic_link_plan_create": [vp, vp, i32, i32, i32, vp],
            "pic_link_plan_run": [vp, i32, vp, vp, vp, f32, vp, vp, vp],
            "pic_link_plan_destroy": [vp],
            "pic_mla_absorb_q": [i32, i32, vp, vp, vp, vp],
            "pic_mla_up_v": [i32, i32, vp, vp, vp, vp],
            "pic_prof_begin": [],
            "pic_prof_begin_sampled": [i32],
            "pic_prof_end": [vp, vp, vp, i32],
            "pic_peak_mfma_bf16": [i32, vp, vp],
            "pic_peak_hbm_read": [vp, i64, vp, vp],
            "pic_peak_hbm_write": [vp, i64, vp, vp],
        }
        for name, args in sig.items():
            fn = getattr(L, name)
            fn.argtypes = args
            fn.restype = ctypes.c_int
        L.pic_status_str.argtypes = [ctypes.c_int]
        L.pic_status_str.restype = ctypes.c_char_p
        L.pic_last_error.argtypes = []
        L.pic_last_error.restype = ctypes.c_char_p
        _lib = L
    return _lib


def header_functions() -> list:
    """Names of the functions include/pic.h declares."""
    text = open(_HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pic_[a-z_]+)\s*\(", text)))


def last_error() -> str:
    return lib().pic_last_error().decode()


def _check(st: int):
    if st != OK:
        raise PicError(st, last_error())


def _ptr(x):
    if x is None:
        return None
    if isinstance(x, int):
        return x
    if isinstance(x, np.ndarray):
        return x.ctypes.data
    return x.data_ptr()          # torch tensor


def _host_i32(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.int32)


def _addr(a: np.ndarray) -> int:
    """Address of a contiguous host array's first byte (a ctypes view of a
    writable buffer costs a third of numpy's .ctypes.data)."""
    try:
        return ctypes.addressof(ctypes.c_char.from_buffer(a))
    except (TypeError, ValueError):      # read-only or empty
        return a.ctypes.data


class Store:
    """A chunk store (pool + hash table) on the current HIP device."""

    def __init__(self, kind: int, dtype: int, n_kv_heads: int, d_k: int, d_v: int, capacity_tokens: int,
                 n_layers: int = 1):
        self.desc = StoreDesc(kind, dtype, n_kv_heads, d_k, d_v, n_layers, capacity_tokens)
        h = ctypes.c_void_p()
        _check(lib().pic_store_create(ctypes.byref(self.desc), ctypes.byref(h)))
        self.handle = h

    def close(self):
        if self.handle:
            _check(lib().pic_store_destroy(self.handle))
            self.handle = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def put(self, chunk_id: int, n_tokens: int, k, v, stream: Optional[int] = None):
        _check(lib().pic_store_put(self.handle, int(chunk_id), int(n_tokens), _ptr(k), _ptr(v), stream))

    def remove(self, chunk_id: int, stream: Optional[int] = None):
        """pic_store_remove: frees the chunk's pages once `stream`'s earlier work is done."""
        _check(lib().pic_store_remove(self.handle, int(chunk_id), stream))

    def derive(self, new_id: int, base_id: int, rows, stream: Optional[int] = None):
        """pic_store_derive: new_id = base_id with private copies of the pages holding `rows`."""
        r = np.ascontiguousarray(rows, dtype=np.int32)
        _check(lib().pic_store_derive(self.handle, int(new_id), int(base_id), int(r.size),
                                      r.ctypes.data if r.size else None, stream))

    def write_rows(self, chunk_id: int, layer: int, rows, k, v, stream: Optional[int] = None):
        """pic_store_write_rows: token-major K / V rows of one layer into a derived chunk."""
        r = np.ascontiguousarray(rows, dtype=np.int32)
        _check(lib().pic_store_write_rows(self.handle, int(chunk_id), int(layer), int(r.size),
                                          r.ctypes.data if r.size else None, _ptr(k), _ptr(v), stream))

    def export(self) -> bytes:
        """pic_store_export: a description of the store another process can import."""
        n = ctypes.c_size_t()
        _check(lib().pic_store_export(self.handle, None, 0, ctypes.byref(n)))
        buf = ctypes.create_string_buffer(n.value)
        _check(lib().pic_store_export(self.handle, buf, n.value, ctypes.byref(n)))
        return buf.raw[:n.value]

    @classmethod
    def import_(cls, blob: bytes) -> "Store":
        """pic_store_import: a read-only store over another process's exported pool."""
        self = cls.__new__(cls)
        self.desc = None
        h = ctypes.c_void_p()
        _check(lib().pic_store_import(blob, len(blob), ctypes.byref(h)))
        self.handle = h
        return self

    def lookup(self, chunk_id: int) -> int:
        n = ctypes.c_int64()
        _check(lib().pic_store_lookup(self.handle, int(chunk_id), ctypes.byref(n)))
        return n.value

    def usage(self):
        u, c, n = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        _check(lib().pic_store_usage(self.handle, ctypes.byref(u), ctypes.byref(c), ctypes.byref(n)))
        return u.value, c.value, n.value


def _req(chunk_offsets, chunk_ids, q_offsets, self_offsets, keep: list, layer: int = 0,
         chunk_starts=None, q_doc_limits=None):
    co = _host_i32(chunk_offsets)
    ids = np.ascontiguousarray(chunk_ids, dtype=np.uint64)
    qo = _host_i32(q_offsets)
    so = _host_i32(self_offsets)
    st = _host_i32(chunk_starts)
    dl = _host_i32(q_doc_limits)
    keep += [co, ids, qo, so, st, dl]
    return LinkReq(len(qo) - 1, int(layer), _addr(co), _addr(ids) if ids.size else None,
                   _addr(qo), None if so is None else _addr(so),
                   None if st is None or not st.size else _addr(st),
                   None if dl is None or not dl.size else _addr(dl))


def link_attn(store: Store, chunk_offsets, chunk_ids, q_offsets, self_offsets, n_q_heads: int, q,
              k_self, v_self, softmax_scale: float, out, lse=None, stream: Optional[int] = None,
              layer: int = 0, chunk_starts=None, q_doc_limits=None):
    """pic_link_attn: prefill-shaped link attention on store layer `layer`."""
    keep: list = []
    req = _req(chunk_offsets, chunk_ids, q_offsets, self_offsets, keep, layer, chunk_starts,
               q_doc_limits)
    _check(lib().pic_link_attn(store.handle, ctypes.byref(req), int(n_q_heads), _ptr(q), _ptr(k_self),
                               _ptr(v_self), float(softmax_scale), _ptr(out), _ptr(lse), stream))


def link_decode(store: Store, chunk_offsets, chunk_ids, q_offsets, self_offsets, n_q_heads: int, q,
                k_self, v_self, softmax_scale: float, out, lse=None, num_splits: int = 0,
                stream: Optional[int] = None, layer: int = 0, chunk_starts=None, q_doc_limits=None):
    """pic_link_decode: decode-shaped link attention with split-K on store layer `layer`."""
    keep: list = []
    req = _req(chunk_offsets, chunk_ids, q_offsets, self_offsets, keep, layer, chunk_starts,
               q_doc_limits)
    _check(lib().pic_link_decode(store.handle, ctypes.byref(req), int(n_q_heads), _ptr(q), _ptr(k_self),
                                 _ptr(v_self), float(softmax_scale), int(num_splits), _ptr(out),
                                 _ptr(lse), stream))


class PreparedCall:
    """pic_link_attn (or pic_link_decode) with its arguments marshalled once:
    the request struct, the host arrays it points at (kept alive here) and
    the tensor addresses. Calling it runs the same C entry point on a stream;
    the tensors must stay allocated and the host arrays unchanged."""

    def __init__(self, decode: bool, store: Store, chunk_offsets, chunk_ids, q_offsets,
                 self_offsets, n_q_heads: int, q, k_self, v_self, softmax_scale: float, out,
                 lse=None, num_splits: int = 0, layer: int = 0, chunk_starts=None,
                 q_doc_limits=None):
        self._store = store
        self._keep: list = []
        self._req = _req(chunk_offsets, chunk_ids, q_offsets, self_offsets, self._keep, layer,
                         chunk_starts, q_doc_limits)
        vp = ctypes.c_void_p
        head = (store.handle, ctypes.byref(self._req), ctypes.c_int32(int(n_q_heads)),
                vp(_ptr(q)), vp(_ptr(k_self)), vp(_ptr(v_self)), ctypes.c_float(float(softmax_scale)))
        tail = (vp(_ptr(out)), vp(_ptr(lse)))
        if decode:
            self._fn = lib().pic_link_decode
            self._args = head + (ctypes.c_int32(int(num_splits)),) + tail
        else:
            self._fn = lib().pic_link_attn
            self._args = head + tail

    def __call__(self, stream: Optional[int] = None):
        if not self._store.handle:
            raise PicError(ERR_INVALID, "the store is closed")
        _check(self._fn(*self._args, stream))


def link_decode_noalloc(store: Store, chunk_offsets, chunk_ids, q_offsets, self_offsets,
                        n_q_heads: int, q, k_self, v_self, softmax_scale: float, out, lse=None,
                        num_splits: int = 0, stream: Optional[int] = None, layer: int = 0,
                        chunk_starts=None, q_doc_limits=None):
    """pic_link_decode_noalloc: pic_link_decode in the library's static scratch."""
    keep: list = []
    req = _req(chunk_offsets, chunk_ids, q_offsets, self_offsets, keep, layer, chunk_starts,
               q_doc_limits)
    _check(lib().pic_link_decode_noalloc(store.handle, ctypes.byref(req), int(n_q_heads), _ptr(q),
                                         _ptr(k_self), _ptr(v_self), float(softmax_scale),
                                         int(num_splits), _ptr(out), _ptr(lse), stream))


def debug_request_order(q_len, self_len, doc_tiles, n_q_heads: int, n_kv_heads: int, cus: int,
                        xcds: int):
    """pic_debug_request_order: the d=128 prefill request order (host only).
    Returns (order, finish) with finish = [heaviest first, returned order]."""
    q_len = np.ascontiguousarray(q_len, dtype=np.int32)
    self_len = np.ascontiguousarray(self_len, dtype=np.int32)
    doc_tiles = np.ascontiguousarray(doc_tiles, dtype=np.int32)
    n = len(q_len)
    order = np.zeros(max(n, 1), np.int32)
    finish = np.zeros(2, np.float64)
    _check(lib().pic_debug_request_order(q_len.ctypes.data, self_len.ctypes.data,
                                         doc_tiles.ctypes.data, n, n_q_heads, n_kv_heads, cus,
                                         xcds, order.ctypes.data, finish.ctypes.data))
    return order[:n], finish


def debug_gather(store: Store, ids, k_out, v_out, stream: Optional[int] = None, layer: int = 0):
    """pic_debug_gather: materialise the concatenation of the listed chunks of one layer."""
    ids = np.ascontiguousarray(ids, dtype=np.uint64)
    _check(lib().pic_debug_gather(store.handle, ids.ctypes.data if ids.size else None, len(ids),
                                  int(layer), _ptr(k_out), _ptr(v_out), stream))


class LinkPlan:
    """pic_link_plan_*: a request batch resolved once, run per layer / decode step."""

    def __init__(self, store: Store, chunk_offsets, chunk_ids, q_offsets, self_offsets, n_q_heads: int,
                 mode: int = PREFILL, num_splits: int = 0, chunk_starts=None, q_doc_limits=None):
        keep: list = []
        req = _req(chunk_offsets, chunk_ids, q_offsets, self_offsets, keep, chunk_starts=chunk_starts,
                   q_doc_limits=q_doc_limits)
        h = ctypes.c_void_p()
        _check(lib().pic_link_plan_create(store.handle, ctypes.byref(req), int(n_q_heads), int(mode),
                                          int(num_splits), ctypes.byref(h)))
        self.handle = h.value
        self.store = store          # the store must outlive the plan

    def run(self, layer: int, q, k_self, v_self, softmax_scale: float, out, lse=None,
            stream: Optional[int] = None):
        _check(lib().pic_link_plan_run(self.handle, int(layer), _ptr(q), _ptr(k_self), _ptr(v_self),
                                       float(softmax_scale), _ptr(out), _ptr(lse), stream))

    def close(self):
        if getattr(self, "handle", None):
            _check(lib().pic_link_plan_destroy(self.handle))
            self.handle = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def mla_absorb_q(n_tokens: int, n_heads: int, q, w_uk_t, q_out, stream: Optional[int] = None):
    """pic_mla_absorb_q: q_out = [W_UK^T q_nope | q_rope] per head (bf16)."""
    _check(lib().pic_mla_absorb_q(int(n_tokens), int(n_heads), _ptr(q), _ptr(w_uk_t), _ptr(q_out), stream))


def mla_up_v(n_tokens: int, n_heads: int, o_lat, w_uv, out, stream: Optional[int] = None):
    """pic_mla_up_v: out = W_UV o_lat per head (bf16)."""
    _check(lib().pic_mla_up_v(int(n_tokens), int(n_heads), _ptr(o_lat), _ptr(w_uv), _ptr(out), stream))


def peak_mfma_bf16(iters: int = 4096, stream: Optional[int] = None) -> float:
    """Achievable bf16 matrix-core rate (TFLOP/s) of this GPU; blocking."""
    out = ctypes.c_double()
    _check(lib().pic_peak_mfma_bf16(int(iters), ctypes.byref(out), stream))
    return out.value


def peak_hbm_read(buf, nbytes: int, stream: Optional[int] = None) -> float:
    """Achievable HBM read rate (GB/s) over device buffer buf; blocking."""
    out = ctypes.c_double()
    _check(lib().pic_peak_hbm_read(_ptr(buf), int(nbytes), ctypes.byref(out), stream))
    return out.value


def peak_hbm_write(buf, nbytes: int, stream: Optional[int] = None) -> float:
    """Achievable HBM write rate (GB/s) over device buffer buf (overwritten); blocking."""
    out = ctypes.c_double()
    _check(lib().pic_peak_hbm_write(_ptr(buf), int(nbytes), ctypes.byref(out), stream))
    return out.value


def prof_begin(every: int = 1):
    """pic_prof_begin_sampled: time one launch of the attention kernel in `every`."""
    _check(lib().pic_prof_begin_sampled(int(every)))


def prof_end():
    """(summed kernel milliseconds, launches, kernel name) since prof_begin()."""
    ms, n = ctypes.c_double(), ctypes.c_int64()
    name = ctypes.create_string_buffer(128)
    _check(lib().pic_prof_end(ctypes.byref(ms), ctypes.byref(n), name, 128))
    return ms.value, n.value, name.value.decode()
