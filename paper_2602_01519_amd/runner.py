"""Puts a seeded workload on the GPU and runs the link path through the C ABI.

Device memory and streams come from torch (plumbing only); every step of the
link path runs in libpic.so. Used by the GPU tests, the smoke check and the
benchmark.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Iterable, Optional

import numpy as np
import torch

from . import pic
from . import workloads as W


def to_device(a: Optional[np.ndarray], device) -> Optional[torch.Tensor]:
    """Raw bytes of a host array on the device (bf16 travels as int16 bit patterns)."""
    if a is None:
        return None
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to(device)


def to_host(t: torch.Tensor, dtype: int) -> np.ndarray:
    """Device output as float64 (bf16 bit patterns widened exactly)."""
    a = t.detach().cpu().numpy()
    if dtype == W.BF16:
        return W.bf16_bits_to_f32(a.view(np.uint16)).astype(np.float64)
    return a.astype(np.float64)


@dataclasses.dataclass
class DeviceWorkload:
    wl: W.Workload
    store: pic.Store
    q: torch.Tensor
    k_self: Optional[torch.Tensor]
    v_self: Optional[torch.Tensor]
    out: torch.Tensor
    lse: torch.Tensor
    chunks: Dict[int, tuple]      # host copies of the chunks kept for the oracle
    _calls: dict = dataclasses.field(default_factory=dict)

    def run(self, stream: Optional[int] = None, decode: Optional[bool] = None, num_splits: int = 0):
        cfg, p = self.wl.cfg, self.wl.plan
        if stream is None:
            stream = torch.cuda.current_stream().cuda_stream
        if decode is None:
            decode = cfg.decode
        key = (bool(decode), int(num_splits))
        call = self._calls.get(key)
        if call is None:           # the call's arguments, marshalled once
            call = pic.PreparedCall(key[0], self.store, p.chunk_offsets, self.wl.link_ids(),
                                    p.q_offsets, p.self_offsets, cfg.n_q_heads, self.q, self.k_self,
                                    self.v_self, float(np.float32(cfg.scale)), self.out, self.lse,
                                    num_splits=key[1])
            self._calls[key] = call
        call(stream)

    def results(self):
        return to_host(self.out, self.wl.cfg.dtype), self.lse.detach().cpu().numpy().astype(np.float64)

    def close(self):
        self.store.close()


def padded(n: int) -> int:
    return (n + 63) // 64 * 64


def upload(wl: W.Workload, device="cuda", keep_host: Optional[Iterable[int]] = None,
           extra_capacity: int = 0) -> DeviceWorkload:
    """Creates a store holding every chunk the workload links and uploads the requests.

    keep_host: store indices whose host copies are kept (None = all).
    """
    cfg = wl.cfg
    used = [int(c) for c in wl.used_chunks()]
    cap = sum(padded(cfg.chunk_length(c)) for c in used) + extra_capacity
    store = pic.Store(cfg.kind, cfg.dtype, cfg.n_kv_heads, cfg.d_k, cfg.d_v, max(cap, 64))
    keep = None if keep_host is None else set(int(x) for x in keep_host)
    chunks = {}
    stream = torch.cuda.current_stream().cuda_stream
    for c in used:
        k, v = W.make_chunk(cfg, c)
        kd, vd = to_device(k, device), to_device(v, device)
        # the put reads kd/vd on torch's current stream, so their memory is
        # only reused by later work on that same stream
        store.put(int(wl.chunk_ids[c]), k.shape[0], kd, vd, stream)
        if keep is None or c in keep:
            chunks[c] = (k, v)
    tq = wl.q.shape[0]
    et = torch.float32 if cfg.dtype == W.F32 else torch.int16
    out = torch.empty((tq, cfg.n_q_heads, cfg.d_v), dtype=et, device=device)
    lse = torch.empty((tq, cfg.n_q_heads), dtype=torch.float32, device=device)
    return DeviceWorkload(wl, store, to_device(wl.q, device), to_device(wl.k_self, device),
                          to_device(wl.v_self, device), out, lse, chunks)
