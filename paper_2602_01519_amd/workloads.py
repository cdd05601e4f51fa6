"""Seeded synthetic inputs for link-stage attention.

This module only draws inputs: shapes, seeds, normal samples, the fp32 -> bf16
round-to-nearest-even of those samples, and which chunks each request links.
It holds none of the attention arithmetic. The HIP path and the fp64 oracle
both consume the arrays it returns, so the two sides see identical bytes.

Recipe (the paper's workloads are LongBench-derived and not available; these
stand in for them with the shapes of its two backbones, Sec. 5.1):
  * every tensor element is N(0, 1) drawn in fp32 with numpy's PCG64, then
    scaled by ``q_std`` for queries, then rounded to bf16 (RNE) for bf16
    configs;
  * each chunk, and each request's query / own-KV block, has its own seed
    (``SeedSequence([cfg.seed, stream, index])``), so any one of them can be
    regenerated alone;
  * chunk lengths, link counts and link order come from one planning stream;
    links within a request are distinct and the draw order is the link order;
  * ``disjoint`` configs give every request its own chunks, so nothing is
    shared across requests (the decode workload is then HBM-honest).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Optional, Sequence, Tuple, Union

import numpy as np

F32, BF16 = 0, 1
GQA, MLA = 0, 1

_STREAM_PLAN, _STREAM_CHUNK, _STREAM_REQ = 0, 1, 2


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); returns uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to fp32 (exact)."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def chunk_id_of(index: int) -> int:
    """Stable 64-bit id for the store's index-th chunk (stands in for a content hash)."""
    z = (int(index) + 1) * 0x9E3779B97F4A7C15 & 0xFFFFFFFFFFFFFFFF
    z ^= z >> 31
    return z or 1


@dataclasses.dataclass(frozen=True)
class LinkConfig:
    name: str
    dtype: int                      # F32 or BF16
    kind: int                       # GQA or MLA
    n_q_heads: int
    n_kv_heads: int
    d_k: int
    d_v: int
    store_chunks: int
    chunk_len: Union[int, Tuple[int, ...]]   # one length, or one per store chunk
    batch: int
    links: Tuple[int, int]          # links per request, inclusive range
    q_len: Union[int, Tuple[int, ...]]       # one value, or one per request
    self_len: Union[int, Tuple[int, ...], None]  # None = cross-only (no own KV)
    q_std: float
    scale: float
    seed: int
    disjoint: bool = False
    decode: bool = False

    def chunk_length(self, i: int) -> int:
        return self.chunk_len if isinstance(self.chunk_len, int) else self.chunk_len[i]

    def q_length(self, r: int) -> int:
        return self.q_len if isinstance(self.q_len, int) else self.q_len[r]

    def self_length(self, r: int) -> int:
        if self.self_len is None:
            return 0
        return self.self_len if isinstance(self.self_len, int) else self.self_len[r]

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == F32 else 2

    def with_(self, **kw) -> "LinkConfig":
        return dataclasses.replace(self, **kw)


_BASE_SEED = 20260201

# The five workloads the measurements are quoted on.
SKINNY_Q = tuple((16, 32, 48)[r % 3] for r in range(32))

CONFIGS = {
    # 4 ordered links out of a 16-chunk store, 32 query tokens with causal own KV, fp32.
    "tiny_f32": LinkConfig("tiny_f32", F32, GQA, 8, 2, 64, 64, 16, 128, 1, (4, 4), 32, 32,
                           1.0, 1.0 / 8.0, _BASE_SEED + 1),
    # Llama-3-8B head shape, 10 links of 512 tokens, 256 query tokens, batch 8.
    "llama_prefill": LinkConfig("llama_prefill", BF16, GQA, 32, 8, 128, 128, 64, 512, 8,
                                (10, 10), 256, 256, 1.0 / math.sqrt(128.0), 1.0, _BASE_SEED + 2),
    # Long RAG link: 8..20 links of 1024 tokens from a 256-chunk store, 512 query tokens.
    "long_rag": LinkConfig("long_rag", BF16, GQA, 32, 8, 128, 128, 256, 1024, 16, (8, 20),
                           512, 512, 1.0 / math.sqrt(128.0), 1.0, _BASE_SEED + 3),
    # Decode: 1 query token over 16 private links of 1024 tokens plus 128 own tokens, batch 64.
    "decode": LinkConfig("decode", BF16, GQA, 32, 8, 128, 128, 1024, 1024, 64, (16, 16), 1,
                         128, 1.0 / math.sqrt(128.0), 1.0, _BASE_SEED + 4, disjoint=True,
                         decode=True),
    # DeepSeek-V2-Lite MLA, absorbed: one latent KV row of 512 + 64 rope dims, 16 heads.
    "mla": LinkConfig("mla", BF16, MLA, 16, 1, 576, 512, 64, 512, 8, (12, 12), 256, 256,
                      1.0, 1.0 / math.sqrt(192.0), _BASE_SEED + 5),
    # The paper's own regime: a few dozen dynamic (question) tokens after 4K-16K cached
    # document tokens. Llama-3-8B head shape, 32 requests each linking 4..16 private
    # chunks of 1024 tokens; question lengths 16 / 32 / 48 tokens, own KV = the question.
    "skinny_rag": LinkConfig("skinny_rag", BF16, GQA, 32, 8, 128, 128, 512, 1024, 32, (4, 16),
                             SKINNY_Q, SKINNY_Q, 1.0 / math.sqrt(128.0), 1.0, _BASE_SEED + 6,
                             disjoint=True),
}


@dataclasses.dataclass
class Plan:
    """Which store chunks each request links, and the per-request token counts."""
    chunk_offsets: np.ndarray   # int32 [B+1]
    chunk_index: np.ndarray     # int64 [sum n]: store positions in link order
    q_offsets: np.ndarray       # int32 [B+1]
    self_offsets: Optional[np.ndarray]  # int32 [B+1] or None

    @property
    def batch(self) -> int:
        return len(self.q_offsets) - 1


def make_plan(cfg: LinkConfig) -> Plan:
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([cfg.seed, _STREAM_PLAN])))
    lo, hi = cfg.links
    counts = rng.integers(lo, hi + 1, size=cfg.batch)
    picks = []
    if cfg.disjoint:
        if int(counts.sum()) > cfg.store_chunks:
            raise ValueError("disjoint plan needs more store chunks")
        perm = rng.permutation(cfg.store_chunks)
        pos = 0
        for n in counts:
            picks.append(perm[pos:pos + n])
            pos += n
    else:
        for n in counts:
            if n > cfg.store_chunks:
                raise ValueError("more links than store chunks")
            picks.append(rng.choice(cfg.store_chunks, size=int(n), replace=False))
    chunk_offsets = np.zeros(cfg.batch + 1, np.int32)
    chunk_offsets[1:] = np.cumsum(counts)
    chunk_index = (np.concatenate(picks) if picks else np.zeros(0)).astype(np.int64)
    q_offsets = np.zeros(cfg.batch + 1, np.int32)
    q_offsets[1:] = np.cumsum([cfg.q_length(r) for r in range(cfg.batch)])
    self_offsets = None
    if cfg.self_len is not None:
        self_offsets = np.zeros(cfg.batch + 1, np.int32)
        self_offsets[1:] = np.cumsum([cfg.self_length(r) for r in range(cfg.batch)])
    return Plan(chunk_offsets, chunk_index, q_offsets, self_offsets)


def _normal(rng, shape, std, dtype):
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return f32_to_bf16_bits(x) if dtype == BF16 else x


def make_chunk(cfg: LinkConfig, index: int, layer: int = 0):
    """KV of the store's index-th chunk in cross-attention layer `layer`, token-major.

    GQA: (k [len, H_kv, d_k], v [len, H_kv, d_v]); MLA: (k [len, 1, d_k], None),
    the value being the first d_v entries of each latent row. Every layer
    draws its own values (layer 0 keeps the single-layer stream).
    """
    entropy = [cfg.seed, _STREAM_CHUNK, index] + ([layer] if layer else [])
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(entropy)))
    n = cfg.chunk_length(index)
    k = _normal(rng, (n, cfg.n_kv_heads, cfg.d_k), 1.0, cfg.dtype)
    v = None if cfg.kind == MLA else _normal(rng, (n, cfg.n_kv_heads, cfg.d_v), 1.0, cfg.dtype)
    return k, v


def make_request(cfg: LinkConfig, plan: Plan, r: int):
    """(q [L_q, H_q, d_k], k_self [L_s, H_kv, d_k] or None, v_self or None) of request r."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([cfg.seed, _STREAM_REQ, r])))
    lq = int(plan.q_offsets[r + 1] - plan.q_offsets[r])
    q = _normal(rng, (lq, cfg.n_q_heads, cfg.d_k), cfg.q_std, cfg.dtype)
    if plan.self_offsets is None:
        return q, None, None
    ls = int(plan.self_offsets[r + 1] - plan.self_offsets[r])
    ks = _normal(rng, (ls, cfg.n_kv_heads, cfg.d_k), 1.0, cfg.dtype)
    vs = None if cfg.kind == MLA else _normal(rng, (ls, cfg.n_kv_heads, cfg.d_v), 1.0, cfg.dtype)
    return q, ks, vs


@dataclasses.dataclass
class Workload:
    cfg: LinkConfig
    plan: Plan
    chunk_ids: np.ndarray            # uint64 [store_chunks]
    q: np.ndarray                    # [Tq, H_q, d_k]
    k_self: Optional[np.ndarray]     # [Ts, H_kv, d_k]
    v_self: Optional[np.ndarray]     # [Ts, H_kv, d_v] (GQA only)

    def link_ids(self) -> np.ndarray:
        return self.chunk_ids[self.plan.chunk_index]

    def used_chunks(self) -> np.ndarray:
        return np.unique(self.plan.chunk_index)


def make_workload(cfg: LinkConfig) -> Workload:
    """Plan plus all per-request tensors; chunk tensors are made on demand by make_chunk."""
    plan = make_plan(cfg)
    qs, kss, vss = [], [], []
    for r in range(cfg.batch):
        q, ks, vs = make_request(cfg, plan, r)
        qs.append(q)
        kss.append(ks)
        vss.append(vs)
    q = np.concatenate(qs) if qs else np.zeros((0, cfg.n_q_heads, cfg.d_k))
    k_self = v_self = None
    if plan.self_offsets is not None:
        k_self = np.concatenate(kss)
        if cfg.kind == GQA:
            v_self = np.concatenate(vss)
    ids = np.array([chunk_id_of(i) for i in range(cfg.store_chunks)], dtype=np.uint64)
    return Workload(cfg, plan, ids, q, k_self, v_self)


def visible_pairs(cfg: LinkConfig, plan: Plan) -> int:
    """Visible (query token, key) pairs per head summed over the batch (masked pairs excluded)."""
    total = 0
    for r in range(plan.batch):
        ld = sum(cfg.chunk_length(int(c)) for c in
                 plan.chunk_index[plan.chunk_offsets[r]:plan.chunk_offsets[r + 1]])
        lq = int(plan.q_offsets[r + 1] - plan.q_offsets[r])
        ls = 0 if plan.self_offsets is None else int(plan.self_offsets[r + 1] - plan.self_offsets[r])
        own = 0
        if plan.self_offsets is not None:
            # row i sees own keys 0 .. i + ls - lq (inclusive)
            own = sum(i + 1 + ls - lq for i in range(lq))
        total += lq * ld + own
    return total


def small_config(name: str, *, dtype=BF16, kind=GQA, n_q_heads=8, n_kv_heads=2, d_k=128, d_v=None,
                 chunk_lens: Sequence[int] = (70, 64, 1, 130), batch=2, links=(1, 3),
                 q_len=(37, 5), self_len=(41, 5), q_std=None, scale=None, seed=7,
                 disjoint=False, decode=False) -> LinkConfig:
    """Small ragged workload for parity and edge-case tests."""
    if d_v is None:
        d_v = d_k if kind == GQA else max(1, d_k - 64)
    if kind == MLA:
        n_kv_heads = 1
    if q_std is None:
        q_std = 1.0 / math.sqrt(d_k) if dtype == BF16 else 1.0
    if scale is None:
        scale = 1.0 if dtype == BF16 else 1.0 / math.sqrt(d_k)
    return LinkConfig(name, dtype, kind, n_q_heads, n_kv_heads, d_k, d_v, len(chunk_lens),
                      tuple(int(x) for x in chunk_lens), batch, tuple(links),
                      q_len if isinstance(q_len, int) else tuple(q_len),
                      self_len if (self_len is None or isinstance(self_len, int)) else tuple(self_len),
                      q_std, scale, seed, disjoint, decode)
