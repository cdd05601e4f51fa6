"""The parity bar can fail: CPU checks with the oracle alone.

At the decode workload's per-request shape (16 linked chunks of 1024 tokens
plus 128 own tokens, H_q 32 / H_kv 8, d 128, bf16), an output that misses one
64-key tile of a request's concatenated keys (the last 64 rows of one linked
chunk) must be rejected, although its element-wise errors stay inside the
max-abs / mean-abs bar (the outputs are ~1e-2, so those bars alone cannot see
it). The same outputs rounded the way the bf16 path rounds (probabilities and
output to bf16, nearest even) must pass, with margin: the relative L2 bar
is 2u = 2^-7 and the rounding model predicts about 0.6u.
"""
import dataclasses

import numpy as np

import oracle
import parity_gate as G
from paper_2602_01519_amd import workloads as W

REQS = 3     # requests of the decode plan used (each one a full-shape request)


def _decode_case():
    cfg = dataclasses.replace(W.CONFIGS["decode"], batch=REQS, store_chunks=REQS * 16)
    wl = W.make_workload(cfg)
    links = []
    for r in range(REQS):
        idx = wl.plan.chunk_index[wl.plan.chunk_offsets[r]:wl.plan.chunk_offsets[r + 1]]
        links.append([W.make_chunk(cfg, int(c)) for c in idx])
    return cfg, wl, links


def _oracle(cfg, wl, links):
    return oracle.link_attn(dtype=cfg.dtype, mla=False, n_q_heads=cfg.n_q_heads, d_v=cfg.d_v,
                            links=links, q=wl.q, q_offsets=wl.plan.q_offsets, k_self=wl.k_self,
                            v_self=wl.v_self, self_offsets=wl.plan.self_offsets,
                            tau=float(np.float32(cfg.scale)))


def _round_bf16(x):
    return W.bf16_bits_to_f32(W.f32_to_bf16_bits(np.asarray(x, np.float32))).astype(np.float64)


def _bf16_rounding_model(cfg, wl, links, r):
    """Request r's output as the bf16 path forms it: fp64 scores, then
    probabilities rounded to bf16, their sum, and the output rounded to bf16.
    An independent numpy restatement used only to check the bar's margin."""
    p = wl.plan
    widen = lambda a: W.bf16_bits_to_f32(a).astype(np.float64)
    k = np.concatenate([widen(kv[0]) for kv in links[r]] +
                       [widen(wl.k_self[p.self_offsets[r]:p.self_offsets[r + 1]])])
    v = np.concatenate([widen(kv[1]) for kv in links[r]] +
                       [widen(wl.v_self[p.self_offsets[r]:p.self_offsets[r + 1]])])
    q = widen(wl.q[p.q_offsets[r]:p.q_offsets[r + 1]])       # one token, decode
    g = cfg.n_q_heads // cfg.n_kv_heads
    out = np.zeros((1, cfg.n_q_heads, cfg.d_v))
    for h in range(cfg.n_q_heads):
        s = cfg.scale * (k[:, h // g, :] @ q[0, h])
        pr = _round_bf16(np.exp(s - s.max()))
        out[0, h] = _round_bf16(pr @ v[:, h // g, :] / pr.sum())
    return out


def test_gate_rejects_one_dropped_tile_at_decode_shape():
    cfg, wl, links = _decode_case()
    ref, ref_lse = _oracle(cfg, wl, links)
    dropped = [list(l) for l in links]
    k, v = dropped[1][7]
    dropped[1][7] = (k[:-64], v[:-64])          # request 1 loses 64 of its 16,512 keys
    out, lse = _oracle(cfg, wl, dropped)
    rows = slice(wl.plan.q_offsets[1], wl.plan.q_offsets[2])
    m = G.metrics(out[rows], ref[rows])
    t = G.TOL[G.BF16]
    # the element-wise bar alone would accept it ...
    assert m["max_abs"] <= t.max_abs and m["mean_abs"] <= t.mean_abs, m
    # ... the relative L2 bar does not, on the request and on the batch
    assert m["rel_l2"] > 4 * t.rel_l2, m
    bad = G.failures(G.BF16, out[rows], ref[rows])
    assert any("relative L2" in b for b in bad), bad
    assert G.failures(G.BF16, out, ref)


def test_bf16_rounding_model_passes_with_margin():
    cfg, wl, links = _decode_case()
    ref, ref_lse = _oracle(cfg, wl, links)
    for r in range(REQS):
        rows = slice(wl.plan.q_offsets[r], wl.plan.q_offsets[r + 1])
        got = _bf16_rounding_model(cfg, wl, links, r)
        m = G.metrics(got, ref[rows])
        assert not G.failures(G.BF16, got, ref[rows]), m
        assert m["rel_l2"] < 0.6 * G.TOL[G.BF16].rel_l2, m     # ~0.6u predicted, bar 2u
    # output rounding alone stays within u per element
    rounded = _round_bf16(ref)
    assert np.all(np.abs(rounded - ref) <= G.U_BF16 * np.abs(ref))
