"""GPU parity for the attention side of post-training PIC with scattered
recomputed tokens (CacheBlend-style: a fifth of every document's tokens are
recomputed at link time; Sec. 2, and Sec. 6.1 runs CacheBlend at 20%). The
token choice and the recompute itself need the model and are not built; the
two attention steps are:

1. the recomputed tokens attend as in a prefill of the concatenated
   documents: token at position P sees linked rows 0..P, the recomputed ones
   among them with their new K/V (pic_store_derive + pic_store_write_rows
   give each document a chunk with those rows replaced, sharing the other
   pages with the cached chunk; pic_link_req.q_doc_limits = P + 1);
2. the question links the patched chunks as usual (prefill, decode, plan).

Each call is compared with the fp64 oracle on the explicitly patched
arrays, to the tolerances of test_gpu_link.py; gathers are bit-exact.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_01519_amd import pic, runner
from paper_2602_01519_amd import workloads as W

from test_gpu_link import compare

pytestmark = pytest.mark.gpu

RATIO = 0.2                     # recomputed share of every document


def stream():
    return torch.cuda.current_stream().cuda_stream


def case_cfg(kind, dtype, d_k, seed):
    d_v = 512 if kind == W.MLA else d_k
    return W.small_config(f"blend_{seed}", kind=kind, dtype=dtype, d_k=d_k, d_v=d_v,
                          n_q_heads=4 if kind == W.MLA else 8, chunk_lens=(130, 200, 64, 250),
                          batch=1, links=(4, 4), q_len=(9,), self_len=(9,), seed=seed)


def dev(x):
    return runner.to_device(x, "cuda")


def pick_rows(rng, n):
    """A seeded fifth of a document's tokens, always including its first."""
    k = max(1, int(round(RATIO * n)))
    return np.unique(np.concatenate([[0], rng.choice(n, k, replace=False)])).astype(np.int32)


def patched(k, v, rows, k_new, v_new):
    k2 = k.copy()
    k2[rows] = k_new
    if v is None:
        return k2, None
    v2 = v.copy()
    v2[rows] = v_new
    return k2, v2


def gather(store, cfg, ids, layer=0):
    n = sum(store.lookup(i) for i in ids)
    et = torch.float32 if cfg.dtype == W.F32 else torch.int16
    k_out = torch.empty((n, cfg.n_kv_heads, cfg.d_k), dtype=et, device="cuda")
    v_out = None if cfg.kind == W.MLA else torch.empty((n, cfg.n_kv_heads, cfg.d_v), dtype=et,
                                                       device="cuda")
    pic.debug_gather(store, ids, k_out, v_out, stream=stream(), layer=layer)
    torch.cuda.synchronize()
    np_t = np.uint16 if cfg.dtype == W.BF16 else np.float32
    k = k_out.cpu().numpy().view(np_t)
    return k, None if v_out is None else v_out.cpu().numpy().view(np_t)


def run_link(store, cfg, co, ids, qo, so, q, ks, vs, lims=None, decode=False, splits=0, layer=0):
    tq = q.shape[0]
    et = torch.float32 if cfg.dtype == W.F32 else torch.int16
    out = torch.empty((tq, cfg.n_q_heads, cfg.d_v), dtype=et, device="cuda")
    lse = torch.empty((tq, cfg.n_q_heads), dtype=torch.float32, device="cuda")
    args = (store, co, np.asarray(ids, np.uint64), qo, so, cfg.n_q_heads, dev(q), dev(ks), dev(vs),
            float(np.float32(cfg.scale)), out, lse)
    if decode:
        pic.link_decode(*args, num_splits=splits, stream=stream(), layer=layer, q_doc_limits=lims)
    else:
        pic.link_attn(*args, stream=stream(), layer=layer, q_doc_limits=lims)
    torch.cuda.synchronize()
    return runner.to_host(out, cfg.dtype), lse.cpu().numpy().astype(np.float64)


def ref_link(cfg, links, q, qo, ks=None, vs=None, so=None, lims=None):
    return oracle.link_attn(dtype=cfg.dtype, mla=cfg.kind == W.MLA, n_q_heads=cfg.n_q_heads,
                            d_v=cfg.d_v, links=links, q=q, q_offsets=qo, k_self=ks, v_self=vs,
                            self_offsets=so, tau=float(np.float32(cfg.scale)), q_doc_limits=lims)


def rand_q(cfg, rng, n, heads=None, width=None, std=None):
    x = rng.standard_normal((n, heads or cfg.n_q_heads, width or cfg.d_k), dtype=np.float32)
    x *= np.float32(cfg.q_std if std is None else std)
    return W.f32_to_bf16_bits(x) if cfg.dtype == W.BF16 else x


CASES = {
    "gqa_bf16": (W.GQA, W.BF16, 128),      # matrix-core flash kernel
    "mla_bf16": (W.MLA, W.BF16, 576),      # MLA kernel
    "gqa_f32": (W.GQA, W.F32, 64),         # vector-ALU kernel
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_blend_recompute_and_link(case):
    kind, dtype, d_k = CASES[case]
    cfg = case_cfg(kind, dtype, d_k, seed=81 + sorted(CASES).index(case))
    n_docs = len(cfg.chunk_len)
    rng = np.random.default_rng(cfg.seed)
    docs = [W.make_chunk(cfg, c) for c in range(n_docs)]
    fresh = [W.make_chunk(cfg, c, layer=1) for c in range(n_docs)]    # stand-in recomputed KV
    rows = [pick_rows(rng, cfg.chunk_length(c)) for c in range(n_docs)]
    new_kv = [(fresh[c][0][rows[c]], None if kind == W.MLA else fresh[c][1][rows[c]])
              for c in range(n_docs)]
    spliced = [patched(*docs[c], rows[c], *new_kv[c]) for c in range(n_docs)]
    print(f"case {case}: rows per doc {[r.size for r in rows]}", flush=True)
    cap = sum(runner.padded(cfg.chunk_length(c)) for c in range(n_docs)) * 2
    store = pic.Store(kind, dtype, cfg.n_kv_heads, cfg.d_k, cfg.d_v, cap)
    try:
        base = [int(W.chunk_id_of(c)) for c in range(n_docs)]
        blend = [int(W.chunk_id_of(500 + c)) for c in range(n_docs)]
        for c in range(n_docs):
            store.put(base[c], cfg.chunk_length(c), dev(docs[c][0]), dev(docs[c][1]), stream())
            store.derive(blend[c], base[c], rows[c], stream())
            store.write_rows(blend[c], 0, rows[c], dev(new_kv[c][0]), dev(new_kv[c][1]), stream())
        torch.cuda.synchronize()
        for c in range(n_docs):           # the derived chunk is patched, the base is not
            k, v = gather(store, cfg, [blend[c]])
            assert np.array_equal(k, spliced[c][0])
            if v is not None:
                assert np.array_equal(v, spliced[c][1])
            k, _ = gather(store, cfg, [base[c]])
            assert np.array_equal(k, docs[c][0])

        # 1. recompute attention: every recomputed token, at its position in
        #    the concatenation, over the patched documents (cross-only)
        starts = np.cumsum([0] + [cfg.chunk_length(c) for c in range(n_docs)])
        pos = np.concatenate([starts[c] + rows[c] for c in range(n_docs)]).astype(np.int32)
        q1 = rand_q(cfg, rng, pos.size)
        co = np.array([0, n_docs], np.int32)
        qo = np.array([0, pos.size], np.int32)
        lims = pos + 1
        out, lse = run_link(store, cfg, co, blend, qo, None, q1, None, None, lims=lims)
        ref, ref_lse = ref_link(cfg, [spliced], q1, qo, lims=lims)
        compare(cfg, out, lse, ref, ref_lse, label=f"{case} recompute")

        # the same queries split over two requests with other link orders
        order2 = [2, 0, 3, 1]
        co2 = np.array([0, n_docs, 2 * n_docs], np.int32)
        half = pos.size // 2
        qo2 = np.array([0, half, pos.size], np.int32)
        lims2 = np.concatenate([lims[:half], rng.integers(0, starts[-1] + 1, pos.size - half)]).astype(np.int32)
        out, lse = run_link(store, cfg, co2, blend + [blend[i] for i in order2], qo2, None, q1, None,
                            None, lims=lims2)
        ref, ref_lse = ref_link(cfg, [spliced, [spliced[i] for i in order2]], q1, qo2, lims=lims2)
        compare(cfg, out, lse, ref, ref_lse, label=f"{case} recompute, two requests")

        # 2. the question over the patched documents, prefill and decode
        lq = cfg.q_length(0)
        q2 = rand_q(cfg, rng, lq)
        ks2 = rand_q(cfg, rng, lq, heads=cfg.n_kv_heads, std=1.0)
        vs2 = None if kind == W.MLA else rand_q(cfg, rng, lq, heads=cfg.n_kv_heads, width=cfg.d_v,
                                                std=1.0)
        so = np.array([0, lq], np.int32)
        out, lse = run_link(store, cfg, co, blend, so, so, q2, ks2, vs2)
        ref, ref_lse = ref_link(cfg, [spliced], q2, so, ks2, vs2, so)
        compare(cfg, out, lse, ref, ref_lse, label=f"{case} question prefill")
        qd = np.array([0, 1], np.int32)
        out, lse = run_link(store, cfg, co, blend, qd, so, q2[-1:], ks2, vs2, decode=True, splits=3)
        ref, ref_lse = ref_link(cfg, [spliced], q2[-1:], qd, ks2, vs2, so)
        compare(cfg, out, lse, ref, ref_lse, label=f"{case} question decode")
    finally:
        store.close()


@pytest.mark.parametrize("case", ["gqa_bf16", "mla_bf16"])
def test_limits_with_starts_over_derived_chunks(case):
    """Per-query limits, page-aligned starts and derived chunks in one call:
    the links read [derived doc 3 from token 128 ; base doc 1 ; derived doc 0
    from token 64], queries see different numbers of those rows."""
    kind, dtype, d_k = CASES[case]
    cfg = case_cfg(kind, dtype, d_k, seed=87)
    n_docs = len(cfg.chunk_len)
    rng = np.random.default_rng(88)
    docs = [W.make_chunk(cfg, c) for c in range(n_docs)]
    fresh = [W.make_chunk(cfg, c, layer=1) for c in range(n_docs)]
    rows = [pick_rows(rng, cfg.chunk_length(c)) for c in range(n_docs)]
    new_kv = [(fresh[c][0][rows[c]], None if kind == W.MLA else fresh[c][1][rows[c]])
              for c in range(n_docs)]
    spliced = [patched(*docs[c], rows[c], *new_kv[c]) for c in range(n_docs)]
    print(f"case {case} limits + starts + derived", flush=True)
    store = pic.Store(kind, dtype, cfg.n_kv_heads, cfg.d_k, cfg.d_v,
                      2 * sum(runner.padded(cfg.chunk_length(c)) for c in range(n_docs)))
    try:
        base = [int(W.chunk_id_of(c)) for c in range(n_docs)]
        blend = [int(W.chunk_id_of(600 + c)) for c in range(n_docs)]
        for c in range(n_docs):
            store.put(base[c], cfg.chunk_length(c), dev(docs[c][0]), dev(docs[c][1]), stream())
            store.derive(blend[c], base[c], rows[c], stream())
            store.write_rows(blend[c], 0, rows[c], dev(new_kv[c][0]), dev(new_kv[c][1]), stream())
        ids = [blend[3], base[1], blend[0]]
        starts = np.array([128, 0, 64], np.int32)
        links = [tuple(None if x is None else x[st:] for x in kv)
                 for kv, st in zip([spliced[3], docs[1], spliced[0]], starts)]
        ld = sum(k.shape[0] for k, _ in links)
        nq = 70
        q = rand_q(cfg, rng, nq)
        lims = rng.integers(0, ld + 1, nq).astype(np.int32)
        lims[:3] = (0, ld, 1)
        qo = np.array([0, nq], np.int32)
        tq = q.shape[0]
        et = torch.float32 if cfg.dtype == W.F32 else torch.int16
        out = torch.empty((tq, cfg.n_q_heads, cfg.d_v), dtype=et, device="cuda")
        lse = torch.empty((tq, cfg.n_q_heads), dtype=torch.float32, device="cuda")
        pic.link_attn(store, np.array([0, 3], np.int32), np.asarray(ids, np.uint64), qo, None,
                      cfg.n_q_heads, dev(q), None, None, float(np.float32(cfg.scale)), out, lse,
                      stream=stream(), chunk_starts=starts, q_doc_limits=lims)
        torch.cuda.synchronize()
        ref, ref_lse = ref_link(cfg, [links], q, qo, lims=lims)
        compare(cfg, runner.to_host(out, cfg.dtype), lse.cpu().numpy().astype(np.float64), ref,
                ref_lse, label=f"{case} limits + starts + derived")
    finally:
        store.close()


@pytest.mark.parametrize("case", ["gqa_bf16", "mla_bf16"])
def test_limits_in_decode_calls(case):
    """Decode-shaped calls with limits: one token per request (the links are
    cut on the host), and several tokens of one request with different
    limits (the GQA decode kernel has no per-row masks: the flash kernel
    takes the call)."""
    kind, dtype, d_k = CASES[case]
    cfg = case_cfg(kind, dtype, d_k, seed=91)
    n_docs = len(cfg.chunk_len)
    rng = np.random.default_rng(92)
    docs = [W.make_chunk(cfg, c) for c in range(n_docs)]
    print(f"case {case} decode limits", flush=True)
    store = pic.Store(kind, dtype, cfg.n_kv_heads, cfg.d_k, cfg.d_v,
                      sum(runner.padded(cfg.chunk_length(c)) for c in range(n_docs)))
    try:
        ids = [int(W.chunk_id_of(c)) for c in range(n_docs)]
        for c in range(n_docs):
            store.put(ids[c], cfg.chunk_length(c), dev(docs[c][0]), dev(docs[c][1]), stream())
        ld = sum(cfg.chunk_length(c) for c in range(n_docs))
        # 5 requests, one token each, own KV of 3 tokens
        B = 5
        co = np.arange(B + 1, dtype=np.int32) * n_docs
        qo = np.arange(B + 1, dtype=np.int32)
        so = np.arange(B + 1, dtype=np.int32) * 3
        q = rand_q(cfg, rng, B)
        ks = rand_q(cfg, rng, 3 * B, heads=cfg.n_kv_heads, std=1.0)
        vs = None if kind == W.MLA else rand_q(cfg, rng, 3 * B, heads=cfg.n_kv_heads, width=cfg.d_v,
                                               std=1.0)
        lims = np.array([0, 1, 129, 331, ld], np.int32)
        out, lse = run_link(store, cfg, co, ids * B, qo, so, q, ks, vs, lims=lims, decode=True)
        ref, ref_lse = ref_link(cfg, [docs] * B, q, qo, ks, vs, so, lims=lims)
        compare(cfg, out, lse, ref, ref_lse, label=f"{case} decode, one token per request")
        # one request, 12 tokens with different limits, own KV 12 tokens
        q = rand_q(cfg, rng, 12)
        ks = rand_q(cfg, rng, 12, heads=cfg.n_kv_heads, std=1.0)
        vs = None if kind == W.MLA else rand_q(cfg, rng, 12, heads=cfg.n_kv_heads, width=cfg.d_v,
                                               std=1.0)
        lims = np.sort(rng.integers(0, ld + 1, 12)).astype(np.int32)
        o12 = np.array([0, 12], np.int32)
        out, lse = run_link(store, cfg, np.array([0, n_docs], np.int32), ids, o12, o12, q, ks, vs,
                            lims=lims, decode=True, splits=4)
        ref, ref_lse = ref_link(cfg, [docs], q, o12, ks, vs, o12, lims=lims)
        compare(cfg, out, lse, ref, ref_lse, label=f"{case} decode, mixed limits")
    finally:
        store.close()


def test_plan_with_limits_over_layers():
    """A link plan carrying per-query limits, run on two store layers."""
    cfg = case_cfg(W.GQA, W.BF16, 128, seed=95)
    n_docs = len(cfg.chunk_len)
    rng = np.random.default_rng(96)
    print("case plan limits", flush=True)
    store = pic.Store(W.GQA, W.BF16, cfg.n_kv_heads, 128, 128,
                      sum(runner.padded(cfg.chunk_length(c)) for c in range(n_docs)), n_layers=2)
    try:
        host = [[W.make_chunk(cfg, c, layer=l) for c in range(n_docs)] for l in range(2)]
        ids = [int(W.chunk_id_of(c)) for c in range(n_docs)]
        for c in range(n_docs):
            k = np.stack([host[l][c][0] for l in range(2)])
            v = np.stack([host[l][c][1] for l in range(2)])
            store.put(ids[c], cfg.chunk_length(c), dev(k), dev(v), stream())
        ld = sum(cfg.chunk_length(c) for c in range(n_docs))
        nq = 40
        q = rand_q(cfg, rng, nq)
        lims = rng.integers(0, ld + 1, nq).astype(np.int32)
        co, qo = np.array([0, n_docs], np.int32), np.array([0, nq], np.int32)
        plan = pic.LinkPlan(store, co, np.asarray(ids, np.uint64), qo, None, cfg.n_q_heads,
                            q_doc_limits=lims)
        try:
            for layer in (1, 0):
                out = torch.empty((nq, cfg.n_q_heads, 128), dtype=torch.int16, device="cuda")
                lse = torch.empty((nq, cfg.n_q_heads), dtype=torch.float32, device="cuda")
                plan.run(layer, dev(q), None, None, float(np.float32(cfg.scale)), out, lse,
                         stream=stream())
                torch.cuda.synchronize()
                ref, ref_lse = ref_link(cfg, [host[layer]], q, qo, lims=lims)
                compare(cfg, runner.to_host(out, cfg.dtype), lse.cpu().numpy().astype(np.float64),
                        ref, ref_lse, label=f"plan layer {layer}")
        finally:
            plan.close()
    finally:
        store.close()


def test_derive_lifecycle_and_errors():
    """Page sharing: a derived chunk holds private copies only of the pages
    with its rows; removing the base keeps the shared pages alive; a page
    shared again by a later derive is no longer writable; and rejected
    arguments leave the store as it was."""
    cfg = case_cfg(W.GQA, W.BF16, 128, seed=97)
    print("case derive lifecycle", flush=True)
    n = 250                                        # 4 pages
    store = pic.Store(W.GQA, W.BF16, cfg.n_kv_heads, 128, 128, 9 * 64, n_layers=2)
    try:
        big = W.small_config("derive_big", d_k=128, chunk_lens=(250,), batch=1, links=(1, 1),
                             q_len=(1,), self_len=(1,), seed=98)
        host = [W.make_chunk(big, 0, layer=l) for l in range(2)]
        A, D1, D2 = (int(W.chunk_id_of(i)) for i in (0, 700, 701))
        store.put(A, n, dev(np.stack([h[0] for h in host])), dev(np.stack([h[1] for h in host])),
                  stream())
        assert store.usage()[0] == 4 * 64
        rows = np.array([3, 70, 71, 249], np.int32)             # pages 0, 1 and 3
        store.derive(D1, A, rows, stream())
        assert store.usage()[0] == 7 * 64 and store.lookup(D1) == n
        rng = np.random.default_rng(99)
        new = [(W.f32_to_bf16_bits(rng.standard_normal((4, 2, 128), dtype=np.float32)),
                W.f32_to_bf16_bits(rng.standard_normal((4, 2, 128), dtype=np.float32))) for _ in range(2)]
        for l in range(2):
            store.write_rows(D1, l, rows, dev(new[l][0]), dev(new[l][1]), stream())
        # page 2 (rows 128..191) is shared with A: not writable
        with pytest.raises(pic.PicError) as e:
            store.write_rows(D1, 0, np.array([130], np.int32), dev(new[0][0][:1]), dev(new[0][1][:1]))
        assert e.value.status == pic.ERR_INVALID
        with pytest.raises(pic.PicError) as e:                   # A was put, not derived
            store.write_rows(A, 0, np.array([3], np.int32), dev(new[0][0][:1]), dev(new[0][1][:1]))
        assert e.value.status == pic.ERR_INVALID
        for bad in ([5, 5], [7, 3], [-1], [250]):
            with pytest.raises(pic.PicError) as e:
                store.derive(int(W.chunk_id_of(702)), A, np.array(bad, np.int32))
            assert e.value.status == pic.ERR_INVALID
        with pytest.raises(pic.PicError) as e:
            store.derive(D1, A, rows)
        assert e.value.status == pic.ERR_EXISTS
        with pytest.raises(pic.PicError) as e:                   # 3 more pages: only 2 free
            store.derive(int(W.chunk_id_of(702)), A, np.array([0, 64, 128], np.int32))
        assert e.value.status == pic.ERR_OOM
        assert store.usage()[0] == 7 * 64 and store.usage()[2] == 2
        torch.cuda.synchronize()
        want = [patched(*host[l], rows, *new[l]) for l in range(2)]
        store.remove(A, stream())                                # D1 keeps page 2 alive
        torch.cuda.synchronize()
        for l in range(2):
            k, v = gather(store, cfg, [D1], layer=l)
            assert np.array_equal(k, want[l][0]) and np.array_equal(v, want[l][1])
        # D2 shares all of D1's pages except page 3: D1's pages 0 and 1 are shared now
        store.derive(D2, D1, np.array([200], np.int32), stream())
        with pytest.raises(pic.PicError) as e:
            store.write_rows(D1, 0, np.array([3], np.int32), dev(new[0][0][:1]), dev(new[0][1][:1]))
        assert e.value.status == pic.ERR_INVALID
        store.write_rows(D1, 1, np.array([249], np.int32), dev(new[0][0][3:]), dev(new[0][1][3:]),
                         stream())                                # page 3 of D1 is still its own
        torch.cuda.synchronize()
        k, v = gather(store, cfg, [D2], layer=1)
        assert np.array_equal(k, want[1][0]) and np.array_equal(v, want[1][1])
        k, v = gather(store, cfg, [D1], layer=1)
        d1_want = patched(*want[1], np.array([249]), new[0][0][3:], new[0][1][3:])
        assert np.array_equal(k, d1_want[0]) and np.array_equal(v, d1_want[1])
        # linking D1 and D2 together matches the oracle on their contents
        # (D1's layer 1 as written on the host: row 249 replaced once more)
        d1_l1 = d1_want
        rng = np.random.default_rng(100)
        q = W.f32_to_bf16_bits(rng.standard_normal((5, cfg.n_q_heads, 128), dtype=np.float32) *
                               np.float32(cfg.q_std))
        qo = np.array([0, 5], np.int32)
        out, lse = run_link(store, cfg, np.array([0, 2], np.int32), [D2, D1], qo, None, q, None, None,
                            layer=1)
        ref, ref_lse = ref_link(cfg, [[want[1], d1_l1]], q, qo)
        compare(cfg, out, lse, ref, ref_lse, label="derived chain")
        store.remove(D1, stream())
        store.remove(D2, stream())
        torch.cuda.synchronize()
        assert store.usage()[2] == 0
        # every page comes back: a 9-page chunk fits
        nine = W.small_config("derive_nine", d_k=128, chunk_lens=(9 * 64,), batch=1, links=(1, 1),
                              q_len=(1,), self_len=(1,), seed=101)
        k9 = [W.make_chunk(nine, 0, layer=l) for l in range(2)]
        store.put(int(W.chunk_id_of(703)), 9 * 64, dev(np.stack([x[0] for x in k9])),
                  dev(np.stack([x[1] for x in k9])), stream())
        assert store.usage()[0] == 9 * 64
    finally:
        store.close()


# Per-query limits on the linked rows over the link tests' seeded shapes
# (every kernel's limit variant: matrix-core d=128 and MLA, generic, decode
# calls), limits drawn uniformly, increasing with the query token (the
# CacheBlend pattern) or mostly full, against the oracle.
def _random_limits(wl, rng):
    cfg, p = wl.cfg, wl.plan
    lims = np.zeros(wl.q.shape[0], np.int32)
    style = rng.integers(0, 3)
    for r in range(cfg.batch):
        ld = sum(cfg.chunk_length(int(c))
                 for c in p.chunk_index[p.chunk_offsets[r]:p.chunk_offsets[r + 1]])
        q0, q1 = int(p.q_offsets[r]), int(p.q_offsets[r + 1])
        if style == 0:
            lims[q0:q1] = rng.integers(0, ld + 1, q1 - q0)
        elif style == 1:
            lims[q0:q1] = np.sort(rng.integers(0, ld + 1, q1 - q0))
        else:
            lims[q0:q1] = np.where(rng.random(q1 - q0) < 0.8, ld, rng.integers(0, ld + 1, q1 - q0))
    return lims


@pytest.mark.parametrize("seed", range(24))
def test_random_limits(seed):
    from test_gpu_link import _sweep_config
    cfg = _sweep_config(seed)
    wl = W.make_workload(cfg)
    lims = _random_limits(wl, np.random.default_rng(7000 + seed))
    print(f"case limits sweep {seed}: {cfg}", flush=True)
    p = wl.plan
    dw = runner.upload(wl)
    try:
        args = (dw.store, p.chunk_offsets, wl.link_ids(), p.q_offsets, p.self_offsets,
                cfg.n_q_heads, dw.q, dw.k_self, dw.v_self, float(np.float32(cfg.scale)), dw.out,
                dw.lse)
        if cfg.decode:
            pic.link_decode(*args, stream=stream(), q_doc_limits=lims)
        else:
            pic.link_attn(*args, stream=stream(), q_doc_limits=lims)
        torch.cuda.synchronize()
        out, lse = dw.results()
        links = oracle.workload_links(wl, dict(dw.chunks))
        ref, ref_lse = oracle.link_attn(
            dtype=cfg.dtype, mla=cfg.kind == W.MLA, n_q_heads=cfg.n_q_heads, d_v=cfg.d_v,
            links=links, q=wl.q, q_offsets=p.q_offsets, k_self=wl.k_self, v_self=wl.v_self,
            self_offsets=p.self_offsets, tau=float(np.float32(cfg.scale)), q_doc_limits=lims)
        compare(cfg, out, lse, ref, ref_lse, label=f"limits sweep {seed}")
    finally:
        dw.close()


# Seeded chains of derived chunks (derive from a base or from a derived
# chunk, bases removed while derived chunks live, rows written into derived
# chunks) against a host model of every chunk's content and of the chunks
# holding each 64-token page: a write is accepted exactly when each of its
# rows lies on a page only that derived chunk holds, every gather is
# bit-exact, and links over the live chunks match the oracle.
@pytest.mark.parametrize("seed", range(6))
def test_random_derive_chains(seed):
    import random
    rnd = random.Random(700 + seed)
    rng = np.random.default_rng(700 + seed)
    kind = W.MLA if seed % 2 else W.GQA
    d_k, d_v = (576, 512) if kind == W.MLA else (128, 128)
    lens = tuple(rnd.randint(1, 600) for _ in range(3))
    cfg = W.small_config(f"derive_rand{seed}", kind=kind, d_k=d_k, d_v=d_v, n_q_heads=8,
                         chunk_lens=lens, batch=1, links=(1, 1), q_len=(9,), self_len=(12,),
                         seed=710 + seed)
    print(f"case derive chains {seed}: {'MLA' if kind == W.MLA else 'GQA'} lens {lens}", flush=True)
    cap = sum(runner.padded(n) for n in lens) + 64 * 8 * 36   # every derive may copy 8 pages
    store = pic.Store(kind, cfg.dtype, cfg.n_kv_heads, d_k, d_v, cap)
    chunks = {}         # id -> [k, v, page ids, derived]
    refs = {}           # page id -> chunks holding it
    next_page = [0]

    def fresh_page():
        next_page[0] += 1
        refs[next_page[0]] = 1
        return next_page[0]

    def new_rows(n):
        k = rand_q(cfg, rng, n, heads=cfg.n_kv_heads, std=1.0)
        v = None if kind == W.MLA else rand_q(cfg, rng, n, heads=cfg.n_kv_heads, width=d_v, std=1.0)
        return k, v

    def write(cid, rows, expect_ok, op):
        k_new, v_new = new_rows(len(rows))
        args = (cid, 0, np.array(rows, np.int32), dev(k_new), None if v_new is None else dev(v_new),
                stream())
        if expect_ok:
            store.write_rows(*args)
            chunks[cid][0][rows] = k_new
            if v_new is not None:
                chunks[cid][1][rows] = v_new
        else:
            with pytest.raises(pic.PicError) as e:
                store.write_rows(*args)
            assert e.value.status == pic.ERR_INVALID, f"op {op}"

    try:
        for c in range(3):
            k, v = W.make_chunk(cfg, c)
            cid = int(W.chunk_id_of(c))
            store.put(cid, lens[c], dev(k), None if v is None else dev(v), stream())
            chunks[cid] = [k, v, [fresh_page() for _ in range(-(-lens[c] // 64))], False]
        next_id = int(W.chunk_id_of(900))
        for op in range(36):
            ids = sorted(chunks)
            r = rnd.random()
            if r < 0.35:
                parent = rnd.choice(ids)
                pk, pv, ppages, _ = chunks[parent]
                n = pk.shape[0]
                rows = sorted(set(rnd.randrange(n) for _ in range(rnd.randint(0, 6)))
                              | ({0} if rnd.random() < 0.3 else set())
                              | ({n - 1} if rnd.random() < 0.3 else set()))
                store.derive(next_id, parent, np.array(rows, np.int32), stream())
                own = {x // 64 for x in rows}
                pages = []
                for i, pg in enumerate(ppages):
                    if i in own:
                        pages.append(fresh_page())
                    else:
                        refs[pg] += 1
                        pages.append(pg)
                chunks[next_id] = [pk.copy(), None if pv is None else pv.copy(), pages, True]
                next_id += 1
            elif r < 0.5 and len(chunks) > 1:
                victim = rnd.choice(ids)
                store.remove(victim, stream())
                for pg in chunks[victim][2]:
                    refs[pg] -= 1
                del chunks[victim]
            elif r < 0.75:
                cid = rnd.choice(ids)
                n = chunks[cid][0].shape[0]
                alone = [x for x in range(n)
                         if chunks[cid][3] and refs[chunks[cid][2][x // 64]] == 1]
                pool = alone if alone and rnd.random() < 0.6 else range(n)
                rows = sorted(rnd.sample(pool, rnd.randint(1, min(8, len(pool)))))
                ok = chunks[cid][3] and all(refs[chunks[cid][2][x // 64]] == 1 for x in rows)
                write(cid, rows, ok, op)
            else:
                cid = rnd.choice(ids)
                k, v = gather(store, cfg, [cid])
                assert np.array_equal(k, chunks[cid][0]), f"op {op}: chunk {cid:#x} K"
                if v is not None:
                    assert np.array_equal(v, chunks[cid][1]), f"op {op}: chunk {cid:#x} V"
            if op % 6 == 5:
                ids = sorted(chunks)
                pick = [rnd.choice(ids) for _ in range(rnd.randint(1, 4))]
                q = rand_q(cfg, rng, 9)
                ks, vs = new_rows(12)
                so = np.array([0, 12], np.int32)
                qo = np.array([0, 9], np.int32)
                co = np.array([0, len(pick)], np.int32)
                out, lse = run_link(store, cfg, co, pick, qo, so, q, ks, vs)
                ref, ref_lse = ref_link(cfg, [[(chunks[i][0], chunks[i][1]) for i in pick]], q, qo,
                                        ks, vs, so)
                compare(cfg, out, lse, ref, ref_lse, label=f"derive chains {seed} op {op}")
        assert store.usage()[2] == len(chunks)
    finally:
        store.close()
