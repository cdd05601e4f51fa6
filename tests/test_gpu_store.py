"""GPU tests of the store's lifecycle: removal, page reuse and chunks split
over several runs of pages (the pool is reserved once, Sec. 5.3; chunks are
placed in 64-token pages, no copy ever moves them). Outputs are compared with
the fp64 oracle to the tolerances of test_gpu_link.py; gathers are bit-exact.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_01519_amd import pic, runner
from paper_2602_01519_amd import workloads as W

from test_gpu_link import compare

pytestmark = pytest.mark.gpu

CFG = W.small_config("store_life", d_k=128, chunk_lens=(130, 64, 200, 70, 250, 64), batch=1,
                     links=(1, 1), q_len=(29,), self_len=(33,), seed=51)


def stream():
    return torch.cuda.current_stream().cuda_stream


def put(store, cfg, c, n_layers=1, st=None):
    ks, vs = [], []
    for l in range(n_layers):
        k, v = W.make_chunk(cfg, c, layer=l)
        ks.append(k)
        vs.append(v)
    kd, vd = runner.to_device(np.stack(ks), "cuda"), runner.to_device(np.stack(vs), "cuda")
    if st is None:
        store.put(int(W.chunk_id_of(c)), ks[0].shape[0], kd, vd, stream())
    else:                              # another stream: wait for the uploads first
        st.wait_stream(torch.cuda.current_stream())
        store.put(int(W.chunk_id_of(c)), ks[0].shape[0], kd, vd, st.cuda_stream)
        st.synchronize()
    return [(ks[l], vs[l]) for l in range(n_layers)]


def link_and_check(store, cfg, idx, host, layer=0, label=""):
    """One request linking chunks idx (store indices) plus own KV, against the oracle."""
    wl = W.make_workload(cfg)
    co = np.array([0, len(idx)], np.int32)
    ids = np.array([W.chunk_id_of(c) for c in idx], np.uint64)
    q, ks, vs = (runner.to_device(x, "cuda") for x in (wl.q, wl.k_self, wl.v_self))
    et = torch.int16
    out = torch.empty((wl.q.shape[0], cfg.n_q_heads, cfg.d_v), dtype=et, device="cuda")
    lse = torch.empty((wl.q.shape[0], cfg.n_q_heads), dtype=torch.float32, device="cuda")
    pic.link_attn(store, co, ids, wl.plan.q_offsets, wl.plan.self_offsets, cfg.n_q_heads, q, ks, vs,
                  float(np.float32(cfg.scale)), out, lse, stream=stream(), layer=layer)
    torch.cuda.synchronize()
    ref, ref_lse = oracle.link_attn(dtype=cfg.dtype, mla=False, n_q_heads=cfg.n_q_heads, d_v=cfg.d_v,
                                    links=[[host[c] for c in idx]], q=wl.q, q_offsets=wl.plan.q_offsets,
                                    k_self=wl.k_self, v_self=wl.v_self,
                                    self_offsets=wl.plan.self_offsets, tau=float(np.float32(cfg.scale)))
    compare(cfg, runner.to_host(out, cfg.dtype), lse.cpu().numpy().astype(np.float64), ref, ref_lse,
            label=label)


def gather_check(store, cfg, idx, host, layer=0):
    n = sum(cfg.chunk_length(c) for c in idx)
    k_out = torch.empty((n, cfg.n_kv_heads, cfg.d_k), dtype=torch.int16, device="cuda")
    v_out = torch.empty((n, cfg.n_kv_heads, cfg.d_v), dtype=torch.int16, device="cuda")
    pic.debug_gather(store, [W.chunk_id_of(c) for c in idx], k_out, v_out, stream=stream(),
                     layer=layer)
    torch.cuda.synchronize()
    assert np.array_equal(k_out.cpu().numpy().view(np.uint16), np.concatenate([host[c][0] for c in idx]))
    assert np.array_equal(v_out.cpu().numpy().view(np.uint16), np.concatenate([host[c][1] for c in idx]))


@pytest.mark.parametrize("n_layers", [1, 2])
def test_chunk_split_over_page_runs(n_layers):
    """Pages: A 130 tok -> 3, B 64 -> 1, C 200 -> 4, D 70 -> 2, one free page.
    Removing B and D leaves runs of 1 and 3 pages; E (250 tok, 4 pages) must
    be split over both, and links through the split match the oracle."""
    print(f"case split runs layers={n_layers}", flush=True)
    store = pic.Store(W.GQA, W.BF16, CFG.n_kv_heads, 128, 128, 11 * 64, n_layers=n_layers)
    try:
        host = [dict() for _ in range(n_layers)]
        for c in (0, 1, 2, 3):
            for l, kv in enumerate(put(store, CFG, c, n_layers)):
                host[l][c] = kv
        assert store.usage() == (10 * 64, 11 * 64, 4)
        store.remove(W.chunk_id_of(1), stream())
        store.remove(W.chunk_id_of(3), stream())
        for l, kv in enumerate(put(store, CFG, 4, n_layers)):
            host[l][4] = kv
        assert store.usage()[1:] == (11 * 64, 3)
        with pytest.raises(pic.PicError) as e:         # full: one page short
            put(store, CFG, 5, n_layers)
        assert e.value.status == pic.ERR_OOM
        for l in range(n_layers):
            gather_check(store, CFG, [4, 0, 2], host[l], layer=l)
            link_and_check(store, CFG, [4, 0, 2, 4], host[l], layer=l, label=f"split layer {l}")
        with pytest.raises(pic.PicError) as e:
            store.lookup(W.chunk_id_of(1))
        assert e.value.status == pic.ERR_NOT_FOUND
    finally:
        store.close()


def test_removed_pages_are_reused_after_their_readers():
    """Link calls reading X are enqueued, X is removed on their stream and Y
    is put, on another stream, into a pool with room only for X's pages: the
    store must hold Y's put back until the link calls are done, whose result
    is X's."""
    print("case reuse after readers", flush=True)
    cfg = CFG
    store = pic.Store(W.GQA, W.BF16, cfg.n_kv_heads, 128, 128, 4 * 64)
    try:
        host = {2: put(store, cfg, 2)[0]}                  # X: 200 tokens, 4 pages, pool full
        wl = W.make_workload(cfg)
        q, ks, vs = (runner.to_device(x, "cuda") for x in (wl.q, wl.k_self, wl.v_self))
        out = torch.empty((wl.q.shape[0], cfg.n_q_heads, cfg.d_v), dtype=torch.int16, device="cuda")
        lse = torch.empty((wl.q.shape[0], cfg.n_q_heads), dtype=torch.float32, device="cuda")
        args = (np.array([0, 1], np.int32), np.array([W.chunk_id_of(2)], np.uint64), wl.plan.q_offsets,
                wl.plan.self_offsets, cfg.n_q_heads, q, ks, vs, float(np.float32(cfg.scale)), out, lse)
        for _ in range(20):                                 # several calls in flight
            pic.link_attn(store, *args, stream=stream())
        store.remove(W.chunk_id_of(2), stream())
        side = torch.cuda.Stream()
        host[4] = put(store, cfg, 4, st=side)[0]            # Y: 250 tokens, the same 4 pages
        torch.cuda.synchronize()
        ref, ref_lse = oracle.link_attn(dtype=cfg.dtype, mla=False, n_q_heads=cfg.n_q_heads,
                                        d_v=cfg.d_v, links=[[host[2]]], q=wl.q,
                                        q_offsets=wl.plan.q_offsets, k_self=wl.k_self,
                                        v_self=wl.v_self, self_offsets=wl.plan.self_offsets,
                                        tau=float(np.float32(cfg.scale)))
        compare(cfg, runner.to_host(out, cfg.dtype), lse.cpu().numpy().astype(np.float64), ref, ref_lse,
                label="X before removal")
        link_and_check(store, cfg, [4], host, label="Y in X's pages")
        gather_check(store, cfg, [4], host)
    finally:
        store.close()


def test_plan_keeps_its_chunks():
    print("case plan refs", flush=True)
    cfg = CFG
    store = pic.Store(W.GQA, W.BF16, cfg.n_kv_heads, 128, 128, 16 * 64)
    try:
        host = {}
        for c in (0, 2):
            host[c] = put(store, cfg, c)[0]
        wl = W.make_workload(cfg)
        plan = pic.LinkPlan(store, np.array([0, 2], np.int32),
                            np.array([W.chunk_id_of(0), W.chunk_id_of(0)], np.uint64),
                            wl.plan.q_offsets, wl.plan.self_offsets, cfg.n_q_heads)
        try:
            with pytest.raises(pic.PicError) as e:
                store.remove(W.chunk_id_of(0))
            assert e.value.status == pic.ERR_INVALID
            store.remove(W.chunk_id_of(2))                # not linked by the plan
        finally:
            plan.close()
        store.remove(W.chunk_id_of(0))                    # plan gone: allowed
        with pytest.raises(pic.PicError) as e:
            store.remove(W.chunk_id_of(0))
        assert e.value.status == pic.ERR_NOT_FOUND
        host[0] = put(store, cfg, 0)[0]                   # a removed id may be put again
        link_and_check(store, cfg, [0], host, label="re-put")
        assert store.usage()[2] == 1
    finally:
        store.close()


# Seeded sequences of puts, removals, gathers and links on a small pool
# (30 pages of 64 tokens, 1 or 2 layers, d 64 or 128), against a host model
# of the pages in use: a put fits exactly when the free pages (those of
# removed chunks included, once their readers are done) cover it, chunks
# may be split over several runs of pages, and every gather is bit-exact and
# every link matches the oracle.
@pytest.mark.parametrize("seed", range(4))
def test_random_put_remove_link(seed):
    import random
    rnd = random.Random(500 + seed)
    n_layers = 1 + seed % 2
    d = (64, 128)[(seed // 2) % 2]
    lens = tuple(rnd.randint(1, 500) for _ in range(12))
    cfg = W.small_config(f"store_rand{seed}", d_k=d, chunk_lens=lens, batch=1, links=(1, 1),
                         q_len=(29,), self_len=(33,), seed=600 + seed)
    cap = 30
    pages = [-(-n // 64) for n in lens]
    print(f"case store sequence {seed}: layers {n_layers} d {d} lens {lens}", flush=True)
    store = pic.Store(W.GQA, W.BF16, cfg.n_kv_heads, d, d, cap * 64, n_layers=n_layers)
    present = {}
    try:
        for op in range(40):
            c = rnd.randrange(len(lens))
            if c in present and rnd.random() < 0.6:
                store.remove(W.chunk_id_of(c), stream())
                del present[c]
            elif c not in present:
                torch.cuda.synchronize()            # removed chunks' readers are done
                free = cap - sum(pages[x] for x in present)
                if free >= pages[c]:
                    present[c] = put(store, cfg, c, n_layers)
                    used = sum(pages[x] for x in present) * 64
                    assert store.usage() == (used, cap * 64, len(present)), f"op {op}"
                else:
                    with pytest.raises(pic.PicError) as e:
                        put(store, cfg, c, n_layers)
                    assert e.value.status == pic.ERR_OOM, f"op {op}"
            assert store.usage()[2] == len(present)
            if op % 5 == 4 and present:
                idx = [rnd.choice(sorted(present)) for _ in range(rnd.randint(1, 5))]
                layer = rnd.randrange(n_layers)
                host = {x: present[x][layer] for x in present}
                gather_check(store, cfg, idx, host, layer=layer)
                link_and_check(store, cfg, idx, host, layer=layer, label=f"seq {seed} op {op}")
    finally:
        store.close()
