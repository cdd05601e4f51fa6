"""GPU parity for the attention side of post-training PIC with selective
recompute (EPIC-style: the first 64 tokens of every document are recomputed
at link time; Sec. 1 and 2.2, Sec. 6.1 runs EPIC with 64 tokens per
document). The recompute itself needs the model and is not built; its two
attention steps are:

1. the recomputed tokens of document r attend to documents 0..r-1 and,
   causally, to themselves: one link call whose request r links documents
   0..r-1 and carries the 64 tokens as its own KV;
2. the question links, for every document, [its recomputed tokens, put as a
   chunk of their own ; the cached chunk from token 64] -- links to
   page-aligned sub-ranges of chunks (pic_link_req.chunk_starts).

Each is compared with the fp64 oracle on the explicitly spliced key/value
arrays, to the tolerances of test_gpu_link.py.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_01519_amd import pic, runner
from paper_2602_01519_amd import workloads as W

from test_gpu_link import compare

pytestmark = pytest.mark.gpu

HEAD = 64        # recomputed tokens per document


def stream():
    return torch.cuda.current_stream().cuda_stream


def case_cfg(kind, dtype, d_k, seed):
    d_v = 512 if kind == W.MLA else d_k
    return W.small_config(f"recompute_{seed}", kind=kind, dtype=dtype, d_k=d_k, d_v=d_v,
                          n_q_heads=4 if kind == W.MLA else 8, chunk_lens=(130, 200, 64, 250),
                          batch=1, links=(4, 4), q_len=(9,), self_len=(9,), seed=seed)


def put_chunk(store, cid, k, v):
    store.put(int(cid), k.shape[0], runner.to_device(k, "cuda"),
              None if v is None else runner.to_device(v, "cuda"), stream())


def run_link(store, cfg, co, ids, qo, so, q, ks, vs, starts=None, decode=False, splits=0):
    tq = q.shape[0]
    et = torch.float32 if cfg.dtype == W.F32 else torch.int16
    out = torch.empty((tq, cfg.n_q_heads, cfg.d_v), dtype=et, device="cuda")
    lse = torch.empty((tq, cfg.n_q_heads), dtype=torch.float32, device="cuda")
    args = (store, co, np.asarray(ids, np.uint64), qo, so, cfg.n_q_heads, runner.to_device(q, "cuda"),
            runner.to_device(ks, "cuda"), runner.to_device(vs, "cuda"), float(np.float32(cfg.scale)),
            out, lse)
    if decode:
        pic.link_decode(*args, num_splits=splits, stream=stream(), chunk_starts=starts)
    else:
        pic.link_attn(*args, stream=stream(), chunk_starts=starts)
    torch.cuda.synchronize()
    return runner.to_host(out, cfg.dtype), lse.cpu().numpy().astype(np.float64)


CASES = {
    "gqa_bf16": (W.GQA, W.BF16, 128),
    "mla_bf16": (W.MLA, W.BF16, 576),
    "gqa_f32": (W.GQA, W.F32, 64),
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_recompute_and_spliced_link(case):
    kind, dtype, d_k = CASES[case]
    cfg = case_cfg(kind, dtype, d_k, seed=61 + sorted(CASES).index(case))
    n_docs = len(cfg.chunk_len)
    docs = [W.make_chunk(cfg, c) for c in range(n_docs)]           # cached caches
    recomp = [W.make_chunk(cfg, c, layer=1) for c in range(n_docs)]  # stand-in recomputed KV
    recomp = [(k[:HEAD], None if v is None else v[:HEAD]) for k, v in recomp]
    print(f"case {case}", flush=True)
    cap = sum(runner.padded(cfg.chunk_length(c)) for c in range(n_docs)) + n_docs * HEAD
    store = pic.Store(kind, dtype, cfg.n_kv_heads, cfg.d_k, cfg.d_v, cap)
    try:
        for c in range(n_docs):
            put_chunk(store, W.chunk_id_of(c), *docs[c])
            put_chunk(store, W.chunk_id_of(1000 + c), *recomp[c])
        rng = np.random.default_rng(cfg.seed)
        cast = (lambda x: W.f32_to_bf16_bits(x)) if dtype == W.BF16 else (lambda x: x)
        qstd = np.float32(cfg.q_std)

        # 1. recompute attention: request r = documents 0..r-1, own KV = the
        #    recomputed tokens of document r, queries = their new queries
        co = np.array([r * (r - 1) // 2 for r in range(n_docs + 1)], np.int32)
        ids = [W.chunk_id_of(c) for r in range(n_docs) for c in range(r)]
        qo = np.arange(n_docs + 1, dtype=np.int32) * HEAD
        q1 = cast(rng.standard_normal((n_docs * HEAD, cfg.n_q_heads, cfg.d_k), dtype=np.float32) * qstd)
        ks = np.concatenate([k for k, _ in recomp])
        vs = None if kind == W.MLA else np.concatenate([v for _, v in recomp])
        out, lse = run_link(store, cfg, co, ids, qo, qo, q1, ks, vs)
        ref, ref_lse = oracle.link_attn(dtype=dtype, mla=kind == W.MLA, n_q_heads=cfg.n_q_heads,
                                        d_v=cfg.d_v, links=[[docs[c] for c in range(r)] for r in range(n_docs)],
                                        q=q1, q_offsets=qo, k_self=ks, v_self=vs, self_offsets=qo,
                                        tau=float(np.float32(cfg.scale)))
        compare(cfg, out, lse, ref, ref_lse, label=f"{case} recompute")

        # 2. the question over spliced documents: [recomputed head ; cached tail]
        # a 64-token document has no tail (a start of 64 would be out of range)
        tails = [c for c in range(n_docs) if cfg.chunk_length(c) > HEAD]
        keep = [i for c in range(n_docs) for i in ((1000 + c, 0), (c, HEAD)) if i[0] >= 1000 or c in tails]
        ids = [W.chunk_id_of(i) for i, _ in keep]
        starts = np.array([s for _, s in keep], np.int32)
        co = np.array([0, len(ids)], np.int32)
        lq = cfg.q_length(0)
        qo, so = np.array([0, lq], np.int32), np.array([0, lq], np.int32)
        q2 = cast(rng.standard_normal((lq, cfg.n_q_heads, cfg.d_k), dtype=np.float32) * qstd)
        ks2 = cast(rng.standard_normal((lq, cfg.n_kv_heads, cfg.d_k), dtype=np.float32))
        vs2 = None if kind == W.MLA else cast(rng.standard_normal((lq, cfg.n_kv_heads, cfg.d_v),
                                                                  dtype=np.float32))
        links = []
        for i, s in keep:
            k, v = recomp[i - 1000] if i >= 1000 else docs[i]
            links.append((k[s:], None if v is None else v[s:]))
        ref, ref_lse = oracle.link_attn(dtype=dtype, mla=kind == W.MLA, n_q_heads=cfg.n_q_heads,
                                        d_v=cfg.d_v, links=[links], q=q2, q_offsets=qo, k_self=ks2,
                                        v_self=vs2, self_offsets=so, tau=float(np.float32(cfg.scale)))
        out, lse = run_link(store, cfg, co, ids, qo, so, q2, ks2, vs2, starts=starts)
        compare(cfg, out, lse, ref, ref_lse, label=f"{case} spliced prefill")
        # the same link as one generated token (decode path)
        qd = np.array([0, 1], np.int32)
        out, lse = run_link(store, cfg, co, ids, qd, so, q2[-1:], ks2, vs2, starts=starts, decode=True,
                            splits=3)
        ref, ref_lse = oracle.link_attn(dtype=dtype, mla=kind == W.MLA, n_q_heads=cfg.n_q_heads,
                                        d_v=cfg.d_v, links=[links], q=q2[-1:], q_offsets=qd, k_self=ks2,
                                        v_self=vs2, self_offsets=so, tau=float(np.float32(cfg.scale)))
        compare(cfg, out, lse, ref, ref_lse, label=f"{case} spliced decode")
    finally:
        store.close()


def test_starts_across_page_runs_and_errors():
    """A chunk split over two runs of pages, linked from tokens 64 and 128
    (both inside and at the boundary of a run), and rejected starts."""
    cfg = case_cfg(W.GQA, W.BF16, 128, seed=71)
    print("case starts across runs", flush=True)
    store = pic.Store(W.GQA, W.BF16, cfg.n_kv_heads, 128, 128, 11 * 64)
    try:
        sizes = {0: 130, 1: 64, 2: 200, 3: 70}             # pages 3, 1, 4, 2 (+1 free)
        big = W.small_config("starts_big", d_k=128, chunk_lens=(130, 64, 200, 70, 250), batch=1,
                             links=(1, 1), q_len=(9,), self_len=(9,), seed=72)
        host = {c: W.make_chunk(big, c) for c in range(5)}
        for c in range(4):
            assert host[c][0].shape[0] == sizes[c]
            put_chunk(store, W.chunk_id_of(c), *host[c])
        store.remove(W.chunk_id_of(1), stream())
        store.remove(W.chunk_id_of(3), stream())
        put_chunk(store, W.chunk_id_of(4), *host[4])       # 250 tokens over runs of 1 and 3 pages
        rng = np.random.default_rng(73)
        lq = 9
        q = W.f32_to_bf16_bits(rng.standard_normal((lq, cfg.n_q_heads, 128), dtype=np.float32) *
                               np.float32(cfg.q_std))
        ks = W.f32_to_bf16_bits(rng.standard_normal((lq, cfg.n_kv_heads, 128), dtype=np.float32))
        vs = W.f32_to_bf16_bits(rng.standard_normal((lq, cfg.n_kv_heads, 128), dtype=np.float32))
        qo = np.array([0, lq], np.int32)
        for starts in ([64, 0, 128], [128, 64, 192]):
            ids = [W.chunk_id_of(4), W.chunk_id_of(0), W.chunk_id_of(4)]
            links = [(host[c][0][s:], host[c][1][s:]) for c, s in zip((4, 0, 4), starts)]
            out, lse = run_link(store, cfg, np.array([0, 3], np.int32), ids, qo, qo, q, ks, vs,
                                starts=np.array(starts, np.int32))
            ref, ref_lse = oracle.link_attn(dtype=W.BF16, mla=False, n_q_heads=cfg.n_q_heads, d_v=128,
                                            links=[links], q=q, q_offsets=qo, k_self=ks, v_self=vs,
                                            self_offsets=qo, tau=float(np.float32(cfg.scale)))
            compare(cfg, out, lse, ref, ref_lse, label=f"starts {starts}")
        for bad in ([32, 0, 0], [-64, 0, 0], [256, 0, 0], [0, 192, 0]):
            with pytest.raises(pic.PicError) as e:
                run_link(store, cfg, np.array([0, 3], np.int32),
                         [W.chunk_id_of(4), W.chunk_id_of(0), W.chunk_id_of(4)], qo, qo, q, ks, vs,
                         starts=np.array(bad, np.int32))
            assert e.value.status == pic.ERR_INVALID
    finally:
        store.close()
