"""Child side of the store hand-over test (test_gpu_ipc.py): runs in a fresh
process spawned on the same GPU, imports the parent's exported store and
runs a link call on it. Not collected by pytest (no test_ prefix)."""
import traceback


def run(cfg, blob, out_q):
    try:
        import numpy as np
        import torch

        import oracle
        import parity_gate as G
        from paper_2602_01519_amd import pic, runner
        from paper_2602_01519_amd import workloads as W

        torch.cuda.set_device(0)
        store = pic.Store.import_(blob)
        wl = W.make_workload(cfg)
        p = wl.plan
        res = {}
        # the chunk index came along, and the store is read-only
        res["lookup"] = store.lookup(int(wl.chunk_ids[int(p.chunk_index[0])]))
        k = torch.zeros((64, cfg.n_kv_heads, cfg.d_k), dtype=torch.int16, device="cuda")
        v = None if cfg.kind == W.MLA else torch.zeros((64, cfg.n_kv_heads, cfg.d_v),
                                                         dtype=torch.int16, device="cuda")
        try:
            store.put(0x5EED, 64, k, v)
            res["put_status"] = 0
        except pic.PicError as e:
            res["put_status"] = e.status
        q = runner.to_device(wl.q, "cuda")
        ks = runner.to_device(wl.k_self, "cuda")
        vs = runner.to_device(wl.v_self, "cuda")
        out = torch.empty((wl.q.shape[0], cfg.n_q_heads, cfg.d_v), dtype=torch.int16, device="cuda")
        lse = torch.empty((wl.q.shape[0], cfg.n_q_heads), dtype=torch.float32, device="cuda")
        pic.link_attn(store, p.chunk_offsets, wl.link_ids(), p.q_offsets, p.self_offsets,
                      cfg.n_q_heads, q, ks, vs, float(np.float32(cfg.scale)), out, lse)
        torch.cuda.synchronize()
        o = runner.to_host(out, cfg.dtype)
        l = lse.cpu().numpy().astype(np.float64)
        chunks = {int(c): W.make_chunk(cfg, int(c)) for c in wl.used_chunks()}
        ref, ref_lse = oracle.run_workload(wl, chunks)
        dt = G.F32 if cfg.dtype == W.F32 else G.BF16
        res["bad"] = G.failures(dt, o, ref, l, ref_lse)
        res["metrics"] = G.metrics(o, ref)
        res["out"] = o
        res["lse"] = l
        store.close()
        out_q.put(res)
    except Exception:
        out_q.put({"error": traceback.format_exc()})
        raise
