"""GPU parity for Comb's layer structure: a store holding the chunk caches of
several cross-attention layers (Sec. 4.2-4.3: L_cross layers interleaved with
the decoder, each attending to its own document K and V), link calls that
name a layer, and link plans that resolve a request batch once and run it per
layer and per decode step. Every output is compared with the fp64 oracle on
that layer's caches, to the tolerances of test_gpu_link.py; the gather hook
is bit-exact per layer.
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from paper_2602_01519_amd import pic, runner
from paper_2602_01519_amd import workloads as W

from test_gpu_link import compare

pytestmark = pytest.mark.gpu

N_LAYERS = 3


def layered_store(cfg, wl, n_layers=N_LAYERS):
    """Store with every chunk the workload links, layer l holding make_chunk(.., layer=l)."""
    used = [int(c) for c in wl.used_chunks()]
    cap = max(64, sum(runner.padded(cfg.chunk_length(c)) for c in used))
    store = pic.Store(cfg.kind, cfg.dtype, cfg.n_kv_heads, cfg.d_k, cfg.d_v, cap, n_layers=n_layers)
    per_layer = [dict() for _ in range(n_layers)]
    stream = torch.cuda.current_stream().cuda_stream
    for c in used:
        ks, vs = [], []
        for l in range(n_layers):
            k, v = W.make_chunk(cfg, c, layer=l)
            per_layer[l][c] = (k, v)
            ks.append(k)
            vs.append(v)
        kd = runner.to_device(np.stack(ks), "cuda")
        vd = None if cfg.kind == W.MLA else runner.to_device(np.stack(vs), "cuda")
        store.put(int(wl.chunk_ids[c]), ks[0].shape[0], kd, vd, stream)
    torch.cuda.synchronize()
    return store, per_layer


def outputs(cfg, tq):
    et = torch.float32 if cfg.dtype == W.F32 else torch.int16
    return (torch.empty((tq, cfg.n_q_heads, cfg.d_v), dtype=et, device="cuda"),
            torch.empty((tq, cfg.n_q_heads), dtype=torch.float32, device="cuda"))


def tensors(wl):
    return (runner.to_device(wl.q, "cuda"), runner.to_device(wl.k_self, "cuda"),
            runner.to_device(wl.v_self, "cuda"))


LAYER_CASES = {
    "gqa_bf16": W.small_config("layers_gqa", d_k=128, chunk_lens=(70, 64, 1, 130), batch=3,
                               links=(1, 3), q_len=(37, 5, 64), self_len=(41, 5, 64), seed=21),
    "mla_bf16": W.small_config("layers_mla", kind=W.MLA, d_k=576, d_v=512, n_q_heads=4,
                               chunk_lens=(70, 64, 130), batch=2, links=(1, 3), q_len=(37, 5),
                               self_len=(41, 5), seed=22),
    "gqa_f32": W.small_config("layers_f32", dtype=W.F32, d_k=64, chunk_lens=(70, 64, 1, 130),
                              batch=2, links=(1, 3), q_len=(9, 3), self_len=(12, 3), seed=23),
}


@pytest.mark.parametrize("case", sorted(LAYER_CASES))
def test_layered_store_link_and_gather(case):
    cfg = LAYER_CASES[case]
    wl = W.make_workload(cfg)
    print(f"case {case}: layers={N_LAYERS}", flush=True)
    store, per_layer = layered_store(cfg, wl)
    try:
        q, ks, vs = tensors(wl)
        p = wl.plan
        for layer in (2, 0, 1):
            out, lse = outputs(cfg, wl.q.shape[0])
            pic.link_attn(store, p.chunk_offsets, wl.link_ids(), p.q_offsets, p.self_offsets,
                          cfg.n_q_heads, q, ks, vs, float(np.float32(cfg.scale)), out, lse,
                          stream=torch.cuda.current_stream().cuda_stream, layer=layer)
            torch.cuda.synchronize()
            ref, ref_lse = oracle.run_workload(wl, per_layer[layer])
            compare(cfg, runner.to_host(out, cfg.dtype), lse.cpu().numpy().astype(np.float64), ref,
                    ref_lse, label=f"{case} layer {layer}")
        # gather of one request's links, per layer, against the host concatenation
        idx = [int(c) for c in p.chunk_index[p.chunk_offsets[0]:p.chunk_offsets[1]]]
        n = sum(cfg.chunk_length(c) for c in idx)
        et = torch.float32 if cfg.dtype == W.F32 else torch.int16
        for layer in range(N_LAYERS):
            k_out = torch.empty((n, cfg.n_kv_heads, cfg.d_k), dtype=et, device="cuda")
            v_out = None if cfg.kind == W.MLA else torch.empty((n, cfg.n_kv_heads, cfg.d_v), dtype=et,
                                                               device="cuda")
            pic.debug_gather(store, [int(wl.chunk_ids[c]) for c in idx], k_out, v_out,
                             stream=torch.cuda.current_stream().cuda_stream, layer=layer)
            torch.cuda.synchronize()
            kh = np.concatenate([per_layer[layer][c][0] for c in idx])
            assert np.array_equal(k_out.cpu().numpy().view(kh.dtype), kh), f"layer {layer} K"
            if v_out is not None:
                vh = np.concatenate([per_layer[layer][c][1] for c in idx])
                assert np.array_equal(v_out.cpu().numpy().view(vh.dtype), vh), f"layer {layer} V"
        with pytest.raises(pic.PicError) as e:
            out, lse = outputs(cfg, wl.q.shape[0])
            pic.link_attn(store, p.chunk_offsets, wl.link_ids(), p.q_offsets, p.self_offsets,
                          cfg.n_q_heads, q, ks, vs, 1.0, out, lse, layer=N_LAYERS)
        assert e.value.status == pic.ERR_INVALID
    finally:
        store.close()


@pytest.mark.parametrize("case", sorted(LAYER_CASES))
def test_plan_runs_every_layer_with_fresh_tensors(case):
    """One plan, runs on several layers with two different sets of query and
    own-KV values (same shapes): each run matches the oracle on its layer."""
    cfg = LAYER_CASES[case]
    wl = W.make_workload(cfg)
    wl2 = W.make_workload(dataclasses.replace(cfg, seed=cfg.seed + 100))   # other q / own KV
    wl2 = dataclasses.replace(wl2, plan=wl.plan)
    assert wl2.q.shape == wl.q.shape
    print(f"case {case}: plan", flush=True)
    store, per_layer = layered_store(cfg, wl)
    p = wl.plan
    plan = pic.LinkPlan(store, p.chunk_offsets, wl.link_ids(), p.q_offsets, p.self_offsets,
                        cfg.n_q_heads)
    try:
        with pytest.raises(pic.PicError) as e:
            store.close()             # refused while the plan lives
        assert e.value.status == pic.ERR_INVALID
        stream = torch.cuda.current_stream().cuda_stream
        for layer, w in [(1, wl), (2, wl2), (0, wl), (1, wl2)]:
            q, ks, vs = tensors(w)
            out, lse = outputs(cfg, w.q.shape[0])
            plan.run(layer, q, ks, vs, float(np.float32(cfg.scale)), out, lse, stream=stream)
            torch.cuda.synchronize()
            ref, ref_lse = oracle.run_workload(w, per_layer[layer])
            compare(cfg, runner.to_host(out, cfg.dtype), lse.cpu().numpy().astype(np.float64), ref,
                    ref_lse, label=f"{case} plan layer {layer}")
        with pytest.raises(pic.PicError) as e:
            plan.run(N_LAYERS, q, ks, vs, 1.0, out, lse)
        assert e.value.status == pic.ERR_INVALID
        with pytest.raises(pic.PicError) as e:
            plan.run(0, q, None, vs, 1.0, out, lse)        # own KV missing
        assert e.value.status == pic.ERR_INVALID
    finally:
        plan.close()
        store.close()


@pytest.mark.parametrize("splits", [0, 3])
def test_decode_plan_cross_only_every_layer(splits):
    """Comb's cross-attention layers during decoding: one generated token per
    request attends to its documents only (Eq. 7-8, no own KV); the plan is
    made once and run for every layer of two decode steps."""
    cfg = W.small_config("layers_decode", d_k=128, chunk_lens=(70, 64, 1, 130, 512), batch=4,
                         links=(1, 4), q_len=1, self_len=None, seed=31, decode=True)
    wl = W.make_workload(cfg)
    print(f"case decode plan splits={splits}", flush=True)
    store, per_layer = layered_store(cfg, wl)
    p = wl.plan
    plan = pic.LinkPlan(store, p.chunk_offsets, wl.link_ids(), p.q_offsets, None, cfg.n_q_heads,
                        mode=pic.DECODE, num_splits=splits)
    try:
        stream = torch.cuda.current_stream().cuda_stream
        for step in range(2):
            w = wl if step == 0 else dataclasses.replace(
                W.make_workload(dataclasses.replace(cfg, seed=cfg.seed + 1)), plan=wl.plan)
            q = runner.to_device(w.q, "cuda")
            for layer in range(N_LAYERS):
                out, lse = outputs(cfg, w.q.shape[0])
                plan.run(layer, q, None, None, float(np.float32(cfg.scale)), out, lse, stream=stream)
                torch.cuda.synchronize()
                ref, ref_lse = oracle.run_workload(w, per_layer[layer])
                compare(cfg, runner.to_host(out, cfg.dtype), lse.cpu().numpy().astype(np.float64),
                        ref, ref_lse, label=f"decode step {step} layer {layer}")
    finally:
        plan.close()
        store.close()


# Link plans over the link tests' seeded shapes (prefill and decode plans, every
# kernel choice, cross-only calls): one plan per shape on a two-layer store,
# run on both layers, each run against the oracle on that layer's caches and
# bit for bit against the direct call on that layer.
@pytest.mark.parametrize("seed", range(24))
def test_random_plans(seed):
    from test_gpu_link import _sweep_config
    cfg = _sweep_config(seed)
    wl = W.make_workload(cfg)
    print(f"case plan sweep {seed}: {cfg}", flush=True)
    store, per_layer = layered_store(cfg, wl, n_layers=2)
    p = wl.plan
    plan = pic.LinkPlan(store, p.chunk_offsets, wl.link_ids(), p.q_offsets, p.self_offsets,
                        cfg.n_q_heads, mode=pic.DECODE if cfg.decode else pic.PREFILL)
    try:
        stream = torch.cuda.current_stream().cuda_stream
        q = runner.to_device(wl.q, "cuda")
        ks = None if wl.k_self is None else runner.to_device(wl.k_self, "cuda")
        vs = None if wl.v_self is None else runner.to_device(wl.v_self, "cuda")
        for layer in (1, 0):
            out, lse = outputs(cfg, wl.q.shape[0])
            plan.run(layer, q, ks, vs, float(np.float32(cfg.scale)), out, lse, stream=stream)
            torch.cuda.synchronize()
            ref, ref_lse = oracle.run_workload(wl, per_layer[layer])
            compare(cfg, runner.to_host(out, cfg.dtype), lse.cpu().numpy().astype(np.float64), ref,
                    ref_lse, label=f"plan sweep {seed} layer {layer}")
            # the direct call on the same layer returns the same bits (same kernels and splits)
            out2, lse2 = outputs(cfg, wl.q.shape[0])
            args = (store, p.chunk_offsets, wl.link_ids(), p.q_offsets, p.self_offsets,
                    cfg.n_q_heads, q, ks, vs, float(np.float32(cfg.scale)), out2, lse2)
            if cfg.decode:
                pic.link_decode(*args, stream=stream, layer=layer)
            else:
                pic.link_attn(*args, stream=stream, layer=layer)
            torch.cuda.synchronize()
            assert torch.equal(out, out2) and torch.equal(lse, lse2), \
                f"layer {layer}: plan and direct call differ"
    finally:
        plan.close()
        store.close()
