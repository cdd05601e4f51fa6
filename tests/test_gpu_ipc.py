"""Store hand-over between processes on one GPU (the PIC manager passing
PICache handles to the inference engine in place, Sec. 5.3): the parent puts
chunks and exports its store; a child process spawned on the same GPU
imports it, links the chunks and is checked against the fp64 oracle; the
parent's own call on the same inputs must give the same bytes."""
import math
import multiprocessing as mp

import numpy as np
import pytest
import torch

import ipc_child
from paper_2602_01519_amd import pic, runner
from paper_2602_01519_amd import workloads as W
from test_gpu_link import compare

pytestmark = pytest.mark.gpu

CASES = {
    "gqa": W.small_config("ipc_gqa", d_k=128, n_q_heads=8, n_kv_heads=2,
                          chunk_lens=(70, 64, 1, 130, 300), batch=3, links=(2, 4),
                          q_len=(37, 5, 16), self_len=(41, 5, 16), seed=41),
    # a small call (tables as a kernel argument, the lean kernel) on the imported store
    "gqa_small": W.small_config("ipc_small", d_k=64, n_q_heads=8, n_kv_heads=2,
                                chunk_lens=(70, 64, 1, 130), batch=2, links=(1, 3),
                                q_len=(9, 3), self_len=(12, 3), seed=45),
    "mla": W.small_config("ipc_mla", kind=W.MLA, n_q_heads=16, d_k=576, d_v=512,
                          chunk_lens=(70, 64, 130), batch=2, links=(1, 3), q_len=(9, 4),
                          self_len=(9, 6), q_std=1.0, scale=1 / math.sqrt(192), seed=43),
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_child_process_links_the_exported_store(case):
    cfg = CASES[case]
    wl = W.make_workload(cfg)
    print(f"case ipc {case}", flush=True)
    dw = runner.upload(wl)
    try:
        blob = dw.store.export()
        ctx = mp.get_context("spawn")
        q = ctx.Queue()
        child = ctx.Process(target=ipc_child.run, args=(cfg, blob, q))
        child.start()
        try:
            res = q.get(timeout=240)
        finally:
            child.join(timeout=60)
        assert "error" not in res, res.get("error")
        assert child.exitcode == 0
        assert res["lookup"] == cfg.chunk_length(int(wl.plan.chunk_index[0]))
        assert res["put_status"] == pic.ERR_INVALID
        assert not res["bad"], res["bad"]
        print(f"ipc {case}: child rel_l2={res['metrics']['rel_l2']:.3e}", flush=True)
        # the parent's own call reads the same pool bytes with the same kernels
        dw.run()
        torch.cuda.synchronize()
        out, lse = dw.results()
        assert np.array_equal(out, res["out"]) and np.array_equal(lse, res["lse"])
    finally:
        dw.close()


def test_export_limits_and_size_query():
    store = pic.Store(W.GQA, W.BF16, 8, 128, 128, 4096)
    k = torch.zeros((100, 8, 128), dtype=torch.int16, device="cuda")
    store.put(7, 100, k, k)
    blob = store.export()
    assert len(blob) > 64
    with pytest.raises(pic.PicError) as e:     # not in the process that exported it
        bad = bytearray(blob)
        bad[0] ^= 0xFF
        pic.Store.import_(bytes(bad))
    assert e.value.status == pic.ERR_INVALID
    store.close()
    # 2 GiB and more: 8 heads * 256 * 2 B = 4 KiB per token, 2^19 tokens = 2 GiB
    big = pic.Store(W.GQA, W.BF16, 8, 128, 128, 1 << 19)
    with pytest.raises(pic.PicError) as e:
        big.export()
    assert e.value.status == pic.ERR_UNSUPPORTED
    big.close()
