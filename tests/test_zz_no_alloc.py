"""pic_link_decode_noalloc (the decode entry point that allocates nothing:
its tables and workspace live in the library's static device scratch)
against pic_link_decode, through the C ABI.

Two calls in a row on one stream, the second with a smaller batch (the
scratch keeps the first call's contents), each compared with
pic_link_decode's output on the same inputs (same kernels and split count,
so the results are identical) and with the fp64 oracle to the parity bar; a
call that needs more than the scratch is rejected before any device work.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_01519_amd import pic, runner
from paper_2602_01519_amd import workloads as W
from test_gpu_link import _sweep_config, compare

pytestmark = pytest.mark.gpu


def _case(batch, seed):
    return W.small_config("noalloc", d_k=128, n_q_heads=32, n_kv_heads=8,
                          chunk_lens=(1024, 700, 64, 1, 300, 512, 1024, 129), batch=batch,
                          links=(2, 6), q_len=tuple((1, 3, 1, 16, 2, 1)[r % 6] for r in range(batch)),
                          self_len=tuple((128, 5, 65, 40, 200, 1)[r % 6] for r in range(batch)),
                          seed=seed, decode=True)


def _run(cfg, splits):
    wl = W.make_workload(cfg)
    dw = runner.upload(wl)
    p = wl.plan
    args = (dw.store, p.chunk_offsets, wl.link_ids(), p.q_offsets, p.self_offsets, cfg.n_q_heads,
            dw.q, dw.k_self, dw.v_self, float(np.float32(cfg.scale)))
    stream = torch.cuda.current_stream().cuda_stream
    try:
        out_n = torch.full_like(dw.out, 77)
        lse_n = torch.full_like(dw.lse, 5.0)
        pic.link_decode_noalloc(*args, out_n, lse_n, num_splits=splits, stream=stream)
        pic.link_decode(*args, dw.out, dw.lse, num_splits=splits, stream=stream)
        torch.cuda.synchronize()
        a, la = runner.to_host(out_n, cfg.dtype), lse_n.cpu().numpy().astype(np.float64)
        b, lb = dw.results()
        assert np.array_equal(a, b) and np.array_equal(la, lb), "differs from pic_link_decode"
        ref, ref_lse = oracle.run_workload(wl, dw.chunks)
        compare(cfg, a, la, ref, ref_lse, label=f"noalloc batch {cfg.batch} splits {splits}")
    finally:
        dw.close()


@pytest.mark.parametrize("splits", [0, 3])
def test_noalloc_matches_decode_twice_shrinking(splits):
    _run(_case(6, 31), splits)
    _run(_case(3, 32), splits)


# The decode-shaped draws of the link tests' seeded sweep (fp32 / bf16, GQA /
# MLA, several head widths and groups, ragged chunks): each through the entry
# point twice in a row, against pic_link_decode and the oracle.
_DECODE_SEEDS = [s for s in range(96) if _sweep_config(s).decode][:12]


@pytest.mark.parametrize("seed", _DECODE_SEEDS)
def test_noalloc_sweep(seed):
    cfg = _sweep_config(seed)
    _run(cfg, 0)
    _run(cfg, 0)


def test_noalloc_rejects_a_call_beyond_the_scratch():
    """140 requests of 128 own tokens need 140 * 128 * 8 * 256 * 2 B = 73 MB of
    own-KV layout, more than the 64 MiB scratch: INVALID, outputs untouched."""
    B, L, hkv, hq, d = 140, 128, 8, 32, 128
    store = pic.Store(W.GQA, W.BF16, hkv, d, d, 64)
    ks = torch.zeros((B * L, hkv, d), dtype=torch.int16, device="cuda")
    vs = torch.zeros_like(ks)
    q = torch.zeros((B, hq, d), dtype=torch.int16, device="cuda")
    out = torch.full((B, hq, d), 1234, dtype=torch.int16, device="cuda")
    lse = torch.full((B, hq), 5.0, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    co = np.zeros(B + 1, np.int32)
    qo = np.arange(B + 1, dtype=np.int32)
    so = np.arange(B + 1, dtype=np.int32) * L
    with pytest.raises(pic.PicError) as e:
        pic.link_decode_noalloc(store, co, np.zeros(0, np.uint64), qo, so, hq, q, ks, vs, 1.0,
                                out, lse)
    assert e.value.status == pic.ERR_INVALID
    assert "scratch" in pic.last_error()
    torch.cuda.synchronize()
    assert bool(torch.all(out == 1234)) and bool(torch.all(lse == 5.0))
    store.close()
