"""GPU parity of the dense MLA projections (pic_mla_absorb_q, pic_mla_up_v)
against the fp64 oracle, and of one absorbed cross-attention layer of the
DeepSeek-V2-Lite backbone end to end (absorb -> link -> up).

Per-element bound of a projection output: the GPU accumulates K products in
fp32 and rounds the result to bf16 (nearest even), so
    |gpu - ref| <= 2^-8 |ref| + (K + 2) 2^-24 sum_k |a_k w_k|,
output rounding plus the worst-case fp32 accumulation error, checked element
by element against the oracle's exact products. The rope part of the absorbed
query is a copy and must be bit-exact. The end-to-end layer is held to the
link bar (bf16: max-abs 2e-2, mean-abs 2e-3), the oracle rounding its
intermediate query and latent output to bf16 where the C ABI hands bf16
tensors from one call to the next.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2602_01519_amd import pic, runner
from paper_2602_01519_amd import workloads as W

pytestmark = pytest.mark.gpu

D_NOPE, D_ROPE, R_LAT, D_V = 128, 64, 512, 128


def bf16(rng, shape, std=1.0):
    return W.f32_to_bf16_bits((rng.standard_normal(shape, dtype=np.float32) * np.float32(std)))


def f64(bits):
    return W.bf16_bits_to_f32(bits).astype(np.float64)


def check_bound(gpu, ref, absum, K, label):
    err = np.abs(gpu - ref)
    lim = 2.0 ** -8 * np.abs(ref) + (K + 2) * 2.0 ** -24 * absum
    worst = np.max(err - lim)
    print(f"{label}: max_abs={err.max():.3e} mean_abs={err.mean():.3e} worst margin={worst:.3e}",
          flush=True)
    assert np.all(err <= lim), f"{label}: {int(np.sum(err > lim))} elements outside the bound"


@pytest.mark.parametrize("T,H", [(37, 3), (1, 16), (2048, 16), (1541, 16), (300, 64), (1000, 64)])
def test_absorb_q(T, H):
    absorb_case(T, H, 1000 + T + H)


def absorb_case(T, H, seed):
    rng = np.random.default_rng(seed)
    q = bf16(rng, (T, H, D_NOPE + D_ROPE))
    w = bf16(rng, (H, R_LAT, D_NOPE), 1 / np.sqrt(D_NOPE))
    print(f"case absorb T={T} H={H}", flush=True)
    qd, wd = runner.to_device(q, "cuda"), runner.to_device(w, "cuda")
    out = torch.empty((T, H, R_LAT + D_ROPE), dtype=torch.int16, device="cuda")
    pic.mla_absorb_q(T, H, qd, wd, out, stream=torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    got_bits = out.cpu().numpy().view(np.uint16)
    ref = oracle.mla_absorb_q(q, w)
    absum = np.einsum("hjd,thd->thj", np.abs(f64(w)), np.abs(f64(q[:, :, :D_NOPE])))
    check_bound(f64(got_bits[:, :, :R_LAT]), ref[:, :, :R_LAT], absum, D_NOPE, f"absorb {T}x{H}")
    assert np.array_equal(got_bits[:, :, R_LAT:], q[:, :, D_NOPE:]), "rope part not copied exactly"


@pytest.mark.parametrize("T,H", [(37, 3), (1, 16), (130, 2), (2048, 16), (1541, 16), (300, 64), (1000, 64)])
def test_up_v(T, H):
    up_case(T, H, 2000 + T + H)


def up_case(T, H, seed):
    rng = np.random.default_rng(seed)
    o = bf16(rng, (T, H, R_LAT))
    w = bf16(rng, (H, D_V, R_LAT), 1 / np.sqrt(R_LAT))
    print(f"case up T={T} H={H}", flush=True)
    od, wd = runner.to_device(o, "cuda"), runner.to_device(w, "cuda")
    out = torch.empty((T, H, D_V), dtype=torch.int16, device="cuda")
    pic.mla_up_v(T, H, od, wd, out, stream=torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    got = f64(out.cpu().numpy().view(np.uint16))
    ref = oracle.mla_up_v(o, w)
    absum = np.einsum("hdr,thr->thd", np.abs(f64(w)), np.abs(f64(o)))
    check_bound(got, ref, absum, R_LAT, f"up {T}x{H}")


# Seeded token and head counts: ragged last token blocks, head counts that do
# and do not divide the XCD count, more heads than CUs per head.
def _sweep_shape(seed):
    import random
    rnd = random.Random(3000 + seed)
    H = rnd.choice([1, 2, 3, 5, 7, 8, 12, 16, 24, 40])
    T = rnd.randint(1, min(6000, 16000 // H))
    return T, H


@pytest.mark.parametrize("seed", range(12))
def test_projection_sweep(seed):
    T, H = _sweep_shape(seed)
    absorb_case(T, H, 4000 + seed)
    up_case(T, H, 5000 + seed)


def test_projection_errors_launch_nothing():
    x = torch.zeros(64, dtype=torch.int16, device="cuda")
    for fn in (pic.mla_absorb_q, pic.mla_up_v):
        for args in [(-1, 1, x, x, x), (1, 0, x, x, x), (1, 1, None, x, x),
                     (1, 1, x.data_ptr() + 2, x, x)]:
            with pytest.raises(pic.PicError) as e:
                fn(*args)
            assert e.value.status == pic.ERR_INVALID
        fn(0, 4, None, None, None)          # no tokens: nothing to do


@pytest.mark.parametrize("own", [False, True])
def test_absorbed_cross_attention_layer_end_to_end(own):
    """q [T,H,192] -> pic_mla_absorb_q -> pic_link_attn on an MLA store of latent
    chunks (cross-only as in Comb's cross-attention layers, Eq. 7-8, or with own
    KV) -> pic_mla_up_v, against the oracle chain."""
    cfg = W.small_config("mla_layer", kind=W.MLA, d_k=R_LAT + D_ROPE, d_v=R_LAT, n_q_heads=16,
                         chunk_lens=(70, 64, 130, 200), batch=3, links=(1, 3), q_len=(37, 5, 64),
                         self_len=(41, 5, 64) if own else None, scale=1 / np.sqrt(192), seed=41)
    wl = W.make_workload(cfg)
    rng = np.random.default_rng(42)
    T, H = wl.q.shape[0], cfg.n_q_heads
    q = bf16(rng, (T, H, D_NOPE + D_ROPE))
    w_uk_t = bf16(rng, (H, R_LAT, D_NOPE), 1 / np.sqrt(D_NOPE))
    w_uv = bf16(rng, (H, D_V, R_LAT), 1 / np.sqrt(R_LAT))
    print(f"case mla layer own={own} T={T}", flush=True)
    dw = runner.upload(wl)
    try:
        stream = torch.cuda.current_stream().cuda_stream
        qd = runner.to_device(q, "cuda")
        q_abs = torch.empty((T, H, R_LAT + D_ROPE), dtype=torch.int16, device="cuda")
        o_lat = torch.empty((T, H, R_LAT), dtype=torch.int16, device="cuda")
        lse = torch.empty((T, H), dtype=torch.float32, device="cuda")
        out = torch.empty((T, H, D_V), dtype=torch.int16, device="cuda")
        pic.mla_absorb_q(T, H, qd, runner.to_device(w_uk_t, "cuda"), q_abs, stream=stream)
        p = wl.plan
        pic.link_attn(dw.store, p.chunk_offsets, wl.link_ids(), p.q_offsets, p.self_offsets, H, q_abs,
                      dw.k_self, None, float(np.float32(cfg.scale)), o_lat, lse, stream=stream)
        pic.mla_up_v(T, H, o_lat, runner.to_device(w_uv, "cuda"), out, stream=stream)
        torch.cuda.synchronize()
        got = f64(out.cpu().numpy().view(np.uint16))
        # oracle chain, bf16 where the ABI passes bf16 between calls
        ref_q = W.f32_to_bf16_bits(oracle.mla_absorb_q(q, w_uk_t).astype(np.float32))
        ref_lat, _ = oracle.link_attn(dtype=W.BF16, mla=True, n_q_heads=H, d_v=R_LAT,
                                      links=oracle.workload_links(wl, dw.chunks), q=ref_q,
                                      q_offsets=p.q_offsets, k_self=wl.k_self, v_self=None,
                                      self_offsets=p.self_offsets, tau=float(np.float32(cfg.scale)))
        ref = oracle.mla_up_v(W.f32_to_bf16_bits(ref_lat.astype(np.float32)), w_uv)
        err = np.abs(got - ref)
        print(f"mla layer own={own}: max_abs={err.max():.3e} mean_abs={err.mean():.3e}", flush=True)
        assert np.all(np.isfinite(got))
        assert err.max() <= 2e-2 and err.mean() <= 2e-3
    finally:
        dw.close()
