"""bench.py's algorithmic work against closed forms of the workloads' shapes
(visible (query, key) pairs only, unique chunk bytes)."""
import importlib.util
import os

from paper_2602_01519_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def bench_module():
    spec = importlib.util.spec_from_file_location("bench", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def test_llama_prefill_flops_closed_form():
    # 8 requests x 32 heads; per (request, head) 256 queries see all 10 x 512
    # document keys and, causally, 1..256 own keys; 2 (d_k + d_v) FLOP per pair
    cfg = W.CONFIGS["llama_prefill"]
    flops, nbytes = bench_module().algorithmic(cfg, W.make_workload(cfg))
    pairs = 256 * 5120 + 256 * 257 // 2
    assert flops == 8 * 32 * pairs * 2 * (128 + 128)
    assert abs(flops - 1.761e11) / 1.761e11 < 1e-3


def test_mla_flops_closed_form():
    # 8 requests x 16 heads, 12 x 512 latent rows, 256 queries causal over
    # 256 own rows, 2 (576 + 512) FLOP per pair
    cfg = W.CONFIGS["mla"]
    flops, _ = bench_module().algorithmic(cfg, W.make_workload(cfg))
    assert flops == 8 * 16 * (256 * 12 * 512 + 256 * 257 // 2) * 2 * (576 + 512)


def test_decode_bytes_closed_form():
    # 64 requests, 16 private chunks of 1024 tokens each (8 heads x 128 x 2
    # bytes x (K + V) per token), 128 own tokens, one query token x 32 heads
    cfg = W.CONFIGS["decode"]
    _, nbytes = bench_module().algorithmic(cfg, W.make_workload(cfg))
    kv_tok = 8 * 128 * 2 * 2
    chunk = 64 * 16 * 1024 * kv_tok
    own = 64 * 128 * kv_tok
    q_out_lse = 64 * 32 * (128 + 128) * 2 + 64 * 32 * 4
    assert nbytes == chunk + own + q_out_lse
