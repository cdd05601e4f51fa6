"""The seeded input generator: determinism, bf16 rounding, plan shapes."""
import math

import numpy as np
import torch

from paper_2602_01519_amd import workloads as W


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(100000).astype(np.float32),
                        np.array([0.0, -0.0, 1.0, -1.5, 3.0e38, 1e-40], np.float32)])
    # ties: exact halfway bit patterns
    ties = (np.arange(1, 2000, dtype=np.uint32) << 16 | 0x8000).view(np.float32)
    x = np.concatenate([x, ties, -ties])
    ours = W.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(ours, ref)
    back = W.bf16_bits_to_f32(ours)
    assert np.array_equal(back, torch.from_numpy(x).to(torch.bfloat16).float().numpy())


def test_same_seed_same_bytes():
    cfg = W.CONFIGS["llama_prefill"]
    a = W.make_chunk(cfg, 5)
    b = W.make_chunk(cfg, 5)
    c = W.make_chunk(cfg, 6)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    assert not np.array_equal(a[0], c[0])
    p1, p2 = W.make_plan(cfg), W.make_plan(cfg)
    assert np.array_equal(p1.chunk_index, p2.chunk_index)


def test_config_shapes():
    c = W.CONFIGS
    p = W.make_plan(c["tiny_f32"])
    assert p.batch == 1 and len(p.chunk_index) == 4 and len(set(p.chunk_index)) == 4
    p = W.make_plan(c["llama_prefill"])
    assert p.batch == 8 and np.all(np.diff(p.chunk_offsets) == 10)
    for r in range(8):
        idx = p.chunk_index[p.chunk_offsets[r]:p.chunk_offsets[r + 1]]
        assert len(set(idx)) == 10
    p = W.make_plan(c["long_rag"])
    n = np.diff(p.chunk_offsets)
    assert p.batch == 16 and n.min() >= 8 and n.max() <= 20
    p = W.make_plan(c["decode"])
    assert p.batch == 64 and len(set(p.chunk_index)) == 1024       # disjoint
    assert np.all(np.diff(p.q_offsets) == 1) and np.all(np.diff(p.self_offsets) == 128)
    p = W.make_plan(c["mla"])
    assert p.batch == 8 and np.all(np.diff(p.chunk_offsets) == 12)
    k, v = W.make_chunk(c["mla"], 0)
    assert k.shape == (512, 1, 576) and v is None


def test_visible_pair_counts():
    cfg = W.CONFIGS["llama_prefill"]
    pairs = W.visible_pairs(cfg, W.make_plan(cfg))
    # 8 requests x (256 x 5120 + sum_{i<256} (i+1))
    assert pairs == 8 * (256 * 5120 + 256 * 257 // 2)
    cfg = W.CONFIGS["decode"]
    assert W.visible_pairs(cfg, W.make_plan(cfg)) == 64 * (16384 + 128)


def test_query_scale():
    cfg = W.CONFIGS["llama_prefill"].with_(batch=1)
    wl = W.make_workload(cfg)
    q = W.bf16_bits_to_f32(wl.q)
    assert abs(q.std() - 1 / math.sqrt(128)) < 2e-3
