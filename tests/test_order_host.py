"""Host-only checks of the request order the planner gives a bf16 d=128
prefill call (pic_debug_request_order; no GPU needed).

The d=128 prefill kernel runs row block j % nrb of group x + n_xcd (j / nrb)
as workgroup j of XCD x (group = request position x kv heads + kv head), and
the hardware starts each workgroup on the first free CU of its XCD. The
reference below simulates that dispatch from the mapping alone, in its own
code: a row block takes its visible tiles (every document tile, then the own
tiles up to the one holding the last own key its last row sees, causal per
Sec. 4.1) plus 1.5. The planner's order must be a permutation, never finish
later than heaviest first, and its reported finish times must be those of
this simulation.
"""
import heapq
import math

import numpy as np
import pytest

from paper_2602_01519_amd import pic
from paper_2602_01519_amd import workloads as W

ROWS = 256   # rows (query token x query head of a GQA group) per workgroup


def simulate(order, q_len, self_len, doc_tiles, n_q, n_kv, cus, xcds):
    group = n_q // n_kv
    batch = len(order)
    nrb = max(1, math.ceil(max(q * group for q in q_len) / ROWS))
    n_groups = math.ceil(batch * n_kv / xcds) * xcds
    worst = 0.0
    for x in range(xcds):
        free = [0.0] * (cus // xcds)
        for j in range(n_groups // xcds * nrb):
            grp, rb = x + xcds * (j // nrb), j % nrb
            if grp >= batch * n_kv:
                continue
            r = order[grp // n_kv]
            rows = q_len[r] * group
            if rb * ROWS >= rows:
                continue
            last_q = min(rows - 1, rb * ROWS + ROWS - 1) // group
            own_last = last_q + self_len[r] - q_len[r]
            tiles = doc_tiles[r] + math.ceil(self_len[r] / 64)
            vis = min(doc_tiles[r] + own_last // 64 + 1, tiles) if own_last >= 0 else doc_tiles[r]
            t = heapq.heappop(free)
            heapq.heappush(free, t + vis + 1.5)
        worst = max(worst, max(free))
    return worst


def heaviest_first(q_len, self_len, doc_tiles):
    w = [(doc_tiles[r] + math.ceil(self_len[r] / 64)) * q_len[r] for r in range(len(q_len))]
    return sorted(range(len(q_len)), key=lambda r: -w[r])   # stable, as the planner's


def check(q_len, self_len, doc_tiles, n_q=32, n_kv=8, cus=256, xcds=8):
    order, finish = pic.debug_request_order(q_len, self_len, doc_tiles, n_q, n_kv, cus, xcds)
    order = [int(x) for x in order]
    assert sorted(order) == list(range(len(q_len)))
    lpt = heaviest_first(q_len, self_len, doc_tiles)
    if finish[0] == 0:          # no search: one round, or XCDs seeing different requests
        assert order == lpt
        return order, finish
    args = (q_len, self_len, doc_tiles, n_q, n_kv, cus, xcds)
    assert finish[0] == pytest.approx(simulate(lpt, *args), abs=1e-9)
    assert finish[1] == pytest.approx(simulate(order, *args), abs=1e-9)
    assert finish[1] <= finish[0]
    return order, finish


def test_long_rag_order():
    """The long_rag batch (16 requests, 8-20 chunks of 1024 tokens, 512 query
    and own tokens): four rounds of row blocks per XCD; the swaps take the
    simulated finish from 957 to 934 tiles (the average is 910)."""
    cfg = W.CONFIGS["long_rag"]
    plan = W.make_plan(cfg)
    links = np.diff(plan.chunk_offsets)
    doc_tiles = [int(n) * (cfg.chunk_len // 64) for n in links]
    q_len = [cfg.q_len] * cfg.batch
    order, finish = check(q_len, q_len, doc_tiles)
    assert finish[0] == pytest.approx(957.0) and finish[1] == pytest.approx(934.0)


def test_one_round_keeps_heaviest_first():
    """llama_prefill's 32 row blocks per XCD fill its 32 CUs once: no search."""
    order, finish = check([256] * 8, [256] * 8, [80, 96, 64, 80, 112, 80, 48, 80])
    assert list(finish) == [0.0, 0.0]


def test_xcds_seeing_different_requests_keep_heaviest_first():
    """With 2 kv heads over 8 XCDs the XCDs see different request sequences;
    the planner keeps heaviest first."""
    order, finish = check([64] * 40, [64] * 40, list(range(1, 41)), n_q=8, n_kv=2)
    assert list(finish) == [0.0, 0.0]


def test_random_batches():
    rng = np.random.default_rng(11)
    searched = 0
    for _ in range(40):
        b = int(rng.integers(3, 49))
        q_len = [int(x) for x in rng.integers(1, 300, size=b)]
        self_len = [q + int(x) for q, x in zip(q_len, rng.integers(0, 200, size=b))]
        doc_tiles = [int(x) for x in rng.integers(0, 300, size=b)]
        _, finish = check(q_len, self_len, doc_tiles)
        searched += finish[0] > 0
    assert searched >= 10


def test_bad_arguments():
    with pytest.raises(pic.PicError):
        pic.debug_request_order([4, -1], [4, 4], [1, 1], 32, 8, 256, 8)
    with pytest.raises(pic.PicError):
        pic.debug_request_order([4], [4], [1], 30, 8, 256, 8)
    with pytest.raises(pic.PicError):
        pic.debug_request_order([4], [4], [1], 32, 8, 250, 8)
