"""fp64 oracle of the dense projections around absorbed MLA link attention
(test infrastructure only: tests, the smoke check and the benchmark's CPU
leg may use it; the product path never does).

DeepSeek-V2-Lite's multi-head latent attention (the MLA backbone of Sec. 5.1)
gives head h, for a latent row c (width r = 512) with rope part k_rope, the
key [W_UK[h] c | k_rope] and the value W_UV[h] c, where W_UK[h] and W_UV[h]
are d x r (d = 128). Since q_nope . (W_UK c) = (W_UK^T q_nope) . c and
sum_j p_j W_UV c_j = W_UV sum_j p_j c_j, attention can run on the latent rows
directly with the absorbed query [W_UK^T q_nope | q_rope] and its latent
output mapped back by W_UV. Each function below is that definition: one fp64
matrix product per head (numpy), nothing else.

Inputs are the bytes the GPU path reads -- bf16 bit patterns (uint16), widened
exactly -- or float arrays used as they are (for chaining oracle steps).
"""
from __future__ import annotations

import numpy as np


def _f64(a: np.ndarray) -> np.ndarray:
    a = np.asarray(a)
    if a.dtype == np.uint16:       # bf16 bit pattern: the high half of an fp32
        return (a.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return a.astype(np.float64)


def mla_absorb_q(q: np.ndarray, w_uk_t: np.ndarray) -> np.ndarray:
    """Absorbed query [T, H, r + rope] from q [T, H, d + rope] and W_UK^T [H, r, d].

    q_out[t, h, :r] = W_UK[h]^T q[t, h, :d]; q_out[t, h, r:] = q[t, h, d:].
    """
    q = _f64(q)
    w = _f64(w_uk_t)
    H, r, d = w.shape
    assert q.ndim == 3 and q.shape[1] == H and q.shape[2] >= d
    lat = np.einsum("hjd,thd->thj", w, q[:, :, :d])
    return np.concatenate([lat, q[:, :, d:]], axis=2)


def mla_up_v(o_lat: np.ndarray, w_uv: np.ndarray) -> np.ndarray:
    """Value-space output [T, H, d] = W_UV[h] o_lat[t, h] from o_lat [T, H, r] and W_UV [H, d, r]."""
    o = _f64(o_lat)
    w = _f64(w_uv)
    H, d, r = w.shape
    assert o.ndim == 3 and o.shape[1] == H and o.shape[2] == r
    return np.einsum("hdr,thr->thd", w, o)
