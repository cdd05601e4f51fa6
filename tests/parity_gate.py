"""The parity bar between the HIP path and the fp64 oracle (shared by every
GPU parity test and by the CPU check that the bar can fail).

Element-wise bar (the stated accuracy requirement): bf16 inputs max-abs
<= 2e-2 and mean-abs <= 2e-3 over the compared outputs; fp32 inputs max-abs
and mean-abs <= 1e-4.

Relative L2 bar, ||out - ref||_2 / ||ref||_2, derived from how the bf16 path
rounds (the kernels accumulate Q K^T and P V in fp32, round the
probabilities P to bf16 before the P V product and the output to bf16; both
roundings are to nearest even, unit roundoff u = 2^-8):
  * the output rounding changes every element by a relative |delta| <= u;
  * the P rounding changes out[i] = sum_j p_j v_j / sum_j p_j (the row sum
    adds the same rounded p_j) by sum_j (p_j / l) delta_j (v_j - out[i]) to
    first order; with independent rounding errors and values drawn
    independently of the scores its root mean square is that of
    sum_j (p_j / l) delta_j v_j, i.e. |out| times an RMS |delta| <= u.
  Each term's RMS is at most u, so ||e|| / ||ref|| <= 2u = 2^-7 holds with
  room; both roundings, RMS relative error of a round to nearest ~u/sqrt(6),
  give about 0.6u = 2.3e-3 in expectation. fp32 path: no bf16 rounding; the
  error is that of fp32 dot products and exponentials (u = 2^-24, scores of
  <= 576 products), bounded here by 1e-5, about 170 u.
  The bar catches what the element-wise one misses at full size, where the
  outputs themselves are ~1e-2: dropping one 64-key tile of a 16,512-key
  decode row moves the output by a relative ~sqrt(64 / 16512) = 0.06.

Log-sum-exp (absolute): fp32 1e-4; bf16 4e-3, because the row sum adds
probabilities rounded to bf16, so ln(sum) can be off by up to
ln(1 + 2^-8) = 3.9e-3 in a row with few visible keys.
"""
from __future__ import annotations

import dataclasses
import json
import os

import numpy as np

F32, BF16 = 0, 1
U_BF16 = 2.0 ** -8


@dataclasses.dataclass(frozen=True)
class Tol:
    max_abs: float
    mean_abs: float
    lse: float
    rel_l2: float


TOL = {F32: Tol(1e-4, 1e-4, 1e-4, 1e-5), BF16: Tol(2e-2, 2e-3, 4e-3, 2 * U_BF16)}


def metrics(out, ref):
    err = np.abs(out - ref)
    nref = float(np.linalg.norm(ref))
    return {
        "max_abs": float(err.max()) if err.size else 0.0,
        "mean_abs": float(err.mean()) if err.size else 0.0,
        "rel_l2": float(np.linalg.norm(err)) / nref if nref > 0 else 0.0,
        "elements": int(err.size),
    }


def failures(dtype, out, ref, lse=None, ref_lse=None):
    """Which parts of the bar (out, ref: float64 arrays of the compared
    outputs; lse, ref_lse optional) are violated: an empty list passes."""
    t = TOL[dtype]
    bad = []
    if not np.all(np.isfinite(out)):
        bad.append("non-finite output")
        return bad
    m = metrics(out, ref)
    if m["max_abs"] > t.max_abs:
        bad.append(f"max abs err {m['max_abs']:.3e} > {t.max_abs:.1e}")
    if m["mean_abs"] > t.mean_abs:
        bad.append(f"mean abs err {m['mean_abs']:.3e} > {t.mean_abs:.1e}")
    if m["rel_l2"] > t.rel_l2:
        bad.append(f"relative L2 err {m['rel_l2']:.3e} > {t.rel_l2:.2e}")
    if lse is not None:
        fin = np.isfinite(ref_lse)
        if not np.array_equal(fin, np.isfinite(lse)):
            bad.append("lse finiteness differs")
        elif not np.all(np.isneginf(lse[~fin])):
            bad.append("lse of an empty key set is not -inf")
        elif fin.any() and np.abs(lse[fin] - ref_lse[fin]).max() > t.lse:
            bad.append(f"lse err {np.abs(lse[fin] - ref_lse[fin]).max():.3e} > {t.lse:.1e}")
    return bad


def record(label, dtype, out, ref):
    """Prints the observed errors against the bar; with PIC_PARITY_LOG set,
    also appends them to that JSON-lines file (the margins DESIGN records)."""
    m = metrics(out, ref)
    t = TOL[dtype]
    m.update(label=label, dtype="f32" if dtype == F32 else "bf16",
             rel_l2_margin=(t.rel_l2 / m["rel_l2"]) if m["rel_l2"] > 0 else None)
    print(f"{label}: max_abs={m['max_abs']:.3e} mean_abs={m['mean_abs']:.3e} "
          f"rel_l2={m['rel_l2']:.3e}", flush=True)
    path = os.environ.get("PIC_PARITY_LOG")
    if path:
        with open(path, "a") as f:
            f.write(json.dumps(m) + "\n")
    return m
