#!/usr/bin/env python3
"""Benchmark of the link-stage attention hot path on one MI355X.

One step = one pic_link_attn (or pic_link_decode) call over the whole batch
of the workload: host chunk-id resolution and chunk-table upload, the
attention kernel, and the split-K combine when used. The chunk store is
filled (compile side, not timed) before the timed region, so every input is
resident in HBM when timing starts.

Default workload: the long-RAG link, the largest single-GPU configuration
(Llama-3-8B head shape H_q 32, H_kv 8, d 128; 16 requests, each linking 8-20
chunks of 1024 tokens from a 256-chunk store, then 512 query tokens with
causal own KV; bf16). Prints one JSON line.

Warm-up: the W untimed steps are extended, if needed, to at least
--min-warmup-s seconds of work. The GPU's core clock ramps up over the first
tens of milliseconds of sustained load; without this, a short warm-up times
partly ramped clocks (measured: 200 vs 175 us per llama_prefill kernel).
The JSON line reports both the requested W and the steps actually run.

Algorithmic work counts visible (query, key) pairs only:
  FLOPs = sum_r H_q (2 d_k + 2 d_v) P_r,  P_r = L_q L_d + sum_{i<L_q} (i + 1 + L_s - L_q)
  bytes = Q + out + lse + own KV + each linked chunk's KV once.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 matrix peak
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E
PEAK_FP32_TFLOPS = 157.3       # MI355X fp32: dense matrix and vector (packed) peaks alike
PROF_EVERY = 5                # timed steps per kernel-timing event pair

# Source file of each attention kernel: a traffic record measured with
# rocprofv3 counters is used only while the kernel source is unchanged.
KERNEL_SOURCES = {
    "link_mfma_d128_kernel": "kernels_mfma_d128.hip",
    "link_decode_d128_kernel": "kernels_decode_d128.hip",
    "link_mla_kernel": "kernels_mla.hip",
    "link_valu_kernel": "kernels_generic.hip",
    "link_small_kernel": "kernels_generic.hip",
    "link_lean_kernel": "kernels_generic.hip",
    "proj_kernel": "kernels_mla_proj.hip",
}
PROFILES = os.path.join(ROOT, "profiles")


def kernel_source_sha(kernel: str):
    import hashlib
    for k, f in KERNEL_SOURCES.items():
        if kernel.startswith(k):
            path = os.path.join(ROOT, "paper_2602_01519_amd", "csrc", f)
            return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]
    return None


def traffic_record(kernel: str, workload: str):
    """HBM bytes per launch from a committed counter record, if still valid."""
    base = kernel.split("<")[0]
    path = os.path.join(PROFILES, f"traffic_{base}_{workload}.json")
    if not os.path.exists(path):
        return None
    rec = json.load(open(path))
    if rec.get("kernel_source_sha") != kernel_source_sha(kernel):
        return None
    return rec.get("hbm_bytes_per_launch")


def _pmc_per_dispatch(csv_path: str, kernel_prefix: str, counter: str):
    import csv
    vals = [float(r["Counter_Value"]) for r in csv.DictReader(open(csv_path))
            if r["Counter_Name"] == counter and kernel_prefix in r["Kernel_Name"]]
    if not vals:
        raise SystemExit(f"no {counter} samples for {kernel_prefix} in {csv_path}")
    return sum(vals) / len(vals)


# HBM bytes from the L2 -> memory request counters of gfx950: reads by request
# size (32, 64 or 128 bytes), writes as 32- or 64-byte requests. (The
# profiler's derived FETCH_SIZE takes 128-byte reads from a counter that
# reads zero on gfx950 and counts them as 64 bytes: a 2 GiB read stream
# shows as 1 GiB.)
RD_COUNTERS = ("TCC_EA0_RDREQ_32B", "TCC_EA0_RDREQ_64B", "TCC_EA0_RDREQ_128B")
WR_COUNTERS = ("TCC_EA0_WRREQ", "TCC_EA0_WRREQ_64B")


def read_bytes(rd_csv: str, kernel_prefix: str):
    n32, n64, n128 = (_pmc_per_dispatch(rd_csv, kernel_prefix, c) for c in RD_COUNTERS)
    return 32 * n32 + 64 * n64 + 128 * n128


def write_bytes(wr_csv: str, kernel_prefix: str):
    wr, wr64 = (_pmc_per_dispatch(wr_csv, kernel_prefix, c) for c in WR_COUNTERS)
    return 32 * (wr - wr64) + 64 * wr64


def summarize_traffic(args):
    """Writes profiles/traffic_<kernel>_<workload>.json from four rocprofv3 --pmc
    CSVs: the read-request counters (RD_COUNTERS) and write-request counters
    (WR_COUNTERS) of the kernel, and the same counters of the streaming-read
    and streaming-write kernels over --calib-mib MiB, which check the byte
    formula on dispatches of known size."""
    rd_csv, wr_csv, calib_rd_csv, calib_wr_csv = args.summarize_traffic
    calib_bytes = args.calib_mib * (1 << 20)
    cr = read_bytes(calib_rd_csv, "peak_read_kernel")
    cw = write_bytes(calib_wr_csv, "peak_write_kernel")
    kr, kw = read_bytes(rd_csv, args.kernel), write_bytes(wr_csv, args.kernel)
    base = args.kernel.split("<")[0]
    name = args.traffic_name or base
    rec = {
        "kernel": args.kernel,
        "workload": args.config,
        "kernel_source_sha": kernel_source_sha(base),
        "counters": list(RD_COUNTERS + WR_COUNTERS),
        "read_bytes": kr, "write_bytes": kw,
        "calib_bytes": calib_bytes, "calib_read_measured": cr, "calib_write_measured": cw,
        "hbm_bytes_per_launch": kr + kw,
    }
    os.makedirs(PROFILES, exist_ok=True)
    out = os.path.join(PROFILES, f"traffic_{name}_{args.config}.json")
    json.dump(rec, open(out, "w"), indent=1)
    print(json.dumps(rec))
    return 0


def stream_calibration(args):
    """--calib read|write: streaming-read (or -write) passes over --calib-mib MiB,
    the known-size dispatches that calibrate the traffic counters; prints the
    measured rates."""
    import torch
    from paper_2602_01519_amd import pic
    n = args.calib_mib * (1 << 20)
    buf = torch.empty(n, dtype=torch.uint8, device="cuda")
    fn = pic.peak_hbm_read if args.calib == "read" else pic.peak_hbm_write
    rates = [fn(buf, n) for _ in range(args.steps)]
    print(json.dumps({"calib": args.calib, "bytes": n, "dispatches": args.steps,
                      "gbs": [round(r, 1) for r in rates]}))
    return 0


def projections(args):
    """--projections: times pic_mla_absorb_q and pic_mla_up_v at the mla
    workload's size (all its query tokens x 16 heads) and prints one JSON line
    per kernel with its HBM roofline (these projections move more bytes than
    they compute). Inputs: seeded N(0,1) activations, N(0,1/K) weights, bf16."""
    import torch
    from paper_2602_01519_amd import pic, runner
    from paper_2602_01519_amd import workloads as W
    cfg = W.CONFIGS["mla"]
    T = sum(cfg.q_length(r) for r in range(cfg.batch))
    H = cfg.n_q_heads
    rng = np.random.default_rng(cfg.seed + 17)
    bf = lambda shape, std=1.0: runner.to_device(
        W.f32_to_bf16_bits(rng.standard_normal(shape, dtype=np.float32) * np.float32(std)), "cuda")
    q, w_uk_t = bf((T, H, 192)), bf((H, 512, 128), 1 / np.sqrt(128))
    o_lat, w_uv = bf((T, H, 512)), bf((H, 128, 512), 1 / np.sqrt(512))
    q_out = torch.empty((T, H, 576), dtype=torch.int16, device="cuda")
    out = torch.empty((T, H, 128), dtype=torch.int16, device="cuda")
    st = torch.cuda.current_stream()
    flops = 2.0 * T * H * 128 * 512
    cases = [("pic_mla_absorb_q", "mla_absorb",
              lambda: pic.mla_absorb_q(T, H, q, w_uk_t, q_out, st.cuda_stream),
              (T * H * (192 + 576) + H * 512 * 128) * 2),
             ("pic_mla_up_v", "mla_up",
              lambda: pic.mla_up_v(T, H, o_lat, w_uv, out, st.cuda_stream),
              (T * H * (512 + 128) + H * 128 * 512) * 2)]
    for name, workload, fn, nbytes in cases:
        t_w = time.perf_counter()
        n_w = 0
        while n_w < args.warmup or time.perf_counter() - t_w < args.min_warmup_s:
            fn()
            n_w += 1
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        for _ in range(args.steps):
            fn()
        e1.record(st)
        torch.cuda.synchronize()
        us = e0.elapsed_time(e1) / args.steps * 1e3
        gbs = nbytes / (us * 1e-6) / 1e9
        print(json.dumps({
            "metric": "MLA projection HBM GB/s (algorithmic bytes) at 1 GPU", "entry": name,
            "value": round(gbs, 1), "unit": "GB/s", "us_per_call": round(us, 3), "steps": args.steps,
            "dtype": "bf16", "data": "synthetic", "config": {"tokens": T, "heads": H},
            "algorithmic_bytes": nbytes, "flops": flops,
            "roofline": {"kernel": "proj_kernel", "bound": "hbm", "achieved": round(gbs, 1),
                         "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
                         "traffic": traffic_record("proj_kernel", workload)}}), flush=True)
    return 0


def algorithmic(cfg, wl):
    from paper_2602_01519_amd import workloads as W
    pairs = W.visible_pairs(cfg, wl.plan)
    flops = pairs * cfg.n_q_heads * (2 * cfg.d_k + 2 * cfg.d_v)
    esz = cfg.elem_bytes
    tq = wl.q.shape[0]
    ts = 0 if wl.k_self is None else wl.k_self.shape[0]
    kv_tok = cfg.n_kv_heads * (cfg.d_k + (cfg.d_v if cfg.kind == W.GQA else 0)) * esz
    chunk_bytes = sum(cfg.chunk_length(int(c)) for c in wl.used_chunks()) * kv_tok
    nbytes = (tq * cfg.n_q_heads * (cfg.d_k + cfg.d_v) * esz + tq * cfg.n_q_heads * 4 +
              ts * kv_tok + chunk_bytes)
    return flops, nbytes


def host_cpu_info():
    """nproc, the affinity mask and the CPU model of the host the oracle ran on."""
    import re
    import subprocess
    aff = sorted(os.sched_getaffinity(0))
    ranges, start = [], None
    for i, c in enumerate(aff):
        if start is None:
            start = c
        if i + 1 == len(aff) or aff[i + 1] != c + 1:
            ranges.append(f"{start}-{c}" if c != start else f"{c}")
            start = None
    model = None
    try:
        txt = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        m = re.search(r"^Model name:\s*(.+)$", txt, re.M)
        model = m.group(1).strip() if m else None
    except (OSError, subprocess.SubprocessError):
        pass
    if model is None and os.path.exists("/proc/cpuinfo"):
        m = re.search(r"^model name\s*:\s*(.+)$", open("/proc/cpuinfo").read(), re.M)
        model = m.group(1).strip() if m else None
    return {"nproc": os.cpu_count(), "affinity": ",".join(ranges), "affinity_cpus": len(aff),
            "model": model}


def single_core_tiny():
    """The oracle on the whole tiny fp32 workload with one OpenMP thread (ms)."""
    import ctypes
    import oracle
    from paper_2602_01519_amd import workloads as W
    cfg = W.CONFIGS["tiny_f32"]
    wl = W.make_workload(cfg)
    chunks = {int(c): W.make_chunk(cfg, int(c)) for c in wl.used_chunks()}
    oracle.num_threads()                      # loads the oracle (and its OpenMP runtime)
    gomp = ctypes.CDLL("libgomp.so.1")
    prev = gomp.omp_get_max_threads()
    gomp.omp_set_num_threads(1)
    try:
        best = None
        for _ in range(3):
            t0 = time.perf_counter()
            oracle.run_workload(wl, chunks)
            dt = (time.perf_counter() - t0) * 1e3
            best = dt if best is None else min(best, dt)
    finally:
        gomp.omp_set_num_threads(prev)
    flops = W.visible_pairs(cfg, wl.plan) * cfg.n_q_heads * (2 * cfg.d_k + 2 * cfg.d_v)
    return {"ms": round(best, 3), "cores": 1, "tflops": flops / (best * 1e-3) / 1e12}


def cpu_baseline(cfg, wl, dw, budget_s: float):
    """Times the fp64 oracle on a bounded sample of whole requests (host cores),
    and checks the GPU output of the sampled requests against it."""
    import oracle
    from paper_2602_01519_amd import workloads as W
    p = wl.plan
    flops_req = []
    for r in range(p.batch):
        sub = W.Plan(p.chunk_offsets[r:r + 2] - p.chunk_offsets[r], p.chunk_index[p.chunk_offsets[r]:p.chunk_offsets[r + 1]],
                     p.q_offsets[r:r + 2] - p.q_offsets[r],
                     None if p.self_offsets is None else p.self_offsets[r:r + 2] - p.self_offsets[r])
        flops_req.append(W.visible_pairs(cfg, sub) * cfg.n_q_heads * (2 * cfg.d_k + 2 * cfg.d_v))
    order = list(range(p.batch))
    done, t_used, flops_done = [], 0.0, 0
    out_gpu, _ = dw.results()
    max_err = 0.0
    for r in order:
        if t_used > budget_s and done:
            break
        idx = p.chunk_index[p.chunk_offsets[r]:p.chunk_offsets[r + 1]]
        links = [[dw.chunks[int(c)] if int(c) in dw.chunks else W.make_chunk(cfg, int(c)) for c in idx]]
        qs = slice(p.q_offsets[r], p.q_offsets[r + 1])
        so = None
        ks = vs = None
        if p.self_offsets is not None:
            ss = slice(p.self_offsets[r], p.self_offsets[r + 1])
            ks = wl.k_self[ss]
            vs = None if wl.v_self is None else wl.v_self[ss]
            so = np.array([0, ss.stop - ss.start], np.int32)
        t0 = time.perf_counter()
        ref, _ = oracle.link_attn(dtype=cfg.dtype, mla=cfg.kind == W.MLA, n_q_heads=cfg.n_q_heads,
                                  d_v=cfg.d_v, links=links, q=wl.q[qs],
                                  q_offsets=np.array([0, qs.stop - qs.start], np.int32), k_self=ks,
                                  v_self=vs, self_offsets=so, tau=float(np.float32(cfg.scale)))
        t_used += time.perf_counter() - t0
        flops_done += flops_req[r]
        done.append(r)
        max_err = max(max_err, float(np.abs(out_gpu[qs] - ref).max()))
    return {
        "value": flops_done / t_used / 1e12,
        "unit": "TFLOP/s",
        "cores": oracle.num_threads(),
        "host": host_cpu_info(),
        "single_core_tiny_f32": single_core_tiny(),
        "kind": "oracle",
        "sample": f"requests {done} of {p.batch} (all query rows and heads), fp64, {t_used:.1f} s",
        "gpu_max_abs_err_on_sample": max_err,
    }


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--no-measured-peaks", action="store_true",
                    help="skip the achievable-peak microbenchmarks (second roofline denominator)")
    ap.add_argument("--min-warmup-s", type=float, default=0.5,
                    help="run untimed warm-up steps for at least this long (clock ramp-up)")
    ap.add_argument("--config", default="long_rag",
                    help="workload: long_rag (default), tiny_f32, llama_prefill, decode, mla, "
                         "skinny_rag")
    ap.add_argument("--flush-mib", type=int, default=0,
                    help="also time K steps each after writing this many MiB of scratch "
                         "(cold last-level cache); reported as step_ms_flushed")
    ap.add_argument("--cpu-budget", type=float, default=15.0,
                    help="seconds of oracle time for the CPU baseline (0 = skip)")
    ap.add_argument("--calib", choices=["read", "write"],
                    help="run streaming-read or -write passes of --calib-mib MiB instead "
                         "(traffic counter calibration)")
    ap.add_argument("--calib-mib", type=int, default=2048)
    ap.add_argument("--summarize-traffic", nargs=4, metavar="CSV",
                    help="kernel read-request csv, kernel write-request csv, and the same "
                         "two for the streaming-read and streaming-write calibration runs")
    ap.add_argument("--kernel", default="link_mfma_d128_kernel")
    ap.add_argument("--traffic-name", default=None,
                    help="file name stem of the traffic record (default: the kernel's base name)")
    ap.add_argument("--projections", action="store_true",
                    help="time the MLA absorption / up-projection kernels instead (one line each)")
    args = ap.parse_args(argv)
    if args.summarize_traffic:
        return summarize_traffic(args)
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              f"(the link path shards by request with no exchange, see the design notes)",
              file=sys.stderr)
        return 2

    import torch
    from paper_2602_01519_amd import pic, runner
    from paper_2602_01519_amd import workloads as W

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    torch.cuda.set_device(0)
    if args.calib:
        return stream_calibration(args)
    if args.projections:
        return projections(args)
    cfg = W.CONFIGS[args.config]
    wl = W.make_workload(cfg)
    keep = set(int(c) for c in wl.plan.chunk_index[wl.plan.chunk_offsets[0]:wl.plan.chunk_offsets[min(4, wl.plan.batch)]])
    dw = runner.upload(wl, keep_host=keep)
    stream = torch.cuda.current_stream()
    warm_run = 0
    t_w = time.perf_counter()
    while warm_run < args.warmup or time.perf_counter() - t_w < args.min_warmup_s:
        for _ in range(max(1, min(args.warmup, 20))):
            dw.run()
            warm_run += 1
        torch.cuda.synchronize()

    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    # HIP events around one attention launch in PROF_EVERY (the event pair
    # adds a few microseconds between kernels), on the launch stream, inside
    # the timed region
    pic.prof_begin(PROF_EVERY)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(args.steps):
        dw.run()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kern_ms, launches, kname = pic.prof_end()
    step_ms = ev0.elapsed_time(ev1) / args.steps
    kern_avg_ms = kern_ms / max(launches, 1)

    # Spread of single steps: a second pass of K steps (after the timed
    # region) with an event at every step boundary; each step's time then
    # also holds one event record.
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    evs[0].record(stream)
    for i in range(args.steps):
        dw.run()
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    per_step = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)])
    step_dist = {"p10": round(float(np.percentile(per_step, 10)), 5),
                 "median": round(float(np.median(per_step)), 5),
                 "p90": round(float(np.percentile(per_step, 90)), 5),
                 "steps": args.steps,
                 "how": "second pass of K steps, one event per step boundary"}
    flushed = None
    if args.flush_mib > 0:
        # Cold-cache steps: before each step, writing a scratch buffer larger
        # than the 256 MB last-level cache evicts the step's inputs; only the
        # call is timed (events right around it).
        scratch = torch.empty(args.flush_mib << 18, dtype=torch.float32, device="cuda")
        cold = []
        for _ in range(args.steps):
            scratch.fill_(1.0)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            dw.run()
            e1.record(stream)
            torch.cuda.synchronize()
            cold.append(e0.elapsed_time(e1))
        cold = np.array(cold)
        flushed = {"flush_mib": args.flush_mib, "p10": round(float(np.percentile(cold, 10)), 5),
                   "median": round(float(np.median(cold)), 5),
                   "p90": round(float(np.percentile(cold, 90)), 5), "steps": args.steps}
        del scratch

    flops, nbytes = algorithmic(cfg, wl)
    tflops = flops / (step_ms * 1e-3) / 1e12
    gbs = nbytes / (step_ms * 1e-3) / 1e9
    if cfg.dtype == W.F32:
        # fp32 products run on the matrix cores in the lean small-call kernel,
        # on the vector ALUs in the generic ones
        bound = "mfma" if kname.startswith("link_lean_kernel") else "alu"
        peak, unit, achieved = PEAK_FP32_TFLOPS, "TFLOP/s", flops / (kern_avg_ms * 1e-3) / 1e12
    elif flops / nbytes < PEAK_BF16_TFLOPS * 1e12 / (PEAK_HBM_GBS * 1e9):
        # below the ridge point (about 312 FLOP/B): decode, and short questions
        # over long documents
        bound, peak, unit, achieved = "hbm", PEAK_HBM_GBS, "GB/s", nbytes / (kern_avg_ms * 1e-3) / 1e9
    else:
        bound, peak, unit, achieved = "mfma", PEAK_BF16_TFLOPS, "TFLOP/s", flops / (kern_avg_ms * 1e-3) / 1e12

    # Achievable peaks on this GPU (after the timed region, at the ramped-up
    # clock): the bf16 matrix-core rate with every SIMD busy, and a streaming
    # read of 2 GiB (far beyond the last-level cache).
    measured = None
    if not args.no_measured_peaks and bound in ("mfma", "hbm") and cfg.dtype != W.F32:
        if bound == "mfma":
            pic.peak_mfma_bf16(64)
            measured = max(pic.peak_mfma_bf16(256) for _ in range(3))
        else:
            buf = torch.empty(2 << 30, dtype=torch.uint8, device="cuda")
            pic.peak_hbm_read(buf, buf.numel())
            measured = max(pic.peak_hbm_read(buf, buf.numel()) for _ in range(3))
            del buf
            torch.cuda.empty_cache()

    cpu = None
    if args.cpu_budget > 0:
        cpu = cpu_baseline(cfg, wl, dw, args.cpu_budget)
    dw.close()

    line = {
        "metric": "link-attn TFLOP/s (algorithmic, visible pairs) at 1 GPU",
        "value": round(tflops, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "warmup_steps_run": warm_run,
        "ms_per_step": round(step_ms, 5),
        "step_ms_dist": step_dist,
        **({"step_ms_flushed": flushed} if flushed else {}),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32" if cfg.dtype == W.F32 else "bf16",
        "data": "synthetic (seeded N(0,1), shapes of the paper's Llama-3.1-8B / DeepSeek-V2-Lite backbones)",
        "config": {
            "workload": cfg.name,
            "batch": cfg.batch,
            "n_q_heads": cfg.n_q_heads,
            "n_kv_heads": cfg.n_kv_heads,
            "d_k": cfg.d_k,
            "d_v": cfg.d_v,
            "links_per_request": list(cfg.links),
            "chunk_tokens": cfg.chunk_len,
            "query_tokens": cfg.q_len,
            "own_tokens": cfg.self_len,
            "entry": "pic_link_decode" if cfg.decode else "pic_link_attn",
        },
        "us_per_request": round(step_ms * 1e3 / cfg.batch, 3),
        "hbm_gbs_algorithmic": round(gbs, 1),
        "hbm_frac": round(gbs / PEAK_HBM_GBS, 4),
        "mfma_frac": round(tflops / PEAK_BF16_TFLOPS, 4) if cfg.dtype == W.BF16 else None,
        "algorithmic_flops_per_step": flops,
        "algorithmic_bytes_per_step": nbytes,
        "wall_s_timed": round(wall, 4),
        "roofline": {
            "kernel": kname,
            "bound": bound,
            "achieved": round(achieved, 3),
            "peak": peak,
            "unit": unit,
            "frac": round(achieved / peak, 4),
            "measured_peak": round(measured, 1) if measured else None,
            "measured_frac": round(achieved / measured, 4) if measured else None,
            "traffic": traffic_record(kname, cfg.name),
            "kernel_avg_us": round(kern_avg_ms * 1e3, 3),
            "launches": launches,
            "launches_timed_every": PROF_EVERY,
        },
        "cpu_baseline": cpu,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
