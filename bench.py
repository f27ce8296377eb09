"""Benchmark: candidate pipeline schedules simulated per second on one MI355X.

Workload: 1,048,576 synthetic candidates of a Nemotron-H-like 52-layer model on P = 8 devices
with M = 64 micro-batches, v in {1, 2} stages per device, four placements and four schedule
policies in equal strata (paper_2509_23722_amd/inputs.py, workload 3). One step = one
octo_sim_batch call over the whole batch, inputs resident in GPU memory. Prints one JSON line.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu] [--headline-only]
                    [--copy-calibration]

The CPU oracle's results are compared with the GPU's for every candidate of the batch; on any
difference the line carries "value": null and the script exits with status 1.
"""
import argparse
import ctypes
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# MI355X (gfx950): 256 CUs x 4 SIMD x 16 lanes at 2.4 GHz -> 32-bit integer VALU lane-ops/s.
PEAK_VALU_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12
HBM_PEAK_GBS = 8000.0
# simulation kernels, in launch order, between the library's measurement boundaries
SIM_KERNELS = ["k_static", "k_sim<2>", "k_sim<1>", "k_sim<8>", "k_afab", "k_sim_mat<2>"]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_nemotron-h-like-52L-P8-M64.json")


def kernel_source_hash():
    h = hashlib.sha256()
    for f in ("octo.hip", "octo_sim.hpp", "octo_device.hpp"):
        with open(os.path.join(ROOT, "paper_2509_23722_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def algorithmic_work(recs, P, M):
    """Per candidate: N ops, E edges of the DAG (queue order N - P, forward and backward chains
    2 (S-1) M, F->B S M, B->W S M when split). Relaxation = one add + one max per edge and one
    add per op (2E + N int64 ops) = 5E + 2N 32-bit lane-ops (add = 2, max = cmp + 2 selects).
    Returns per-candidate (int64 ops, lane-ops) arrays."""
    v = recs[:, 1].astype(np.int64)
    split = recs[:, 0] == 3
    S = P * v
    N = np.where(split, 3, 2) * S * M
    E = (N - P) + 2 * (S - 1) * M + S * M + np.where(split, S * M, 0)
    return 2 * E + N, 5 * E + 2 * N


def static_class_mask(recs, P, v_max):
    """Candidates that the library evaluates with a static round schedule: no moves, not AFAB,
    v = 1, or v = 2 with looped, blocked or V-shape stage pairs (the structure classes)."""
    pol, v, npert = recs[:, 0], recs[:, 1], recs[:, 2]
    s_max = P * v_max
    dev = recs[:, 3 + s_max:3 + 2 * s_max].astype(np.int64)
    ok = (pol != 0) & (npert == 0)
    st = ok & (v == 1)
    if v_max >= 2:
        i = np.arange(P)
        lp = (dev[:, i] == dev[:, i + P]).all(axis=1)
        bl = (dev[:, 2 * i] == dev[:, 2 * i + 1]).all(axis=1)
        vs = (dev[:, i] == dev[:, 2 * P - 1 - i]).all(axis=1)
        st |= ok & (v == 2) & (lp | bl | vs)
    return st


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def host_threads():
    """Threads for the oracle: the CPUs this process may run on, at most 16 (the host share of
    one GPU on the benchmark machines)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def gpipe_sweep_lane_ops(recs, P, M):
    """Work a GPipe row sweep needs per candidate: every op takes one input (its row's producer,
    or its own device clock), so one add for the input's arrival, one max against the clock and
    one add for the duration: 7 32-bit lane-ops per op (N = 2 S M ops, all fused)."""
    v = recs[:, 1].astype(np.int64)
    return 7 * 2 * P * v * M


def hip_events(n):
    hip = ctypes.CDLL("libamdhip64.so")
    hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
    hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                        ctypes.c_void_p]
    hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
    evs = []
    for _ in range(n):
        e = ctypes.c_void_p()
        if hip.hipEventCreate(ctypes.byref(e)) != 0:
            raise RuntimeError("hipEventCreate failed")
        evs.append(e.value)
    return hip, evs


def copy_calibration(torch):
    """A plain device copy of known size, for scaling the HBM counters."""
    nbytes = 1 << 30
    x = torch.empty(nbytes // 8, dtype=torch.int64, device="cuda:0").fill_(1)
    y = torch.empty_like(x)
    torch.cuda.synchronize()
    for _ in range(3):
        y.copy_(x)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes": nbytes, "launches": 3}), flush=True)


def time_variant(torch, _lib, call, n, steps, warmup, kernels=True):
    """Time `call` (one batch evaluation) like the headline: wall clock over `steps` calls after
    `warmup`, and (kernels) each simulation kernel by the library's HIP events, which only the
    batch-evaluation entry points record. Returns (candidates/s, ms per call, {kernel: ms})."""
    for _ in range(warmup):
        call()
    torch.cuda.synchronize()
    if not kernels:
        t0 = time.perf_counter()
        for _ in range(steps):
            call()
        torch.cuda.synchronize()
        secs = time.perf_counter() - t0
        return round(n * steps / secs, 1), round(secs / steps * 1e3, 4), {}
    nb = len(SIM_KERNELS) + 1
    hip, evs = hip_events(nb * steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(steps):
        _lib.profile_events(evs[nb * k:nb * (k + 1)])
        call()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    _lib.profile_events([])
    km = np.zeros((steps, len(SIM_KERNELS)))
    for k in range(steps):
        for j in range(len(SIM_KERNELS)):
            f = ctypes.c_float()
            hip.hipEventElapsedTime(ctypes.byref(f), evs[nb * k + j], evs[nb * k + j + 1])
            km[k, j] = f.value
    for e in evs:
        hip.hipEventDestroy(e)
    return (round(n * steps / (t1 - t0), 1), round((t1 - t0) / steps * 1e3, 4),
            {k: round(float(x), 4) for k, x in zip(SIM_KERNELS, km.mean(axis=0))})


def time_w_advance(torch, _lib, inputs, w, costs, link, mem, recs_np, dev, warmup, steps,
                   with_cpu):
    """Selective W advancing (octo_advance_w) on the batch's first 65,536 split-backward (ZB)
    candidates, each given 255 move slots, under one capacity for all devices: the 40th
    percentile of the candidates' largest peaks."""
    zb = recs_np[recs_np[:, 0] == inputs.POLICY["ZB"]][:65536]
    mp = 255
    stride = inputs.record_stride(w.P, w.v_max, mp)
    r_np = np.zeros((len(zb), stride), np.uint8)
    r_np[:, :zb.shape[1]] = zb
    n = len(r_np)
    prob = _lib.problem(w.L, w.P, w.v_max, w.M, stride, mp)
    r = torch.from_numpy(r_np).to(dev)
    _, _, pk0 = _lib.sim_batch_mem(prob, costs, mem, link, r)
    cap_np = np.full(w.P, int(np.percentile(pk0.max(dim=1).values.cpu().numpy(), 40)), np.int64)
    cap = torch.from_numpy(cap_np).to(dev)
    out = torch.empty_like(r)
    for _ in range(max(warmup, 1)):
        res = _lib.advance_w(prob, costs, mem, cap, link, r, out_candidates=out)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        res = _lib.advance_w(prob, costs, mem, cap, link, r, out_candidates=out)
    torch.cuda.synchronize()
    secs = (time.perf_counter() - t0) / steps
    o_rec, o_ms, o_bub, o_pk = (x.cpu().numpy() for x in res)
    fit0 = int(((pk0.cpu().numpy() <= cap_np).all(axis=1)).sum())
    fit1 = int(((o_pk <= cap_np).all(axis=1) & (o_ms > 0)).sum())
    adv = o_rec[:, 2].astype(np.int64) - r_np[:, 2]
    res = {"value": round(n / secs, 1), "unit": "candidates/s", "ms_per_call": round(secs * 1e3, 3),
           "candidates": n, "move_slots": mp, "capacity_bytes": int(cap_np[0]),
           "fit_before": fit0, "fit_after": fit1, "mean_advances": round(float(adv.mean()), 2),
           "cpu_baseline": None}
    if with_cpu:
        from oracle import octoref
        sample = np.arange(0, n, 32)
        threads = min(16, os.cpu_count() or 1)
        rprob = octoref.problem(w.L, w.P, w.v_max, w.M, stride, mp)
        c0 = time.perf_counter()
        rr = octoref.advance_w(rprob, inputs.layer_costs(w), inputs.layer_mem(w),
                               cap_np, inputs.link_matrix(w.P, w.link_ns), r_np[sample],
                               nthreads=threads)
        c1 = time.perf_counter()
        same = bool((rr[0] == o_rec[sample]).all() and (rr[1] == o_ms[sample]).all() and
                    (rr[3] == o_pk[sample]).all())
        res["cpu_baseline"] = {"value": round(len(sample) / (c1 - c0), 1), "unit": "candidates/s",
                               "cores": threads, "kind": "oracle",
                               "sample": f"every 32nd of the same candidates ({len(sample)})",
                               "parity_on_sample": same}
    return res


def time_alg1(torch, _lib, inputs, w, costs, link, recs_np, dev, warmup, steps, with_cpu):
    """Algorithm 1 (octo_alg1_tune: bubble-aware phases, overlap-aware insertions in the
    scheduling phase) on 4,096 records of the batch (every 256th), widened to four move slots,
    32 iterations per call; the unit of work is one iteration of one record's search (phase
    choice, its whole neighbourhood evaluated, best kept). Beside it, the random-search variant
    (octo_alg1_tune_ex with random phases, the same insertions) on the same records: rate,
    gain, and the iterations each variant gave each phase."""
    n, iters, mp = 4096, 32, 4
    base = recs_np[::len(recs_np) // n][:n]
    stride = inputs.record_stride(w.P, w.v_max, mp)
    r_np = np.zeros((n, stride), np.uint8)
    r_np[:, :base.shape[1]] = base
    prob = _lib.problem(w.L, w.P, w.v_max, w.M, stride, mp)
    r0 = torch.from_numpy(r_np).to(dev)
    r = torch.empty_like(r0)
    for _ in range(max(warmup, 1)):
        r.copy_(r0)
        res = _lib.alg1_tune(prob, costs, link, r, iters)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        r.copy_(r0)
        res = _lib.alg1_tune(prob, costs, link, r, iters)
    torch.cuda.synchronize()
    secs = (time.perf_counter() - t0) / steps
    o_rec, o_ms = r.cpu().numpy(), res[0].cpu().numpy()
    stats = res[2].cpu().numpy()
    ms0 = _lib.sim_batch(prob, costs, link, r0)[0].cpu().numpy()
    ok = ms0 > 0
    out = {"value": round(n * iters / secs, 1), "unit": "record-iterations/s",
           "ms_per_call": round(secs * 1e3, 3), "records": n, "iterations": iters,
           "move_slots": mp, "searched_iterations": int(stats[:, 3].sum()),
           "kept_moves": {"partition": int(stats[:, 0].sum()), "placement": int(stats[:, 1].sum()),
                          "schedule": int(stats[:, 2].sum())},
           "mean_makespan_gain": round(float(1 - (o_ms[ok] / ms0[ok]).mean()), 4),
           "cpu_baseline": None}
    # the phase iterations of the bubble-aware search, then the random-search variant
    flags = _lib.A1_INSERT
    r.copy_(r0)
    pit = _lib.alg1_tune_ex(prob, costs, link, r, iters, flags)[3].cpu().numpy()
    out["phase_iterations"] = {k: int(x) for k, x in zip(("partition", "placement", "schedule"), pit.sum(axis=0))}
    for _ in range(max(warmup, 1)):
        r.copy_(r0)
        rres = _lib.alg1_tune_ex(prob, costs, link, r, iters, flags | _lib.A1_RANDOM, 20250929)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        r.copy_(r0)
        rres = _lib.alg1_tune_ex(prob, costs, link, r, iters, flags | _lib.A1_RANDOM, 20250929)
    torch.cuda.synchronize()
    rsecs = (time.perf_counter() - t0) / steps
    r_ms, r_pit = rres[0].cpu().numpy(), rres[3].cpu().numpy()
    out["random_phases"] = {
        "value": round(n * iters / rsecs, 1), "unit": "record-iterations/s",
        "ms_per_call": round(rsecs * 1e3, 3), "seed": 20250929,
        "mean_makespan_gain": round(float(1 - (r_ms[ok] / ms0[ok]).mean()), 4),
        "phase_iterations": {k: int(x) for k, x in zip(("partition", "placement", "schedule"), r_pit.sum(axis=0))}}
    if with_cpu:
        from oracle import alg1 as A
        from oracle import octoref
        sample = np.arange(0, n, 256)
        threads = min(16, os.cpu_count() or 1)
        rprob = octoref.problem(w.L, w.P, w.v_max, w.M, stride, mp)
        c0 = time.perf_counter()
        rr = A.tune(rprob, inputs.layer_costs(w), inputs.link_matrix(w.P, w.link_ns),
                    r_np[sample], iters, nthreads=threads)
        c1 = time.perf_counter()
        same = bool((rr[0] == o_rec[sample]).all() and (rr[1] == o_ms[sample]).all() and
                    (rr[3] == stats[sample, :3]).all() and (rr[4] == stats[sample, 3]).all())
        out["cpu_baseline"] = {"value": round(len(sample) * iters / (c1 - c0), 1),
                               "unit": "record-iterations/s", "cores": threads, "kind": "oracle",
                               "sample": f"every 256th of the same records ({len(sample)})",
                               "parity_on_sample": same}
    return out


def time_tuner(torch, _lib, inputs, warmup, steps, with_cpu):
    """The local-search tuner (octo_tune_step) on its own workload: 96 layers, P = 32, M = 256,
    v = 2, 4,096 chains; one job = step 0 (generate and evaluate) plus 64 move steps, every
    chain re-simulated at every step. The unit of work is one chain-step (one candidate
    evaluated and accepted or rejected)."""
    w = inputs.WORKLOADS[5]
    dev = torch.device("cuda:0")
    recs_np = inputs.tuner_chains(w)
    n = recs_np.shape[0]
    prob = _lib.problem(w.L, w.P, w.v_max, w.M, recs_np.shape[1], 0)
    costs_np, link_np = inputs.layer_costs(w), inputs.link_matrix(w.P, w.link_ns)
    costs = torch.from_numpy(costs_np).to(dev)
    link = torch.from_numpy(link_np).to(dev)
    c0_np = np.zeros((n, _lib.chain_stride(prob)), np.uint8)
    c0_np[:, :recs_np.shape[1]] = recs_np
    c0 = torch.from_numpy(c0_np).to(dev)
    chains = torch.empty_like(c0)
    queues = torch.empty((n, w.P, _lib.queue_capacity(prob)), dtype=torch.int16, device=dev)

    def job():
        chains.copy_(c0)
        for t in range(w.steps + 1):
            _lib.tune_step(prob, costs, link, chains, queues, w.seed, t)

    for _ in range(max(warmup, 1)):
        job()
    torch.cuda.synchronize()
    hip, evs = hip_events(2)
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    t0 = time.perf_counter()
    hip.hipEventRecord(evs[0], stream)
    for _ in range(steps):
        job()
    hip.hipEventRecord(evs[1], stream)
    torch.cuda.synchronize()
    secs = (time.perf_counter() - t0) / steps
    f = ctypes.c_float()
    hip.hipEventElapsedTime(ctypes.byref(f), evs[0], evs[1])
    ev_secs = f.value * 1e-3 / steps
    for e in evs:
        hip.hipEventDestroy(e)
    g_ms, g_acc, _ = _lib.chain_state(chains, prob)
    g_ms, g_acc = g_ms.numpy(), g_acc.numpy()
    init_ms = _lib.sim_batch(prob, costs, link, torch.from_numpy(recs_np).to(dev))[0]
    init_ms = init_ms.cpu().numpy()
    ok = (init_ms > 0) & (g_ms > 0)
    evals = n * (w.steps + 1)
    out = {"value": round(evals / secs, 1), "unit": "chain-steps/s",
           "ms_per_job": round(secs * 1e3, 3), "ms_per_job_events": round(ev_secs * 1e3, 3),
           "chains": n, "steps": w.steps + 1, "workload": w.name,
           "accepted_moves": int(g_acc.sum()),
           "mean_makespan_gain": round(float(1 - (g_ms[ok] / init_ms[ok]).mean()), 4),
           "cpu_baseline": None}
    if with_cpu:
        from oracle import octoref
        sample = np.arange(0, n, 16)
        threads = min(16, os.cpu_count() or 1)
        rprob = octoref.problem(w.L, w.P, w.v_max, w.M, recs_np.shape[1], 0)
        t1 = time.perf_counter()
        rr = octoref.tune_chains(rprob, costs_np, link_np, recs_np, sample, w.seed, w.steps,
                                 nthreads=threads)
        t2 = time.perf_counter()
        g_rec = chains.cpu().numpy()[:, :recs_np.shape[1]]
        same = bool((rr[0] == g_rec[sample]).all() and (rr[1] == g_ms[sample]).all() and
                    (rr[3] == g_acc[sample]).all())
        out["cpu_baseline"] = {"value": round(len(sample) * (w.steps + 1) / (t2 - t1), 1),
                               "unit": "chain-steps/s", "cores": threads, "kind": "oracle",
                               "sample": f"every 16th chain of the same job ({len(sample)} "
                                         f"chains x {w.steps + 1} steps)",
                               "parity_on_sample": same}
    return out


def time_strata(torch, _lib, prob, costs, link, recs_np, dev, steps, warmup):
    """octo_sim_batch on each (v, policy) stratum of the batch on its own (131,072 candidates
    each), timed like the headline: wall clock over `steps` calls."""
    names = {0: "AFAB", 1: "1F1B", 2: "I1F1B", 3: "ZB"}
    out = {}
    for v in (1, 2):
        for p in range(4):
            sel = (recs_np[:, 1] == v) & (recs_np[:, 0] == p)
            if not sel.any():
                continue
            r = torch.from_numpy(np.ascontiguousarray(recs_np[sel])).to(dev)
            m = torch.empty(r.shape[0], dtype=torch.int64, device=dev)
            b = torch.empty((r.shape[0], prob.P), dtype=torch.int64, device=dev)
            rate, ms_, _ = time_variant(torch, _lib,
                                        lambda: _lib.sim_batch(prob, costs, link, r, m, b),
                                        r.shape[0], steps, warmup, kernels=False)
            out[f"v{v}_{names[p]}"] = {"candidates": int(sel.sum()), "ms_per_call": ms_,
                                       "candidates_per_s": rate}
    return out


def time_transfers(torch, recs_np, P, step_ms):
    """Host <-> device copies a caller starting from host memory would add per batch: the
    records in, makespans and bubbles out (pinned host buffers), and the rate they imply."""
    n = recs_np.shape[0]
    h_in = torch.from_numpy(recs_np).pin_memory()
    d_in = torch.empty(h_in.shape, dtype=torch.uint8, device="cuda:0")
    d_out = torch.empty((n, 1 + P), dtype=torch.int64, device="cuda:0")
    h_out = torch.empty((n, 1 + P), dtype=torch.int64, pin_memory=True)
    e = [torch.cuda.Event(enable_timing=True) for _ in range(4)]
    reps = 10
    for _ in range(2):
        d_in.copy_(h_in, non_blocking=True)
        h_out.copy_(d_out, non_blocking=True)
    torch.cuda.synchronize()
    e[0].record()
    for _ in range(reps):
        d_in.copy_(h_in, non_blocking=True)
    e[1].record()
    for _ in range(reps):
        h_out.copy_(d_out, non_blocking=True)
    e[2].record()
    torch.cuda.synchronize()
    h2d = e[0].elapsed_time(e[1]) / reps
    d2h = e[1].elapsed_time(e[2]) / reps
    return {"h2d_bytes": int(recs_np.nbytes), "h2d_ms": round(h2d, 4),
            "h2d_gbs": round(recs_np.nbytes / (h2d * 1e-3) / 1e9, 2),
            "d2h_bytes": int(n * (1 + P) * 8), "d2h_ms": round(d2h, 4),
            "d2h_gbs": round(n * (1 + P) * 8 / (d2h * 1e-3) / 1e9, 2),
            "pcie_inclusive_candidates_per_s": round(n / ((h2d + step_ms + d2h) * 1e-3), 1)}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU-oracle baseline leg")
    ap.add_argument("--copy-calibration", action="store_true")
    ap.add_argument("--headline-only", action="store_true",
                    help="time only the headline call (for kernel traces: every simulation "
                         "kernel dispatch is then a headline one); no other legs, no oracle")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: the batch is split across GPUs by candidate "
              f"range with no communication in the hot loop, so --gpus {args.gpus} is not run "
              f"here.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2509_23722_amd import _lib, inputs

    if args.copy_calibration:
        copy_calibration(torch)
        return

    dev = torch.device("cuda:0")
    w = inputs.WORKLOADS[3]
    costs_np, link_np = inputs.layer_costs(w), inputs.link_matrix(w.P, w.link_ns)
    recs_np = inputs.candidates(w)
    n = recs_np.shape[0]
    prob = _lib.problem(w.L, w.P, w.v_max, w.M, recs_np.shape[1], w.max_pert)
    costs = torch.from_numpy(costs_np).to(dev)
    link = torch.from_numpy(link_np).to(dev)
    recs = torch.from_numpy(recs_np).to(dev)
    ms = torch.empty(n, dtype=torch.int64, device=dev)
    bub = torch.empty((n, w.P), dtype=torch.int64, device=dev)

    for _ in range(args.warmup):
        _lib.sim_batch(prob, costs, link, recs, ms, bub)
    torch.cuda.synchronize()

    nb = len(SIM_KERNELS) + 1
    hip, evs = hip_events(nb * args.steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(args.steps):
        _lib.profile_events(evs[nb * k:nb * (k + 1)])
        _lib.sim_batch(prob, costs, link, recs, ms, bub)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    _lib.profile_events([])
    kern_ms = np.zeros((args.steps, len(SIM_KERNELS)))
    for k in range(args.steps):
        for j in range(len(SIM_KERNELS)):
            f = ctypes.c_float()
            hip.hipEventElapsedTime(ctypes.byref(f), evs[nb * k + j], evs[nb * k + j + 1])
            kern_ms[k, j] = f.value
    for e in evs:
        hip.hipEventDestroy(e)

    secs = t1 - t0
    value = n * args.steps / secs
    gms, gbub = ms.cpu().numpy(), bub.cpu().numpy()  # the headline call's results
    ms_per_step = secs / args.steps * 1e3
    per_kernel_ms = kern_ms.mean(axis=0)
    int64_c, lane_c = algorithmic_work(recs_np, w.P, w.M)
    v, pol = recs_np[:, 1], recs_np[:, 0]
    # candidates each simulation kernel handles (no moves in this workload)
    stat = static_class_mask(recs_np, w.P, w.v_max)
    sets = [stat, (v == 2) & (pol != 0) & ~stat, (v == 1) & (pol != 0) & ~stat,
            (v >= 3) & (pol != 0), pol == 0, np.zeros(n, dtype=bool)]
    # the dominant kernel: the one that takes longest
    dom = int(np.argmax(per_kernel_ms))
    dom_ms = float(per_kernel_ms[dom])
    dom_set = sets[dom]
    dom_lane_ops = int(lane_c[dom_set].sum())
    achieved = dom_lane_ops / (dom_ms * 1e-3) / 1e12
    n_dom = int(dom_set.sum())
    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        t = json.load(open(TRAFFIC_FILE))
        tk = re.sub(r", (false|0)>$", ">", str(t.get("kernel", "")))
        if t.get("kernel_source_sha") == kernel_source_hash() and tk == SIM_KERNELS[dom]:
            traffic = t.get("hbm_bytes_per_launch")
    all_ms = float(per_kernel_ms.sum())
    # every kernel priced by its own work: the generated-queue kernels by the DAG relaxation
    # count, k_afab by what a GPipe row sweep needs
    lane_all = lane_c.copy()
    lane_all[pol == 0] = gpipe_sweep_lane_ops(recs_np[pol == 0], w.P, w.M)
    # per stratum: the candidates each simulation kernel handles, at that kernel's rate
    names = ["static_schedules", "v2_generated", "v1_generated", "v3plus_generated", "gpipe_all_v",
             "with_moves"]
    strata = {}
    for name, kname, sel, kms in zip(names, SIM_KERNELS, sets, per_kernel_ms):
        cnt = int(sel.sum())
        if cnt:
            work = int(lane_all[sel].sum())
            strata[name] = {"kernel": kname, "candidates": cnt, "ms": round(float(kms), 4),
                            "candidates_per_s": round(cnt / (float(kms) * 1e-3), 1),
                            "alg_lane_ops": work,
                            "frac": round(work / (float(kms) * 1e-3) / 1e12 / PEAK_VALU_TOPS, 5)}
            if kname == "k_afab":
                strata[name]["work_priced_as"] = (
                    "the GPipe row sweep (an add, a max and an add per op); the kernel evaluates "
                    "each row as an envelope of at most eight lines, fewer operations for the "
                    "same times")
    roofline = {
        "bound": "alu", "achieved": round(achieved, 3), "peak": round(PEAK_VALU_TOPS, 2),
        "unit": "Tops/s (32-bit VALU lane-ops)", "frac": round(achieved / PEAK_VALU_TOPS, 5),
        "traffic": traffic, "kernel": SIM_KERNELS[dom], "kernel_ms": round(dom_ms, 4),
        "kernel_candidates": n_dom, "alg_lane_ops_per_launch": dom_lane_ops,
        "alg_int64_ops_per_launch": int(int64_c[dom_set].sum()),
        "hbm_alg_gbs": round(n_dom * (recs_np.shape[1] + 8 + 8 * w.P) / (dom_ms * 1e-3) / 1e9, 2),
        "hbm_peak_gbs": HBM_PEAK_GBS,
        "sim_kernels_ms": {k: round(float(x), 4) for k, x in zip(SIM_KERNELS, per_kernel_ms)},
        "all_sim_kernels_frac": round(int(lane_all.sum()) / (all_ms * 1e-3) / 1e12 /
                                      PEAK_VALU_TOPS, 5),
        "strata": strata,
    }
    out = {
        "metric": "candidate schedules simulated/sec at P=8,M=64",
        "value": round(value, 1), "unit": "candidates/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "int64", "data": "synthetic",
        "config": {"workload": w.name, "candidates": n, "P": w.P, "M": w.M, "L": w.L,
                   "v": [1, 2], "policies": ["AFAB", "1F1B", "I1F1B", "ZB"],
                   "placements": list(inputs.PLACEMENTS), "seed": w.seed},
        "roofline": roofline,
    }
    if args.headline_only:
        print(json.dumps(out), flush=True)
        return

    out["strata_v_policy"] = time_strata(torch, _lib, prob, costs, link, recs_np, dev,
                                         args.steps, args.warmup)
    out["transfers"] = time_transfers(torch, recs_np, w.P, ms_per_step)

    # the same batch with the memory model (peak bytes per device), timed the same way
    mem = torch.from_numpy(inputs.layer_mem(w)).to(dev)
    peak = torch.empty((n, w.P), dtype=torch.int64, device=dev)
    v_, t_, k_ = time_variant(
        torch, _lib, lambda: _lib.sim_batch_mem(prob, costs, mem, link, recs, ms, bub, peak), n,
        args.steps, args.warmup)
    memory_model = {"value": v_, "unit": "candidates/s", "ms_per_step": t_, "sim_kernels_ms": k_,
                    "layer_mem": "inputs.layer_mem (per-type activation and static bytes)"}

    # with communication accounting (nodes, overlap)
    comm = torch.empty((n, 4), dtype=torch.int64, device=dev)
    v_, t_, k_ = time_variant(
        torch, _lib, lambda: _lib.sim_batch_comm(prob, costs, link, recs, ms, bub, comm), n,
        args.steps, args.warmup)
    cm_np = comm.cpu().numpy()
    comm_model = {
        "value": v_, "unit": "candidates/s", "ms_per_step": t_, "sim_kernels_ms": k_,
        "overlap_rate_nodes": round(float(cm_np[:, 1].sum() / max(cm_np[:, 0].sum(), 1)), 4),
        "overlap_rate_time": round(float(cm_np[:, 3].sum() / max(cm_np[:, 2].sum(), 1)), 4),
    }

    # with serialised links (one transfer at a time per directed link)
    sms = torch.empty_like(ms)
    sbub = torch.empty_like(bub)
    v_, t_, k_ = time_variant(
        torch, _lib, lambda: _lib.sim_batch_serial(prob, costs, link, recs, sms, sbub), n,
        args.steps, args.warmup)
    s_np = sms.cpu().numpy()
    serial_links = {"value": v_, "unit": "candidates/s", "ms_per_step": t_, "sim_kernels_ms": k_,
                    "makespan_changed": int((s_np != ms.cpu().numpy()).sum())}

    # with blocking rendezvous transfers (receive before the consumer, send after the producer)
    rms_ = torch.empty_like(ms)
    rbub_ = torch.empty_like(bub)
    v_, t_, k_ = time_variant(
        torch, _lib, lambda: _lib.sim_batch_rdv(prob, costs, link, recs, rms_, rbub_), n,
        args.steps, args.warmup)
    r_np = rms_.cpu().numpy()
    rendezvous = {"value": v_, "unit": "candidates/s", "ms_per_step": t_, "sim_kernels_ms": k_,
                  "deadlocked": int((r_np == -1).sum()), "completed": int((r_np > 0).sum())}

    # the reordered coordination (deadlock-free): every 16th candidate of the batch
    sub = recs[::16].contiguous()
    ns = sub.shape[0]
    oms = torch.empty(ns, dtype=torch.int64, device=dev)
    obub = torch.empty((ns, w.P), dtype=torch.int64, device=dev)
    v_, t_, _ = time_variant(
        torch, _lib, lambda: _lib.sim_batch_ordered(prob, costs, link, sub, oms, obub), ns,
        args.steps, args.warmup, kernels=False)
    o_np = oms.cpu().numpy()
    ordered = {"value": v_, "unit": "candidates/s", "ms_per_step": t_, "candidates": ns,
               "sample": "every 16th candidate of the batch", "deadlocked": int((o_np == -1).sum()),
               "mean_slowdown_vs_async": round(float((o_np / ms[::16].cpu().numpy()).mean()), 4)}

    # the executor's three-step reordering with handshake transfers, on the same sample
    rst = torch.empty((ns, 2), dtype=torch.int64, device=dev)
    v_, t_, _ = time_variant(
        torch, _lib, lambda: _lib.sim_batch_reorder(prob, costs, link, sub, oms, obub, rst), ns,
        args.steps, args.warmup, kernels=False)
    o_np, st_np = oms.cpu().numpy(), rst.cpu().numpy()
    reorder = {"value": v_, "unit": "candidates/s", "ms_per_step": t_, "candidates": ns,
               "sample": "every 16th candidate of the batch", "deadlocked": int((o_np == -1).sum()),
               "mean_slowdown_vs_async": round(float((o_np / ms[::16].cpu().numpy()).mean()), 4),
               "mean_transfers": round(float(st_np[:, 0].mean()), 1),
               "mean_mismatched_receives": round(float(st_np[:, 1].mean()), 1)}

    w_advance = time_w_advance(torch, _lib, inputs, w, costs, link, mem, recs_np, dev,
                               args.warmup, min(args.steps, 3), not args.no_cpu)
    alg1 = time_alg1(torch, _lib, inputs, w, costs, link, recs_np, dev, args.warmup,
                     min(args.steps, 3), not args.no_cpu)
    tuner = time_tuner(torch, _lib, inputs, args.warmup, min(args.steps, 3), not args.no_cpu)
    cpu, parity_ok = None, True
    if not args.no_cpu:
        from oracle import octoref
        threads = host_threads()
        rprob = octoref.problem(w.L, w.P, w.v_max, w.M, recs_np.shape[1], w.max_pert)
        # the whole batch on every thread the process may use: the baseline rate and the
        # parity check of every candidate
        c0 = time.perf_counter()
        rms, rbub = octoref.sim_batch(rprob, costs_np, link_np, recs_np, nthreads=threads)
        c1 = time.perf_counter()
        bad = (rms != gms) | (rbub != gbub).any(axis=1)
        parity_ok = not bad.any()
        # one thread on every 16th candidate (all strata; about as long as the full run)
        sample = np.arange(0, n, 16)
        c2 = time.perf_counter()
        octoref.sim_batch(rprob, costs_np, link_np, recs_np[sample], nthreads=1)
        c3 = time.perf_counter()
        cpu = {"value": round(n / (c1 - c0), 1), "unit": "candidates/s", "cores": threads,
               "kind": "oracle",
               "sample": f"the whole batch ({n} candidates, {c1 - c0:.2f} s wall on {threads} "
                         f"threads)",
               "single_thread": {"value": round(len(sample) / (c3 - c2), 1),
                                 "unit": "candidates/s",
                                 "sample": f"every 16th candidate ({len(sample)}, "
                                           f"{c3 - c2:.2f} s on one thread)"},
               "cpu_model": cpu_model(), "os_cpu_count": os.cpu_count(),
               "parity_every_candidate": parity_ok, "mismatches": int(bad.sum())}
        if not parity_ok:
            i = int(np.nonzero(bad)[0][0])
            print(f"bench: {int(bad.sum())} of {n} GPU results differ from the oracle; first "
                  f"{i}: gpu {gms[i]} oracle {rms[i]}", file=sys.stderr)

    if not parity_ok:
        out["value"] = None
    out.update({
        "cpu_baseline": cpu,
        "memory_model": memory_model,
        "comm_model": comm_model,
        "serial_links": serial_links,
        "rendezvous": rendezvous,
        "ordered": ordered,
        "reorder": reorder,
        "w_advance": w_advance,
        "alg1": alg1,
        "tuner": tuner,
    })
    print(json.dumps(out), flush=True)
    if not parity_ok:
        sys.exit(1)


if __name__ == "__main__":
    main()
