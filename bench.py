"""Benchmark of the device-side LSTM while-loop: forward + gradient loop.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]

One step = lstm_loop_fwd (save_for_backward) + lstm_loop_bwd over one batch
of synthetic input already resident in device memory.  Prints one JSON line:
throughput in timesteps*sequences per second (sum of the sequence lengths per
step / step time), the matrix-core utilisation against the dense peak of the
operand type, the time per loop iteration, a roofline entry for the dominant
kernel (timed with HIP events on the launch stream inside the timed region),
and the CPU oracle timed on a bounded sample of the same workload.
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

METRIC = "LSTM fwd+bwd timesteps·seqs/sec at H=1024; MFMA util; per-iteration µs"
PEAK = {"bf16": 2.5e15, "f32": 157.3e12}     # MI355X dense matrix-core peaks, flop/s


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="lstm_b128_h1024_tmax200_varlen_bf16")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="target CPU work of the oracle baseline sample (0 = skip)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="after the benchmark, a plain device copy of MIB MiB, five "
                         "times (scale of the memory counters)")
    return ap.parse_args()


def stage_flops(w, sum_len):
    """Algorithmic flops per launch of each stage (per layer)."""
    H, G2 = w.H, 2.0 * w.gates     # 2 flops per multiply-add, G gate blocks
    out = {}
    for l in range(w.layers):
        I = w.I if l == 0 else w.H
        out.setdefault("fwd_loop", []).append(G2 * H * H * sum_len)
        out.setdefault("bwd_loop", []).append(G2 * H * H * sum_len)
        out.setdefault("input_proj", []).append(G2 * H * I * sum_len)
        out.setdefault("dw", []).append(G2 * H * (I + H) * sum_len)
        out.setdefault("dx", []).append(G2 * H * I * sum_len)
    return {k: float(np.mean(v)) for k, v in out.items()}


def _blas_threads():
    try:
        from threadpoolctl import threadpool_info
        return max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:
        return None


def cpu_baseline(w, inp, target_s, precision="fp32", threads=None):
    """The oracle as it is, in its batched masked form (BLAS products per
    step, hand-written gradient loop) on the full batch: the first T_s loop
    iterations when the whole run would take longer than `target_s`, else the
    whole run repeated up to about `target_s` seconds.  precision "fp32" is
    the float32 form; "bf16" the bfloat16-emulating float64 form the parity
    tests use.  threads: BLAS threads (None: every core available to the
    process)."""
    import oracle
    from threadpoolctl import threadpool_limits
    avail = len(os.sched_getaffinity(0))
    nthr = avail if threads is None else threads
    dt_in = np.float32 if precision == "fp32" else np.float64

    def run(Ts):
        sl = np.minimum(inp["seq_len"], Ts)
        x = inp["x"][:Ts].astype(dt_in)
        dy = inp["dy"][:Ts].astype(dt_in) if inp["dy"] is not None else None
        Ws = [a.astype(dt_in) for a in inp["W"]]
        bs = [a.astype(dt_in) for a in inp["bias"]]
        h0, c0 = inp["h0"].astype(dt_in), inp["c0"].astype(dt_in)
        dhT, dcT = inp["dhT"].astype(dt_in), inp["dcT"].astype(dt_in)
        t0 = time.perf_counter()
        if w.cell in ("rnn", "gru"):
            fwd, bwd = ((oracle.stacked_rnn_forward, oracle.stacked_rnn_backward) if w.cell == "rnn"
                        else (oracle.stacked_gru_forward, oracle.stacked_gru_backward))
            _, _, tapes = fwd(x, sl, Ws, bs, h0, precision)
            bwd(tapes, dy, dhT)
        elif w.cell == "act":
            _, _, _, tapes = oracle.stacked_act_forward(x, sl, Ws, bs, h0, c0, precision, w.ponder_max)
            oracle.stacked_act_backward(tapes, dy, dhT, dcT)
        else:
            fwd, bwd = ((oracle.stacked_skip_forward, oracle.stacked_skip_backward) if w.cell == "skip"
                        else (oracle.stacked_forward, oracle.stacked_backward))
            y, hT, cT, tapes = fwd(x, sl, Ws, bs, h0, c0, precision)
            bwd(tapes, dy, dhT, dcT)
        return time.perf_counter() - t0, int(sl.sum())

    with threadpool_limits(limits=nthr):
        used = _blas_threads() or nthr
        T_eff = int(inp["seq_len"].max())
        dt, _ = run(2)
        Ts = int(max(2, min(T_eff, target_s / max(dt / 2, 1e-6))))
        dt, n = run(Ts)
        reps = 1
        if Ts == T_eff:
            while dt < target_s and reps < 16:
                d2, n2 = run(Ts)
                dt += d2
                n += n2
                reps += 1
    what = (f"first {Ts} of {T_eff} loop iterations" if Ts < T_eff
            else f"all {T_eff} loop iterations, {reps} runs")
    form = ("float32 batched masked form (BLAS)" if precision == "fp32"
            else "bfloat16-emulating float64 batched masked form")
    return {"value": n / dt, "unit": "timesteps·seqs/s", "cores": int(used),
            "cores_available": avail, "kind": "oracle",
            "sample": f"full batch B={w.B}, {what} ({n} timesteps*seqs), oracle {form}, "
                      f"fwd+bwd, {dt:.1f} s on {used} BLAS thread(s) of {avail} cores available"}


# HBM traffic of the loop kernels, from rocprofv3 PMC runs (FETCH_SIZE and
# WRITE_SIZE per dispatch, scaled by the same counters on a plain copy).  The
# figures are used only while the kernel source they were taken on is
# unchanged.
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "pmc_traffic.md")
LOOP_STAGES = ("fwd_loop", "bwd_loop")


def source_hash(rels):
    """Hash of the kernel sources (a list of repository-relative paths)."""
    import hashlib
    h = hashlib.sha256()
    for rel in rels:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def recorded_traffic(kernel, workload):
    """Bytes per launch recorded for (kernel, workload), or None."""
    if kernel not in LOOP_STAGES or not os.path.exists(TRAFFIC_FILE):
        return None
    text = open(TRAFFIC_FILE).read()
    if "```json" not in text:
        return None
    block = text.split("```json", 1)[1].split("```", 1)[0]
    try:
        rec = json.loads(block)
    except ValueError:
        return None
    ent = rec.get("entries", {}).get(f"{kernel}/{workload}")
    if not ent or not ent.get("sources") or ent.get("source_sha256_16") != source_hash(ent["sources"]):
        return None
    return float(ent["bytes_per_launch"])


def pinned_copy_peak(nbytes, streams=1, reps=5):
    """Host-link rate of plain copies between pinned host memory and device
    memory: GB/s for device-to-host and host-to-device, each direction alone,
    `streams` copies of nbytes in flight at once (one per stream)."""
    import torch
    n = nbytes // 4
    dev = [torch.ones(n, dtype=torch.float32, device="cuda:0") for _ in range(streams)]
    host = [torch.empty(n, dtype=torch.float32, pin_memory=True) for _ in range(streams)]
    ss = [torch.cuda.Stream() for _ in range(streams)]
    out = {}
    for name in ("d2h", "h2d"):
        best = 0.0
        for _ in range(reps):
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for i in range(streams):
                with torch.cuda.stream(ss[i]):
                    if name == "d2h":
                        host[i].copy_(dev[i], non_blocking=True)
                    else:
                        dev[i].copy_(host[i], non_blocking=True)
            torch.cuda.synchronize()
            best = max(best, streams * nbytes / (time.perf_counter() - t0) / 1e9)
        out[name] = best
    return out


def copy_calibration(mib):
    """A plain device copy of `mib` MiB, five times (for counter scaling)."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4, "launches": 5}),
          file=sys.stderr, flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the data-parallel split over GPUs is described, not run)", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_1805_01772_amd import lstmloop, workloads as wl
    from paper_1805_01772_amd.runner import DeviceCase

    w = wl.BY_NAME[args.workload]
    inp = wl.generate(w)
    sum_len = int(inp["seq_len"].sum())
    T_eff = int(inp["seq_len"].max())
    dc = DeviceCase(inp, w.H, w.I, w.layers, w.dtype, device="cuda:0", cell=w.cell,
                    ponder_max=w.ponder_max)
    plan_kw = {}
    if w.spill:   # stack swapped to pinned host memory through a ring of 4 chunks of 32 steps
        C = 32
        plan_kw = dict(spill=1, spill_chunk_steps=C,
                       device_stack_budget_bytes=4 * C * w.B * 5 * w.H * 4)

    def timed(kw, timing, steps=None, per_step_events=False):
        steps = steps or args.steps
        plan = dc.plan(**kw)
        for _ in range(args.warmup):
            dc.fwd(plan)
            dc.bwd(plan)
        torch.cuda.synchronize()
        if plan.status_sync() != 0:
            raise RuntimeError("device error during warmup")
        plan.set_timing(timing)
        stream = torch.cuda.current_stream()
        # an event after every step only where per-step times are wanted (each
        # costs a few microseconds of stream time)
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1 if per_step_events else 2)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        evs[0].record(stream)
        for k in range(steps):
            dc.fwd(plan)
            dc.bwd(plan)
            if per_step_events:
                evs[k + 1].record(stream)
        if not per_step_events:
            evs[1].record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        per_step = [evs[k].elapsed_time(evs[k + 1]) for k in range(len(evs) - 1)]
        stages = plan.read_timing()
        plan.set_timing(False)
        err = plan.status_sync()
        if err:
            raise RuntimeError(f"device error word {err}")
        geom, sbytes = plan.geometry(), plan.stack_bytes()
        plan.close()
        return evs[0].elapsed_time(evs[-1]), wall, stages, geom, sbytes, per_step

    # Stage breakdown from a pass of its own: every stage's event pair costs
    # a few microseconds of stream time, so the timed region below records
    # only the dominant kernel's stage (the roofline's launch duration).
    breakdown_steps = min(args.steps, 10)
    stages_all = timed(plan_kw, True, breakdown_steps)[2]
    dom = max(("fwd_loop", "bwd_loop", "input_proj", "dw", "dx"), key=lambda k: stages_all[k][0])
    gpu_ms, wall, stages, geom, sbytes, _ = timed(plan_kw, [dom])
    # the spread of single steps, from a pass of its own with an event after
    # every step and no stage events
    per_step = timed(plan_kw, False, breakdown_steps, per_step_events=True)[5]
    spill = None
    if w.spill:
        res_ms = timed({}, False)[0]
        nch = -(-w.T_max // C)
        moved = 2 * sbytes[1]   # the chunks evicted from the device ring go out once and come back once
        # the alternative to swapping: push c_t only, recompute each chunk's
        # gates in the gradient pass (two products over the chunk's rows)
        rc = timed({"recompute": 1, "spill_chunk_steps": C}, False)
        slot_bytes = C * w.B * 5 * w.H * 4
        peak1 = pinned_copy_peak(slot_bytes, 1)
        peak2 = pinned_copy_peak(slot_bytes, 2)
        link = moved / (gpu_ms / args.steps / 1e3) / 1e9
        spill = {"chunk_steps": C, "ring_slots": 4, "device_stack_bytes": sbytes[0],
                 "host_stack_bytes": sbytes[1], "ms_per_step_resident": res_ms / args.steps,
                 "ms_per_step_recompute": rc[0] / args.steps, "device_stack_bytes_recompute": rc[4][0],
                 "overlap_efficiency": (res_ms / args.steps) / (gpu_ms / args.steps),
                 "host_link_GBps": link,
                 "pinned_copy_peak_GBps": {"chunk_bytes": slot_bytes, "one_stream": peak1,
                                           "two_streams": peak2},
                 "host_link_fraction_of_peak": link / max(peak1["d2h"], peak1["h2d"], 1e-9),
                 "seconds_at_peak": moved / 2 / peak1["d2h"] / 1e9 + moved / 2 / peak1["h2d"] / 1e9}

    ms_per_step = gpu_ms / args.steps
    value = sum_len / (ms_per_step / 1e3)
    flops = wl.algorithmic_flops(w, inp["seq_len"])
    mfma_util = flops / (ms_per_step / 1e3) / PEAK[w.dtype]
    sflops = stage_flops(w, sum_len)
    per_launch = {k: (ms / n if n else 0.0) for k, (ms, n) in stages.items()}
    achieved = sflops[dom] / (per_launch[dom] / 1e3) / 1e12
    peak_tf = PEAK[w.dtype] / 1e12
    measured_peak = lstmloop.ll_measure_mfma_peak(w.dtype, 32)
    measured_16 = lstmloop.ll_measure_mfma_peak(w.dtype, 16)
    # what a loop over T_eff (or T_max) padded steps would execute: every
    # sequence runs every step (a static unroll to the longest sequence)
    padded = {f"T_{n}": sum(6.0 * w.gates * w.H * ((w.I if l == 0 else w.H) + w.H) * w.B * T
                            for l in range(w.layers)) for n, T in (("eff", T_eff), ("max", w.T_max))}
    q = np.percentile(per_step, [5, 50, 95])
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "timesteps·seqs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "I": w.I, "H": w.H, "T_max": w.T_max,
                   "layers": w.layers, "cell": w.cell, "seq_len": f"U{{{w.len_lo}..{w.len_hi}}}",
                   "sum_len": sum_len, "T_eff": T_eff, "loop_workgroups": geom["workgroups"],
                   "units_per_workgroup": geom["units_per_workgroup"]},
        "mfma_util": mfma_util,
        "mfma_util_of_measured_peak": flops / (ms_per_step / 1e3) / (measured_peak * 1e12),
        "measured_mfma_peak_tflops": measured_peak,
        "measured_mfma_rate_16x16_tflops": measured_16,
        "step_ms": {"median": q[1], "p5": q[0], "p95": q[2],
                    "from": f"separate pass of {breakdown_steps} steps with an event after each"},
        "padded_flops_per_step": padded,
        "flops_skipped_vs_padded_T_eff": 1.0 - flops / padded["T_eff"],
        "per_iteration_us": ms_per_step * 1e3 / T_eff if T_eff else None,
        "algorithmic_tflops": flops / (ms_per_step / 1e3) / 1e12,
        "host_wall_ms_per_step": wall * 1e3 / args.steps,
        "stage_ms_per_step": {k: ms / breakdown_steps for k, (ms, n) in stages_all.items()},
        "stage_timing": f"separate pass of {breakdown_steps} steps with every stage's events",
        "roofline": {"bound": "mfma", "kernel": dom, "achieved": achieved, "peak": peak_tf,
                     "unit": "TFLOP/s", "frac": achieved / peak_tf,
                     "frac_of_measured_peak": achieved / measured_peak,
                     "traffic": recorded_traffic(dom, w.name),
                     "traffic_source": "stored record in profiles/pmc_traffic.md (two rocprofv3 "
                                       "--pmc passes, FETCH_SIZE and WRITE_SIZE, scaled by a plain "
                                       "copy), used only while the kernel sources hash to the "
                                       "recorded value, else null",
                     "per_launch_ms": per_launch[dom],
                     "algorithmic_flops_per_launch": sflops[dom]},
    }
    if spill:
        out["spill"] = spill
    if args.cpu_seconds > 0:
        # the float32 form on every core available to the process, and on one
        # core; the bfloat16-emulating form (the parity reference) for context
        out["cpu_baseline"] = cpu_baseline(w, inp, args.cpu_seconds)
        out["cpu_baseline_1core"] = cpu_baseline(w, inp, args.cpu_seconds / 3, threads=1)
        if w.dtype == "bf16":
            out["cpu_baseline_bf16_emulating"] = cpu_baseline(w, inp, args.cpu_seconds / 3,
                                                              precision="bf16")
    print(json.dumps(out), flush=True)
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)


if __name__ == "__main__":
    main()
