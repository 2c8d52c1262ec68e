"""Throughput of the variable-length LSTM time loop on one MI355X.

python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu]

A step is one forward of the whole path (length preparation, input
projection over all valid time steps, on-device time loop) on one batch of the
seeded synthetic workload, with inputs resident in HBM.  W untimed forwards,
then exactly K timed forwards between device synchronisations.  Prints one
JSON line.

value        valid seq*steps/s = sum of lengths / mean forward time
roofline     the loop kernel (the dominant kernel): algorithmic recurrent
             FLOPs (8 H^2 per valid seq*step) per launch / its mean launch
             duration from HIP events recorded by the library on the
             forward's stream, against the dense bf16 (or fp32) MFMA peak
cpu_baseline the fp64 oracle on a bounded sample of the same workload, timed
             on this host's cores; per_config: the oracle on the smaller
             whole workloads, on one thread and on every core

Side legs on the same workload (not part of value): forward_seq (the forward
that also writes the output sequence), forward_stop (termination computed
from the state by a halting read-out), cells (the GRU and tanh RNN cells),
train_step (the forward for training and the backward pass), per_step_path
(the host-driven comparison loop), tiny_f32 (the launch-bound small case) and
configs (every workload shape: the on-device loop against the per-step path).
Each has a --no-* flag.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import workloads  # noqa: E402

PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}  # MI355X dense MFMA
LOOP_SOURCE = os.path.join(ROOT, "paper_1810_08061_amd", "csrc", "persistent.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "loop_{workload}_traffic.json")
HBM_PEAK_GBS = 8000.0
METRIC = "valid seq·steps/sec + MFMA util; speedup of on-device loop vs per-step launch"
DEFAULT_WORKLOAD = "large2048_bf16"


def _log(*a):
    print(*a, file=sys.stderr, flush=True)


def to_device(inp, torch, cell="lstm"):
    """Device tensors in the C ABI's argument order; GRU and RNN have no c0."""
    if inp.dtype == workloads.BF16:
        conv = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).cuda().view(torch.bfloat16)
    else:
        conv = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    f32 = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
    head = (conv(inp.x), torch.from_numpy(np.ascontiguousarray(inp.lengths, np.int32)).cuda(),
            conv(inp.W), conv(inp.U), f32(inp.b), f32(inp.h0))
    return head if cell != "lstm" else (*head, f32(inp.c0))


def time_forwards(torch, ld, model, dev, steps, warmup, out):
    """Mean/std forward time (s) over `steps` forwards, and mean per-phase times."""
    for _ in range(warmup):
        model.forward(*dev, out_h=out[0], out_c=out[1])
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    per, loop_ns, inproj_ns, prep_ns = [], [], [], []
    for _ in range(steps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        model.forward(*dev, out_h=out[0], out_c=out[1])
        e1.record(stream)
        e1.synchronize()
        per.append(e0.elapsed_time(e1) * 1e-3)
        loop_ns.append(model.query(ld.Q_TIME_LOOP_NS))
        inproj_ns.append(model.query(ld.Q_TIME_INPROJ_NS))
        prep_ns.append(model.query(ld.Q_TIME_PREP_NS))
    torch.cuda.synchronize()
    return (float(np.mean(per)), float(np.std(per)), float(np.mean(loop_ns)) * 1e-9,
            float(np.mean(inproj_ns)) * 1e-9, float(np.mean(prep_ns)) * 1e-9)


def time_whole(torch, model, dev, steps, warmup, out):
    """Wall time of exactly `steps` back-to-back forwards (host clock, synchronised)."""
    for _ in range(warmup):
        model.forward(*dev, out_h=out[0], out_c=out[1])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        model.forward(*dev, out_h=out[0], out_c=out[1])
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) / steps


def loop_source_sha256():
    with open(LOOP_SOURCE, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic(workload):
    """HBM bytes per launch of the loop kernel from the committed rocprofv3
    counter summary, or None when absent or taken from another kernel source."""
    path = TRAFFIC_FILE.format(workload=workload)
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_sha256") != loop_source_sha256():
        return None
    return rec.get("bytes_per_launch")


def copy_calibration(torch, mib=512, reps=5):
    """A plain device copy of known size, for scaling FETCH_SIZE/WRITE_SIZE."""
    n = mib * (1 << 20) // 4
    a = torch.ones(n, device="cuda")
    b = torch.empty_like(a)
    for _ in range(reps):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_each_way": n * 4, "dispatches": reps}), flush=True)


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(inp, budget_rows_steps):
    """Time the fp64 oracle on a sample of the workload's rows whose lengths
    sum to about `budget_rows_steps` (all host cores)."""
    import oracle
    order = np.argsort(-inp.lengths, kind="stable")
    # take rows from the middle of the length distribution so the sample's
    # per-step row count resembles the workload's
    mid = len(order) // 4
    rows, total = [], 0
    for r in list(order[mid:]) + list(order[:mid]):
        if total >= budget_rows_steps:
            break
        rows.append(int(r))
        total += int(inp.lengths[r])
    threads = oracle.max_threads()
    t0 = time.perf_counter()
    oracle.forward_inputs(inp, rows=rows, threads=threads)
    dt = time.perf_counter() - t0
    return {"value": total / dt, "unit": "seq·steps/s", "cores": threads, "kind": "oracle",
            "sample": f"{len(rows)} of {inp.B} rows of the workload (sum of lengths {total}), "
                      f"fp64 C oracle, OpenMP over rows, {dt:.1f} s"}


# the smaller workloads timed whole: on one thread (the first three) and on
# every core (the first four); the largest stays sampled (cpu_baseline)
CPU_ONE_THREAD = ("tiny_f32", "lstm256_f32", "lstm512_bf16")
CPU_ALL_CORES = ("tiny_f32", "lstm256_f32", "lstm512_bf16", "skewed1024_bf16")


def cpu_per_config(skip):
    """The fp64 oracle on whole workloads, in valid seq*steps/s."""
    import oracle
    threads = oracle.max_threads()
    out = {}
    for name in workloads.ORDER:
        if name == skip or name not in CPU_ALL_CORES:
            continue
        inp = workloads.workload_inputs(name)
        sumL = int(inp.lengths.sum())
        rec = {"sum_lengths": sumL}
        for th, key in ((1, "one_thread"), (threads, "all_cores")):
            if th == 1 and name not in CPU_ONE_THREAD:
                continue
            _log(f"cpu baseline (oracle), {name}, {th} thread(s)")
            t0 = time.perf_counter()
            oracle.forward_inputs(inp, threads=th)
            dt = time.perf_counter() - t0
            rec[key] = {"value": sumL / dt, "seconds": dt, "threads": th}
        out[name] = rec
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD, choices=workloads.ORDER)
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--no-cpu-configs", action="store_true",
                    help="skip timing the oracle on the smaller whole workloads")
    ap.add_argument("--cpu-budget", type=int, default=24000,
                    help="seq*steps of the oracle sample (about 10-30 s on a host)")
    ap.add_argument("--per-step-reps", type=int, default=3,
                    help="forwards of the per-step path to time (0: skip)")
    ap.add_argument("--no-tiny", action="store_true", help="skip the tiny_f32 launch-overhead leg")
    ap.add_argument("--no-seq", action="store_true",
                    help="skip timing the forward that also writes the output sequence")
    ap.add_argument("--no-cells", action="store_true",
                    help="skip timing the GRU and RNN cells on the same workload shape")
    ap.add_argument("--no-stop", action="store_true",
                    help="skip timing the loop with termination computed from the state")
    ap.add_argument("--no-train", action="store_true",
                    help="skip timing the forward for training and the backward pass")
    ap.add_argument("--no-configs", action="store_true",
                    help="skip the persistent vs per-step comparison over every workload shape")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain copy of known size (for scaling HBM counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path "
              "(the batch would shard across GPUs with no exchange inside the loop).",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_1810_08061_amd as ld

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.copy_calibration:
        copy_calibration(torch)
        return
    w = workloads.WORKLOADS[args.workload]
    _log(f"generating {args.workload}")
    inp = workloads.workload_inputs(args.workload)
    sumL = int(inp.lengths.sum())
    max_len = int(inp.lengths.max())
    dev = to_device(inp, torch)
    out = (torch.empty((w.B, w.H), device="cuda"), torch.empty((w.B, w.H), device="cuda"))

    _log("persistent path")
    model = ld.LstmDyn(w.B, w.D, w.H, w.T, w.dtype, "persistent")
    model.set_option(ld.OPT_TIMING, 1)
    t_fwd, t_std, t_loop, t_inproj, t_prep = time_forwards(torch, ld, model, dev, args.steps,
                                                           args.warmup, out)
    assert model.query(ld.Q_LAST_STATUS) == ld.OK
    launches = model.query(ld.Q_LAUNCHES_PER_FORWARD)
    groups = model.query(ld.Q_GROUPS)
    model.set_option(ld.OPT_TIMING, 0)
    t_wall = time_whole(torch, model, dev, args.steps, 1, out)

    seq_leg = None
    if not args.no_seq:
        # the same forward, also writing out_seq [B, T, H] (zeros past each length)
        _log("persistent path with the output sequence")
        out_seq = torch.empty((w.B, w.T, w.H), device="cuda")
        for _ in range(2):
            model.forward_seq(*dev, out_h=out[0], out_c=out[1], out_seq=out_seq)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(5):
            model.forward_seq(*dev, out_h=out[0], out_c=out[1], out_seq=out_seq)
        torch.cuda.synchronize()
        t_seq = (time.perf_counter() - t0) / 5
        seq_leg = {"ms_per_forward": t_seq * 1e3, "launches_per_forward": model.query(ld.Q_LAUNCHES_PER_FORWARD),
                   "out_seq_bytes": 4 * w.B * w.T * w.H}
        del out_seq

    cell_legs = None
    if not args.no_cells:
        # the same shapes, lengths and x with the GRU and the tanh RNN cells
        # (their weights are repacked on the device into the four-block
        # layout every forward); recurrent FLOPs per valid seq*step: 6H^2 (GRU),
        # 2H^2 (RNN)
        cell_legs = {}
        for cell, rec_per_h2 in (("gru", 6.0), ("rnn", 2.0)):
            _log(f"persistent path, {cell} cell")
            cin = workloads.cell_workload_inputs(cell, args.workload)
            assert np.array_equal(cin.lengths, inp.lengths)
            cdev = to_device(cin, torch, cell=cell)
            cm = ld.LstmDyn(w.B, w.D, w.H, w.T, w.dtype, "persistent", cell=cell)
            cm.set_option(ld.OPT_TIMING, 1)
            c_fwd, c_std, c_loop, c_inproj, c_prep = time_forwards(torch, ld, cm, cdev, args.steps,
                                                                   args.warmup, out)
            assert cm.query(ld.Q_LAST_STATUS) == ld.OK
            c_rec = rec_per_h2 * w.H * w.H * sumL
            cell_legs[cell] = {
                "value": sumL / c_fwd, "unit": "seq·steps/s", "ms_per_forward": c_fwd * 1e3,
                "ms_per_forward_std": c_std * 1e3,
                "phases_ms": {"prep_and_pack": c_prep * 1e3, "input_projection": c_inproj * 1e3,
                              "loop": c_loop * 1e3},
                "loop_algorithmic_tflops": c_rec / c_loop / 1e12,
                "loop_frac": c_rec / c_loop / 1e12 / PEAK_TFLOPS[w.dtype],
                "launches_per_forward": cm.query(ld.Q_LAUNCHES_PER_FORWARD)}
            if not args.no_train:
                # the cell's training step: forward for training, then the
                # backward from a random upstream gradient of the final h
                cdh = torch.from_numpy(np.random.default_rng(6).standard_normal((w.B, w.H))
                                       .astype(np.float32)).cuda()
                for _ in range(2):
                    cm.forward_train(*cdev, out_h=out[0], out_c=out[1])
                    cm.backward(*cdev, None, cdh)
                torch.cuda.synchronize()
                tf = tb = 0.0
                for _ in range(3):
                    t0 = time.perf_counter()
                    cm.forward_train(*cdev, out_h=out[0], out_c=out[1])
                    torch.cuda.synchronize()
                    t1 = time.perf_counter()
                    cm.backward(*cdev, None, cdh)
                    torch.cuda.synchronize()
                    tf += t1 - t0
                    tb += time.perf_counter() - t1
                cell_legs[cell]["train_step"] = {
                    "forward_train_ms": tf / 3 * 1e3, "backward_ms": tb / 3 * 1e3,
                    "step_ms": (tf + tb) / 3 * 1e3, "value": sumL / ((tf + tb) / 3),
                    "unit": "seq·steps/s"}
            cm.close()
            del cdev, cin

    stop_leg = None
    if not args.no_stop:
        # the same forward with a halting read-out v . h + c > 0 ending rows
        # before their caps (v ~ N(0, 1/H) from seed 900, c = -0.5); the
        # loop leaves on the device once no row runs
        _log("persistent path, termination from the state")
        v = (np.random.default_rng(900).standard_normal(w.H) / np.sqrt(w.H)).astype(np.float32)
        vd = torch.from_numpy(v).cuda()
        steps = torch.empty((w.B,), dtype=torch.int32, device="cuda")
        for _ in range(2):
            model.forward_stop(*dev[:6], dev[6], vd, -0.5, out_h=out[0], out_c=out[1], out_steps=steps)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(5):
            model.forward_stop(*dev[:6], dev[6], vd, -0.5, out_h=out[0], out_c=out[1], out_steps=steps)
        torch.cuda.synchronize()
        t_stop = (time.perf_counter() - t0) / 5
        st = steps.cpu().numpy()
        stop_leg = {"ms_per_forward": t_stop * 1e3, "stop_c": -0.5,
                    "loop_steps_run": model.query(ld.Q_STEPS_EXECUTED), "loop_bound": max_len,
                    "rows_ended_early": int((st < inp.lengths).sum()),
                    "valid_seq_steps_run": int(st.sum()),
                    "launches_per_forward": model.query(ld.Q_LAUNCHES_PER_FORWARD)}

    train_leg = None
    if not args.no_train:
        # one training step of the loop: the forward that keeps its state, then
        # the backward pass (gradients of x, W, U, b, h0, c0) from random
        # upstream gradients of the final state
        _log("forward for training + backward")
        rng = np.random.default_rng(5)
        dh = torch.from_numpy(rng.standard_normal((w.B, w.H)).astype(np.float32)).cuda()
        dc = torch.from_numpy(rng.standard_normal((w.B, w.H)).astype(np.float32)).cuda()
        for _ in range(2):
            model.forward_train(*dev, out_h=out[0], out_c=out[1])
            model.backward(*dev, dh, dc)
        torch.cuda.synchronize()
        tf = tb = 0.0
        reps = 3
        for _ in range(reps):
            t0 = time.perf_counter()
            model.forward_train(*dev, out_h=out[0], out_c=out[1])
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            model.backward(*dev, dh, dc)
            torch.cuda.synchronize()
            tf += t1 - t0
            tb += time.perf_counter() - t1
        tf, tb = tf / reps, tb / reps
        train_leg = {"forward_train_ms": tf * 1e3, "backward_ms": tb * 1e3,
                     "step_ms": (tf + tb) * 1e3, "value": sumL / (tf + tb), "unit": "seq·steps/s",
                     "backward_launches": model.query(ld.Q_LAUNCHES_PER_FORWARD),
                     "backward_algorithmic_tflops": 16.0 * w.H * (w.D + w.H) * sumL / tb / 1e12}

    per_step = None
    if args.per_step_reps > 0:
        _log("per-step path")
        ps = ld.LstmDyn(w.B, w.D, w.H, w.T, w.dtype, "per_step")
        t_ps = time_whole(torch, ps, dev, args.per_step_reps, 1, out)
        per_step = {"ms_per_step": t_ps * 1e3, "launches_per_forward": ps.query(ld.Q_LAUNCHES_PER_FORWARD),
                    "speedup_of_persistent": t_ps / t_wall}
        ps.close()

    tiny = None
    if not args.no_tiny:
        # smallest workload: where the per-step launch overhead dominates
        tw = workloads.WORKLOADS["tiny_f32"]
        tin = workloads.workload_inputs("tiny_f32")
        tdev = to_device(tin, torch)
        tout = (torch.empty((tw.B, tw.H), device="cuda"), torch.empty((tw.B, tw.H), device="cuda"))
        tm = ld.LstmDyn(tw.B, tw.D, tw.H, tw.T, tw.dtype, "persistent")
        t_tiny = time_whole(torch, tm, tdev, 200, 20, tout)
        tps = ld.LstmDyn(tw.B, tw.D, tw.H, tw.T, tw.dtype, "per_step")
        t_tiny_ps = time_whole(torch, tps, tdev, 50, 5, tout)
        tiny = {"persistent_us": t_tiny * 1e6, "per_step_us": t_tiny_ps * 1e6,
                "speedup_of_persistent": t_tiny_ps / t_tiny,
                "launches_per_forward": tm.query(ld.Q_LAUNCHES_PER_FORWARD)}
        tm.close()
        tps.close()

    per_shape = None
    if not args.no_configs:
        # every workload shape: the forward with the loop on the device
        # against the per-step path (one host launch pair per step), both
        # timed back to back on the host clock between synchronisations
        per_shape = {}
        for name in workloads.ORDER:
            cw = workloads.WORKLOADS[name]
            _log(f"persistent vs per-step, {name}")
            if name == args.workload:
                cin, cdev, cout = inp, dev, out
            else:
                cin = workloads.workload_inputs(name)
                cdev = to_device(cin, torch)
                cout = (torch.empty((cw.B, cw.H), device="cuda"), torch.empty((cw.B, cw.H), device="cuda"))
            cL = int(cin.lengths.sum())
            cm = ld.LstmDyn(cw.B, cw.D, cw.H, cw.T, cw.dtype, "persistent")
            t_p = time_whole(torch, cm, cdev, 50 if cw.H <= 512 else 10, 3, cout)
            assert cm.query(ld.Q_LAST_STATUS) == ld.OK
            cps = ld.LstmDyn(cw.B, cw.D, cw.H, cw.T, cw.dtype, "per_step")
            t_s = time_whole(torch, cps, cdev, 10 if cw.H <= 512 else 2, 1, cout)
            per_shape[name] = {"value": cL / t_p, "unit": "seq·steps/s", "dtype": cw.dtype,
                             "sum_lengths": cL, "max_len": int(cin.lengths.max()),
                             "persistent_ms": t_p * 1e3, "per_step_ms": t_s * 1e3,
                             "speedup_of_persistent": t_s / t_p,
                             "launches_persistent": cm.query(ld.Q_LAUNCHES_PER_FORWARD),
                             "launches_per_step": cps.query(ld.Q_LAUNCHES_PER_FORWARD),
                             "mfma_frac_forward": 8.0 * cw.H * (cw.D + cw.H) * cL / t_p / 1e12
                             / PEAK_TFLOPS[cw.dtype]}
            cm.close()
            cps.close()

    dt = w.dtype
    flops_fwd = 8.0 * w.H * (w.D + w.H) * sumL
    flops_rec = 8.0 * w.H * w.H * sumL
    flops_in = 8.0 * w.H * w.D * sumL
    e = 2 if dt == workloads.BF16 else 4
    bytes_alg = sumL * w.D * e + 4 * w.H * (w.D + w.H) * e + 16 * w.H + 16 * w.B * w.H + 4 * w.B
    peak = PEAK_TFLOPS[dt]
    achieved = flops_rec / t_loop / 1e12
    traffic = measured_traffic(args.workload)
    line = {
        "metric": METRIC,
        "value": sumL / t_fwd,
        "unit": "seq·steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": t_fwd * 1e3,
        "ms_per_step_std": t_std * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": dt,
        "data": "synthetic (seeded generator; random-init weights)",
        "config": {"workload": args.workload, "B": w.B, "D": w.D, "H": w.H, "T_max": w.T,
                   "lengths": list(map(str, w.lengths)), "sum_lengths": sumL, "max_len": max_len,
                   "parallelism": "none (1 GPU)", "persistent_groups": groups},
        "roofline": {"bound": "mfma", "kernel": "persistent time loop (recurrent h U, gates)",
                     "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                     "frac": achieved / peak, "traffic": traffic,
                     "algorithmic_flops_per_launch": flops_rec,
                     "mean_launch_ms": t_loop * 1e3},
        "mfma_frac_forward": flops_fwd / t_fwd / 1e12 / peak,
        # algorithmic bytes (valid x, W, U, b, states, lengths) over the forward
        "hbm_frac_forward_algorithmic": bytes_alg / t_fwd / 1e9 / HBM_PEAK_GBS,
        # the loop kernel's counted HBM bytes (committed rocprofv3 record) over
        # its mean launch time
        "hbm_frac_loop_measured": (traffic / t_loop / 1e9 / HBM_PEAK_GBS) if traffic else None,
        "phases_ms": {"prep": t_prep * 1e3, "input_projection": t_inproj * 1e3,
                      "loop": t_loop * 1e3},
        "input_projection_tflops": flops_in / t_inproj / 1e12,
        "launches_per_forward": launches,
        "wall_ms_per_step": t_wall * 1e3,
        "per_step_path": per_step,
        "forward_seq": seq_leg,
        "forward_stop": stop_leg,
        "train_step": train_leg,
        "cells": cell_legs,
        "tiny_f32": tiny,
        "configs": per_shape,
    }
    if not args.no_cpu:
        _log("cpu baseline (oracle)")
        cb = cpu_baseline(inp, args.cpu_budget)
        cb["host"] = {"cpu_model": cpu_model(), "nproc": os.cpu_count(),
                      "affinity": len(os.sched_getaffinity(0))}
        if not args.no_cpu_configs:
            cb["per_config"] = cpu_per_config(skip=None)
        line["cpu_baseline"] = cb
    print(json.dumps(line), flush=True)
    model.close()


if __name__ == "__main__":
    main()
