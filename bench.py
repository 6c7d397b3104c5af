#!/usr/bin/env python3
"""Online surrogate-training throughput on one MI355X.

One step is one pass of the whole hot path on one batch: a put of one chunk of
streamed samples into the GPU reservoir (eviction of seen samples once full),
a batch draw with replacement and its gather, and one train step of the MLP
surrogate (forward, fused MSE, backward, Adam).  Workload: 100x100 heat fields
from an FTCS solver, 1000 simulations x 100 steps, MLP 6-256-256-10000 fp32,
batch 1024, reservoir of 100,000 samples (threshold 16,667), chunks of the
100 concurrent simulations' current time step.  The whole ensemble is first
streamed through the schedule (untimed), then the stream wraps around so
every timed put replaces seen samples.

Prints one JSON line.  `value` is samples processed per second by the train
step (batch size x steps / time), measured with HIP events on the work stream
over the timed steps.  `roofline` reports the dominant kernel's algorithmic
rate against MI355X's datasheet peak, from HIP events around that kernel in
the same timed region.  `cpu_baseline` times the plain fp64 CPU oracle on a
bounded sample of the same workload on this host.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_FP32_MFMA = 157.3e12      # MI355X dense fp32 matrix peak, FLOP/s
PEAK_HBM = 8.0e12              # MI355X HBM3E, bytes/s


def parse_args():
    p = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=2000)
    p.add_argument("--warmup", type=int, default=50)
    p.add_argument("--config", default="heat-100x100")
    p.add_argument("--profile-steps", type=int, default=200,
                   help="steps of the per-kernel breakdown pass (all phases timed)")
    p.add_argument("--cpu-seconds", type=float, default=15.0,
                   help="target duration of the CPU-oracle baseline sample (0 disables it)")
    p.add_argument("--out", default=None, help="also write the JSON line to this file")
    return p.parse_args()


def gemm_flops(w) -> float:
    """Algorithmic flops of one output-layer GEMM launch: 2 B H D."""
    return 2.0 * w.batch * w.widths[-2] * w.widths[-1]


def kernel_table(w, phases_ms: dict, res_ms: dict) -> dict:
    """Average duration and algorithmic rate of each timed phase."""
    out = {}
    D, B, H = w.widths[-1], w.batch, w.widths[-2]
    n_params = w.n_params()
    for name, (ms, n) in phases_ms.items():
        avg = ms / max(n, 1)
        row = {"avg_us": round(avg * 1e3, 2), "launches": n}
        if name in ("fwd_output", "wgrad_output", "igrad_output"):
            rate = gemm_flops(w) / (avg * 1e-3)
            row.update(achieved_tflops=round(rate / 1e12, 2), frac_fp32_mfma=round(rate / PEAK_FP32_MFMA, 4))
        if name == "adam":
            rate = 28.0 * n_params / (avg * 1e-3)
            row.update(achieved_gbs=round(rate / 1e9, 1), frac_hbm=round(rate / PEAK_HBM, 4))
        out[name] = row
    x_dim = w.widths[0]
    for name, (ms, n) in res_ms.items():
        avg = ms / max(n, 1)
        row = {"avg_us": round(avg * 1e3, 2), "launches": n}
        if name == "gather":
            byts = 2.0 * B * (D + x_dim) * 4
            row.update(achieved_gbs=round(byts / (avg * 1e-3) / 1e9, 1), frac_hbm=round(byts / (avg * 1e-3) / PEAK_HBM, 4))
        if name == "put_copy":
            byts = 2.0 * w.wave * (D + x_dim) * 4
            row.update(achieved_gbs=round(byts / (avg * 1e-3) / 1e9, 1), frac_hbm=round(byts / (avg * 1e-3) / PEAK_HBM, 4))
        out["reservoir_" + name] = row
    return out


def cpu_baseline(w, inputs, fields, seconds: float) -> dict:
    """The fp64 oracle (put + draw + train step) on this host, bounded in time."""
    from oracle import mlp
    from oracle.reservoir import OK, Reservoir
    from oracle.runner import chunk_arrays
    try:
        import threadpoolctl
        blas = threadpoolctl.threadpool_info()
        blas_threads = max((b.get("num_threads", 1) for b in blas), default=1)
    except Exception:  # pragma: no cover
        blas_threads = 1
    res = Reservoir(w.capacity, w.threshold, inputs.shape[-1], fields.shape[-1], w.reservoir_seed)
    chunk = 0
    while res.N <= w.threshold:                     # fill past the threshold (untimed)
        res.put(*chunk_arrays(w, inputs, fields, chunk))
        chunk += 1
    params = mlp.init_params(w.widths, w.init_seed)
    opt = mlp.Adam(lr=w.lr)
    steps = 0
    t0 = time.perf_counter()
    while steps < 2 or time.perf_counter() - t0 < seconds:
        res.put(*chunk_arrays(w, inputs, fields, chunk % w.n_chunks))
        chunk += 1
        st, slots, xb, ub, _ = res.sample_batch(w.batch)
        assert st == OK
        loss, grads = mlp.loss_and_grads(params, xb, ub)
        params = opt.step(params, grads)
        steps += 1
    dt = time.perf_counter() - t0
    return {"value": round(w.batch * steps / dt, 2), "unit": "samples/s",
            "cores": blas_threads, "kind": "oracle",
            "sample": f"{steps} steps (put {w.wave} rows + draw {w.batch} + fp64 train step) on a reservoir "
                      f"filled past its threshold with the first {chunk - steps} chunks; "
                      f"{len(os.sched_getaffinity(0))} host cores visible, numpy BLAS threads {blas_threads}",
            "ms_per_step": round(dt / steps * 1e3, 1)}


def main():
    args = parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} (WORLD_SIZE {world}) is not supported: "
              "this build has no multi-GPU path.", file=sys.stderr)
        sys.exit(2)

    import torch

    from fixtures import configs, heat
    from paper_2309_16743_amd._abi import SURROGATE_PHASES
    from paper_2309_16743_amd.online import OnlineTrainer

    if args.config not in configs.ALL or configs.ALL[args.config].precision != "fp32":
        print(f"unsupported config {args.config}", file=sys.stderr)
        sys.exit(2)
    w = configs.ALL[args.config]
    t_gen = time.perf_counter()
    X = heat.sample_parameters(w.n_sims, w.data_seed)
    inputs = heat.inputs_for(X, w.tau)
    fields = heat.heat_fields(X, w.grid, w.tau)
    t_gen = time.perf_counter() - t_gen
    print(f"[bench] generated {fields.nbytes / 1e9:.1f} GB of {w.grid}x{w.grid} fields in {t_gen:.1f} s",
          file=sys.stderr, flush=True)

    dev = torch.device("cuda:0")
    inputs_d = torch.from_numpy(inputs).to(dev)
    fields_d = torch.from_numpy(fields).to(dev)
    stream = torch.cuda.Stream(device=dev)
    with torch.cuda.stream(stream):
        tr = OnlineTrainer(w.widths, w.batch, w.capacity, w.threshold, w.wave, w.tau, inputs_d, fields_d,
                           w.reservoir_seed, w.init_seed, lr=w.lr, stream=stream)
        # stream the whole ensemble through the schedule (untimed), then warm up
        for _ in range(w.n_chunks):
            tr.iterate()
        for _ in range(args.warmup):
            assert tr.iterate(wrap=True)
        torch.cuda.synchronize()
        print(f"[bench] setup done: {tr.steps_done} train steps, reservoir {tr.res.stats()['n']} samples",
              file=sys.stderr, flush=True)

        # per-kernel breakdown pass (every phase timed)
        kp = max(args.profile_steps, 1)
        tr.sur.timing_begin(list(SURROGATE_PHASES), kp)
        tr.res.timing_begin(["put_assign", "put_copy", "select", "gather"], 2 * kp)
        for _ in range(kp):
            tr.iterate(wrap=True)
        breakdown = kernel_table(w, tr.sur.timing_end(), tr.res.timing_end())
        gemm_phases = ("fwd_output", "wgrad_output", "igrad_output")
        dominant = max(gemm_phases, key=lambda p: breakdown[p]["avg_us"])

        # timed region: K steps; HIP events around the dominant kernel and the gather
        K = args.steps
        tr.sur.timing_begin([dominant], K)
        tr.res.timing_begin(["gather"], 2 * K)
        n_win = K // 10
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(n_win + 2)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        ev[0].record(stream)
        for i in range(K):
            tr.iterate(wrap=True)
            if (i + 1) % 10 == 0 and (i + 1) // 10 <= n_win:
                ev[(i + 1) // 10].record(stream)
        ev[-1].record(stream)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        gpu_ms = ev[0].elapsed_time(ev[-1])
        windows = [ev[j].elapsed_time(ev[j + 1]) for j in range(n_win)]
        dom_ms, dom_n = tr.sur.timing_end()[dominant]
        g_ms, g_n = tr.res.timing_end()["gather"]
        loss = float(tr.loss.item())

    ms_per_step = gpu_ms / K
    value = w.batch * K / (gpu_ms * 1e-3)
    win_sps = [10 * w.batch / (t * 1e-3) for t in windows] if windows else [value]
    dom_avg_s = dom_ms / dom_n * 1e-3
    achieved = gemm_flops(w) / dom_avg_s
    gather_avg_s = g_ms / g_n * 1e-3
    gather_rate = 2.0 * w.batch * (w.widths[-1] + w.widths[0]) * 4 / gather_avg_s

    line = {
        "metric": "surrogate train samples/s at 1 MI355X; MFMA util of output layer; reservoir GB/s",
        "value": round(value, 1),
        "unit": "samples/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "fields": f"FTCS heat {w.grid}x{w.grid}, {w.n_sims} sims x {w.tau} steps",
                   "widths": list(w.widths), "batch": w.batch, "capacity": w.capacity,
                   "threshold": w.threshold, "put_rows_per_step": w.wave},
        "roofline": {"bound": "mfma", "kernel": f"gemm_f32 ({dominant})", "achieved": round(achieved / 1e12, 2),
                     "peak": PEAK_FP32_MFMA / 1e12, "unit": "TFLOP/s", "frac": round(achieved / PEAK_FP32_MFMA, 4),
                     "traffic": None, "per_launch_flops": gemm_flops(w), "avg_us": round(dom_avg_s * 1e6, 2)},
        "reservoir_gather": {"achieved": round(gather_rate / 1e9, 1), "unit": "GB/s",
                             "frac_hbm": round(gather_rate / PEAK_HBM, 4), "avg_us": round(gather_avg_s * 1e6, 2)},
        "windows_of_10": {"median_samples_s": round(float(np.median(win_sps)), 1),
                          "mean_samples_s": round(float(np.mean(win_sps)), 1), "n": len(win_sps)},
        "wall_s": round(wall, 3),
        "last_loss": loss,
        "kernels": breakdown,
        "cpu_baseline": None,
    }
    tr.close()
    del inputs_d, fields_d
    torch.cuda.empty_cache()
    if args.cpu_seconds > 0:
        line["cpu_baseline"] = cpu_baseline(w, inputs, fields, args.cpu_seconds)
    text = json.dumps(line)
    print(text, flush=True)
    if args.out:
        with open(args.out, "w") as f:
            f.write(text + "\n")


if __name__ == "__main__":
    main()
