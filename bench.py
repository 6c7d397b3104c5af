#!/usr/bin/env python3
"""Online surrogate-training throughput on one MI355X.

One step is one pass of the whole hot path on one batch: a put of one chunk of
streamed samples into the GPU reservoir (replacing seen samples once full), a
batch draw with replacement and its gather, and one train step of the MLP
surrogate (forward, fused MSE, backward, Adam).  The reservoir's put, draw and
gather for the next batch run on a second stream while the current batch
trains (two batch buffers, ordered by events), as the paper's aggregator and
training threads run concurrently; --one-stream runs everything on one stream,
as does a workload whose batch targets are under 1 MiB (tiny-16x16), where the
step is launch-latency-bound and two cross-stream waits cost more than the
overlap gains; there the train step is captured once as a HIP graph and
replayed each step (--no-graph launches its kernels every step).

Default workload (--config deep-sine-1000x1000): 1000x1000 fields (smooth
sine-mode stand-ins for heat solutions, generated on the GPU), MLP
6-2048-2048-2048-1,000,000 with bf16 GEMMs, fp32 master weights and Adam,
batch 1024, a reservoir of 30,000 samples (120 GB) with threshold 5,000.  The
reservoir is filled with generated chunks (untimed); during the timed steps
8 producer streams (the paper's clients) each put chunks of 64 samples, one
put per step in turn, concurrently with training ("mode B"); the same steps
are then timed again with production suspended ("mode A", --prefilled makes
it the headline).  --config sine-1000x1000: 6-1024-1024-1,000,000, batch
512, 20,000 samples (80 GB), the same schedule.

--config heat-100x100: 100x100 heat fields from an FTCS solver, 1000
simulations x 100 steps, MLP 6-256-256-10000 fp32, batch 1024, reservoir of
100,000 samples (threshold 16,667), chunks of the 100 concurrent simulations'
current time step.  The whole ensemble is first streamed through the
schedule (untimed), then the stream wraps around so every timed put replaces
seen samples.  --config tiny-16x16: the same at 16x16 (latency-bound).

--config stress-100k-rows: the reservoir alone with rows of 100,000 floats,
capacity 50,000 (20 GB slab), threshold 10,000, 64 producer streams putting
chunks of 256 rows and one consumer drawing batches of 256 into a batch
buffer; `value` is then the reservoir's data rate in GB/s (rows accepted by
puts plus rows gathered, each moved once in and once out) over the timed
iterations (one put and one draw each).

Prints one JSON line.  `value` is samples processed per second by the train
step (batch size x steps / time), from HIP events on the work stream over the
timed steps.  `roofline` reports the dominant kernel's algorithmic rate
against MI355X's datasheet peak, from HIP events that the library hands to
that kernel's launch (hipExtLaunchKernel stamps them with the kernel's own
start and end) on the stream it runs on, inside the same timed region (the
only launches there that carry events; a replayed train step carries none,
and then its kernels are timed as below); `output_layer` does the same for
the three output-layer GEMMs and `reservoir` for the put copies and the
gather, on eager steps right after the timed region.  `cpu_baseline` times the
plain fp64 CPU oracle on a bounded sample of the same workload on this host.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np
from typing import Optional

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_FP32_MFMA = 157.3e12      # MI355X dense fp32 matrix peak, FLOP/s
PEAK_BF16_MFMA = 2.5e15        # MI355X dense bf16 matrix peak, FLOP/s
PEAK_HBM = 8.0e12              # MI355X HBM3E, bytes/s
METRIC = "surrogate train samples/s at 1 MI355X; MFMA util of output layer; reservoir GB/s"


def parse_args():
    p = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=None, help="timed steps (default 2000 fp32, 100 bf16)")
    p.add_argument("--warmup", type=int, default=None, help="untimed steps before timing (default 50 / 5)")
    p.add_argument("--config", default="deep-sine-1000x1000")
    p.add_argument("--producers", type=int, default=8,
                   help="1000x1000 workloads: producer streams the timed puts come from, one put per step in turn")
    p.add_argument("--policy-comparison", action="store_true",
                   help="instead of the throughput benchmark: stream the heat-100x100 ensemble once through the "
                        "Reservoir, FIRO and FIFO buffers and report train steps and samples/s per buffer")
    p.add_argument("--prefilled", action="store_true",
                   help="no puts in the timed steps: draws and train steps on the reservoir as the setup left it "
                        "(the paper's throughput with production suspended); default: one put per step")
    p.add_argument("--gathered-targets", action="store_true",
                   help="gather the batch's field rows into a batch buffer before the train step (default: the "
                        "output layer's forward reads them in place from the reservoir through the drawn slots)")
    p.add_argument("--no-graph", action="store_true",
                   help="one-stream workloads: launch every train step's kernels instead of replaying the "
                        "step captured as a HIP graph")
    p.add_argument("--one-stream", action="store_true",
                   help="run the reservoir and the train step on one stream (default: the reservoir's put, draw "
                        "and gather of the next batch overlap the current train step on a second stream, unless "
                        "a batch's targets are under 1 MiB: then the step is launch-latency-bound and the two "
                        "cross-stream waits per step cost more than the overlap gains, so one stream is used)")
    p.add_argument("--profile-steps", type=int, default=None,
                   help="steps of the per-kernel breakdown pass (all phases timed)")
    p.add_argument("--cpu-seconds", type=float, default=15.0,
                   help="target duration of the CPU-oracle baseline sample (0 disables it)")
    p.add_argument("--out", default=None, help="also write the JSON line to this file")
    p.add_argument("--pmc-calibration", action="store_true",
                   help="first run a reference elementwise kernel of known traffic (1 GiB read, 1 GiB written) "
                        "for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE")
    p.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"), default=None,
                   help="no GPU work: turn the counter CSVs of two rocprofv3 --pmc runs (FETCH_SIZE, WRITE_SIZE) of "
                        "this workload with --pmc-calibration into per-launch HBM bytes of its dominant kernel "
                        "(--kernel) and record them in profiles/hbm_traffic.json")
    p.add_argument("--library-reference", action="store_true",
                   help="instead of the benchmark: time torch's own GEMMs (hipBLASLt / rocBLAS) on this workload's "
                        "three output-layer products, without epilogues, for comparison with the library's kernels")
    p.add_argument("--kernel", default=None, help="roofline kernel label for --summarize-pmc")
    p.add_argument("--pmc-command", default="", help="command line recorded with --summarize-pmc")
    return p.parse_args()


# ---------------------------------------------------------------- HBM traffic from PMC counters
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")
CAL_FLOATS = 1 << 28                                 # reference kernel: 1 GiB read + 1 GiB written


def pmc_calibration():
    """Elementwise negation of 2^28 floats, three launches: it moves exactly
    the bytes of a copy, so its counter readings scale the others."""
    import torch
    a = torch.ones(CAL_FLOATS, device="cuda:0")
    b = torch.empty_like(a)
    for _ in range(3):
        torch.neg(a, out=b)
    torch.cuda.synchronize()
    del a, b
    torch.cuda.empty_cache()


SMALL_STEP_BYTES = 1 << 20


def one_stream(args, w) -> bool:
    """Whether the reservoir work runs on the train step's stream."""
    return args.one_stream or w.batch * w.widths[-1] * 4 < SMALL_STEP_BYTES


def stream_mode(args, w) -> str:
    if args.one_stream:
        return "one stream"
    if one_stream(args, w):
        return "one stream (a batch's targets are under 1 MiB: latency-bound step)"
    return "overlapped with the train step"


def kernel_sources(label: str):
    csrc = os.path.join(ROOT, "paper_2309_16743_amd", "csrc")
    files = ["common.h"]
    if label.startswith("gemm_fp32"):
        files += ["adam.h", "gemm_f32.h", "surrogate.hip"]
    elif label.startswith("gemm_bf16"):
        files += ["adam.h", "gemm_bf16.h", "surrogate.hip"]
    elif label == "adam_kernel":
        files += ["adam.h", "surrogate.hip"]
    else:
        files += ["reservoir.hip", "philox.h"]
    return [os.path.join(csrc, f) for f in files]


def sources_hash(label: str) -> str:
    import hashlib
    h = hashlib.sha256()
    for f in kernel_sources(label):
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def kernel_matches(label: str, name: str) -> bool:
    """Whether a rocprofv3 kernel name is the kernel behind a roofline label."""
    if label in ("adam_kernel", "gather_kernel", "gather_x_kernel", "put_copy_kernel"):
        return f"ot::{label}(" in name
    phase = label.split("(")[1].rstrip(")")
    if phase == "wgrad_output + fused Adam":       # bf16 weight gradient with the Adam epilogue
        return "gemm_bf16_pipe_kernel<" in name and "(ot::LayB)1, (ot::LayB)1, (ot::EpiB)6" in name
    if label.startswith("gemm_fp32"):
        lay = {"fwd_output": "(ot::Lay)0, (ot::Lay)0", "wgrad_output": "(ot::Lay)1, (ot::Lay)1",
               "igrad_output": "(ot::Lay)0, (ot::Lay)1"}[phase]
        return "gemm_f32_kernel<" in name and lay in name and name.split(">(")[0].endswith(", 1")
    lay = {"fwd_output": "(ot::LayB)0, (ot::LayB)0", "wgrad_output": "(ot::LayB)1, (ot::LayB)1",
           "igrad_output": "(ot::LayB)0, (ot::LayB)1"}[phase]
    return ("gemm_bf16_pipe_kernel<" in name or "gemm_bf16_pp_kernel<" in name) and lay in name


def traffic_for(workload: str, label: str):
    """Recorded HBM bytes per launch, or None if absent or the kernel's sources changed since."""
    try:
        with open(TRAFFIC_FILE) as f:
            db = json.load(f)
    except (OSError, ValueError):
        return None
    e = db.get(f"{workload} / {label}")
    if not e or e.get("sources_sha256") != sources_hash(label):
        return None
    return e["bytes_per_launch"]


def summarize_pmc(fetch_dir: str, write_dir: str, workload: str, label: str, command: str) -> dict:
    import csv
    import glob

    def rows(d, counter):
        files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
        if not files:
            raise SystemExit(f"no counter_collection.csv under {d}")
        out = []
        for fn in files:
            with open(fn) as f:
                for r in csv.DictReader(f):
                    if r["Counter_Name"] == counter:
                        out.append((r["Kernel_Name"], float(r["Counter_Value"])))
        return out

    def per_dispatch_kb(rs, pred):
        v = [x for n, x in rs if pred(n)]
        if not v:
            raise SystemExit("no matching dispatches")
        return float(np.median(v)), len(v)

    fr, wr = rows(fetch_dir, "FETCH_SIZE"), rows(write_dir, "WRITE_SIZE")
    cal = lambda n: "neg_kernel" in n
    cal_f, n_cf = per_dispatch_kb(fr, cal)
    cal_w, n_cw = per_dispatch_kb(wr, cal)
    cal_bytes = CAL_FLOATS * 4
    sf, sw = cal_bytes / (cal_f * 1024), cal_bytes / (cal_w * 1024)
    k_f, n_f = per_dispatch_kb(fr, lambda n: kernel_matches(label, n))
    k_w, n_w = per_dispatch_kb(wr, lambda n: kernel_matches(label, n))
    entry = {"workload": workload, "kernel": label,
             "fetch_kib_per_launch": round(k_f, 1), "write_kib_per_launch": round(k_w, 1),
             "launches": [n_f, n_w],
             "calibration": {"kernel": "elementwise negation of 2^28 fp32 (1 GiB read, 1 GiB written)",
                             "fetch_kib": round(cal_f, 1), "write_kib": round(cal_w, 1),
                             "fetch_scale": round(sf, 4), "write_scale": round(sw, 4)},
             "bytes_per_launch": round(k_f * 1024 * sf + k_w * 1024 * sw),
             "sources_sha256": sources_hash(label), "command": command}
    try:
        with open(TRAFFIC_FILE) as f:
            db = json.load(f)
    except (OSError, ValueError):
        db = {}
    db[f"{workload} / {label}"] = entry
    with open(TRAFFIC_FILE, "w") as f:
        json.dump(db, f, indent=1, sort_keys=True)
        f.write("\n")
    return entry


def gemm_flops(w) -> float:
    """Algorithmic flops of one output-layer GEMM launch: 2 B H D."""
    return 2.0 * w.batch * w.widths[-2] * w.widths[-1]


def out_weights(w) -> int:
    """Weights of the output layer (H x D), whose Adam update is fused into the
    weight-gradient GEMM (bf16) or its split-K reduction (fp32)."""
    return w.widths[-2] * w.widths[-1]


def adam_bytes(w) -> float:
    """Algorithmic bytes of the standalone Adam launch over every parameter
    except the output-layer weights: read p, g, m, v; write p, m, v (+ the
    bf16 weight copy in mixed precision)."""
    return (28.0 + (2.0 if w.precision == "bf16" else 0.0)) * (w.n_params() - out_weights(w))


def fused_adam_bytes(w) -> float:
    """Algorithmic bytes of the output layer's fused weight update: read p, m,
    v and write p, m, v (+ the bf16 copy) of its H x D weights, and read its
    operands dY (B x D) and A (B x H) once."""
    e = 2.0 if w.precision == "bf16" else 4.0
    per = 24.0 + (2.0 if w.precision == "bf16" else 0.0)
    return per * out_weights(w) + e * w.batch * (w.widths[-1] + w.widths[-2])


GATHERED_TARGETS = False         # --gathered-targets


def gather_bytes(w, targets: Optional[bool] = None) -> float:
    """Bytes the batch gather moves (read from the slab, written to the batch
    buffer): the input rows, plus the field rows when the targets are gathered
    too (--gathered-targets); otherwise the forward reads them in place."""
    targets = GATHERED_TARGETS if targets is None else targets
    return 2.0 * w.batch * ((w.widths[-1] if targets else 0) + w.widths[0]) * 4


def put_bytes(w) -> float:
    return 2.0 * w.wave * (w.widths[-1] + w.widths[0]) * 4


def kernel_table(w, phases_ms: dict, res_ms: dict) -> dict:
    """Average duration and algorithmic rate of each timed phase."""
    peak_mfma = PEAK_BF16_MFMA if w.precision == "bf16" else PEAK_FP32_MFMA
    out = {}
    for name, (ms, n) in phases_ms.items():
        avg = ms / max(n, 1)
        row = {"avg_us": round(avg * 1e3, 2), "launches": n}
        if name in ("fwd_output", "wgrad_output", "igrad_output"):
            rate = gemm_flops(w) / (avg * 1e-3)
            row.update(achieved_tflops=round(rate / 1e12, 2), frac_mfma=round(rate / peak_mfma, 4))
        if (name == "wgrad_output" and w.precision == "bf16") or (name == "wgrad_reduce" and w.precision == "fp32"):
            rate = fused_adam_bytes(w) / (avg * 1e-3)     # the phase that applies the fused Adam update
            row.update(fused_adam=True, achieved_gbs=round(rate / 1e9, 1), frac_hbm=round(rate / PEAK_HBM, 4))
        if name == "adam":
            rate = adam_bytes(w) / (avg * 1e-3)
            row.update(achieved_gbs=round(rate / 1e9, 1), frac_hbm=round(rate / PEAK_HBM, 4))
        out[name] = row
    for name, (ms, n) in res_ms.items():
        avg = ms / max(n, 1)
        row = {"avg_us": round(avg * 1e3, 2), "launches": n}
        byts = {"gather": gather_bytes(w), "put_copy": put_bytes(w)}.get(name)
        if byts:
            rate = byts / (avg * 1e-3)
            row.update(achieved_gbs=round(rate / 1e9, 1), frac_hbm=round(rate / PEAK_HBM, 4))
        out["reservoir_" + name] = row
    return out


def roofline_entry(w, phase: str, avg_s: float) -> dict:
    """Roofline object for the dominant kernel (per-launch algorithmic work / duration).
    traffic: HBM bytes per launch from rocprofv3 counters (profiles/hbm_traffic.json),
    None when not measured for this kernel as it now stands."""
    if phase == "wgrad_output" and w.precision == "bf16":
        # weight gradient with Adam in its epilogue: 26 B per output weight against 2 B H D flop
        work = fused_adam_bytes(w)
        label = "gemm_bf16 (wgrad_output + fused Adam)"
        return {"bound": "hbm", "kernel": label,
                "achieved": round(work / avg_s / 1e9, 1), "peak": PEAK_HBM / 1e9, "unit": "GB/s",
                "frac": round(work / avg_s / PEAK_HBM, 4), "traffic": traffic_for(w.name, label),
                "per_launch_bytes": work, "per_launch_flops": gemm_flops(w),
                "mfma_frac": round(gemm_flops(w) / avg_s / PEAK_BF16_MFMA, 4), "avg_us": round(avg_s * 1e6, 2)}
    if phase in ("fwd_output", "wgrad_output", "igrad_output"):
        peak = PEAK_BF16_MFMA if w.precision == "bf16" else PEAK_FP32_MFMA
        work = gemm_flops(w)
        label = f"gemm_{w.precision} ({phase})"
        return {"bound": "mfma", "kernel": label,
                "achieved": round(work / avg_s / 1e12, 2), "peak": peak / 1e12, "unit": "TFLOP/s",
                "frac": round(work / avg_s / peak, 4), "traffic": traffic_for(w.name, label),
                "per_launch_flops": work, "avg_us": round(avg_s * 1e6, 2)}
    work = {"adam": adam_bytes(w), "gather": gather_bytes(w)}[phase]
    label = "adam_kernel" if phase == "adam" else ("gather_kernel" if GATHERED_TARGETS else "gather_x_kernel")
    return {"bound": "hbm", "kernel": label,
            "achieved": round(work / avg_s / 1e9, 1), "peak": PEAK_HBM / 1e9, "unit": "GB/s",
            "frac": round(work / avg_s / PEAK_HBM, 4), "traffic": traffic_for(w.name, label),
            "per_launch_bytes": work, "avg_us": round(avg_s * 1e6, 2)}


def achievable_rates(precision: str) -> dict:
    """Rates this GPU reaches outside the library, measured live for context:
    a device-to-device copy of 1 GiB (read + write) and torch's GEMM on
    8192 x 8192 x 8192 in the workload's precision."""
    import torch
    dev = torch.device("cuda:0")

    def avg_ms(fn, it):
        fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(it):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / it

    a = torch.empty(CAL_FLOATS, device=dev)
    b = torch.empty_like(a)
    a.fill_(1.0)
    copy_gbs = 2 * CAL_FLOATS * 4 / (avg_ms(lambda: b.copy_(a), 5) * 1e-3) / 1e9
    del a, b
    dt = torch.float32 if precision == "fp32" else torch.bfloat16
    torch.backends.cuda.matmul.allow_tf32 = False
    x = torch.ones(8192, 8192, device=dev, dtype=dt)
    ms = avg_ms(lambda: torch.matmul(x, x), 3 if precision == "fp32" else 10)
    del x
    torch.cuda.empty_cache()
    return {"hbm_copy_gbs": round(copy_gbs, 1), "gemm_tflops": round(2 * 8192 ** 3 / (ms * 1e-3) / 1e12, 1),
            "gemm": f"torch.matmul 8192^3 {'fp32' if precision == 'fp32' else 'bf16'}"}


def with_achievable(roof: dict, ach: dict) -> dict:
    """Adds the fraction of the live-measured achievable rate of the same unit."""
    ref = ach["hbm_copy_gbs"] if roof["unit"] == "GB/s" else ach["gemm_tflops"]
    out = dict(roof)
    out["frac_achievable"] = round(roof["achieved"] / ref, 4)
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


def _blas_threads() -> int:
    try:
        import threadpoolctl
        return max((b.get("num_threads", 1) for b in threadpoolctl.threadpool_info()), default=1)
    except Exception:  # pragma: no cover
        return 1


def linear_extrapolation(d1: float, t1: float, d2: float, t2: float, d: float):
    """(a, b, t(d)) of the line t = a + b d through (d1, t1) and (d2, t2)."""
    b = (t2 - t1) / (d2 - d1)
    a = t1 - b * d1
    return a, b, a + b * d


def cpu_baseline_field(w, seconds: float) -> dict:
    """The fp64 oracle's whole step at a 1000x1000 workload on this host.

    Train step (bf16-rounding fp64 oracle): the hidden layers at full width,
    the output layer at two slices of D (D/400 and D/200 outputs); a step's
    time is a + b d in the output width d (every output-layer cost -- its
    GEMMs, roundings and Adam -- is linear in d, the hidden layers are the
    constant a), so the two timings give the full-width step without scaling
    the hidden layers.  Reservoir (oracle put of one chunk + draw of a batch
    with its gather) at the full row length on a host reservoir of B + 2 x
    chunk rows (the per-step work does not depend on the capacity)."""
    from fixtures import synthetic
    from oracle import mlp
    from oracle.reservoir import OK, Reservoir
    blas_threads = _blas_threads()
    rng = np.random.default_rng(0)
    X = np.concatenate([rng.uniform(100, 500, (w.batch, 5)), rng.uniform(0.01, 1.0, (w.batch, 1))], axis=1)
    D = w.widths[-1]
    timings = []
    budget = seconds / 3
    for f in (400, 200):
        d = D // f
        widths = list(w.widths[:-1]) + [d]
        params = mlp.init_params(widths, w.init_seed)
        U = rng.uniform(100, 500, (w.batch, d))
        opt = mlp.Adam(lr=w.lr)
        loss, grads = mlp.loss_and_grads(params, X, U, bf16=True)        # untimed first step
        params = opt.step(params, grads)
        steps = 0
        t0 = time.perf_counter()
        while steps < 1 or time.perf_counter() - t0 < budget:
            loss, grads = mlp.loss_and_grads(params, X, U, bf16=True)
            params = opt.step(params, grads)
            steps += 1
        timings.append((d, (time.perf_counter() - t0) / steps, steps))
        del params, grads, opt, U
    (d1, t1, n1), (d2, t2, n2) = timings
    a, b, t_train = linear_extrapolation(d1, t1, d2, t2, D)
    # reservoir ops at the full row length: a draw (with its gather) on a
    # reservoir filled with unseen samples, then a put that replaces seen ones
    C = w.batch + 2 * w.wave
    res = Reservoir(C, w.batch, w.widths[0], D, w.reservoir_seed)
    keys = np.arange(w.wave)
    px = np.concatenate([rng.uniform(100, 500, (w.wave, 5)), np.full((w.wave, 1), 0.5)], axis=1).astype(np.float32)
    pu = synthetic.hash_rows(keys, D).astype(np.float32)
    while res.N < C:                                   # fill (untimed)
        res.put(px, pu)
    steps = 0
    t0 = time.perf_counter()
    while steps < 1 or time.perf_counter() - t0 < budget:
        st, slots, xb, ub, _ = res.sample_batch(w.batch)
        assert st == OK
        del xb, ub
        _, acc, _, _ = res.put(px, pu)
        assert acc == w.wave
        steps += 1
    t_res = (time.perf_counter() - t0) / steps
    del res
    t_step = t_train + t_res
    return {"value": round(w.batch / t_step, 3), "unit": "samples/s", "cores": blas_threads, "kind": "oracle",
            "sample": f"fp64 oracle (bf16 rounding points) train steps of {'-'.join(map(str, w.widths[:-1]))} with "
                      f"output slices of {d1} ({n1} steps, {t1:.3f} s each) and {d2} ({n2} steps, {t2:.3f} s) "
                      f"outputs, the step time extrapolated linearly in the output width to {D} "
                      f"(hidden layers {a:.3f} s + {b * 1e6:.3f} us per output unit); plus {steps} oracle "
                      f"iterations of draw {w.batch} with gather + put {w.wave} rows of {D} floats on a host "
                      f"reservoir of {C} rows ({t_res:.3f} s each); numpy BLAS threads {blas_threads}, "
                      f"{len(os.sched_getaffinity(0))} host cores visible; reservoir copies one thread",
            "ms_per_step": round(t_step * 1e3, 1), "train_ms": round(t_train * 1e3, 1),
            "reservoir_ms": round(t_res * 1e3, 1)}


def timed_region(tr, w, K, profile_steps, stream, wrap_put):
    """Breakdown pass (all phases), then K timed steps with events on the
    dominant kernel, then eager steps that time the other output-layer GEMMs,
    the put copies and the gather."""
    import torch

    from paper_2309_16743_amd._abi import SURROGATE_PHASES
    kp = max(profile_steps, 1)
    tr.sur.timing_begin(list(SURROGATE_PHASES), kp)
    tr.res.timing_begin(["put_assign", "put_copy", "select", "gather"], 2 * kp)
    tr.serialize = True             # breakdown with the reservoir and train step one after the other
    graph = getattr(tr, "graph", False)
    tr.graph_active = False          # phase events come from eager launches (a replayed step records none)
    for _ in range(kp):
        wrap_put()
        assert tr.sample_and_train()
    breakdown = kernel_table(w, tr.sur.timing_end(), tr.res.timing_end())
    tr.serialize = False
    tr.graph_active = graph
    candidates = ("fwd_output", "wgrad_output", "igrad_output", "adam", "reservoir_gather")
    dominant = max((c for c in candidates if c in breakdown), key=lambda p: breakdown[p]["avg_us"])
    dom_phase = "gather" if dominant == "reservoir_gather" else dominant

    # timed region: HIP events on the launches of the dominant kernel only
    # (each event pair on a launch costs host time and a few microseconds of
    # GPU time between kernels, which would show in a short step); the other
    # output-layer GEMMs, the put copies and the gather are timed on eager
    # steps right after the timed region.  A train step replayed as a graph
    # records no phase events, so then the dominant kernel is timed there too.
    out_phases = [p for p in ("fwd_output", "wgrad_output", "igrad_output") if p in breakdown]
    sur_phases = [p for p in SURROGATE_PHASES if p in out_phases or p == dom_phase]
    live = not graph
    if live:
        if dom_phase == "gather":
            tr.res.timing_begin(["gather"], 2 * K)
        else:
            tr.sur.timing_begin([dom_phase], K)
    n_win = K // 10
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(n_win + 2)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev[0].record(stream)
    if tr.overlap:
        tr.res_stream.wait_event(ev[0])     # reservoir work of the timed steps starts after the first event
    for i in range(K):
        wrap_put()
        assert tr.sample_and_train()
        if (i + 1) % 10 == 0 and (i + 1) // 10 <= n_win:
            ev[(i + 1) // 10].record(stream)
    ev[-1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = ev[0].elapsed_time(ev[-1])
    windows = [ev[j].elapsed_time(ev[j + 1]) for j in range(n_win)]
    live_t = {}
    if live:
        live_t = tr.res.timing_end() if dom_phase == "gather" else tr.sur.timing_end()
    kt = min(K, 200)
    tr.graph_active = False
    post_sur = [p for p in sur_phases if not (live and p == dom_phase)]
    if post_sur:
        tr.sur.timing_begin(post_sur, kt)
    tr.res.timing_begin(["put_copy", "gather"], 2 * kt)
    for _ in range(kt):
        wrap_put()
        assert tr.sample_and_train()
    sur_t = tr.sur.timing_end() if post_sur else {}
    res_t = tr.res.timing_end()
    tr.graph_active = graph
    if live and dom_phase == "gather":
        res_t["gather"] = live_t["gather"]
    elif live:
        sur_t[dom_phase] = live_t[dom_phase]
    g_ms, g_n = res_t["gather"]
    phase_avg_s = {p: sur_t[p][0] / sur_t[p][1] * 1e-3 for p in sur_phases if p in sur_t}
    put_avg_s = res_t["put_copy"][0] / res_t["put_copy"][1] * 1e-3 if "put_copy" in res_t else None
    dom_avg_s = g_ms / g_n * 1e-3 if dom_phase == "gather" else phase_avg_s[dom_phase]
    achievable = achievable_rates(w.precision)      # after the timed region, which it does not disturb
    return dict(gpu_ms=gpu_ms, wall=wall, windows=windows, breakdown=breakdown, dom_phase=dom_phase,
                achievable=achievable, dom_avg_s=dom_avg_s, gather_avg_s=g_ms / g_n * 1e-3,
                phase_avg_s=phase_avg_s, put_avg_s=put_avg_s, loss=float(tr.loss.item()))


def steps_rate(tr, w, K, stream, wrap_put) -> dict:
    """Samples/s of K more steps, HIP events on the work stream."""
    import torch
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    e0.record(stream)
    if tr.overlap:
        tr.res_stream.wait_event(e0)
    for _ in range(K):
        wrap_put()
        assert tr.sample_and_train()
    e1.record(stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1)
    return {"value": round(w.batch * K / (ms * 1e-3), 1), "unit": "samples/s", "steps": K,
            "ms_per_step": round(ms / K, 4)}


def output_layer_entry(w, phase_avg_s: dict) -> dict:
    """Rates of the output layer's three GEMMs (the dominant one measured in
    the timed region, the others on the eager steps that follow it):
    forward (+ fused MSE) and input gradient against the MFMA peak of their
    precision; the weight gradient too, and in bf16, where it applies Adam to
    the output weights in its epilogue, also against HBM."""
    peak = PEAK_BF16_MFMA if w.precision == "bf16" else PEAK_FP32_MFMA
    out = {}
    for p in ("fwd_output", "igrad_output", "wgrad_output"):
        if p not in phase_avg_s:
            continue
        t = phase_avg_s[p]
        e = {"avg_us": round(t * 1e6, 2), "tflops": round(gemm_flops(w) / t / 1e12, 1),
             "frac_mfma": round(gemm_flops(w) / t / peak, 4)}
        if p == "wgrad_output" and w.precision == "bf16":
            e.update(fused_adam=True, achieved_gbs=round(fused_adam_bytes(w) / t / 1e9, 1),
                     frac_hbm=round(fused_adam_bytes(w) / t / PEAK_HBM, 4))
        out[p] = e
    out["peak_tflops"] = peak / 1e12
    return out


def reservoir_entry(w, r) -> dict:
    """Put copies (whole rows into the slab: the reservoir's bandwidth at this
    shape) and the batch gather, timed on the eager steps that follow the
    timed region (in it when the gather is the dominant kernel)."""
    g_rate = gather_bytes(w) / r["gather_avg_s"]
    out = {"gather": {"achieved": round(g_rate / 1e9, 1), "unit": "GB/s", "frac_hbm": round(g_rate / PEAK_HBM, 4),
                      "avg_us": round(r["gather_avg_s"] * 1e6, 2), "bytes_per_launch": gather_bytes(w),
                      "rows": "input rows only (the targets are read in place by the forward)"
                      if not GATHERED_TARGETS else "input and field rows"}}
    if r.get("put_avg_s"):
        p_rate = put_bytes(w) / r["put_avg_s"]
        out["put_copy"] = {"achieved": round(p_rate / 1e9, 1), "unit": "GB/s", "frac_hbm": round(p_rate / PEAK_HBM, 4),
                           "avg_us": round(r["put_avg_s"] * 1e6, 2), "bytes_per_launch": put_bytes(w),
                           "rows": f"{w.wave} whole rows read from the producer and written to the slab"}
    return out


def result_line(w, args, K, warmup, r, config: dict) -> dict:
    value = w.batch * K / (r["gpu_ms"] * 1e-3)
    win_sps = [10 * w.batch / (t * 1e-3) for t in r["windows"]] if r["windows"] else [value]
    return {
        "metric": METRIC, "value": round(value, 1), "unit": "samples/s", "n_gpus": 1, "steps": K,
        "warmup": warmup, "ms_per_step": round(r["gpu_ms"] / K, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32" if w.precision == "fp32" else "bf16",
        "data": "synthetic", "config": config,
        "roofline": with_achievable(roofline_entry(w, r["dom_phase"], r["dom_avg_s"]), r["achievable"]),
        "achievable": r["achievable"],
        "output_layer": output_layer_entry(w, r["phase_avg_s"]),
        "reservoir": reservoir_entry(w, r),
        "windows_of_10": {"median_samples_s": round(float(np.median(win_sps)), 1),
                          "mean_samples_s": round(float(np.mean(win_sps)), 1), "n": len(win_sps)},
        "wall_s": round(r["wall"], 3), "last_loss": r["loss"], "kernels": r["breakdown"], "cpu_baseline": None,
    }


def instrumentation(tr, w, stream) -> dict:
    """Training instrumentation of Sec. 3.1 and 4.3-4.4, measured after the
    timed region: one validation pass (surrogate_eval_loss) over 10 held-out
    simulations (the paper's validation set size), timed with events on the
    training stream; the repetition histogram of the run so far; and one
    synchronous checkpoint of reservoir and surrogate to host memory."""
    import torch

    from fixtures import heat
    Xv = heat.sample_parameters(10, w.data_seed + 1000)
    iv = torch.from_numpy(heat.inputs_for(Xv, w.tau).reshape(-1, w.widths[0])).to(tr.xb.device)
    fv = torch.from_numpy(heat.heat_fields(Xv, w.grid, w.tau).reshape(-1, w.widths[-1])).to(tr.xb.device)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    tr.validate(iv, fv)                        # warm
    e0.record(stream)
    val = tr.validate(iv, fv)
    e1.record(stream)
    torch.cuda.synchronize()
    h = tr.repetition_histogram()
    last = int(np.max(np.nonzero(h)[0])) if h.any() else 0
    t0 = time.perf_counter()
    ck = tr.checkpoint()                       # synchronous snapshot to host memory
    t_ck = time.perf_counter() - t0
    ck_bytes = sum(int(v.nbytes) for v in ck.values())
    del ck
    return {"validation": {"rows": int(iv.shape[0]), "ms": round(e0.elapsed_time(e1), 3),
                           "loss": round(float(val.item()), 4)},
            "checkpoint": {"bytes": ck_bytes, "s": round(t_ck, 3), "gb_per_s": round(ck_bytes / t_ck / 1e9, 2)},
            "repetition_histogram": {"draws_per_sample": h[:last + 1].tolist(),
                                     "last_bin_is_tail": last == len(h) - 1}}


def run_heat(args, w):
    import torch

    from fixtures import heat
    from paper_2309_16743_amd.online import OnlineTrainer
    K = args.steps or 2000
    warmup = 50 if args.warmup is None else args.warmup
    t_gen = time.perf_counter()
    X = heat.sample_parameters(w.n_sims, w.data_seed)
    inputs = heat.inputs_for(X, w.tau)
    fields = heat.heat_fields(X, w.grid, w.tau)
    print(f"[bench] generated {fields.nbytes / 1e9:.1f} GB of {w.grid}x{w.grid} fields in "
          f"{time.perf_counter() - t_gen:.1f} s", file=sys.stderr, flush=True)
    dev = torch.device("cuda:0")
    inputs_d = torch.from_numpy(inputs).to(dev)
    fields_d = torch.from_numpy(fields).to(dev)
    stream = torch.cuda.Stream(device=dev)
    with torch.cuda.stream(stream):
        graph = one_stream(args, w) and not args.gathered_targets and not args.no_graph
        tr = OnlineTrainer(w.widths, w.batch, w.capacity, w.threshold, w.wave, w.tau, inputs_d, fields_d,
                           w.reservoir_seed, w.init_seed, lr=w.lr, stream=stream, overlap=not one_stream(args, w),
                           fused_targets=not args.gathered_targets, graph=graph)
        for _ in range(w.n_chunks):             # stream the ensemble once (untimed)
            tr.iterate()
        for _ in range(warmup):
            assert tr.iterate(wrap=True)
        torch.cuda.synchronize()
        print(f"[bench] setup done: {tr.steps_done} train steps, reservoir {tr.res.stats()['n']} samples",
              file=sys.stderr, flush=True)
        r = timed_region(tr, w, K, args.profile_steps or 200, stream, (lambda: None) if args.prefilled else (lambda: tr.put_next(wrap=True)))
        instr = instrumentation(tr, w, stream)
    config = {"workload": w.name, "fields": f"FTCS heat {w.grid}x{w.grid}, {w.n_sims} sims x {w.tau} steps",
              "widths": list(w.widths), "batch": w.batch, "capacity": w.capacity, "threshold": w.threshold,
              "put_rows_per_step": w.wave, "precision": w.precision,
              "reservoir_stream": stream_mode(args, w),
              "targets": "gathered into a batch buffer" if args.gathered_targets
              else "read in place from the reservoir by the forward (inputs gathered)",
              "timed_puts": "none (pre-filled reservoir)" if args.prefilled else "one per step",
              "train_step": ("captured once as a HIP graph and replayed (Adam's step counter in device memory; "
                             "the reservoir's calls eager); its kernels and the reservoir's copies timed on eager "
                             "steps after the timed region")
              if graph else "kernels launched per step"}
    line = result_line(w, args, K, warmup, r, config)
    line["instrumentation"] = instr
    tr.close()
    del inputs_d, fields_d
    torch.cuda.empty_cache()
    if args.cpu_seconds > 0:
        line["cpu_baseline"] = cpu_baseline(w, inputs, fields, args.cpu_seconds)
    return line


def run_policy_comparison(args, w):
    """The paper's buffer comparison (Sec. 4.3, Fig. 2 / Table 1) on this
    workload's production schedule: the whole ensemble is streamed once through
    each buffer (one put of the wave's rows per iteration, then a train step
    whenever the buffer yields a batch), then reception ends and the buffer is
    drained.  Reports per policy the train steps, trained samples, GPU time and
    trained samples/s; the Reservoir repeats samples, so it trains more batches
    from the same production."""
    import torch

    from fixtures import heat
    from paper_2309_16743_amd import OT_POLICY_FIFO, OT_POLICY_FIRO, OT_POLICY_RESERVOIR
    from paper_2309_16743_amd.online import OnlineTrainer
    X = heat.sample_parameters(w.n_sims, w.data_seed)
    inputs = heat.inputs_for(X, w.tau)
    fields = heat.heat_fields(X, w.grid, w.tau)
    dev = torch.device("cuda:0")
    inputs_d = torch.from_numpy(inputs).to(dev)
    fields_d = torch.from_numpy(fields).to(dev)
    stream = torch.cuda.Stream(device=dev)
    out = {}
    for name, policy in (("reservoir", OT_POLICY_RESERVOIR), ("firo", OT_POLICY_FIRO), ("fifo", OT_POLICY_FIFO)):
        with torch.cuda.stream(stream):
            tr = OnlineTrainer(w.widths, w.batch, w.capacity, w.threshold, w.wave, w.tau, inputs_d, fields_d,
                               w.reservoir_seed, w.init_seed, lr=w.lr, stream=stream, policy=policy)
            e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
            torch.cuda.synchronize()
            e0.record(stream)
            steps_stream = 0
            for _ in range(w.n_chunks):
                steps_stream += int(tr.iterate())
            e1.record(stream)
            tr.res.end_reception()
            steps_drain = 0
            while tr.sample_and_train():
                steps_drain += 1
            e2.record(stream)
            torch.cuda.synchronize()
            st = tr.res.stats()
            steps = steps_stream + steps_drain
            ms = e0.elapsed_time(e2)
            out[name] = {"train_steps": steps, "steps_while_streaming": steps_stream, "steps_draining": steps_drain,
                         "trained_samples": st["total_draws"], "produced_samples": st["total_put"],
                         "batches_per_1000_produced": round(1000.0 * steps / max(st["total_put"], 1), 2),
                         "gpu_ms": round(ms, 2), "streaming_ms": round(e0.elapsed_time(e1), 2),
                         "samples_per_s": round(st["total_draws"] / (ms * 1e-3), 1),
                         "last_loss": float(tr.loss.item())}
            tr.close()
    return {"metric": "buffer comparison: trained samples per produced sample and samples/s (Sec. 4.3)",
            "workload": w.name, "production": f"{w.n_chunks} puts of {w.wave} rows (the ensemble once), "
                                              f"then end of reception and drain",
            "batch": w.batch, "capacity": w.capacity, "threshold": w.threshold, "policies": out}


def run_field(args, w):
    import torch

    from fixtures import heat, synthetic
    from paper_2309_16743_amd import OT_BF16
    from paper_2309_16743_amd.online import OnlineTrainer
    K = args.steps or 100
    warmup = 5 if args.warmup is None else args.warmup
    dev = torch.device("cuda:0")
    n, D = w.grid, w.widths[-1]
    X = torch.from_numpy(heat.sample_parameters(w.n_sims, w.data_seed)).to(dev)
    basis = synthetic.sine_mode_basis_torch(n, w.data_seed, dev)
    stream = torch.cuda.Stream(device=dev)

    def gen_chunk(c, xbuf, ubuf):
        wv, k = divmod(c % w.n_chunks, w.tau)
        sims = X[wv * w.wave:(wv + 1) * w.wave]
        t = torch.full((w.wave,), 0.01 * (k + 1), device=dev, dtype=torch.float64)
        synthetic.sine_mode_fields_torch(sims, t, w.data_seed, basis, out=ubuf)
        xbuf[:, :5] = sims.to(torch.float32)
        xbuf[:, 5] = t.to(torch.float32)

    P = max(1, args.producers)
    producers = [torch.cuda.Stream(device=dev) for _ in range(P)]    # default priority, like every stream here
    with torch.cuda.stream(stream):
        pool = max(P, 8)                        # pre-generated chunks the timed puts cycle through
        pool_x = [torch.empty(w.wave, 8, device=dev)[:, :6] for _ in range(pool)]
        pool_u = [torch.empty(w.wave, D, device=dev) for _ in range(pool)]
        first_pool_chunk = w.n_chunks // 2
        for i in range(pool):
            gen_chunk(first_pool_chunk + i, pool_x[i], pool_u[i])
        tr = OnlineTrainer(w.widths, w.batch, w.capacity, w.threshold, w.wave, w.tau, None, None,
                           w.reservoir_seed, w.init_seed, precision=OT_BF16, lr=w.lr, stream=stream,
                           chunk_fn=lambda c: (pool_x[c % pool], pool_u[c % pool]), n_chunks=1 << 40, device=dev,
                           overlap=not one_stream(args, w), fused_targets=not args.gathered_targets,
                           put_streams=producers)
        fx = torch.empty(w.wave, 8, device=dev)[:, :6]
        fu = torch.empty(w.wave, D, device=dev)
        t_fill = time.perf_counter()
        n_stored, c = 0, 0
        while n_stored < w.capacity:            # fill with generated chunks (untimed), drawing once past T
            gen_chunk(c, fx, fu)
            tr.res.put(fx, fu, stream=stream)
            n_stored = min(w.capacity, n_stored + w.wave)
            c += 1
            if n_stored > w.threshold:
                tr.sample_only()
        for _ in range(warmup):
            tr.put_next(wrap=True)
            assert tr.sample_and_train()
        torch.cuda.synchronize()
        print(f"[bench] filled {n_stored} samples ({n_stored * D * 4 / 1e9:.0f} GB) in "
              f"{time.perf_counter() - t_fill:.1f} s; {tr.steps_done} warm-up steps",
              file=sys.stderr, flush=True)
        put = (lambda: None) if args.prefilled else (lambda: tr.put_next(wrap=True))
        r = timed_region(tr, w, K, args.profile_steps or 20, stream, put)
        # the other mode, same steps: production suspended (mode A) or running (mode B)
        other = steps_rate(tr, w, K, stream, (lambda: tr.put_next(wrap=True)) if args.prefilled else (lambda: None))
    mode_b = f"{P} producer streams, one put of {w.wave} samples per step in turn, concurrent with training"
    mode_a = "production suspended: draws and train steps on the filled reservoir"
    config = {"workload": w.name, "fields": f"sine-mode {n}x{n}, {w.n_sims} sims x {w.tau} steps",
              "widths": list(w.widths), "batch": w.batch, "capacity": w.capacity, "threshold": w.threshold,
              "put_rows_per_step": 0 if args.prefilled else w.wave, "precision": w.precision,
              "reservoir_stream": stream_mode(args, w),
              "targets": "gathered into a batch buffer" if args.gathered_targets
              else "read in place from the reservoir by the forward (inputs gathered)",
              "timed_puts": ("mode A: " + mode_a) if args.prefilled else ("mode B: " + mode_b)}
    line = result_line(w, args, K, warmup, r, config)
    other.update(mode=("B: " + mode_b) if args.prefilled else ("A: " + mode_a))
    line["other_mode"] = other
    tr.close()
    torch.cuda.empty_cache()
    if args.cpu_seconds > 0:
        line["cpu_baseline"] = cpu_baseline_field(w, args.cpu_seconds)
    return line


def cpu_baseline_stress(w, seconds: float) -> dict:
    """The oracle reservoir (put + draw + gather of 100,000-float rows) on this
    host at a reduced capacity of 5,000 rows (2 GB slab), timed in steady state."""
    from fixtures import synthetic
    from oracle.reservoir import OK, Reservoir
    C, T, D, k, B = 5000, 1000, w.row_len, w.chunk, w.batch
    res = Reservoir(C, T, 6, D, w.reservoir_seed)
    pool = [(synthetic.hash_inputs(np.arange(i * k, (i + 1) * k)), synthetic.hash_rows(np.arange(i * k, (i + 1) * k), D))
            for i in range(2)]
    i = 0
    while res.N < C:                                 # fill (untimed), drawing once past the threshold
        res.put(*pool[i % 2])
        if res.N > T:
            res.sample_batch(B)
        i += 1
    rows_in = rows_out = steps = 0
    t0 = time.perf_counter()
    while steps < 2 or time.perf_counter() - t0 < seconds:
        _, a, _, _ = res.put(*pool[i % 2])
        st, slots, _, _, _ = res.sample_batch(B)
        assert st == OK
        rows_in += a
        rows_out += len(slots)
        i += 1
        steps += 1
    dt = time.perf_counter() - t0
    row_bytes = 2 * (D + 6) * 4
    return {"value": round((rows_in + rows_out) * row_bytes / dt / 1e9, 3), "unit": "GB/s", "cores": 1,
            "kind": "oracle",
            "sample": f"{steps} iterations of put {k} rows + draw {B} rows (with gather) on a host reservoir of "
                      f"capacity {C} (reduced from {w.capacity}; 2 GB slab) in steady state; numpy row copies, "
                      f"one thread; {rows_in} rows accepted, {rows_out} drawn"}


def run_stress(args):
    """Reservoir-only workload: 100,000-float rows, 64 producer streams, one consumer."""
    import torch

    from fixtures import configs, synthetic
    from paper_2309_16743_amd import OT_OK, Reservoir
    w = configs.STRESS
    K = args.steps or 2000
    warmup = 20 if args.warmup is None else args.warmup
    dev = torch.device("cuda:0")
    D, k, B, P = w.row_len, w.chunk, w.batch, w.producers
    order = torch.cuda.Stream(device=dev)
    cons = torch.cuda.Stream(device=dev)
    streams = [torch.cuda.Stream(device=dev) for _ in range(P)]
    res = Reservoir(w.capacity, w.threshold, 6, D, w.reservoir_seed, order_stream=order)
    xs, us = [], []
    for p, s in enumerate(streams):                  # one chunk per producer stream (hash rows; untimed)
        with torch.cuda.stream(s):
            keys = torch.arange(p * k, (p + 1) * k, device=dev, dtype=torch.int64)
            u = torch.empty(k, D, device=dev)
            synthetic.hash_rows_torch(keys, D, out=u)
            x = torch.empty(k, 8, device=dev)[:, :6]
            x.copy_(synthetic.hash_inputs_torch(keys, 6))
        xs.append(x)
        us.append(u)
    slots = torch.empty(B, dtype=torch.int32, device=dev)
    xb = torch.empty(B, 8, device=dev)[:, :6]
    ub = torch.empty(B, D, device=dev)
    torch.cuda.synchronize()
    row_bytes = 2 * (D + 6) * 4                      # read the source row + write the slab row (u and x)

    # fill: 195 whole chunks from the producer streams, every row accepted
    n_fill = w.capacity // k
    res.timing_begin(["put_copy"], n_fill)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(order)
    for i in range(n_fill):
        res.put(xs[i % P], us[i % P], stream=streams[i % P])
    e1.record(order)
    torch.cuda.synchronize()
    fill_ms = e0.elapsed_time(e1)
    fill_copy_ms, fill_copies = res.timing_end()["put_copy"]
    fill_rate = n_fill * k * row_bytes / (fill_ms * 1e-3)

    # steady state: each iteration, one producer stream puts a chunk (replacing seen rows once full)
    # and the consumer draws a batch with its gather
    def iteration(i, direct=False):
        res.put(xs[i % P], us[i % P], stream=order if direct else streams[i % P], accepted=acc[i:i + 1])
        st, _, _ = res.sample_batch(B, slots, x_out=xb, u_out=ub, stream=order if direct else cons)
        assert st == OT_OK

    def timed(first, direct, timing):
        torch.cuda.synchronize()
        s0 = res.stats()
        if timing:
            res.timing_begin(["put_copy", "gather"], 2 * K + 8)
        t_wall = time.perf_counter()
        e0.record(order)
        for i in range(first, first + K):
            iteration(i, direct)
        e1.record(order)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t_wall
        tim = res.timing_end() if timing else None
        s1 = res.stats()
        rows_in = int(acc[first:first + K].sum().item())
        assert s1["total_put"] - s0["total_put"] == rows_in and s1["total_draws"] - s0["total_draws"] == B * K
        return e0.elapsed_time(e1), wall, rows_in, tim

    acc = torch.zeros(2 * K + warmup, dtype=torch.int64, device=dev)
    for i in range(warmup):
        iteration(i)
    gpu_ms, wall, rows_in, tim = timed(warmup, False, True)
    d_ms, d_wall, d_rows_in, _ = timed(warmup + K, True, False)
    rows_out = B * K
    total_bytes = (rows_in + rows_out) * row_bytes
    value = total_bytes / (gpu_ms * 1e-3) / 1e9
    direct_rate = (d_rows_in + rows_out) * row_bytes / (d_ms * 1e-3) / 1e9
    g_ms, g_n = tim["gather"]
    c_ms, c_n = tim["put_copy"]
    assert g_n == K and c_n == K
    g_avg = g_ms * 1e-3 / g_n
    g_rate = B * row_bytes / g_avg
    put_rate = rows_in * row_bytes / (c_ms * 1e-3)
    dom = "gather" if g_ms >= c_ms else "put_copy"
    ach = achievable_rates("fp32")
    if dom == "gather":
        roof = {"bound": "hbm", "kernel": "gather_kernel", "achieved": round(g_rate / 1e9, 1), "peak": PEAK_HBM / 1e9,
                "unit": "GB/s", "frac": round(g_rate / PEAK_HBM, 4), "traffic": traffic_for(w.name, "gather_kernel"),
                "per_launch_bytes": B * row_bytes, "avg_us": round(g_avg * 1e6, 2)}
    else:
        c_avg = c_ms * 1e-3 / c_n
        roof = {"bound": "hbm", "kernel": "put_copy_kernel", "achieved": round(put_rate / 1e9, 1),
                "peak": PEAK_HBM / 1e9, "unit": "GB/s", "frac": round(put_rate / PEAK_HBM, 4),
                "traffic": traffic_for(w.name, "put_copy_kernel"),
                "per_launch_bytes": round(rows_in * row_bytes / c_n), "avg_us": round(c_avg * 1e6, 2)}
    line = {
        "metric": METRIC, "value": round(value, 1), "unit": "GB/s", "n_gpus": 1, "steps": K, "warmup": warmup,
        "ms_per_step": round(gpu_ms / K, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32", "data": "synthetic",
        "config": {"workload": w.name, "row_floats": D, "capacity": w.capacity, "threshold": w.threshold,
                   "producer_streams": P, "chunk": k, "batch": B,
                   "rows": "hash rows (value = hash of the row key, exact in fp32)"},
        "roofline": with_achievable(roof, ach),
        "achievable": ach,
        "put": {"achieved": round(put_rate / 1e9, 1), "unit": "GB/s", "frac_hbm": round(put_rate / PEAK_HBM, 4),
                "rows_accepted": rows_in, "rows_offered": k * K, "copy_ms": round(c_ms, 3)},
        "gather": {"achieved": round(g_rate / 1e9, 1), "unit": "GB/s", "frac_hbm": round(g_rate / PEAK_HBM, 4),
                   "rows": rows_out, "avg_us": round(g_avg * 1e6, 2)},
        "same_stream": {"achieved": round(direct_rate, 1), "unit": "GB/s", "ms_per_step": round(d_ms / K, 4),
                        "note": "the same iterations issued on the reservoir's ordering stream (no cross-stream "
                                "events)"},
        "host_s_per_step": round(wall / K, 6),
        "fill": {"achieved": round(fill_rate / 1e9, 1), "unit": "GB/s", "puts": n_fill,
                 "copy_avg_us": round(fill_copy_ms * 1e3 / fill_copies, 2), "ms": round(fill_ms, 3)},
        "wall_s": round(wall, 3), "cpu_baseline": None,
    }
    res.close()
    del xs, us, ub
    torch.cuda.empty_cache()
    if args.cpu_seconds > 0:
        line["cpu_baseline"] = cpu_baseline_stress(w, args.cpu_seconds)
    return line


def run_library_reference(w) -> dict:
    """torch.matmul on the output layer's forward (A W^T), weight-gradient
    (dY^T A) and input-gradient (dY W) shapes of workload w, in its GEMM
    precision, plus a square 8192 product; plain products without the fused
    epilogues of the library's kernels.  Comparison only."""
    import torch
    dev = torch.device("cuda:0")
    dt = torch.float32 if w.precision == "fp32" else torch.bfloat16
    torch.backends.cuda.matmul.allow_tf32 = False
    B, H, D = w.batch, w.widths[-2], w.widths[-1]
    g = torch.Generator(device=dev)
    g.manual_seed(0)
    A = torch.randn(B, H, device=dev, generator=g).to(dt)
    W = torch.randn(D, H, device=dev, generator=g).to(dt)
    dY = torch.randn(B, D, device=dev, generator=g).to(dt)

    def avg_us(fn, it):
        for _ in range(3):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(it):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e3 / it

    it = 50 if w.precision == "fp32" else 10
    flop = 2.0 * B * H * D
    peak = PEAK_FP32_MFMA if w.precision == "fp32" else PEAK_BF16_MFMA
    out = {}
    for name, fn in (("fwd_output", lambda: torch.matmul(A, W.t())), ("wgrad_output", lambda: torch.matmul(dY.t(), A)),
                     ("igrad_output", lambda: torch.matmul(dY, W))):
        us = avg_us(fn, it)
        out[name] = {"avg_us": round(us, 2), "tflops": round(flop / us / 1e6, 1), "frac": round(flop / us * 1e6 / peak, 4)}
    del A, W, dY
    torch.cuda.empty_cache()
    X = torch.randn(8192, 8192, device=dev, generator=g).to(dt)
    us = avg_us(lambda: torch.matmul(X, X), 10)
    out["square_8192"] = {"avg_us": round(us, 1), "tflops": round(2 * 8192 ** 3 / us / 1e6, 1),
                          "frac": round(2 * 8192 ** 3 / us * 1e6 / peak, 4)}
    return {"metric": "torch GEMM reference on the output-layer shapes (no epilogues)", "workload": w.name,
            "dtype": "f32" if w.precision == "fp32" else "bf16", "shapes": {"B": B, "H": H, "D": D},
            "torch": torch.__version__, "gemms": out}


def main():
    global GATHERED_TARGETS
    args = parse_args()
    GATHERED_TARGETS = args.gathered_targets
    if args.summarize_pmc:
        if not args.kernel:
            raise SystemExit("--summarize-pmc needs --kernel")
        e = summarize_pmc(args.summarize_pmc[0], args.summarize_pmc[1], args.config, args.kernel, args.pmc_command)
        print(json.dumps(e))
        return
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} (WORLD_SIZE {world}) is not supported: "
              "the library has no multi-GPU path (one reservoir and one surrogate per GPU).", file=sys.stderr)
        sys.exit(2)
    from fixtures import configs
    if args.pmc_calibration:
        pmc_calibration()
    if args.config == configs.STRESS.name:
        line = run_stress(args)
    else:
        if args.config not in configs.ALL:
            print(f"unknown config {args.config}; choose from {sorted(configs.ALL) + [configs.STRESS.name]}",
                  file=sys.stderr)
            sys.exit(2)
        w = configs.ALL[args.config]
        if args.library_reference:
            line = run_library_reference(w)
        elif args.policy_comparison:
            if w.fields != "ftcs":
                print("--policy-comparison streams an FTCS ensemble (tiny-16x16 or heat-100x100)", file=sys.stderr)
                sys.exit(2)
            line = run_policy_comparison(args, w)
        else:
            line = run_heat(args, w) if w.fields == "ftcs" else run_field(args, w)
    text = json.dumps(line)
    print(text, flush=True)
    if args.out:
        with open(args.out, "w") as f:
            f.write(text + "\n")


if __name__ == "__main__":
    main()
