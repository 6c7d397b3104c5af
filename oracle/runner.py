"""Deterministic online-training loop of the oracle.

One server process of the paper (Sec. 3.1) runs an aggregator thread that puts
received time steps into the training buffer and a training thread that draws
batches from it and trains.  The oracle serialises the two: iteration i puts
chunk i of the streamed ensemble (while chunks remain), then draws a batch of
B and, if the buffer answered with a batch, runs one train step (forward, MSE,
backward, Adam).  The GPU path is driven by the same loop, so both see the
same ticket sequence.

run_to_drain() streams the whole schedule through any of the three buffers
and then drains it after the end of reception.

Training instrumentation of Sec. 4.4-4.5, optional:
  * learning-rate schedule: the rate starts at lr0 and is halved every
    `every_samples` trained samples down to a floor lr_min (the paper halves
    1e-3 every 1000 batches of 10, i.e. every 10,000 samples, to 2.5e-4); the
    rate of a step is set from the samples trained before it;
  * validation: the mean squared error of the current surrogate on held-out
    simulations, every `validate_every` train steps, taken after that step;
  * repetition histogram: how many times each sample that entered the buffer
    was drawn (residents and samples that left alike).
"""
from __future__ import annotations

from typing import Dict, Iterable, Optional

import numpy as np

from fixtures.configs import Workload, chunk_for_iteration

from .mlp import Adam, init_params, loss_and_grads, mse, predict
from .reservoir import NOT_READY, OK, Reservoir


def halving_lr(lr0: float, samples_trained: int, every_samples: int, lr_min: float) -> float:
    """lr0 halved once per completed block of every_samples trained samples, floored at lr_min."""
    return max(lr0 * 0.5 ** (samples_trained // every_samples), lr_min)


def repetition_histogram(res, length: int) -> np.ndarray:
    """h[k] = number of samples that entered the buffer and were drawn k times
    (k >= length - 1 counted in the last bin)."""
    h = np.zeros(length, np.int64)
    for k, c in res.evict_hist.items():
        h[min(k, length - 1)] += c
    for s in res.occ:
        h[min(int(res.seen_count[s]), length - 1)] += 1
    return h


def run_to_drain(w: Workload, inputs: np.ndarray, fields: np.ndarray, buffer) -> Dict:
    """The whole production schedule through `buffer` (a Reservoir, FIFOBuffer
    or FIROBuffer built by the caller), then the end of reception and the
    drain (Sec. 3.2.3): iteration i puts chunk i and trains on a batch when the
    buffer yields one; after the last chunk, end_reception and train on every
    batch the buffer yields until it answers EMPTY (the last one may be short).
    Returns the trace (losses, slots, batch sizes, final parameters)."""
    params = init_params(w.widths, w.init_seed)
    opt = Adam(lr=w.lr)
    trace = dict(losses=[], slots=[], sizes=[])

    def train(xb, ub, slots):
        nonlocal params
        loss, grads = loss_and_grads(params, xb, ub)
        params = opt.step(params, grads)
        trace["losses"].append(loss)
        trace["slots"].append(np.array(slots, dtype=np.int64))
        trace["sizes"].append(len(slots))

    for chunk in range(w.n_chunks):
        xs, us = chunk_arrays(w, inputs, fields, chunk)
        buffer.put(xs, us)
        st, slots, xb, ub, _ = buffer.sample_batch(w.batch)
        if st == OK:
            train(xb, ub, slots)
    buffer.end_reception()
    while True:
        st, slots, xb, ub, _ = buffer.sample_batch(w.batch)
        if st != OK:
            break
        train(xb, ub, slots)
    trace["params"] = params
    return trace


def chunk_arrays(w: Workload, inputs: np.ndarray, fields: np.ndarray, chunk: int):
    """(x rows, u rows) of one chunk from per-simulation arrays (S, tau, .)."""
    rows = w.chunk_rows(chunk)
    sims = np.array([s for s, _ in rows])
    ks = np.array([k for _, k in rows])
    return inputs[sims, ks], fields[sims, ks]


def run(w: Workload, inputs: np.ndarray, fields: np.ndarray, n_steps: int,
        params=None, bf16: Optional[bool] = None, keep_grads: Iterable[int] = (),
        lr: Optional[float] = None, lr_halving: Optional[tuple] = None,
        validation: Optional[tuple] = None, state_fp32: bool = False) -> Dict:
    """Run the schedule until n_steps train steps are done; return the trace.
    lr_halving: (every_samples, lr_min); validation: (X_val, U_val, every);
    state_fp32: parameters and Adam moments stored in fp32 between steps
    (Adam.state_dtype).  For each step in keep_grads the trace holds its
    gradients, the parameters after it and the batch (X, U) it trained on."""
    if bf16 is None:
        bf16 = w.precision == "bf16"
    res = Reservoir(w.capacity, w.threshold, inputs.shape[-1], fields.shape[-1], w.reservoir_seed)
    if params is None:
        params = init_params(w.widths, w.init_seed)
    lr0 = w.lr if lr is None else lr
    opt = Adam(lr=lr0, state_dtype=np.float32 if state_fp32 else None)
    keep = set(keep_grads)
    trace = dict(losses=[], slots=[], tickets=[], put_accepted=[], grads={}, params_at={}, batches={}, lrs=[],
                 val_losses={})
    i = done = 0
    while done < n_steps:
        chunk = chunk_for_iteration(w, i)
        if chunk is not None:
            xs, us = chunk_arrays(w, inputs, fields, chunk)
            _, acc, _, _ = res.put(xs, us)
            trace["put_accepted"].append(acc)
        st, slots, xb, ub, ticket = res.sample_batch(w.batch)
        if st == OK:
            if lr_halving is not None:
                opt.lr = halving_lr(lr0, done * w.batch, *lr_halving)
            trace["lrs"].append(opt.lr)
            loss, grads = loss_and_grads(params, xb, ub, bf16=bf16)
            params = opt.step(params, grads)
            done += 1
            if validation is not None and done % validation[2] == 0:
                Xv, Uv = validation[0], validation[1]
                trace["val_losses"][done] = mse(predict(params, Xv, bf16=bf16), Uv)
            trace["losses"].append(loss)
            trace["slots"].append(np.array(slots, dtype=np.int64))
            trace["tickets"].append(ticket)
            if done in keep:
                trace["grads"][done] = grads
                trace["params_at"][done] = params
                trace["batches"][done] = (xb, ub)
        elif st == NOT_READY and chunk is None:
            raise RuntimeError("schedule ran out of data before the buffer became ready")
        i += 1
    trace["params"] = params
    trace["adam"] = opt
    trace["reservoir"] = res
    trace["iterations"] = i
    return trace
