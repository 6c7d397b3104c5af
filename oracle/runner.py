"""Deterministic online-training loop of the oracle.

One server process of the paper (Sec. 3.1) runs an aggregator thread that puts
received time steps into the training buffer and a training thread that draws
batches from it and trains.  The oracle serialises the two: iteration i puts
chunk i of the streamed ensemble (while chunks remain), then draws a batch of
B and, if the buffer answered with a batch, runs one train step (forward, MSE,
backward, Adam).  The GPU path is driven by the same loop, so both see the
same ticket sequence.
"""
from __future__ import annotations

from typing import Dict, Iterable, Optional

import numpy as np

from fixtures.configs import Workload, chunk_for_iteration

from .mlp import Adam, init_params, loss_and_grads
from .reservoir import NOT_READY, OK, Reservoir


def chunk_arrays(w: Workload, inputs: np.ndarray, fields: np.ndarray, chunk: int):
    """(x rows, u rows) of one chunk from per-simulation arrays (S, tau, .)."""
    rows = w.chunk_rows(chunk)
    sims = np.array([s for s, _ in rows])
    ks = np.array([k for _, k in rows])
    return inputs[sims, ks], fields[sims, ks]


def run(w: Workload, inputs: np.ndarray, fields: np.ndarray, n_steps: int,
        params=None, bf16: Optional[bool] = None, keep_grads: Iterable[int] = (),
        lr: Optional[float] = None) -> Dict:
    """Run the schedule until n_steps train steps are done; return the trace."""
    if bf16 is None:
        bf16 = w.precision == "bf16"
    res = Reservoir(w.capacity, w.threshold, inputs.shape[-1], fields.shape[-1], w.reservoir_seed)
    if params is None:
        params = init_params(w.widths, w.init_seed)
    opt = Adam(lr=w.lr if lr is None else lr)
    keep = set(keep_grads)
    trace = dict(losses=[], slots=[], tickets=[], put_accepted=[], grads={}, params_at={})
    i = done = 0
    while done < n_steps:
        chunk = chunk_for_iteration(w, i)
        if chunk is not None:
            xs, us = chunk_arrays(w, inputs, fields, chunk)
            _, acc, _, _ = res.put(xs, us)
            trace["put_accepted"].append(acc)
        st, slots, xb, ub, ticket = res.sample_batch(w.batch)
        if st == OK:
            loss, grads = loss_and_grads(params, xb, ub, bf16=bf16)
            params = opt.step(params, grads)
            done += 1
            trace["losses"].append(loss)
            trace["slots"].append(np.array(slots, dtype=np.int64))
            trace["tickets"].append(ticket)
            if done in keep:
                trace["grads"][done] = grads
                trace["params_at"][done] = params
        elif st == NOT_READY and chunk is None:
            raise RuntimeError("schedule ran out of data before the buffer became ready")
        i += 1
    trace["params"] = params
    trace["adam"] = opt
    trace["reservoir"] = res
    trace["iterations"] = i
    return trace
