"""Online training loop over the library: one aggregator put and one training
step per iteration, as the paper's server runs a data-aggregator thread that
fills the buffer and a training thread that draws batches from it (Sec. 3.1).

By default all work is enqueued on one HIP stream.  With graph=True (one
stream only) the train step is captured once as a HIP graph, with Adam's
step counter in device memory (surrogate_set_device_step), and replayed for
every later step of full batches: the reservoir's calls stay eager, the train
step costs one launch.  With overlap=True the
reservoir (put, draw, gather) runs on its own ordering stream and the train
step on the trainer's stream, with two batch buffers: the draw and gather of
batch i + 1 run while batch i trains, as the paper's two threads do.  Events
order the streams: train step i waits for gather i, and gather i + 2 waits for
train step i to release its buffer.  The sequence of reservoir operations (and
so every drawn slot) is the same as on one stream.
"""
from __future__ import annotations

import contextlib
from dataclasses import dataclass
from typing import Callable, Optional

import numpy as np
import torch

from . import OT_FP32, OT_BF16, OT_OK, OT_POLICY_RESERVOIR, Reservoir, Surrogate


def _round_up(v: int, m: int) -> int:
    return (v + m - 1) // m * m


class ReceptionLog:
    """Log of received messages per client (Sec. 3.1: the server keeps one, so
    that after a client restart the messages it already received are
    discarded).  A message is a (client, time step) key; it counts as received
    once a put accepted its row.  Acceptance is known on the device (the
    Reservoir accepts a prefix that depends on its unseen count), so each put
    leaves its accepted count in a device word and the log resolves those
    counts only when a key that was offered before arrives again: new keys
    never wait for the device.

    put_stream: the stream the puts run on (the reservoir's ordering stream).
    The counts are cleared and read back on that stream, so a read waits for
    every put enqueued before it, whichever stream is current (None: counts
    in host memory, for host-only use)."""

    def __init__(self, device, put_stream: Optional[torch.cuda.Stream] = None):
        self.received = set()
        self.offered = set()
        self.pending = []                  # (keys of one put in row order, index into the device counts)
        self.put_stream = put_stream
        with self._on_put_stream():
            self.counts = torch.zeros(4096, dtype=torch.int64, device=device)
        self.next_count = 0

    def _on_put_stream(self):
        return torch.cuda.stream(self.put_stream) if self.put_stream is not None else contextlib.nullcontext()

    def count_slot(self) -> torch.Tensor:
        """Device int64 word for the next put's accepted count."""
        if self.next_count == len(self.counts):
            self.resolve()
        i = self.next_count
        self.next_count += 1
        return self.counts[i:i + 1]

    def record(self, keys, count_slot_index: int) -> None:
        self.offered.update(keys)
        self.pending.append((list(keys), count_slot_index))

    def resolve(self) -> None:
        """Read the pending accepted counts (waits for the puts)."""
        if self.pending:
            with self._on_put_stream():                   # ordered after the puts that write the counts
                a = self.counts[:self.next_count].cpu().tolist()
            for keys, i in self.pending:
                self.received.update(keys[:a[i]])
                self.offered.difference_update(keys[a[i]:])     # refused rows may come again
            self.pending = []
        self.next_count = 0

    def new_rows(self, keys) -> np.ndarray:
        """Mask of the rows whose keys were not received yet."""
        if not any(k in self.offered for k in keys):
            return np.ones(len(keys), dtype=bool)
        self.resolve()
        return np.array([k not in self.received for k in keys], dtype=bool)

    def keys(self) -> np.ndarray:
        self.resolve()
        return np.array(sorted(self.received), dtype=np.int64).reshape(-1, 2)


@dataclass(frozen=True)
class HalvingLR:
    """Learning-rate schedule of Sec. 4.4-4.5: start at lr0, halve once per
    every_samples trained samples, never below lr_min (the paper: 1e-3 halved
    every 10,000 samples down to 2.5e-4).  Called with the number of samples
    trained before a step, returns that step's rate."""
    lr0: float = 1e-3
    every_samples: int = 10_000
    lr_min: float = 2.5e-4

    def __call__(self, samples_trained: int) -> float:
        return max(self.lr0 * 0.5 ** (samples_trained // self.every_samples), self.lr_min)


class OnlineTrainer:
    """Streams chunks of an ensemble into a reservoir and trains.

    Either inputs: (S, tau, x_dim) and fields: (S, tau, D) fp32 device tensors
    (chunk c holds time step (c mod tau) of the `wave` simulations of wave
    c // tau), or chunk_fn(c) -> (x rows, u rows) device tensors for chunks
    0 .. n_chunks - 1 (rows with unit column stride, leading dimension a
    multiple of 4).
    """

    def __init__(self, widths, batch: int, capacity: int, threshold: int, wave: int, tau: int,
                 inputs: Optional[torch.Tensor], fields: Optional[torch.Tensor], reservoir_seed: int,
                 init_seed: int, precision: int = OT_FP32, lr: float = 1e-3,
                 stream: Optional[torch.cuda.Stream] = None, record_steps: int = 0,
                 chunk_fn: Optional[Callable] = None, n_chunks: int = 0, device=None, flags: int = 0,
                 overlap: bool = False, policy: int = OT_POLICY_RESERVOIR,
                 lr_schedule: Optional[Callable[[int], float]] = None, reception_log: bool = False,
                 fused_targets: bool = True, put_streams: Optional[list] = None, graph: bool = False):
        self.stream = stream if stream is not None else torch.cuda.current_stream()
        self.widths = tuple(widths)
        self.batch, self.wave, self.tau = batch, wave, tau
        self.inputs, self.fields = inputs, fields
        self.chunk_fn = chunk_fn
        if chunk_fn is None:
            self.n_sims = inputs.shape[0]
            self.n_chunks = (self.n_sims // wave) * tau
            dev = inputs.device
        else:
            self.n_chunks = n_chunks
            dev = device
        x_dim, d = widths[0], widths[-1]
        self.overlap = overlap
        # default-priority stream of its own for the reservoir when overlapping
        self.res_stream = torch.cuda.Stream(device=dev) if overlap else self.stream
        self.res = Reservoir(capacity, threshold, x_dim, d, reservoir_seed, order_stream=self.res_stream,
                             policy=policy)
        self.sur = Surrogate(widths, precision=precision, lr=lr, seed=init_seed, max_batch=batch, flags=flags)
        nbuf = 2 if overlap else 1
        # fused_targets: the train step reads the batch's field rows in place
        # from the reservoir's slab through the drawn slots (only the input
        # rows are gathered); a put then waits until the train step before it
        # has read its targets (targets_read), since it may overwrite them
        self.fused_targets = fused_targets
        self.xbufs = [torch.empty(batch, _round_up(x_dim, 4), device=dev)[:, :x_dim] for _ in range(nbuf)]
        self.ubufs = [] if fused_targets else [torch.empty(batch, _round_up(d, 4), device=dev)[:, :d]
                                               for _ in range(nbuf)]
        self.slotbufs = [torch.empty(batch, dtype=torch.int32, device=dev) for _ in range(nbuf)]
        self.xb = self.xbufs[0]
        self.ub = None if fused_targets else self.ubufs[0]
        _, _, self.u_slab, self.ldu_slab = self.res.slab()
        self.targets_read = torch.cuda.Event()
        self.targets_read_recorded = False
        self._targets_waited = False
        self.ready = [torch.cuda.Event() for _ in range(nbuf)]      # gather into buffer j done
        self.released = [torch.cuda.Event() for _ in range(nbuf)]   # train step on buffer j done
        self.released_recorded = [False] * nbuf
        # serialize=True (overlap mode only): each put waits for the train
        # step before it, so per-kernel timings are not inflated by the other
        # stream's kernels (used for breakdowns, not for throughput)
        self.serialize = False
        self._train_done = torch.cuda.Event() if overlap else None
        self.slots = self.slotbufs[0]
        self.record_steps = record_steps
        self.slot_log = torch.empty((max(record_steps, 1), batch), dtype=torch.int32, device=dev)
        self.loss_log = torch.zeros(max(record_steps, 1), device=dev)
        self.loss = torch.zeros(1, device=dev)
        self.accepted = torch.zeros(1, dtype=torch.int64, device=dev)
        self.iteration = 0
        self.steps_done = 0
        self.chunk_cursor = 0
        self.lr_schedule = lr_schedule
        self.lr = lr
        self.val_loss = torch.zeros(1, device=dev)
        self.log = ReceptionLog(dev, self.res_stream) if reception_log else None
        # producer streams (the paper's clients): chunk c is put from put_streams[c mod P];
        # default: the reservoir's own stream
        self.put_streams = list(put_streams) if put_streams else None
        if graph and (overlap or not fused_targets or lr_schedule is not None):
            raise ValueError("graph=True needs one stream, targets read in place and a constant learning rate")
        self.graph = graph
        self.graph_active = graph        # callers may run eager steps (e.g. with phase timing) meanwhile
        self._graph = None
        self._graph_warm = False

    def chunk_views(self, c: int):
        if self.chunk_fn is not None:
            return self.chunk_fn(c)
        w, k = divmod(c % self.n_chunks, self.tau)
        s0 = w * self.wave
        return self.inputs[s0:s0 + self.wave, k, :], self.fields[s0:s0 + self.wave, k, :]

    def chunk_keys(self, c: int):
        """(client, time step) message keys of the rows of chunk c."""
        if self.chunk_fn is not None:
            return [(c, i) for i in range(self.wave)]
        w, k = divmod(c % self.n_chunks, self.tau)
        return [(w * self.wave + s, k) for s in range(self.wave)]

    def put_next(self, wrap: bool = False) -> bool:
        """Put the next chunk; after the last chunk, wrap around only if asked."""
        if self.chunk_cursor >= self.n_chunks and not wrap:
            return False
        self.offer_chunk(self.chunk_cursor)
        self.chunk_cursor += 1
        return True

    def offer_chunk(self, c: int) -> None:
        """Put the rows of chunk c (with a reception log: only rows not received before)."""
        x, u = self.chunk_views(c)
        if self.overlap and self.serialize:
            self._train_done.record(self.stream)
            self.res_stream.wait_event(self._train_done)
        self._wait_targets_read()                 # a put may overwrite rows the last train step reads
        put_stream = self.put_streams[c % len(self.put_streams)] if self.put_streams else self.res_stream
        if self.log is None:
            self.res.put(x, u, stream=put_stream, accepted=self.accepted)
            return
        keys = self.chunk_keys(c)
        keep = self.log.new_rows(keys)
        i = 0
        while i < len(keys):                      # one put per run of consecutive new rows
            if not keep[i]:
                i += 1
                continue
            j = i
            while j < len(keys) and keep[j]:
                j += 1
            slot = self.log.count_slot()
            self.res.put(x[i:j], u[i:j], stream=put_stream, accepted=slot)
            self.log.record(keys[i:j], self.log.next_count - 1)
            i = j

    def sample_only(self) -> bool:
        """Draw a batch without gathering or training (marks samples seen)."""
        st, _, _ = self.res.sample_batch(self.batch, self.slots, stream=self.res_stream)
        return st == OT_OK

    def _wait_targets_read(self) -> None:
        """Overlapped fused mode: order the reservoir stream after the last
        train step's targets_read event (once per recording).  That event
        follows, on the training stream, every earlier train step, so the
        buffers of the step two back are free after it too."""
        if self.overlap and self.fused_targets and self.targets_read_recorded and not self._targets_waited:
            self.res_stream.wait_event(self.targets_read)
            self._targets_waited = True

    def sample_and_train(self) -> bool:
        rec = self.steps_done < self.record_steps
        j = self.steps_done % len(self.xbufs)
        # a graph replays on the buffers it was captured with: its slots are copied to the log afterwards
        slots = self.slot_log[self.steps_done] if rec and not self.graph else self.slotbufs[j]
        xb = self.xbufs[j]
        ub = None if self.fused_targets else self.ubufs[j]
        # the step two back has finished with buffer j
        if self.overlap and not self.fused_targets and self.released_recorded[j]:
            self.res_stream.wait_event(self.released[j])
        self._wait_targets_read()
        st, n, _ = self.res.sample_batch(self.batch, slots, x_out=xb, u_out=ub, stream=self.res_stream)
        if st != OT_OK:
            return False
        if n < self.batch:                                    # short last batch of a drain
            xb, slots = xb[:n], slots[:n]
            ub = None if ub is None else ub[:n]
        if self.overlap:
            self.ready[j].record(self.res_stream)
            self.stream.wait_event(self.ready[j])
        loss = self.loss_log[self.steps_done:self.steps_done + 1] if rec else self.loss
        if self.lr_schedule is not None:
            lr = self.lr_schedule(self.steps_done * self.batch)
            if lr != self.lr:
                self.sur.set_lr(lr)       # host-side rate, taken by the next enqueued step
                self.lr = lr
        if self.graph and self.graph_active and n == self.batch:
            self._graph_step(xb, slots, loss)
        elif self.fused_targets:
            self.sur.train_step_rows(xb, self.u_slab, self.ldu_slab, slots, self.res.capacity, stream=self.stream,
                                     loss=loss, targets_read=self.targets_read if self.overlap else None)
            self.targets_read_recorded = self.overlap
            self._targets_waited = False
        else:
            self.sur.train_step(xb, ub, stream=self.stream, loss=loss)
        if self.overlap and not self.fused_targets:
            self.released[j].record(self.stream)
            self.released_recorded[j] = True
        if rec and self.graph:
            with torch.cuda.stream(self.stream):
                self.slot_log[self.steps_done, :n].copy_(slots)
        self.steps_done += 1
        return True

    def _graph_step(self, xb, slots, loss) -> None:
        """The train step as a replay of its captured launches (captured at the
        second call, on this trainer's buffers, which the replays reuse; the
        first runs eagerly, so that the step's workspaces exist before capture,
        which allows no allocation)."""
        if not self._graph_warm:
            self._graph_warm = True
            self.sur.train_step_rows(xb, self.u_slab, self.ldu_slab, slots, self.res.capacity, stream=self.stream,
                                     loss=loss)
            return
        if self._graph is None:
            torch.cuda.synchronize()
            self.sur.set_device_step(True)
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                self.sur.train_step_rows(xb, self.u_slab, self.ldu_slab, slots, self.res.capacity,
                                         stream=torch.cuda.current_stream(), loss=self.loss)
            self._graph = g
        with torch.cuda.stream(self.stream):
            self._graph.replay()
            if loss.data_ptr() != self.loss.data_ptr():
                loss.copy_(self.loss)

    def iterate(self, wrap: bool = False) -> bool:
        """One iteration of the schedule; returns whether a train step ran."""
        self.put_next(wrap)
        trained = self.sample_and_train()
        self.iteration += 1
        return trained

    def run(self, n_steps: int, wrap: bool = False) -> None:
        target = self.steps_done + n_steps
        while self.steps_done < target:
            if self.chunk_cursor >= self.n_chunks and not wrap and self.res.stats()["n"] <= self.res.threshold:
                raise RuntimeError("schedule ran out of data before the buffer became ready")
            self.iterate(wrap)

    def validate(self, x: torch.Tensor, u: torch.Tensor, out: Optional[torch.Tensor] = None) -> torch.Tensor:
        """Validation MSE of the current surrogate on held-out rows x -> u,
        enqueued on the training stream after the steps so far (Sec. 4.4
        validates on the training thread).  Returns the device scalar."""
        out = self.val_loss if out is None else out
        self.sur.eval_loss(x, u, out, stream=self.stream)
        return out

    def repetition_histogram(self) -> np.ndarray:
        """h[k] = samples that entered the buffer and were drawn k times so far
        (samples that left the buffer and residents; the last bin collects
        the tail), as the paper's histogram of repetitions (Sec. 4.3)."""
        seen, _, hist = self.res.read_meta()
        h = hist.astype(np.int64).copy()
        resident = seen[seen >= 0]
        np.add.at(h, np.minimum(resident, len(h) - 1), 1)
        return h

    def checkpoint(self) -> dict:
        """Synchronous snapshot of the whole online-training state: reservoir,
        surrogate (parameters and Adam state), the loop's counters and
        learning rate, and the reception log.  Arrays only (np.savez-able)."""
        torch.cuda.synchronize()
        state = np.array([self.chunk_cursor, self.steps_done, self.iteration], dtype=np.int64)
        out = {"reservoir": self.res.checkpoint(), "surrogate": self.sur.checkpoint(), "loop": state,
               "lr": np.array([self.lr], dtype=np.float64)}
        if self.log is not None:
            out["received"] = self.log.keys()
        return out

    def restore(self, ckpt: dict) -> None:
        """Continue from a checkpoint() of a trainer built with the same arguments."""
        torch.cuda.synchronize()
        self.res.restore(ckpt["reservoir"])
        self.sur.restore(ckpt["surrogate"])
        self.chunk_cursor, self.steps_done, self.iteration = (int(v) for v in ckpt["loop"])
        self.lr = float(ckpt["lr"][0])
        self.released_recorded = [False] * len(self.released_recorded)
        self.targets_read_recorded = False
        if self.log is not None:
            self.log = ReceptionLog(self.xb.device, self.res_stream)
            self.log.received = {tuple(int(v) for v in k) for k in ckpt.get("received", np.zeros((0, 2)))}
            self.log.offered = set(self.log.received)

    def close(self):
        self.res.close()
        self.sur.close()
