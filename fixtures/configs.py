"""The five workloads: shapes, seeds, reservoir sizes and the streaming schedule.

Shapes follow the paper's use case (Sec. 4.1-4.3: 6 inputs, fields of n*n fp32
values, MLP with ReLU hidden layers and an identity output, Adam with lr 1e-3,
capacity 6,000 with threshold 1,000 for the paper's own runs).  Where a
workload gives no threshold, T = max(B, round(C/6)), the paper's
capacity/threshold ratio (Sec. 4.3) floored at one batch.

Streaming schedule: simulations run in waves of `wave` concurrent clients (the
paper's runs use series of 100 concurrent clients, Sec. 4.3); chunk i carries
time step k = (i mod tau) + 1 of every simulation of wave i // tau, in
simulation order.  Iteration i puts chunk i (while chunks remain), then draws a
batch and trains if the reservoir holds more than T samples.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Tuple


@dataclass(frozen=True)
class Workload:
    name: str
    grid: int                      # field is grid x grid fp32 values
    tau: int                       # time steps per simulation
    n_sims: int
    widths: Tuple[int, ...]        # MLP widths, input first
    precision: str                 # "fp32" or "bf16"
    batch: int
    capacity: int
    threshold: int
    steps: int                     # train steps of the workload
    wave: int                      # concurrent simulations (rows per chunk)
    data_seed: int
    init_seed: int
    reservoir_seed: int
    fields: str = "ftcs"           # "ftcs" | "sine" | "hash"
    lr: float = 1e-3

    @property
    def d(self) -> int:
        return self.widths[-1]

    @property
    def n_chunks(self) -> int:
        return (self.n_sims // self.wave) * self.tau

    def chunk_rows(self, i: int) -> List[Tuple[int, int]]:
        """(simulation, step index k-1) of every row of chunk i, in put order."""
        w, k = divmod(i, self.tau)
        return [(w * self.wave + s, k) for s in range(self.wave)]

    def n_params(self) -> int:
        return sum(self.widths[l + 1] * (self.widths[l] + 1) for l in range(len(self.widths) - 1))


def _thr(batch: int, capacity: int) -> int:
    return max(batch, int(round(capacity / 6)))


TINY = Workload(
    name="tiny-16x16", grid=16, tau=10, n_sims=8, widths=(6, 64, 64, 256), precision="fp32",
    batch=32, capacity=64, threshold=_thr(32, 64), steps=100, wave=8,
    data_seed=0, init_seed=1, reservoir_seed=0)

HEAT100 = Workload(
    name="heat-100x100", grid=100, tau=100, n_sims=1000, widths=(6, 256, 256, 10000), precision="fp32",
    batch=1024, capacity=100_000, threshold=_thr(1024, 100_000), steps=2000, wave=100,
    data_seed=2, init_seed=3, reservoir_seed=2)

FIELD1M = Workload(
    name="sine-1000x1000", grid=1000, tau=100, n_sims=10_000, widths=(6, 1024, 1024, 1_000_000),
    precision="bf16", batch=512, capacity=20_000, threshold=_thr(512, 20_000), steps=200, wave=64,
    data_seed=4, init_seed=5, reservoir_seed=4, fields="sine")

DEEP1M = Workload(
    name="deep-sine-1000x1000", grid=1000, tau=100, n_sims=10_000, widths=(6, 2048, 2048, 2048, 1_000_000),
    precision="bf16", batch=1024, capacity=30_000, threshold=_thr(1024, 30_000), steps=200, wave=64,
    data_seed=7, init_seed=8, reservoir_seed=7, fields="sine")


@dataclass(frozen=True)
class StressWorkload:
    """Reservoir-only stress: rows of row_len fp32, many producers, one consumer."""
    name: str = "stress-100k-rows"
    row_len: int = 100_000
    capacity: int = 50_000
    threshold: int = 10_000
    producers: int = 64
    chunk: int = 256
    batch: int = 256
    reservoir_seed: int = 6


STRESS = StressWorkload()

ALL = {w.name: w for w in (TINY, HEAT100, FIELD1M, DEEP1M)}


def chunk_for_iteration(w: Workload, i: int) -> Optional[int]:
    """Chunk put at iteration i, or None once the ensemble has been streamed."""
    return i if i < w.n_chunks else None
