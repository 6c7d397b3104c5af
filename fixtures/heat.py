"""Explicit 5-point (FTCS) solver for the 2-D heat equation, used as a data source.

The paper's use case (Sec. 4.1, Eq. 2) is the heat equation dT/dt = alpha*lap(T)
on a square with a constant initial temperature T_IC and four constant
Dirichlet boundary temperatures (T_x1 at x=0, T_x2 at x=L, T_y1 at y=0,
T_y2 at y=L).  The five temperatures are drawn uniformly in [100, 500] K and,
together with the time t, form the 6 inputs of the surrogate; the output is the
discretised field u_X^t (Sec. 4.1; Eq. 1 defines the mapping X -> {u_X^t}).

The paper's own solver is implicit Euler on 1000x1000.  This fixture is the
nondimensional forward-time centred-space scheme

    u+[i,j] = u[i,j] + r * (u[i+1,j] + u[i-1,j] + u[i,j+1] + u[i,j-1] - 4 u[i,j])

on an n x n interior with ghost Dirichlet values (row i=0 holds T_x1, i=n+1
holds T_x2, column j=0 holds T_y1, j=n+1 holds T_y2; the corners are never
read).  r = alpha*dt/h^2 = 0.2 (stable for r <= 1/4).  The solver works in
fp64 and the stored samples are rounded to fp32, as the paper's clients convert
64-bit solver output to 32 bits before sending it (Sec. 3.2.2).

Samples are the post-step states k = 1..tau; the surrogate's time input for
step k is t = 0.01*k (the paper's 100 steps of 0.01 s, Sec. 4.1).
"""
from __future__ import annotations

import numpy as np

R_DEFAULT = 0.2
DT_LABEL = 0.01


def sample_parameters(n_sims: int, seed: int) -> np.ndarray:
    """X = (T_IC, T_x1, T_y1, T_x2, T_y2) ~ U(100, 500) K, shape (n_sims, 5), fp64.

    Monte Carlo draws of the experimental design (Sec. 3.1 lists Monte Carlo
    among the supported designs; Sec. 4.1 fixes the range [100, 500] K).
    """
    rng = np.random.default_rng(seed)
    return rng.uniform(100.0, 500.0, size=(n_sims, 5))


def ftcs_run(u0: np.ndarray, bc: np.ndarray, r: float, n_steps: int) -> np.ndarray:
    """Advance fields with FTCS and return every post-step interior state.

    u0: (S, n, n) interior initial fields.  bc: (S, 4) boundary values ordered
    (T_x1, T_y1, T_x2, T_y2).  Returns (n_steps, S, n, n) fp64, entry k-1 being
    the state after k steps.
    """
    u0 = np.asarray(u0, dtype=np.float64)
    bc = np.asarray(bc, dtype=np.float64)
    s, n, n2 = u0.shape
    assert n == n2 and bc.shape == (s, 4)
    g = np.empty((s, n + 2, n + 2), dtype=np.float64)
    g[:, 1:-1, 1:-1] = u0
    g[:, 0, :] = bc[:, 0, None]        # i = 0   : x = 0 boundary, T_x1
    g[:, :, 0] = bc[:, 1, None]        # j = 0   : y = 0 boundary, T_y1
    g[:, n + 1, :] = bc[:, 2, None]    # i = n+1 : x = L boundary, T_x2
    g[:, :, n + 1] = bc[:, 3, None]    # j = n+1 : y = L boundary, T_y2
    out = np.empty((n_steps, s, n, n), dtype=np.float64)
    for k in range(n_steps):
        c = g[:, 1:-1, 1:-1]
        lap = g[:, 2:, 1:-1] + g[:, :-2, 1:-1] + g[:, 1:-1, 2:] + g[:, 1:-1, :-2] - 4.0 * c
        g[:, 1:-1, 1:-1] = c + r * lap
        out[k] = g[:, 1:-1, 1:-1]
    return out


def heat_fields(X: np.ndarray, n: int, tau: int, r: float = R_DEFAULT,
                sims_per_block: int = 32, threads: int = 0) -> np.ndarray:
    """Fields u_X^k for k = 1..tau of every simulation, fp32, shape (S, tau, n*n).

    X rows are (T_IC, T_x1, T_y1, T_x2, T_y2); the initial field is T_IC
    everywhere.  Simulations are advanced in independent blocks (bounded
    memory), on `threads` worker threads (0: one per available core).
    """
    import concurrent.futures as cf
    import os
    X = np.asarray(X, dtype=np.float64)
    s = X.shape[0]
    out = np.empty((s, tau, n * n), dtype=np.float32)

    def block(b0):
        xb = X[b0:b0 + sims_per_block]
        u0 = np.broadcast_to(xb[:, 0, None, None], (xb.shape[0], n, n))
        states = ftcs_run(u0, xb[:, 1:5], r, tau)             # (tau, sb, n, n)
        out[b0:b0 + xb.shape[0]] = states.transpose(1, 0, 2, 3).reshape(xb.shape[0], tau, n * n)

    starts = list(range(0, s, sims_per_block))
    workers = threads or min(16, len(os.sched_getaffinity(0)))
    if workers <= 1 or len(starts) == 1:
        for b0 in starts:
            block(b0)
    else:
        with cf.ThreadPoolExecutor(max_workers=workers) as ex:
            list(ex.map(block, starts))
    return out


def inputs_for(X: np.ndarray, tau: int) -> np.ndarray:
    """Surrogate inputs (X, t) for k = 1..tau, fp32, shape (S, tau, 6)."""
    X = np.asarray(X, dtype=np.float64)
    s = X.shape[0]
    t = DT_LABEL * np.arange(1, tau + 1, dtype=np.float64)
    out = np.empty((s, tau, 6), dtype=np.float64)
    out[:, :, :5] = X[:, None, :]
    out[:, :, 5] = t[None, :]
    return out.astype(np.float32)
