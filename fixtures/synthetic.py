"""Cheap seeded stand-ins for the paper's 1000x1000 heat fields and for stress rows.

sine_mode_fields: smooth fields shaped like heat-equation solutions, a mean level
plus 8 separable Dirichlet sine modes decaying as exp(-pi^2 (p^2 + q^2) t) (the
eigen-solutions of Eq. 2 on the unit square).  They replace the paper's
implicit 1000x1000 solver (Sec. 4.1) where running a solver per sample would be
too costly; the values stay in [100, 500] like the paper's temperatures.

hash_rows: integer-valued rows, exact in fp32, whose content is a function of a
row key, so that any row read back from the reservoir can be checked against
the key it was stored under.
"""
from __future__ import annotations

import numpy as np

N_MODES = 8


def sine_mode_table(seed: int):
    """Seeded mode table: integer wave numbers p, q in [1, 8], signs, driver columns."""
    rng = np.random.default_rng(seed)
    p = rng.integers(1, 9, N_MODES)
    q = rng.integers(1, 9, N_MODES)
    sgn = rng.choice(np.array([-1.0, 1.0]), N_MODES)
    col = rng.integers(0, 5, N_MODES)
    return p, q, sgn, col


def sine_mode_fields(X: np.ndarray, t: np.ndarray, n: int, seed: int) -> np.ndarray:
    """Fields for inputs (X_i, t_i), fp32, shape (len(X), n*n).

    u(x, y) = m + sum_q a_q exp(-pi^2 (p_q^2 + q_q^2) t) sin(p_q pi x) sin(q_q pi y)
    with x_i = i/(n+1), i = 1..n (row index i is x, column index j is y),
    m = mean of the 5 temperatures, and a_q = A sgn_q (X[col_q] - 100)/400 / 8
    where A = min(m - 100, 500 - m); hence every value lies in [100, 500].
    """
    X = np.asarray(X, dtype=np.float64)
    t = np.asarray(t, dtype=np.float64)
    p, q, sgn, col = sine_mode_table(seed)
    xs = np.arange(1, n + 1, dtype=np.float64) / (n + 1)
    sx = np.sin(np.pi * np.outer(p, xs))          # (8, n)
    sy = np.sin(np.pi * np.outer(q, xs))          # (8, n)
    out = np.empty((X.shape[0], n * n), dtype=np.float32)
    for s in range(X.shape[0]):
        m = X[s].mean()
        amp = min(m - 100.0, 500.0 - m)
        a = amp * sgn * (X[s, col] - 100.0) / 400.0 / N_MODES
        a = a * np.exp(-np.pi ** 2 * (p ** 2 + q ** 2) * t[s])
        field = m + (a[:, None] * sx).T @ sy        # (n, n)
        out[s] = field.reshape(-1).astype(np.float32)
    return out


HASH_MUL_KEY = 2654435761
HASH_MUL_COL = 40503
HASH_MOD = 1 << 24


def hash_values(keys: np.ndarray, cols: np.ndarray) -> np.ndarray:
    """Columns `cols` of the hash rows of `keys`: fp32, shape (len(keys), len(cols))."""
    keys = np.asarray(keys, dtype=np.uint64)
    c = np.asarray(cols, dtype=np.uint64)
    v = (keys[:, None] * np.uint64(HASH_MUL_KEY) + c[None, :] * np.uint64(HASH_MUL_COL)) % np.uint64(HASH_MOD)
    return v.astype(np.float32)


def hash_rows(keys: np.ndarray, d: int) -> np.ndarray:
    """u[c] = float((key * 2654435761 + c * 40503) mod 2^24), fp32, shape (len(keys), d)."""
    return hash_values(keys, np.arange(d))


def hash_inputs(keys: np.ndarray, x_dim: int = 6) -> np.ndarray:
    """x = (key mod 2^24, key >> 24, 0, ...), fp32, shape (len(keys), x_dim)."""
    keys = np.asarray(keys, dtype=np.int64)
    out = np.zeros((keys.shape[0], x_dim), dtype=np.float32)
    out[:, 0] = (keys % HASH_MOD).astype(np.float32)
    if x_dim > 1:
        out[:, 1] = (keys >> 24).astype(np.float32)
    return out


def sine_mode_basis_torch(n: int, seed: int, device):
    """(8, n*n) fp32 device tensor of the separable modes sin(p pi x) sin(q pi y)."""
    import torch
    p, q, _, _ = sine_mode_table(seed)
    xs = torch.arange(1, n + 1, device=device, dtype=torch.float32) / (n + 1)
    pt = torch.tensor(p, device=device, dtype=torch.float32)
    qt = torch.tensor(q, device=device, dtype=torch.float32)
    sx = torch.sin(torch.pi * pt[:, None] * xs[None, :])
    sy = torch.sin(torch.pi * qt[:, None] * xs[None, :])
    return (sx[:, :, None] * sy[:, None, :]).reshape(N_MODES, n * n)


def sine_mode_fields_torch(X, t, seed: int, basis, out=None):
    """sine_mode_fields on the GPU with torch (fp32 arithmetic): same formula,
    values agree with the numpy version to fp32 rounding.  Benchmark inputs
    only; parity tests use the numpy version.  X: (S, 5), t: (S,) device
    tensors; basis from sine_mode_basis_torch."""
    import torch
    p, q, sgn, col = sine_mode_table(seed)
    dev = X.device
    pt = torch.tensor(p, device=dev, dtype=torch.float32)
    qt = torch.tensor(q, device=dev, dtype=torch.float32)
    Xf = X.to(torch.float32)
    m = Xf.mean(dim=1)
    amp = torch.minimum(m - 100.0, 500.0 - m)
    a = amp[:, None] * torch.tensor(sgn, device=dev, dtype=torch.float32)[None, :] \
        * (Xf[:, torch.tensor(col, device=dev)] - 100.0) / 400.0 / N_MODES
    a = a * torch.exp(-(torch.pi ** 2) * (pt ** 2 + qt ** 2)[None, :] * t.to(torch.float32)[:, None])
    res = torch.addmm(m[:, None].expand(-1, basis.shape[1]), a, basis) if out is None else \
        torch.addmm(m[:, None].expand(-1, basis.shape[1]), a, basis, out=out)
    return res


def hash_rows_torch(keys, d: int, out=None):
    """hash_rows on the GPU with torch int64 arithmetic (exact for keys < 2^31):
    (len(keys), d) fp32.  keys: int64 device tensor; out: optional (len(keys), >= d)
    fp32 view whose first d columns are written."""
    import torch
    keys = keys.to(torch.int64)
    c = torch.arange(d, device=keys.device, dtype=torch.int64)
    v = ((keys[:, None] * HASH_MUL_KEY) % HASH_MOD + (c[None, :] * HASH_MUL_COL) % HASH_MOD) % HASH_MOD
    if out is None:
        return v.to(torch.float32)
    out[:, :d].copy_(v)
    return out


def hash_inputs_torch(keys, x_dim: int = 6):
    """hash_inputs on the GPU: (len(keys), x_dim) fp32."""
    import torch
    keys = keys.to(torch.int64)
    out = torch.zeros(keys.shape[0], x_dim, device=keys.device, dtype=torch.float32)
    out[:, 0] = (keys % HASH_MOD).to(torch.float32)
    if x_dim > 1:
        out[:, 1] = (keys >> 24).to(torch.float32)
    return out
