"""Pins of the input fixtures: FTCS heat solver, sine-mode fields, hash rows, workloads.

FTCS (Sec. 4.1, Eq. 2): a discrete eigenmode with zero boundaries decays by
exactly lambda = 1 - 4r[sin^2(p pi/(2(n+1))) + sin^2(q pi/(2(n+1)))] per step;
under refinement at fixed r the discrete solution converges to the separable
continuous solution exp(-pi^2 (p^2 + q^2) t) sin(p pi x) sin(q pi y) at second
order in h; equal temperatures stay constant; values stay within the range of
the data (maximum principle, r <= 1/4); swapping T_x1 and T_x2 mirrors the field.
"""
import numpy as np
import pytest

from fixtures import configs, heat, synthetic


def _mode(n, p, q):
    i = np.arange(1, n + 1) / (n + 1)
    return np.outer(np.sin(p * np.pi * i), np.sin(q * np.pi * i))


@pytest.mark.parametrize("n,p,q", [(16, 1, 1), (16, 3, 2), (31, 5, 7)])
def test_discrete_eigenmode_exact(n, p, q):
    r, steps = 0.2, 25
    u0 = _mode(n, p, q)[None]
    out = heat.ftcs_run(u0, np.zeros((1, 4)), r, steps)
    lam = 1 - 4 * r * (np.sin(p * np.pi / (2 * (n + 1))) ** 2 + np.sin(q * np.pi / (2 * (n + 1))) ** 2)
    for k in range(steps):
        assert np.max(np.abs(out[k, 0] - lam ** (k + 1) * u0[0])) < 1e-13


def test_continuous_closed_form_second_order():
    p, q, r, t_end = 1, 2, 0.2, 0.02
    errs = []
    for n in (15, 31, 63):
        h = 1.0 / (n + 1)
        steps = int(round(t_end / (r * h * h)))
        t = steps * r * h * h
        out = heat.ftcs_run(_mode(n, p, q)[None], np.zeros((1, 4)), r, steps)
        exact = np.exp(-np.pi ** 2 * (p * p + q * q) * t) * _mode(n, p, q)
        errs.append(np.max(np.abs(out[-1, 0] - exact)))
    rates = [np.log2(errs[i] / errs[i + 1]) for i in range(2)]
    assert all(1.8 < k < 2.2 for k in rates), (errs, rates)


def test_constant_field_and_bounds_and_mirror():
    X = np.array([[300.0] * 5, [100.0, 500.0, 200.0, 400.0, 250.0], [450.0, 120.0, 480.0, 130.0, 300.0]])
    f = heat.heat_fields(X, n=12, tau=30)
    assert np.all(f[0] == np.float32(300.0))
    for s in (1, 2):
        assert f[s].min() >= X[s].min() - 1e-3 and f[s].max() <= X[s].max() + 1e-3
    Xm = X[1].copy()
    Xm[1], Xm[3] = X[1][3], X[1][1]              # swap T_x1 and T_x2
    g = heat.heat_fields(Xm[None], n=12, tau=30)
    a = f[1].reshape(30, 12, 12)
    b = g[0].reshape(30, 12, 12)
    assert np.max(np.abs(a - b[:, ::-1, :])) < 1e-3


def test_parameters_and_inputs():
    X = heat.sample_parameters(8, seed=0)
    assert X.shape == (8, 5) and X.min() >= 100 and X.max() < 500
    assert np.array_equal(X, np.random.default_rng(0).uniform(100, 500, (8, 5)))
    inp = heat.inputs_for(X, 10)
    assert inp.shape == (8, 10, 6) and inp.dtype == np.float32
    assert np.allclose(inp[:, :, 5], 0.01 * np.arange(1, 11)[None, :])


def test_sine_fields_range_and_modes():
    rng = np.random.default_rng(1)
    X = rng.uniform(100, 500, (20, 5))
    t = rng.uniform(0.01, 1.0, 20)
    f = synthetic.sine_mode_fields(X, t, n=40, seed=4)
    assert f.shape == (20, 1600) and f.dtype == np.float32
    assert f.min() >= 100 - 1e-3 and f.max() <= 500 + 1e-3
    # equal temperatures -> zero amplitude -> constant field at that temperature
    c = synthetic.sine_mode_fields(np.full((1, 5), 100.0), np.array([0.5]), n=8, seed=4)
    assert np.all(c == 100.0)


def test_hash_rows_exact():
    keys = np.array([0, 1, 12345678901])
    r = synthetic.hash_rows(keys, 70)
    for i, k in enumerate(keys):
        for c in (0, 1, 69):
            assert r[i, c] == float((int(k) * 2654435761 + c * 40503) % (1 << 24))
    assert np.all(r < 2 ** 24) and np.all(r == np.floor(r))


def test_workloads():
    w = configs.TINY
    assert w.threshold == 32 and w.n_chunks == 10 and w.chunk_rows(3) == [(s, 3) for s in range(8)]
    assert configs.HEAT100.threshold == 16667 and configs.HEAT100.n_chunks == 1000
    assert configs.FIELD1M.n_params() == 1_026_056_768
    assert configs.DEEP1M.n_params() == 2_057_407_040
    assert configs.HEAT100.n_params() == 2_637_584
