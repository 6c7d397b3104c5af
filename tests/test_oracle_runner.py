"""The oracle's online loop on the 16x16 workload, and the oracle's isolation."""
import ast
import os

import numpy as np

from fixtures import configs, heat
from oracle import mlp, runner

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def tiny_data():
    w = configs.TINY
    X = heat.sample_parameters(w.n_sims, w.data_seed)
    return w, heat.inputs_for(X, w.tau), heat.heat_fields(X, w.grid, w.tau)


def test_tiny_schedule_and_learning():
    w, inputs, fields = tiny_data()
    tr = runner.run(w, inputs, fields, n_steps=100)
    res = tr["reservoir"]
    res.check_invariants()
    # first batch once N = 40 > T = 32 (iteration 4); chunks 8 and 9 replace seen items
    assert tr["tickets"][0] == 5                      # 5 puts took tickets 0..4
    assert res.total_put == 80 and res.total_evicted == 16 and res.N == 64
    assert tr["iterations"] == 104
    assert len(tr["losses"]) == 100
    assert np.mean(tr["losses"][-10:]) < 0.5 * np.mean(tr["losses"][:10])


def test_oracle_never_imports_the_gpu_package():
    """The oracle imports nothing of the HIP path; where it uses torch (CPU
    fp64 products of the column-chunked output layer) it never places a
    tensor on a device."""
    for fn in os.listdir(os.path.join(ROOT, "oracle")):
        if not fn.endswith(".py"):
            continue
        src = open(os.path.join(ROOT, "oracle", fn)).read()
        tree = ast.parse(src)
        for node in ast.walk(tree):
            names = []
            if isinstance(node, ast.Import):
                names = [a.name for a in node.names]
            elif isinstance(node, ast.ImportFrom):
                names = [node.module or ""]
            for n in names:
                assert not n.startswith("paper_2309_16743_amd"), (fn, n)
                assert n in ("torch",) or not n.startswith("torch"), (fn, n)
        assert "cuda" not in src and "device" not in src, fn


def test_halving_schedule_closed_form():
    """Sec. 4.5: 1e-3 halved every 10,000 trained samples, floored at 2.5e-4."""
    lr = lambda n: runner.halving_lr(1e-3, n, 10_000, 2.5e-4)
    assert [lr(n) for n in (0, 9_999, 10_000, 19_999, 20_000, 30_000, 10**6)] == \
        [1e-3, 1e-3, 5e-4, 5e-4, 2.5e-4, 2.5e-4, 2.5e-4]
    from paper_2309_16743_amd.online import HalvingLR      # the trainer's schedule, same printed values
    h = HalvingLR()
    assert [h(n) for n in (0, 9_999, 10_000, 20_000, 10**6)] == [1e-3, 1e-3, 5e-4, 2.5e-4, 2.5e-4]


def test_schedule_validation_and_repetition_histogram():
    w, inputs, fields = tiny_data()
    Xv = heat.sample_parameters(2, 99)
    iv, fv = heat.inputs_for(Xv, w.tau).reshape(-1, 6), heat.heat_fields(Xv, w.grid, w.tau).reshape(-1, 256)
    tr = runner.run(w, inputs, fields, n_steps=100, lr_halving=(640, 2.5e-4), validation=(iv, fv, 25))
    # 32 samples per step: the rate halves after steps 20 and 40, then stays at the floor
    assert tr["lrs"][:21] == [1e-3] * 20 + [5e-4] and tr["lrs"][40:] == [2.5e-4] * 60
    assert sorted(tr["val_losses"]) == [25, 50, 75, 100]
    assert all(np.isfinite(v) and v > 0 for v in tr["val_losses"].values())
    # validation follows the step it is taken at: the last one sees the final parameters
    assert tr["val_losses"][100] == mlp.mse(mlp.predict(tr["params"], iv), fv)
    res = tr["reservoir"]
    h = runner.repetition_histogram(res, 256)
    assert h.sum() == res.total_put                                  # every sample that entered, once
    assert int((np.arange(256) * h).sum()) == res.total_draws       # every draw, once


def test_run_to_drain_uses_every_sample_once_with_fifo_and_firo():
    """FIFO and FIRO through the whole 16x16 schedule and the drain: every
    produced sample is trained on exactly once (the slots of each sample id
    are never repeated), batches are full except possibly the last, and the
    Reservoir trains on more batches from the same production."""
    from oracle.buffers import FIFOBuffer, FIROBuffer
    from oracle.reservoir import Reservoir
    w, inputs, fields = tiny_data()
    n = w.n_chunks * w.wave
    res = {}
    for name, cls in (("fifo", FIFOBuffer), ("firo", FIROBuffer), ("reservoir", Reservoir)):
        buf = cls(w.capacity, w.threshold, inputs.shape[-1], fields.shape[-1], w.reservoir_seed)
        tr = runner.run_to_drain(w, inputs, fields, buf)
        res[name] = tr
        assert all(np.isfinite(tr["losses"]))
        if name != "reservoir":
            assert sum(tr["sizes"]) == n
            assert all(s == w.batch for s in tr["sizes"][:-1])
            assert buf.total_draws == n and buf.N == 0
    assert len(res["reservoir"]["losses"]) > len(res["fifo"]["losses"])
