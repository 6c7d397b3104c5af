"""The oracle's online loop on the 16x16 workload, and the oracle's isolation."""
import ast
import os

import numpy as np

from fixtures import configs, heat
from oracle import runner

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
    for fn in os.listdir(os.path.join(ROOT, "oracle")):
        if not fn.endswith(".py"):
            continue
        tree = ast.parse(open(os.path.join(ROOT, "oracle", fn)).read())
        for node in ast.walk(tree):
            names = []
            if isinstance(node, ast.Import):
                names = [a.name for a in node.names]
            elif isinstance(node, ast.ImportFrom):
                names = [node.module or ""]
            for n in names:
                assert not n.startswith("paper_2309_16743_amd"), (fn, n)
                assert not n.startswith("torch"), (fn, n)
