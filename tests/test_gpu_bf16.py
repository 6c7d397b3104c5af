"""Mixed-precision (bf16 operands, fp32 accumulation / master weights / Adam)
surrogate against the oracle's bf16 mode, which rounds exactly the operands the
GPU rounds (activations of layers >= 2, the weight copy, dY and every dZ) and
accumulates in fp64.  Tolerance: 2e-2 relative L2 per tensor."""
import numpy as np
import pytest
import torch

from fixtures import configs, heat
from oracle import mlp, runner

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
TOL = 2e-2


def rel(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-30))


def padded_from(arr):
    rows, d = arr.shape
    ld = (d + 7) // 8 * 8
    t = torch.zeros(rows, ld, device=DEV)[:, :d]
    t.copy_(torch.from_numpy(np.ascontiguousarray(arr, dtype=np.float32)))
    return t


def problem(widths, B, seed):
    rng = np.random.default_rng(seed)
    params = []
    for l in range(len(widths) - 1):
        fi, fo = widths[l], widths[l + 1]
        bound = 1 / np.sqrt(fi)
        params.append((rng.uniform(-bound, bound, (fo, fi)).astype(np.float32).astype(np.float64),
                       rng.uniform(-bound, bound, fo).astype(np.float32).astype(np.float64)))
    X = np.concatenate([rng.uniform(100, 500, (B, 5)), rng.uniform(0.01, 1.0, (B, 1))], axis=1)
    U = rng.uniform(100, 500, (B, widths[-1]))
    return params, X.astype(np.float32), U.astype(np.float32)


def make_gpu(widths, params, B, flags=0):
    from paper_2309_16743_amd import OT_BF16, Surrogate
    s = Surrogate(widths, precision=OT_BF16, max_batch=B, seed=0, flags=flags)
    for l, (W, b) in enumerate(params):
        s.set_params(l, W.astype(np.float32), b.astype(np.float32))
    return s


SHAPES = [
    ((6, 64, 64, 256), 32),
    ((6, 100, 77, 1001), 50),          # ragged widths, 64 x 64 tiles, partial tiles
    ((6, 256, 256, 4000), 128),        # split-K input gradient
    ((6, 128, 128, 128, 300), 64),     # three hidden layers
    ((6, 512, 512, 20000), 512),       # pipelined 256 x 128 kernel, the bf16 workloads' batch
    ((6, 512, 512, 30001), 320),       # pipelined kernel with ragged M and N (clamped edges)
    ((6, 1024, 1024, 69984), 512),     # split-K pipelined input gradient (63 splits, ragged last split)
    ((6, 2048, 2048, 2048, 4096), 1024),   # the deep 1000x1000 net's hidden widths and batch
    ((6, 16, 16, 1), 1),               # one sample, one output
    ((6, 40, 24, 9), 3),               # three samples, ragged narrow widths
]


@pytest.mark.parametrize("widths,B", SHAPES)
def test_one_train_step_bf16(widths, B):
    """Kept gradients: loss, every gradient and every parameter after Adam
    against the oracle.  Fused output-layer Adam (the default): every
    parameter against the oracle, and against the kept-gradient step within
    1e-5 (the fused GEMM never splits k, the stored one may, so the gradient
    sums can differ in rounding order)."""
    from paper_2309_16743_amd import OT_SURROGATE_KEEP_GRADS
    print(f"bf16 one train step widths={widths} B={B}", flush=True)
    params, X, U = problem(widths, B, seed=sum(widths) + B)
    s = make_gpu(widths, params, B, flags=OT_SURROGATE_KEEP_GRADS)
    f = make_gpu(widths, params, B)
    Xd, Ud = padded_from(X), padded_from(U)
    loss, loss_f = torch.zeros(1, device=DEV), torch.zeros(1, device=DEV)
    s.train_step(Xd, Ud, loss=loss)
    f.train_step(Xd, Ud, loss=loss_f)
    torch.cuda.synchronize()
    o_loss, o_grads = mlp.loss_and_grads(params, X.astype(np.float64), U.astype(np.float64), bf16=True)
    o_new = mlp.Adam(lr=1e-3).step(params, o_grads)
    assert abs(loss.item() - o_loss) / o_loss < 1e-3
    assert loss_f.item() == loss.item()
    for l in range(len(widths) - 1):
        gW, gb = s.get_grads(l)
        assert rel(gW, o_grads[l][0]) < TOL, (l, rel(gW, o_grads[l][0]))
        assert rel(gb, o_grads[l][1]) < TOL, (l, rel(gb, o_grads[l][1]))
        W, b = s.get_params(l)
        assert rel(W, o_new[l][0]) < TOL and rel(b, o_new[l][1]) < TOL
        Wf, bf = f.get_params(l)
        assert rel(Wf, o_new[l][0]) < TOL and rel(bf, o_new[l][1]) < TOL
        assert rel(Wf, W) < 1e-5 and rel(bf, b) < 1e-5, (l, rel(Wf, W))
    s.close()
    f.close()


@pytest.mark.parametrize("widths,n", [((6, 64, 64, 256), 40), ((6, 100, 77, 1001), 77)])
def test_predict_bf16(widths, n):
    params, X, _ = problem(widths, n, seed=5)
    s = make_gpu(widths, params, 32)
    Y = padded_from(np.zeros((n, widths[-1]), np.float32))
    s.predict(padded_from(X), Y)
    torch.cuda.synchronize()
    assert rel(Y.cpu().numpy(), mlp.predict(params, X.astype(np.float64), bf16=True)) < 1e-3
    s.close()


def test_tiny_workload_100_steps_bf16():
    from paper_2309_16743_amd import OT_BF16
    from paper_2309_16743_amd.online import OnlineTrainer
    w = configs.TINY
    X = heat.sample_parameters(w.n_sims, w.data_seed)
    inputs = heat.inputs_for(X, w.tau)
    fields = heat.heat_fields(X, w.grid, w.tau)
    ref = runner.run(w, inputs, fields, n_steps=100, bf16=True)
    tr = OnlineTrainer(w.widths, w.batch, w.capacity, w.threshold, w.wave, w.tau,
                       torch.from_numpy(inputs).to(DEV), torch.from_numpy(fields).to(DEV),
                       w.reservoir_seed, w.init_seed, precision=OT_BF16, lr=w.lr, record_steps=100)
    tr.run(100)
    torch.cuda.synchronize()
    slots = tr.slot_log.cpu().numpy()
    for i in range(100):
        assert np.array_equal(slots[i], ref["slots"][i]), i
    assert rel(tr.loss_log.cpu().numpy(), ref["losses"]) < TOL
    for l in range(3):
        W, b = tr.sur.get_params(l)
        assert rel(W, ref["params"][l][0]) < TOL and rel(b, ref["params"][l][1]) < TOL
    tr.close()


def test_full_width_output_rows_bf16():
    """6-1024-1024-1,000,000 at batch 512 (the 1000x1000 workload's net): one
    train step from the library's own Philox initialisation; the oracle
    recomputes, for sampled output units j, dY[:, j], dW_L[j, :], db_L[j] and the
    updated W_L[j, :] from its own initialisation of those rows."""
    from paper_2309_16743_amd import OT_BF16, OT_SURROGATE_KEEP_GRADS, Surrogate
    widths, B, seed = (6, 1024, 1024, 1_000_000), 512, 5
    rng = np.random.default_rng(11)
    X = np.concatenate([rng.uniform(100, 500, (B, 5)), rng.uniform(0.01, 1.0, (B, 1))], axis=1).astype(np.float32)
    U = rng.uniform(100, 500, (B, widths[-1])).astype(np.float32)
    s = Surrogate(widths, precision=OT_BF16, max_batch=B, seed=seed, flags=OT_SURROGATE_KEEP_GRADS)
    f = Surrogate(widths, precision=OT_BF16, max_batch=B, seed=seed)      # fused output-layer Adam
    Ud = torch.from_numpy(U).to(DEV)
    Xd = padded_from(X)
    loss = torch.zeros(1, device=DEV)
    s.train_step(Xd, Ud, loss=loss)
    f.train_step(Xd, Ud)
    torch.cuda.synchronize()
    del Ud
    # hidden layers from the oracle's own initialisation
    p_hidden = mlp.init_params(widths[:3], seed)
    Zs, As, _ = mlp.forward(p_hidden + [(np.zeros((1, widths[2])), np.zeros(1))], X.astype(np.float64), bf16=True)
    A2b = mlp.bf16_round(As[2])                          # bf16 operand of the output layer
    js = np.array([0, 1, 777, 123457, 500000, 999999])
    Wj, bj = mlp.init_rows(widths, seed, 2, js)
    Y = A2b @ mlp.bf16_round(Wj).T + bj                  # (B, len(js))
    R = Y - U[:, js].astype(np.float64)
    dY = mlp.bf16_round(2.0 * R / (B * widths[-1]))
    dWj = dY.T @ A2b
    dbj = dY.sum(axis=0)
    gW, gb = s.get_grads(2)
    assert rel(gW[js], dWj) < TOL and rel(gb[js], dbj) < TOL
    W, b = s.get_params(2)
    newW = Wj - 1e-3 * dWj / (np.abs(dWj) + 1e-8)
    assert rel(W[js], newW) < TOL
    Wf, bf = f.get_params(2)
    assert rel(Wf[js], newW) < TOL
    # neither step splits the 512-deep k range here: same sums, same Adam
    assert np.array_equal(Wf, W) and np.array_equal(bf, b)
    s.close()
    f.close()


def test_full_width_targets_in_place_bf16():
    """6-1024-1024-1,000,000 at batch 512 with the targets read in place from
    a 600-row array through row indices (the benchmark's path): the same loss
    and the same parameters, bit for bit, as the step on the gathered rows."""
    from paper_2309_16743_amd import OT_BF16, Surrogate
    widths, B, seed, n_rows = (6, 1024, 1024, 1_000_000), 512, 5, 600
    rng = np.random.default_rng(12)
    X = np.concatenate([rng.uniform(100, 500, (B, 5)), rng.uniform(0.01, 1.0, (B, 1))], axis=1).astype(np.float32)
    slab = torch.empty(n_rows, widths[-1], device=DEV)
    slab.uniform_(100, 500, generator=torch.Generator(device=DEV).manual_seed(3))
    rows = torch.from_numpy(rng.integers(0, n_rows, B).astype(np.int32)).to(DEV)
    a = Surrogate(widths, precision=OT_BF16, max_batch=B, seed=seed)
    g = Surrogate(widths, precision=OT_BF16, max_batch=B, seed=seed)
    Xd = padded_from(X)
    la, lg = torch.zeros(1, device=DEV), torch.zeros(1, device=DEV)
    a.train_step_rows(Xd, slab.data_ptr(), widths[-1], rows, n_rows, loss=la)
    gathered = slab[rows.long()]
    g.train_step(Xd, gathered, loss=lg)
    torch.cuda.synchronize()
    del gathered
    assert la.item() == lg.item()
    for l in range(3):
        Wa, ba = a.get_params(l)
        Wg, bg = g.get_params(l)
        assert np.array_equal(Wa, Wg) and np.array_equal(ba, bg), l
    a.close()
    g.close()


def test_mid_size_online_schedule_bf16():
    """A 6-512-512-19,600 bf16 net (140x140 heat fields) at batch 512 through
    the online loop as the benchmark runs it (two streams, targets read in
    place, pipelined GEMM kernels, output-layer Adam fused into its weight
    gradient), with a 700-slot reservoir so that puts evict during the run:
    10 steps, slots bit-exact, loss series and final parameters within 2e-2
    relative L2 of the oracle's bf16 mode."""
    import dataclasses
    from paper_2309_16743_amd import OT_BF16
    from paper_2309_16743_amd.online import OnlineTrainer
    w = dataclasses.replace(configs.HEAT100, grid=140, n_sims=24, wave=24, widths=(6, 512, 512, 19600),
                            precision="bf16", batch=512, capacity=700, threshold=512)
    print(f"bf16 mid-size online schedule widths={w.widths} B={w.batch} C={w.capacity}", flush=True)
    X = heat.sample_parameters(w.n_sims, w.data_seed)
    inputs = heat.inputs_for(X, w.tau)
    fields = heat.heat_fields(X, w.grid, w.tau)
    n = 10
    ref = runner.run(w, inputs, fields, n_steps=n)
    tr = OnlineTrainer(w.widths, w.batch, w.capacity, w.threshold, w.wave, w.tau,
                       torch.from_numpy(inputs).to(DEV), torch.from_numpy(fields).to(DEV),
                       w.reservoir_seed, w.init_seed, precision=OT_BF16, lr=w.lr, record_steps=n, overlap=True)
    tr.run(n)
    torch.cuda.synchronize()
    assert tr.res.stats()["total_evicted"] > 0
    slots = tr.slot_log.cpu().numpy()
    for i in range(n):
        assert np.array_equal(slots[i], ref["slots"][i]), i
    assert rel(tr.loss_log.cpu().numpy(), ref["losses"]) < TOL
    for l in range(3):
        W, b = tr.sur.get_params(l)
        assert rel(W, ref["params"][l][0]) < TOL and rel(b, ref["params"][l][1]) < TOL
    tr.close()
