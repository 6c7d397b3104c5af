"""Pins of the oracle's surrogate: loss, gradients, Adam, bf16 rounding, init.

* gradients: central finite differences of the fp64 loss on tiny nets, at
  points kept away from ReLU kinks; and torch fp64 autograd of the same net;
* Adam: the step-1 closed form (m_hat = g, v_hat = g^2, so the update is
  -lr * g / (|g| + eps)), and 100 steps against torch.optim.Adam in fp64;
* MSE: hand-computed values;
* bf16 rounding: hand cases at ties and against torch's bfloat16 conversion.
"""
import numpy as np
import pytest
import torch

from oracle import mlp


def tiny_problem(widths=(6, 5, 4, 3), b=4, seed=0):
    rng = np.random.default_rng(seed)
    params = [(rng.normal(size=(widths[l + 1], widths[l])), rng.normal(size=widths[l + 1]))
              for l in range(len(widths) - 1)]
    X = rng.normal(size=(b, widths[0]))
    U = rng.normal(size=(b, widths[-1]))
    return params, X, U


def test_mse_hand_values():
    Y = np.array([[1.0, 2.0, 3.0], [0.0, -1.0, 4.0]])
    U = np.array([[1.0, 0.0, 1.0], [1.0, 1.0, 1.0]])
    # residuals 0,2,2,-1,-2,3 -> squares 0,4,4,1,4,9 = 22 over 6 entries
    assert mlp.mse(Y, U) == pytest.approx(22.0 / 6.0, rel=0, abs=1e-15)
    params = [(np.array([[1.0, 0.0], [0.0, 2.0]]), np.array([0.5, -1.0]))]
    loss, grads = mlp.loss_and_grads(params, np.array([[1.0, 1.0]]), np.array([[0.0, 0.0]]))
    # Y = (1.5, 1.0): loss (2.25 + 1)/2 ; dY = 2R/2 = R -> dW = R^T x, db = R
    assert loss == pytest.approx(1.625, abs=1e-15)
    assert np.allclose(grads[0][1], [1.5, 1.0]) and np.allclose(grads[0][0], [[1.5, 1.5], [1.0, 1.0]])


def _away_from_kinks(params, X, margin):
    Zs, _, _ = mlp.forward(params, X)
    return all(np.min(np.abs(Z)) > margin for Z in Zs[:-1])


@pytest.mark.parametrize("widths,seed", [((6, 5, 4, 3), 0), ((6, 7, 7, 2), 1), ((3, 4, 5, 6, 2), 2)])
def test_gradients_central_differences(widths, seed):
    for s in range(seed, seed + 50):
        params, X, U = tiny_problem(widths, seed=s)
        if _away_from_kinks(params, X, 1e-3):
            break
    else:
        pytest.fail("no kink-free draw")
    loss, grads = mlp.loss_and_grads(params, X, U)
    for l, (W, b) in enumerate(params):
        for which, P in ((0, W), (1, b)):
            num = np.zeros_like(P)
            for idx in np.ndindex(P.shape):
                h = 1e-6 * max(1.0, abs(P[idx]))
                old = P[idx]
                P[idx] = old + h
                lp = mlp.mse(mlp.forward(params, X)[2], U)
                P[idx] = old - h
                lm = mlp.mse(mlp.forward(params, X)[2], U)
                P[idx] = old
                num[idx] = (lp - lm) / (2 * h)
            ana = grads[l][which]
            err = np.linalg.norm(ana - num) / max(np.linalg.norm(num), 1e-30)
            assert err < 1e-6, (l, which, err)


def test_finite_differences_catch_a_dropped_mask():
    """Planted mistake: back-propagating through ReLU without its mask must fail the FD check."""
    params, X, U = tiny_problem((6, 5, 4, 3), seed=3)
    Zs, As, Y = mlp.forward(params, X)
    dY = 2 * (Y - U) / U.size
    dA = dY @ params[2][0]
    wrong_dW1 = dA.T @ As[1]                  # missing (Z > 0)
    _, grads = mlp.loss_and_grads(params, X, U)
    assert not np.allclose(wrong_dW1, grads[1][0])


def test_against_torch_autograd_fp64():
    params, X, U = tiny_problem((6, 16, 16, 9), b=7, seed=5)
    loss, grads = mlp.loss_and_grads(params, X, U)
    tp = [(torch.tensor(W, requires_grad=True), torch.tensor(b, requires_grad=True)) for W, b in params]
    a = torch.tensor(X)
    for l, (W, b) in enumerate(tp):
        a = a @ W.T + b
        if l < len(tp) - 1:
            a = torch.relu(a)
    tl = torch.nn.functional.mse_loss(a, torch.tensor(U))
    tl.backward()
    assert abs(tl.item() - loss) < 1e-12 * max(1.0, abs(loss))
    for (W, b), (gW, gb) in zip(tp, grads):
        assert np.allclose(W.grad.numpy(), gW, rtol=1e-12, atol=1e-14)
        assert np.allclose(b.grad.numpy(), gb, rtol=1e-12, atol=1e-14)


def test_adam_step_one_closed_form():
    params, X, U = tiny_problem(seed=7)
    loss, grads = mlp.loss_and_grads(params, X, U)
    opt = mlp.Adam(lr=1e-3)
    new = opt.step(params, grads)
    for (W, b), (gW, gb), (nW, nb) in zip(params, grads, new):
        assert np.allclose(nW - W, -1e-3 * gW / (np.abs(gW) + 1e-8), rtol=1e-12, atol=1e-18)
        assert np.allclose(nb - b, -1e-3 * gb / (np.abs(gb) + 1e-8), rtol=1e-12, atol=1e-18)


def test_adam_100_steps_against_torch():
    params, X, U = tiny_problem((6, 8, 8, 5), b=6, seed=9)
    rng = np.random.default_rng(1)
    opt = mlp.Adam(lr=1e-3)
    tp = [torch.tensor(p.copy(), requires_grad=True) for W, b in params for p in (W, b)]
    topt = torch.optim.Adam(tp, lr=1e-3, betas=(0.9, 0.999), eps=1e-8)
    for step in range(100):
        g = [(rng.normal(size=W.shape), rng.normal(size=b.shape)) for W, b in params]
        params = opt.step(params, g)
        for t, gg in zip(tp, [x for pair in g for x in pair]):
            t.grad = torch.tensor(gg)
        topt.step()
    ours = [x for pair in params for x in pair]
    for a, t in zip(ours, tp):
        assert np.max(np.abs(a - t.detach().numpy())) < 1e-12


def test_bf16_round_cases():
    one = 1.0
    ulp = 2.0 ** -7                                           # bf16 spacing at 1
    vals = np.array([one, one + ulp / 2, one + 3 * ulp / 2, one + ulp / 4, one + 3 * ulp / 4, -2.5, 0.0, 3e38])
    exp = np.array([one, one, one + 2 * ulp, one, one + ulp, -2.5, 0.0, None], dtype=object)
    got = mlp.bf16_round(vals)
    for g, e in zip(got[:-1], exp[:-1]):
        assert g == e                                          # ties to even, below/above half
    rng = np.random.default_rng(0)
    x = (rng.normal(size=10000) * 10.0 ** rng.integers(-8, 8, 10000)).astype(np.float32)
    ref = torch.tensor(x).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(mlp.bf16_round(x.astype(np.float64)), ref)


def test_init_params_bounds_and_rows():
    widths = (6, 33, 17, 40)
    params = mlp.init_params(widths, seed=3)
    for l, (W, b) in enumerate(params):
        bound = 1 / np.sqrt(widths[l])
        assert W.shape == (widths[l + 1], widths[l]) and b.shape == (widths[l + 1],)
        assert np.max(np.abs(W)) <= bound and np.max(np.abs(b)) <= bound
        assert np.all(W.astype(np.float32).astype(np.float64) == W)
    rows = np.array([0, 5, 39])
    Wr, br = mlp.init_rows(widths, 3, 2, rows)
    assert np.array_equal(Wr, params[2][0][rows]) and np.array_equal(br, params[2][1][rows])
