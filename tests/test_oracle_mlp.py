"""Pins of the oracle's surrogate: loss, gradients, Adam, bf16 rounding, init.

* gradients: central finite differences of the fp64 loss on tiny nets, at
  points kept away from ReLU kinks; and torch fp64 autograd of the same net;
* Adam: the step-1 closed form (m_hat = g, v_hat = g^2, so the update is
  -lr * g / (|g| + eps)), and 100 steps against torch.optim.Adam in fp64;
* MSE: hand-computed values;
* bf16 rounding: hand cases at ties and against torch's bfloat16 conversion;
* bf16 mode: a hand-worked example in which each rounding point of the
  mixed-precision reading changes the result (planted misplacements of those
  points must fail it), equality with fp64 mode where every value is
  bf16-representable, and closeness to fp64 mode on a workload-shaped net.
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


# ---- bf16 mode (the mixed-precision reading of Sec. 4.1's bf16 workloads) ---------------
#
# A one-hidden-layer net, batch 1, input width 1, two hidden units (the second
# dead), one output, worked by hand.  bf16 has 8 significant bits; in [1, 2)
# its spacing is u = 2^-7 = 0.0078125, in [0.5, 1) it is 2^-8.
#   x = 1.005859375 = 1 + 0.75u            (bf16: 1.0078125; layer 1 is fp32, so unrounded)
#   W1 = [[1], [-1]], b1 = [0.25, 0]       -> Z1 = [1.255859375, -1.005859375]
#   A1 = [1.255859375, 0]                  -> bf16(A1) = [1.2578125, 0]   (32.75u -> 33u)
#   W2 = [[1.005859375, 5]], b2 = [0]      -> bf16(W2) = [[1.0078125, 5]]
#   Y = 1.2578125 * 1.0078125 = 1.26763916015625
#   U = 0.5166015625 (bf16 would give 0.515625; targets stay fp32)
#   R = Y - U = 0.75103759765625; loss = R^2 (B D = 1) = 151413025 / 2^28
#   dY = 2R = 1.5020751953125              -> bf16 1.5    (64.27u -> 64u)
#   db2 = 1.5 (sum of the rounded dY)
#   dW2 = dY * bf16(A1) = [1.5 * 1.2578125, 0] = [1.88671875, 0]
#   dA1 = dY * bf16(W2) = [1.51171875, 7.5]; mask [1, 0] -> [1.51171875, 0]
#   dZ1 = bf16 -> 1.515625                 (65.5u: a tie, to even 66u)
#   dW1 = dZ1 * x = 1.515625 * 1.005859375 = 1.524505615234375; db1 = [1.515625, 0]
HAND_PARAMS = [(np.array([[1.0], [-1.0]]), np.array([0.25, 0.0])),
               (np.array([[1.005859375, 5.0]]), np.array([0.0]))]
HAND_X = np.array([[1.005859375]])
HAND_U = np.array([[0.5166015625]])
HAND_LOSS = 151413025 / 2 ** 28
HAND_GRADS = [(np.array([[1.524505615234375], [0.0]]), np.array([1.515625, 0.0])),
              (np.array([[1.88671875, 0.0]]), np.array([1.5]))]


def _hand_result(rounded=None):
    loss, grads = mlp.loss_and_grads(HAND_PARAMS, HAND_X, HAND_U, bf16=True, rounded=rounded)
    return loss, grads


def _equals_hand(loss, grads):
    return loss == HAND_LOSS and all(np.array_equal(g[i], h[i]) for g, h in zip(grads, HAND_GRADS)
                                     for i in range(2))


def test_bf16_hand_worked_one_hidden_layer():
    loss, grads = _hand_result()
    assert loss == HAND_LOSS
    for (dW, db), (hW, hb) in zip(grads, HAND_GRADS):
        assert np.array_equal(dW, hW) and np.array_equal(db, hb)
    Y = mlp.predict(HAND_PARAMS, HAND_X, bf16=True)
    assert Y[0, 0] == 1.26763916015625
    # fp64 mode on the same net gives other values: every rounding is visible here
    loss64, grads64 = mlp.loss_and_grads(HAND_PARAMS, HAND_X, HAND_U)
    assert loss64 != HAND_LOSS and not np.array_equal(grads64[0][0], HAND_GRADS[0][0])


# Each plant moves one rounding point of the bf16 reading; the quantities the
# hand example says it changes must change.
PLANTED = {
    "no dZ rounding": (mlp.BF16_ROUNDED - {"dZ"}, "dW1 from 1.51171875 instead of 1.515625"),
    "no dY rounding": (mlp.BF16_ROUNDED - {"dY"}, "db2 = 1.5020751953125"),
    "no activation rounding": (mlp.BF16_ROUNDED - {"act"}, "Y from A1 = 1.255859375"),
    "no weight rounding": (mlp.BF16_ROUNDED - {"weight"}, "Y from W2 = 1.005859375"),
    "rounded layer-1 input": (mlp.BF16_ROUNDED | {"input"}, "dW1 = 1.515625 * 1.0078125"),
    "rounded targets": (mlp.BF16_ROUNDED | {"target"}, "R from U = 0.515625"),
    "db from unrounded dY": (mlp.BF16_ROUNDED | {"db_raw"}, "db2 = 1.5020751953125"),
}


@pytest.mark.parametrize("name", sorted(PLANTED))
def test_bf16_planted_rounding_mistakes_fail_the_hand_example(name):
    rounded, what = PLANTED[name]
    loss, grads = _hand_result(rounded)
    assert not _equals_hand(loss, grads), f"{name} ({what}) not detected"


def test_bf16_planted_mistakes_hit_the_predicted_quantity():
    _, g = _hand_result(PLANTED["no dZ rounding"][0])
    assert g[0][0][0, 0] == 1.51171875 * 1.005859375
    assert np.array_equal(g[1][0], HAND_GRADS[1][0]) and np.array_equal(g[1][1], HAND_GRADS[1][1])
    _, g = _hand_result(PLANTED["rounded layer-1 input"][0])
    assert g[0][0][0, 0] == 1.515625 * 1.0078125
    _, g = _hand_result(PLANTED["db from unrounded dY"][0])
    assert g[1][1][0] == 1.5020751953125 and np.array_equal(g[1][0], HAND_GRADS[1][0])
    loss, _ = _hand_result(PLANTED["rounded targets"][0])
    assert loss == (1.26763916015625 - 0.515625) ** 2
    loss, _ = _hand_result(PLANTED["no activation rounding"][0])
    assert loss == (1.255859375 * 1.0078125 - 0.5166015625) ** 2


def _bf16_exact(v):
    return np.array_equal(mlp.bf16_round(v), v)


def test_bf16_mode_equals_fp64_when_every_value_is_representable():
    """Small-integer nets with B*D a power of two: every operand, product sum
    and gradient is exact in bf16 and in fp64, so the two modes agree bit for
    bit (a dropped term, a wrong scale or an extra rounding would differ)."""
    rng = np.random.default_rng(11)
    checked = 0
    for trial in range(400):
        widths = (3, 4, 4, 2)
        b = 4                                   # B * D = 8
        params = [(rng.integers(-1, 2, size=(widths[l + 1], widths[l])).astype(np.float64),
                   rng.integers(-2, 3, size=widths[l + 1]).astype(np.float64)) for l in range(3)]
        X = rng.integers(0, 4, size=(b, widths[0])).astype(np.float64)
        U = rng.integers(-8, 9, size=(b, widths[-1])).astype(np.float64)
        Zs, As, Y = mlp.forward(params, X)
        loss64, g64 = mlp.loss_and_grads(params, X, U)
        R = Y - U
        dY = 2.0 * R / R.size
        dA = dY @ params[2][0]
        dZ2 = dA * (Zs[1] > 0)
        dZ1 = (dZ2 @ params[1][0]) * (Zs[0] > 0)
        values = list(Zs) + list(As) + [dY, dA, dZ2, dZ1] + [a for pair in g64 for a in pair]
        if not all(_bf16_exact(v) for v in values) or np.count_nonzero(R) == 0 or np.count_nonzero(dZ1) == 0:
            continue
        loss, g = mlp.loss_and_grads(params, X, U, bf16=True)
        assert loss == loss64
        for (a, c), (d, e) in zip(g, g64):
            assert np.array_equal(a, d) and np.array_equal(c, e)
        checked += 1
        if checked == 20:
            break
    assert checked == 20


def test_bf16_mode_close_to_fp64():
    """bf16 against pure fp64 on a net shaped like the 16x16 workload (values
    ~1e2 like the paper's temperatures): one bf16 rounding is <= 2^-9
    relative, so per-tensor relative L2 differences of a few 2^-8 at most."""
    widths = (6, 64, 64, 256)
    params = mlp.init_params(widths, seed=1)
    rng = np.random.default_rng(3)
    X = np.concatenate([rng.uniform(100, 500, (32, 5)), rng.uniform(0.01, 0.1, (32, 1))], axis=1)
    U = rng.uniform(100, 500, (32, 256))
    loss, g = mlp.loss_and_grads(params, X, U, bf16=True)
    loss64, g64 = mlp.loss_and_grads(params, X, U)
    rels = [abs(loss - loss64) / loss64]
    for (a, c), (d, e) in zip(g, g64):
        rels += [np.linalg.norm(a - d) / np.linalg.norm(d), np.linalg.norm(c - e) / np.linalg.norm(e)]
    print("bf16 vs fp64 relative L2 (loss, dW1, db1, dW2, db2, dW3, db3):", ["%.2e" % r for r in rels])
    assert max(rels) < 2e-2
    assert rels[0] > 0                         # the modes do differ


# ---- the output layer by column chunks (full-width parity checks use it) -------------------
def test_bf16_round_torch_equals_bf16_round():
    rng = np.random.default_rng(4)
    x = rng.normal(size=200000) * 10.0 ** rng.integers(-20, 20, 200000)
    ulp = 2.0 ** -7
    ties = np.array([1 + ulp / 2, 1 + 3 * ulp / 2, -(1 + ulp / 2), 3 * (1 + ulp / 2), 0.0, -0.0])
    for v in (x, ties):
        got = mlp.bf16_round_torch(torch.from_numpy(v)).numpy()
        assert np.array_equal(got, mlp.bf16_round(v))


@pytest.mark.parametrize("bf16,rounded", [(False, None), (True, None), (True, mlp.BF16_ROUNDED - {"dY"}),
                                          (True, mlp.BF16_ROUNDED | {"db_raw", "target"})])
def test_output_layer_by_columns_equals_loss_and_grads(bf16, rounded):
    """Column chunks (ragged last chunk) + hidden_grads reproduce loss_and_grads:
    loss, every hidden gradient, the output bias gradient and sampled output
    weight-gradient rows, up to the order of fp64 sums; with planted rounding
    points too, so the chunked path honours each point."""
    widths, B = (6, 40, 32, 1000), 24
    rng = np.random.default_rng(8)
    params = [(rng.uniform(-0.3, 0.3, (widths[l + 1], widths[l])), rng.uniform(-0.3, 0.3, widths[l + 1]))
              for l in range(3)]
    X = np.concatenate([rng.uniform(100, 500, (B, 5)), rng.uniform(0.01, 1, (B, 1))], axis=1)
    U = rng.uniform(100, 500, (B, widths[-1]))
    loss, grads = mlp.loss_and_grads(params, X, U, bf16=bf16, rounded=rounded)
    Zs, As, Ah = mlp.forward(params[:2], X, bf16=bf16, rounded=rounded)
    A_top = np.maximum(Ah, 0.0)
    W3, b3 = params[2]
    rows = np.array([0, 5, 128, 999])
    l2, dA, db, dWr = mlp.output_layer_by_columns(A_top, lambda a, b: W3[a:b], b3, lambda a, b: U[:, a:b],
                                                  widths[-1], 128, bf16=bf16, rows=rows, rounded=rounded)
    assert abs(l2 - loss) <= 1e-12 * loss
    assert np.allclose(db, grads[2][1], rtol=1e-12, atol=1e-18)
    assert np.allclose(dWr, grads[2][0][rows], rtol=1e-12, atol=1e-18)
    hg = mlp.hidden_grads(params[:2], Zs, dA, As, bf16=bf16, rounded=rounded)
    for (a, c), (d, e) in zip(hg, grads[:2]):
        assert np.allclose(a, d, rtol=1e-10, atol=1e-16) and np.allclose(c, e, rtol=1e-10, atol=1e-16)


def test_adam_fp32_state_rounds_only_what_it_stores():
    """state_dtype=float32: parameters and moments are fp32 values after a
    step, each the fp64 step's result rounded once; fp64 mode is unchanged."""
    params, X, U = tiny_problem((6, 8, 8, 5), b=6, seed=13)
    params = [(W.astype(np.float32).astype(np.float64), b.astype(np.float32).astype(np.float64)) for W, b in params]
    a64, a32 = mlp.Adam(lr=1e-3), mlp.Adam(lr=1e-3, state_dtype=np.float32)
    p64, p32 = params, params
    for _ in range(3):
        _, g = mlp.loss_and_grads(p64, X, U)
        q64 = a64.step(p64, g)
        m_prev, v_prev = [tuple(x.copy() for x in t) for t in a32.m] or None, [tuple(x.copy() for x in t) for t in a32.v] or None
        q32 = a32.step(p32, mlp.loss_and_grads(p32, X, U)[1])
        for pair in q32 + a32.m + a32.v:
            for x in pair:
                assert np.array_equal(x.astype(np.float32).astype(np.float64), x)
        p64, p32 = q64, q32
    # one step from the same fp32 state: the rounded result is the fp64 result rounded
    b64, b32 = mlp.Adam(lr=1e-3), mlp.Adam(lr=1e-3, state_dtype=np.float32)
    _, g = mlp.loss_and_grads(params, X, U)
    r64, r32 = b64.step(params, g), b32.step(params, g)
    for (W64, c64), (W32, c32) in zip(r64, r32):
        assert np.array_equal(W64.astype(np.float32).astype(np.float64), W32)
        assert np.array_equal(c64.astype(np.float32).astype(np.float64), c32)
