"""Fully-connected surrogate, MSE loss, back-propagation and Adam (oracle side, fp64).

What the paper fixes (Sec. 4.1): the direct surrogate maps the 6 inputs (X, t)
to the whole field u_X^t (Eq. 1 and Sec. 2); it is a multilayer perceptron
with ReLU hidden layers trained with Adam at learning rate 1e-3; the training
and validation metric is the mean squared error (Sec. 4.4-4.6).

Readings where the paper is silent (each is listed with its reason in the
design notes):
  * the output layer is the identity (a field of temperatures, no squashing);
  * the loss is the mean of (Y - U)^2 over all B*D entries;
  * Adam (Kingma and Ba, 2015, Algorithm 1) with beta1 = 0.9, beta2 = 0.999,
    eps = 1e-8, bias correction, no weight decay, t counted from 1;
  * ReLU'(0) = 0;
  * weights W_l are stored out x in, row-major; Z_l = A_{l-1} W_l^T + b_l;
  * initialisation U(-1/sqrt(fan_in), +1/sqrt(fan_in)) for W and b, drawn from
    Philox4x64-10 (kind INIT, counter (e, layer), e = flat index over W then b)
    and rounded to fp32.

bf16 mode mirrors the rounding points of the mixed-precision path: layer 1
(K = 6 raw inputs) stays fp32 in the forward pass; the operands of every other
forward GEMM (activations A_{l-1}, the bf16 copy of W_l) are rounded to bf16
(round to nearest even from fp32); the output-layer gradient dY is rounded to
bf16 before the backward GEMMs, as is every back-propagated dZ_l; bias
gradients are sums of those rounded values; Adam works on fp32 master weights
and fp32 gradients.  All accumulation here is fp64.  The rounding points are
named (BF16_ROUNDED below) so that a test can switch one of them, which is how
the tests plant a misplaced rounding point in this module.

Pins: central finite differences of the loss on tiny nets, torch fp64
autograd of the same net, Adam's step-1 closed form (-lr * sign(g) up to eps),
hand-computed MSE values; bf16 mode: a hand-worked one-hidden-layer example
in which every rounding point changes the result, equality with fp64 mode on
nets whose values are all bf16-representable, and closeness to fp64 mode.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Tuple

import numpy as np

from .philox import init_uniform_vec

Params = List[Tuple[np.ndarray, np.ndarray]]


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round to bf16 (8 significant bits), nearest-even, via the fp32 value; fp64 out.

    An fp32 bit pattern keeps its top 16 bits after adding 0x7FFF plus the
    lowest kept bit (round half to even); NaN is not expected here.
    """
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    bits = f.view(np.uint32).astype(np.uint64)
    lsb = (bits >> np.uint64(16)) & np.uint64(1)
    rounded = ((bits + np.uint64(0x7FFF) + lsb) >> np.uint64(16)) << np.uint64(16)
    return rounded.astype(np.uint32).view(np.float32).astype(np.float64)


def init_params(widths, seed: int) -> Params:
    """Seeded U(+-1/sqrt(fan_in)) initialisation, fp32 values held in fp64."""
    params: Params = []
    for l in range(len(widths) - 1):
        fan_in, fan_out = widths[l], widths[l + 1]
        n_w = fan_out * fan_in
        e = np.arange(n_w + fan_out, dtype=np.uint64)
        bound = 1.0 / np.sqrt(float(fan_in))
        vals = (init_uniform_vec(seed, e, l) * bound).astype(np.float32).astype(np.float64)
        params.append((vals[:n_w].reshape(fan_out, fan_in).copy(), vals[n_w:].copy()))
    return params


def init_rows(widths, seed: int, layer: int, rows) -> Tuple[np.ndarray, np.ndarray]:
    """Initial W[rows, :] and b[rows] of one layer without materialising the layer."""
    fan_in, fan_out = widths[layer], widths[layer + 1]
    rows = np.asarray(rows, dtype=np.int64)
    bound = 1.0 / np.sqrt(float(fan_in))
    e = (rows[:, None] * fan_in + np.arange(fan_in)[None, :]).reshape(-1).astype(np.uint64)
    w = (init_uniform_vec(seed, e, layer) * bound).astype(np.float32).astype(np.float64)
    eb = (fan_out * fan_in + rows).astype(np.uint64)
    b = (init_uniform_vec(seed, eb, layer) * bound).astype(np.float32).astype(np.float64)
    return w.reshape(len(rows), fan_in), b


# Rounding points of bf16 mode (the mixed-precision reading of Sec. 4.1's
# "bf16 GEMMs with fp32 master weights"):
#   "act"    - activations A_l (l >= 1) where a GEMM reads them (the forward of
#              layer l + 1 and the weight gradient of layer l + 1);
#   "weight" - the bf16 copy of W_l (l >= 2) read by the forward and by the
#              input gradient;
#   "dY"     - the output gradient 2 (Y - U) / (B D);
#   "dZ"     - every back-propagated dZ_l (after the ReLU mask).
# Bias gradients are column sums of the rounded dY / dZ.  Points that bf16 mode
# leaves unrounded, named only so that a test can plant them as mistakes:
#   "input"  - layer 1's input X and W_1 (layer 1 runs in fp32);
#   "target" - the targets U;
#   "db_raw" - bias gradients summed from dY / dZ before rounding.
BF16_ROUNDED = frozenset({"act", "weight", "dY", "dZ"})


def _rounder(bf16: bool, rounded):
    points = (BF16_ROUNDED if rounded is None else frozenset(rounded)) if bf16 else frozenset()

    def rnd(point: str, v: np.ndarray) -> np.ndarray:
        return bf16_round(v) if point in points else v
    return rnd, points


def forward(params: Params, X: np.ndarray, bf16: bool = False, rounded=None):
    """Return (Zs, As, Y): pre-activations, activations (As[0] = X), output.

    rounded: the bf16 rounding points (default BF16_ROUNDED; tests only)."""
    rnd, _ = _rounder(bf16, rounded)
    A = np.asarray(X, dtype=np.float64)
    As, Zs = [A], []
    L = len(params)
    for l, (W, b) in enumerate(params):
        if l > 0:
            Z = rnd("act", A) @ rnd("weight", W).T + b
        else:
            Z = rnd("input", A) @ rnd("input", W).T + b
        Zs.append(Z)
        if l < L - 1:
            A = np.maximum(Z, 0.0)
            As.append(A)
    return Zs, As, Zs[-1]


def mse(Y: np.ndarray, U: np.ndarray) -> float:
    """Mean over all entries of (Y - U)^2."""
    R = np.asarray(Y, dtype=np.float64) - np.asarray(U, dtype=np.float64)
    return float(np.sum(R * R) / R.size)


def loss_and_grads(params: Params, X: np.ndarray, U: np.ndarray, bf16: bool = False, rounded=None):
    """MSE loss and its gradients with respect to every W_l and b_l.

    rounded: the bf16 rounding points (default BF16_ROUNDED; tests only)."""
    rnd, points = _rounder(bf16, rounded)
    Zs, As, Y = forward(params, X, bf16=bf16, rounded=rounded)
    U = rnd("target", np.asarray(U, dtype=np.float64))
    R = Y - U
    loss = float(np.sum(R * R) / R.size)
    dZ_raw = 2.0 * R / R.size                 # dLoss/dY
    dZ = rnd("dY", dZ_raw)
    return loss, _backprop(params, Zs, As, dZ, dZ_raw, rnd, points)


def _backprop(params: Params, Zs, As, dZ, dZ_raw, rnd, points) -> Params:
    """Gradients of every layer of `params`, from dLoss/dZ of the last one
    (dZ as the GEMMs read it, dZ_raw before rounding), layer by layer down."""
    L = len(params)
    grads: Params = [None] * L                # type: ignore[list-item]
    for l in range(L - 1, -1, -1):
        W = params[l][0]
        A_in = rnd("act", As[l]) if l > 0 else rnd("input", As[l])
        dW = dZ.T @ A_in
        db = (dZ_raw if "db_raw" in points else dZ).sum(axis=0)
        grads[l] = (dW, db)
        if l > 0:
            dA = dZ @ rnd("weight", W)
            dZ_raw = dA * (Zs[l - 1] > 0.0)
            dZ = rnd("dZ", dZ_raw)
    return grads


def hidden_grads(params: Params, Zs, dA: np.ndarray, As, bf16: bool = False, rounded=None) -> Params:
    """Gradients of the hidden layers `params` given dLoss/dA of the last of
    them: the part of loss_and_grads below the output layer, for callers that
    form the output layer's input gradient dA themselves (by column chunks at
    full output width, output_layer_by_columns).  Zs, As: forward(params, X)
    of the hidden layers alone (Zs[-1] is the last hidden pre-activation)."""
    rnd, points = _rounder(bf16, rounded)
    dZ_raw = np.asarray(dA, dtype=np.float64) * (Zs[-1] > 0.0)
    return _backprop(params, Zs, As, rnd("dZ", dZ_raw), dZ_raw, rnd, points)


def output_layer_by_columns(A_in: np.ndarray, weight_rows, bias: np.ndarray, target_cols, D: int, chunk: int,
                            bf16: bool = False, rows=(), rounded=None):
    """The output layer's share of loss_and_grads, formed over column chunks
    of the D outputs so that a 10^6-wide layer need not be held at once:
    A_in (B x H) is the last hidden activation (before rounding);
    weight_rows(j0, j1) and target_cols(j0, j1) give W_L[j0:j1] (j1 - j0 x H)
    and U[:, j0:j1].  Returns (loss, dA_in, db, dW rows) with dA_in = dY W_L
    (what hidden_grads takes), db (D) and dW_L[rows] (len(rows) x H).  Each
    chunk applies the same rounding points as loss_and_grads; the sums over
    chunks (loss, dA_in) are fp64, in chunk order.  torch CPU fp64 carries
    the products and the elementwise steps (multi-threaded)."""
    import torch
    rnd, points = _rounder(bf16, rounded)

    def trnd(point, t):
        return bf16_round_torch(t) if point in points else t

    A = torch.from_numpy(np.asarray(A_in, dtype=np.float64))
    B, H = A.shape
    Ar = trnd("act", A)
    rows = np.asarray(rows, dtype=np.int64)
    loss_sum = 0.0
    dA = torch.zeros(B, H, dtype=torch.float64)
    db = np.zeros(D)
    dW_rows = np.zeros((len(rows), H))
    for j0 in range(0, D, chunk):
        j1 = min(D, j0 + chunk)
        W = trnd("weight", torch.from_numpy(np.asarray(weight_rows(j0, j1))).to(torch.float64))
        U = trnd("target", torch.from_numpy(np.asarray(target_cols(j0, j1))).to(torch.float64))
        R = torch.addmm(torch.from_numpy(np.asarray(bias[j0:j1], dtype=np.float64)), Ar, W.T)
        R.sub_(U)
        loss_sum += float(torch.sum(R * R))
        dY_raw = R.mul_(2.0).div_(B * D)         # 2 R / (B D), as loss_and_grads forms it
        dY = trnd("dY", dY_raw)
        dA.addmm_(dY, W)
        db[j0:j1] = (dY_raw if "db_raw" in points else dY).sum(dim=0).numpy()
        sel = (rows >= j0) & (rows < j1)
        if sel.any():
            dW_rows[sel] = (dY[:, torch.from_numpy(rows[sel] - j0)].T @ Ar).numpy()
    return loss_sum / (B * D), dA.numpy(), db, dW_rows


def bf16_round_torch(t):
    """bf16_round on a torch fp64 CPU tensor (the same bit operation: round the
    fp32 value half to even at its 16th bit), fp64 out."""
    import torch
    b = t.to(torch.float32).view(torch.int32)
    lsb = torch.bitwise_and(torch.bitwise_right_shift(b, 16), 1)
    b = b.add_(0x7FFF).add_(lsb)
    b = torch.bitwise_and(b, -65536, out=b)
    return b.view(torch.float32).to(torch.float64)


@dataclass
class Adam:
    """Adam with bias correction (Kingma and Ba, 2015, Algorithm 1).

    state_dtype: None keeps parameters and moments in fp64; np.float32 rounds
    them to fp32 after every step, as a path that stores fp32 master weights
    and moments does.  The arithmetic of a step is fp64 either way; the
    rounded variant exists to measure how far fp32 storage alone moves a long
    run (the sensitivity of a comparison after many steps)."""
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    t: int = 0
    m: list = field(default_factory=list)
    v: list = field(default_factory=list)
    state_dtype: object = None

    def step(self, params: Params, grads: Params) -> Params:
        if not self.m:
            self.m = [(np.zeros_like(W), np.zeros_like(b)) for W, b in params]
            self.v = [(np.zeros_like(W), np.zeros_like(b)) for W, b in params]
        self.t += 1
        c1 = 1.0 - self.beta1 ** self.t
        c2 = 1.0 - self.beta2 ** self.t
        out: Params = []
        for l, ((W, b), (gW, gb)) in enumerate(zip(params, grads)):
            new = []
            for i, (p, g) in enumerate(((W, gW), (b, gb))):
                m = self.beta1 * self.m[l][i] + (1.0 - self.beta1) * g
                v = self.beta2 * self.v[l][i] + (1.0 - self.beta2) * g * g
                q = p - self.lr * (m / c1) / (np.sqrt(v / c2) + self.eps)
                if self.state_dtype is not None:
                    m, v, q = (np.asarray(a).astype(self.state_dtype).astype(np.float64) for a in (m, v, q))
                self._store(l, i, m, v)
                new.append(q)
            out.append((new[0], new[1]))
        return out

    def _store(self, l, i, m, v):
        ms, vs = list(self.m[l]), list(self.v[l])
        ms[i], vs[i] = m, v
        self.m[l], self.v[l] = tuple(ms), tuple(vs)


def predict(params: Params, X: np.ndarray, bf16: bool = False, rounded=None) -> np.ndarray:
    """Surrogate output f_theta(X, t) for each input row."""
    return forward(params, X, bf16=bf16, rounded=rounded)[2]
