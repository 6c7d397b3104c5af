"""surrogate_predict_noalloc (the prediction entry point that allocates
nothing) against surrogate_predict: same kernels and plans, so the outputs
must agree bit for bit; two calls in a row, the second with fewer rows, so the
second reuses the scratch the first wrote with another layout; a request
larger than the scratch is refused without touching the output."""
import numpy as np
import pytest
import torch

from oracle import mlp

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def padded(rows, d, fill=0.0):
    ld = (d + 3) // 4 * 4
    return torch.full((rows, ld), fill, device=DEV)[:, :d]


def inputs(n, seed):
    rng = np.random.default_rng(seed)
    x = np.concatenate([rng.uniform(100, 500, (n, 5)), rng.uniform(0.01, 1.0, (n, 1))], axis=1)
    t = padded(n, 6)
    t.copy_(torch.from_numpy(x.astype(np.float32)))
    return t, x


@pytest.mark.parametrize("widths,precision,rows", [
    ((6, 64, 64, 256), "fp32", (100, 37)),          # narrow hidden layers (fused hidden-layer kernel)
    ((6, 300, 200, 5000), "fp32", (64, 20)),         # GEMM hidden layer and output, both split over k
    ((6, 128, 128, 1000), "bf16", (200, 50)),
    ((6, 256, 256, 256, 3000), "bf16", (96, 33)),
])
def test_predict_noalloc_matches_predict(widths, precision, rows):
    from paper_2309_16743_amd import OT_BF16, OT_FP32, Surrogate
    prec = OT_BF16 if precision == "bf16" else OT_FP32
    s = Surrogate(widths, precision=prec, seed=5, max_batch=max(rows))
    for i, n in enumerate(rows):
        x, xh = inputs(n, 10 + i)
        y_ref = padded(n, widths[-1], np.nan)
        y_na = padded(n, widths[-1], np.nan)
        s.predict(x, y_ref)
        s.predict_noalloc(x, y_na)
        torch.cuda.synchronize()
        a, b = y_ref.cpu().numpy(), y_na.cpu().numpy()
        assert np.isfinite(b).all()
        assert np.array_equal(a, b), f"call {i} ({n} rows) differs from surrogate_predict"
    # and the last call against the oracle's prediction with the surrogate's parameters
    params = [tuple(p.astype(np.float64) for p in s.get_params(l)) for l in range(len(widths) - 1)]
    ref = mlp.predict(params, xh, bf16=(precision == "bf16"))
    rel = np.linalg.norm(b - ref) / np.linalg.norm(ref)
    assert rel < (1e-3 if precision == "bf16" else 1e-5), rel
    s.close()


def test_predict_noalloc_two_surrogates_share_the_scratch_in_stream_order():
    from paper_2309_16743_amd import Surrogate
    s1 = Surrogate((6, 64, 64, 256), seed=1, max_batch=64)
    s2 = Surrogate((6, 300, 200, 5000), seed=2, max_batch=64)
    x, _ = inputs(64, 3)
    y1a, y1b = padded(64, 256), padded(64, 256)
    y2a, y2b = padded(64, 5000), padded(64, 5000)
    s1.predict(x, y1a)
    s2.predict(x, y2a)
    s1.predict_noalloc(x, y1b)                 # one stream: the second call waits for the first
    s2.predict_noalloc(x, y2b)
    torch.cuda.synchronize()
    assert np.array_equal(y1a.cpu().numpy(), y1b.cpu().numpy())
    assert np.array_equal(y2a.cpu().numpy(), y2b.cpu().numpy())
    s1.close()
    s2.close()


def test_predict_noalloc_refuses_rows_beyond_the_scratch():
    from paper_2309_16743_amd import OT_E_INVAL, OTError, Surrogate
    from paper_2309_16743_amd._abi import OT_PREDICT_NOALLOC_SCRATCH_BYTES
    widths = (6, 4096, 4096, 16)                # 32 KB of fp32 activations per row
    s = Surrogate(widths, seed=4, max_batch=1024)   # predict then runs the half below as one chunk too
    n = OT_PREDICT_NOALLOC_SCRATCH_BYTES // (2 * 4096 * 4) + 1
    x, _ = inputs(n, 6)
    y = padded(n, 16, 7.0)
    with pytest.raises(OTError) as e:
        s.predict_noalloc(x, y)
    assert e.value.status == OT_E_INVAL and "scratch" in str(e.value)
    torch.cuda.synchronize()
    assert (y.cpu().numpy() == 7.0).all()
    # half of it fits (activations plus the output layer's split-K partials)
    m = n // 2
    y2, y3 = padded(m, 16), padded(m, 16)
    s.predict_noalloc(x[:m], y2)
    s.predict(x[:m], y3)
    torch.cuda.synchronize()
    assert np.array_equal(y2.cpu().numpy(), y3.cpu().numpy())
    s.close()
