"""Checkpoint / restart (Sec. 3.1: the server is checkpointed and a failed
server restarts from its last checkpoint; the server's per-client log of
received messages discards what restarted clients send again).

* A run checkpointed mid-stream and restarted into fresh objects, with every
  client resending its time steps from the start, continues bit for bit like
  the uninterrupted run: same tickets, slots, losses and parameters (resent
  messages received before the checkpoint are discarded without a ticket;
  those received after it are accepted again).
* Reservoir checkpoints of all three buffer policies restore into a fresh
  buffer that answers a later operation sequence exactly like the original.
* Blobs of another shape or policy, or truncated ones, are refused and leave
  the target unchanged."""
import numpy as np
import pytest
import torch

from fixtures import configs, heat
from fixtures.synthetic import hash_inputs, hash_rows
from oracle import runner

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def make_trainer(w, inputs, fields, **kw):
    from paper_2309_16743_amd.online import OnlineTrainer
    return OnlineTrainer(w.widths, w.batch, w.capacity, w.threshold, w.wave, w.tau,
                         torch.from_numpy(inputs).to(DEV), torch.from_numpy(fields).to(DEV),
                         w.reservoir_seed, w.init_seed, lr=w.lr, record_steps=200, reception_log=True, **kw)


@pytest.mark.parametrize("precision,overlap,ckpt_iter", [
    ("fp32", False, 7), ("bf16", False, 7), ("fp32", True, 7), ("bf16", True, 7),
    ("fp32", True, 3), ("fp32", False, 3)])
def test_restart_from_checkpoint_with_resent_messages(precision, overlap, ckpt_iter):
    """ckpt_iter 7: the checkpoint is taken after training started (iteration 4);
    3: before the buffer reached its threshold.  overlap: puts and draws on the
    reservoir's own stream, so the log reads accepted counts across streams."""
    from paper_2309_16743_amd import OT_BF16, OT_FP32
    w = configs.TINY
    X = heat.sample_parameters(w.n_sims, w.data_seed)
    inputs, fields = heat.inputs_for(X, w.tau), heat.heat_fields(X, w.grid, w.tau)
    prec = OT_BF16 if precision == "bf16" else OT_FP32
    a = make_trainer(w, inputs, fields, precision=prec, overlap=overlap)
    for _ in range(ckpt_iter):                           # chunks 0..ckpt_iter-1 put, training from iteration 4
        a.iterate()
    ckpt = a.checkpoint()
    steps_at_ckpt = a.steps_done
    for _ in range(3):
        a.iterate()
    a.offer_chunk(ckpt_iter + 1)                         # a restarted client resends: discarded, no ticket
    assert a.res.stats()["next_ticket"] == ckpt_iter + 3 + a.steps_done
    while a.steps_done < 60:
        a.iterate()
    torch.cuda.synchronize()

    b = make_trainer(w, inputs, fields, precision=prec, overlap=overlap)
    b.restore(ckpt)
    tickets0 = b.res.stats()["next_ticket"]
    for c in range(ckpt_iter):                           # every client starts again from its first step
        b.offer_chunk(c)
    assert b.res.stats()["next_ticket"] == tickets0     # all of them were received before the checkpoint
    while b.steps_done < 60:
        b.iterate()
    torch.cuda.synchronize()
    sa, sb = a.slot_log.cpu().numpy(), b.slot_log.cpu().numpy()
    assert np.array_equal(sa[steps_at_ckpt:60], sb[steps_at_ckpt:60])
    la, lb = a.loss_log.cpu().numpy(), b.loss_log.cpu().numpy()
    assert np.array_equal(la[steps_at_ckpt:60], lb[steps_at_ckpt:60])
    for l in range(3):
        for x, y in zip(a.sur.get_params(l), b.sur.get_params(l)):
            assert np.array_equal(x, y)
    assert a.res.stats() == b.res.stats()
    ra, rb = a.res.read_meta(), b.res.read_meta()
    for x, y in zip(ra, rb):
        assert np.array_equal(x, y)
    if precision == "fp32":                              # the restarted run's draws are the oracle's
        ref = runner.run(w, inputs, fields, n_steps=60)
        for i in range(steps_at_ckpt, 60):
            assert np.array_equal(sb[i], ref["slots"][i]), i
    a.close()
    b.close()


def padded(rows, d):
    ld = (d + 3) // 4 * 4
    return torch.zeros(rows, ld, device=DEV)[:, :d]


def run_ops(g, rng, n_ops, d, key0):
    """A seeded sequence of puts and batches; returns what the buffer answered."""
    out = []
    key = key0
    acc = torch.zeros(1, dtype=torch.int64, device=DEV)
    for _ in range(n_ops):
        if rng.random() < 0.5:
            k = int(rng.integers(1, 30))
            keys = np.arange(key, key + k)
            ud, xd = padded(k, d), padded(k, 6)
            ud.copy_(torch.from_numpy(hash_rows(keys, d)))
            xd.copy_(torch.from_numpy(hash_inputs(keys)))
            t = g.put(xd, ud, accepted=acc)
            torch.cuda.synchronize()
            out.append(("put", t, int(acc.item())))
            key += int(acc.item())
        else:
            b = int(rng.integers(1, 25))
            slots = torch.empty(b, dtype=torch.int32, device=DEV)
            ub = padded(b, d)
            st, n, t = g.sample_batch(b, slots, u_out=ub)
            torch.cuda.synchronize()
            out.append(("batch", st, t, slots[:n].cpu().numpy().tolist(), ub[:n].cpu().numpy().tobytes()))
    return out, key


@pytest.mark.parametrize("policy", [0, 1, 2])
def test_reservoir_checkpoint_round_trip(policy):
    from paper_2309_16743_amd import Reservoir
    C, T, d = 80, 12, 300
    g = Reservoir(C, T, 6, d, 13, policy=policy)
    _, key = run_ops(g, np.random.default_rng(1), 60, d, 0)
    blob = g.checkpoint()
    cont_a, _ = run_ops(g, np.random.default_rng(2), 60, d, key)
    h = Reservoir(C, T, 6, d, 999, policy=policy)        # another seed: the checkpoint carries the key
    h.restore(blob)
    cont_b, _ = run_ops(h, np.random.default_rng(2), 60, d, key)
    assert cont_a == cont_b
    assert g.stats() == h.stats()
    for x, y in zip(g.read_meta(), h.read_meta()):
        assert np.array_equal(x, y)
    g.close()
    h.close()


def test_restore_refuses_foreign_or_truncated_blobs():
    from paper_2309_16743_amd import OTError, Reservoir, Surrogate
    g = Reservoir(32, 4, 6, 64, 1)
    g.put(None, padded(10, 64))
    blob = g.checkpoint()
    before = g.stats()
    for other in (Reservoir(33, 4, 6, 64, 1), Reservoir(32, 4, 6, 64, 1, policy=2)):
        with pytest.raises(OTError):
            other.restore(blob)
        other.close()
    with pytest.raises(OTError):
        g.restore(blob[:-4])
    with pytest.raises(OTError):
        g.restore(np.zeros_like(blob))
    assert g.stats() == before
    s = Surrogate((6, 16, 8), max_batch=8)
    sb = s.checkpoint()
    with pytest.raises(OTError):
        Surrogate((6, 16, 9), max_batch=8).restore(sb)
    with pytest.raises(OTError):
        s.restore(sb[:-1])
    with pytest.raises(OTError):
        g.restore(sb)
    g.close()
    s.close()
