"""The reservoir at its stress shape: rows of 100,000 floats, capacity 50,000
(a 20 GB slab), threshold 10,000, 64 producer streams (8 host threads x 8
streams) putting chunks of 256 hash rows while the consumer draws batches of
256.  Replaying the recorded ticket order in the oracle (metadata only; the
key of the row held by each slot is tracked on the host from the slots the
oracle's puts return) must give the same accepted counts, the same slots for
every batch, the same seen counts, sample ids and eviction histogram, and
every gathered row must be the hash row of the key stored in its slot
(checked on sampled columns)."""
import threading

import numpy as np
import pytest
import torch

from fixtures import configs
from fixtures.synthetic import hash_inputs, hash_inputs_torch, hash_rows_torch, hash_values
from oracle import reservoir as orv
from tests.reservoir_checks import compare_meta

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")
COLS = np.array([0, 1, 4097, 50000, 99999])


def test_stress_shape_concurrent_producers_replay():
    from paper_2309_16743_amd import OT_NOT_READY, OT_OK, Reservoir
    w = configs.STRESS
    D, k, B = w.row_len, w.chunk, w.batch
    n_threads, per_thread, puts_per_stream = 8, 8, 8          # 64 streams, 512 puts
    n_puts = n_threads * per_thread * puts_per_stream
    print(f"stress reservoir C={w.capacity} T={w.threshold} row={D} puts={n_puts}", flush=True)
    g = Reservoir(w.capacity, w.threshold, 6, D, w.reservoir_seed)
    acc = torch.zeros(n_puts, dtype=torch.int64, device=DEV)
    log, lock = [], threading.Lock()
    done = threading.Event()

    def producer(t):
        streams = [torch.cuda.Stream(device=DEV) for _ in range(per_thread)]
        bufs = [(torch.empty(k, 8, device=DEV)[:, :6], torch.empty(k, D, device=DEV)) for _ in range(per_thread)]
        for i in range(puts_per_stream):
            for j, s in enumerate(streams):
                q = (t * per_thread + j) * puts_per_stream + i        # put index; its rows have keys q k + r
                with torch.cuda.stream(s):
                    keys = torch.arange(q * k, (q + 1) * k, device=DEV, dtype=torch.int64)
                    xb_, ub_ = bufs[j]
                    hash_rows_torch(keys, D, out=ub_)
                    xb_.copy_(hash_inputs_torch(keys, 6))
                    ticket = g.put(xb_, ub_, stream=s, accepted=acc[q:q + 1])
                with lock:
                    log.append((ticket, "put", q))
        for s in streams:
            s.synchronize()

    threads = [threading.Thread(target=producer, args=(t,)) for t in range(n_threads)]
    for th in threads:
        th.start()
    cons = torch.cuda.Stream(device=DEV)
    slots = torch.empty(B, dtype=torch.int32, device=DEV)
    xb = torch.empty(B, 8, device=DEV)[:, :6]
    ub = torch.empty(B, D, device=DEV)
    cols = torch.from_numpy(COLS).to(DEV)
    batches = []
    while any(th.is_alive() for th in threads) and len(batches) < 4000:
        st, n, t = g.sample_batch(B, slots, x_out=xb, u_out=ub, stream=cons)
        if st == OT_NOT_READY:
            continue
        assert st == OT_OK and n == B
        with torch.cuda.stream(cons):
            batches.append((t, slots.cpu().numpy(), xb.cpu().numpy(), ub[:, cols].cpu().numpy()))
    for th in threads:
        th.join()
    torch.cuda.synchronize()
    acc_h = acc.cpu().numpy()
    print(f"{len(log)} puts, {len(batches)} batches; replaying in ticket order", flush=True)
    assert len(batches) > 0

    o = orv.Reservoir(w.capacity, w.threshold, 6, D, w.reservoir_seed, store_rows=False)
    key_of_slot = np.full(w.capacity, -1, np.int64)
    events = sorted([(t, "put", q) for t, _, q in log] + [(b[0], "sample", i) for i, b in enumerate(batches)])
    for t, kind, idx in events:
        if kind == "put":
            st, a, ot_, oslots = o.put(None, None, k=k)
            assert ot_ == t and a == acc_h[idx], (t, a, acc_h[idx])
            key_of_slot[np.array(oslots, dtype=np.int64)] = idx * k + np.arange(a)
        else:
            st, oslots, _, _, ot_ = o.sample_batch(B)
            assert st == orv.OK and ot_ == t
            _, s_g, x_g, u_g = batches[idx]
            assert np.array_equal(s_g, np.array(oslots, dtype=np.int32)), t
            keys = key_of_slot[s_g]
            assert (keys >= 0).all()
            assert np.array_equal(u_g, hash_values(keys, COLS)), t
            assert np.array_equal(x_g, hash_inputs(keys, 6)), t
    o.check_invariants()
    compare_meta(g, o, g.stats()["hist_len"])
    g.close()
