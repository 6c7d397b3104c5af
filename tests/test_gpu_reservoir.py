"""GPU reservoir against the oracle reservoir: bit-exact slots, seen counts,
sample ids, eviction histogram and gathered rows, over seeded operation
sequences that fill, evict and drain the buffer; statuses; concurrent
producers replayed in ticket order."""
import threading

import numpy as np
import pytest
import torch

from fixtures.synthetic import hash_inputs, hash_rows
from oracle import reservoir as orv
from tests.reservoir_checks import compare_meta

pytestmark = pytest.mark.gpu

DEV = torch.device("cuda:0")


def padded(rows, d):
    """Device tensor (rows, d) whose leading dimension is a multiple of 4."""
    ld = (d + 3) // 4 * 4
    return torch.zeros(rows, ld, device=DEV)[:, :d]


@pytest.mark.parametrize("C,T,d,seed,ops", [
    (64, 32, 256, 0, 60),        # the 16x16 workload's reservoir
    (97, 10, 1003, 5, 80),       # ragged row length, prime capacity
    (300, 50, 4099, 9, 60),      # rows longer than one copy segment
    (1, 0, 1, 3, 40),            # one slot, no watermark, one-float rows
    (2, 1, 5, 4, 50),            # two slots: every put past the first evicts
])
def test_sequence_bit_exact(C, T, d, seed, ops):
    from paper_2309_16743_amd import OT_NOT_READY, OT_OK, Reservoir
    print(f"reservoir sequence C={C} T={T} d={d} seed={seed}", flush=True)
    rng = np.random.default_rng(seed)
    g = Reservoir(C, T, 6, d, seed)
    o = orv.Reservoir(C, T, 6, d, seed)
    key = 0
    acc = torch.zeros(1, dtype=torch.int64, device=DEV)
    for step in range(ops):
        if rng.random() < 0.5:
            k = int(rng.integers(0, 40))
            keys = np.arange(key, key + k)
            u = hash_rows(keys, d)
            x = hash_inputs(keys)
            ud = padded(k, d)
            xd = padded(k, 6)
            if k:
                ud.copy_(torch.from_numpy(u))
                xd.copy_(torch.from_numpy(x))
            t = g.put(xd if k else None, ud if k else None, accepted=acc)
            _, a, ot_, _ = o.put(x, u, k=k)
            assert t == ot_
            torch.cuda.synchronize()
            assert int(acc.item()) == a
            key += a
        else:
            b = int(rng.integers(1, 70))
            slots = torch.empty(b, dtype=torch.int32, device=DEV)
            ub = padded(b, d)
            xb = padded(b, 6)
            st, n, t = g.sample_batch(b, slots, x_out=xb, u_out=ub)
            ost, oslots, ox, ou, ot_ = o.sample_batch(b)
            assert st == ost
            if st == OT_OK:
                assert t == ot_
                torch.cuda.synchronize()
                assert np.array_equal(slots.cpu().numpy(), np.array(oslots))
                assert np.array_equal(ub.cpu().numpy(), ou)
                assert np.array_equal(xb.cpu().numpy(), ox)
            else:
                assert st == OT_NOT_READY
        if step % 10 == 9:
            compare_meta(g, o, 64)
    compare_meta(g, o, 64)
    assert o.total_evicted > 0
    # drain after reception ends
    g.end_reception()
    o.end_reception()
    while True:
        b = int(rng.integers(1, 40))
        slots = torch.empty(b, dtype=torch.int32, device=DEV)
        ub = padded(b, d)
        st, n, t = g.sample_batch(b, slots, u_out=ub)
        ost, oslots, _, ou, _ = o.sample_batch(b)
        assert st == ost
        if st != OT_OK:
            break
        torch.cuda.synchronize()
        assert n == len(oslots)
        assert np.array_equal(slots[:n].cpu().numpy(), np.array(oslots))
        assert np.array_equal(ub[:n].cpu().numpy(), ou)
        compare_meta(g, o, 64)
    assert o.N == 0
    g.close()


def test_statuses():
    from paper_2309_16743_amd import OT_EMPTY, OT_NOT_READY, OT_OK, OTError, Reservoir
    g = Reservoir(8, 4, 6, 16, 1)
    slots = torch.empty(4, dtype=torch.int32, device=DEV)
    assert g.sample_batch(4, slots)[0] == OT_NOT_READY
    u = padded(5, 16)
    g.put(None, u)
    assert g.sample_batch(4, slots)[0] == OT_OK
    assert g.stats()["next_ticket"] == 2
    g.end_reception()
    with pytest.raises(OTError):
        g.put(None, u)
    while g.sample_batch(4, slots)[0] == OT_OK:
        pass
    assert g.sample_batch(4, slots)[0] == OT_EMPTY
    with pytest.raises(OTError):
        g.sample_batch(0, slots)
    g.close()


def test_full_of_unseen_accepts_nothing():
    from paper_2309_16743_amd import Reservoir
    g = Reservoir(16, 0, 6, 8, 2)
    acc = torch.zeros(1, dtype=torch.int64, device=DEV)
    g.put(None, padded(16, 8), accepted=acc)
    g.put(None, padded(5, 8), accepted=acc)
    torch.cuda.synchronize()
    assert acc.item() == 0
    st = g.stats()
    assert st["n"] == 16 and st["unseen"] == 16 and st["total_put"] == 16
    g.close()


def test_concurrent_producers_replay_in_ticket_order():
    """Several host threads put on their own streams while the consumer draws;
    replaying the recorded ticket order in the oracle gives identical state."""
    from paper_2309_16743_amd import OT_OK, Reservoir
    C, T, d, seed = 200, 40, 512, 11
    g = Reservoir(C, T, 6, d, seed)
    log = []
    lock = threading.Lock()
    n_prod, puts_each, k = 4, 12, 16

    def producer(p):
        s = torch.cuda.Stream()
        for i in range(puts_each):
            keys = np.arange((p * puts_each + i) * k, (p * puts_each + i + 1) * k)
            with torch.cuda.stream(s):
                ud = padded(k, d)
                ud.copy_(torch.from_numpy(hash_rows(keys, d)), non_blocking=False)
                t = g.put(None, ud, stream=s)
            s.synchronize()
            with lock:
                log.append((t, "put", keys))

    threads = [threading.Thread(target=producer, args=(p,)) for p in range(n_prod)]
    for th in threads:
        th.start()
    cons = []
    for _ in range(40):
        slots = torch.empty(32, dtype=torch.int32, device=DEV)
        ub = padded(32, d)
        st, n, t = g.sample_batch(32, slots, u_out=ub)
        if st == OT_OK:
            torch.cuda.synchronize()
            cons.append((t, slots.cpu().numpy(), ub.cpu().numpy()))
    for th in threads:
        th.join()
    o = orv.Reservoir(C, T, 6, d, seed)
    events = sorted([(t, "put", keys) for t, _, keys in log] + [(t, "sample", None) for t, _, _ in cons],
                    key=lambda e: e[0])
    by_ticket = {t: (s, u) for t, s, u in cons}
    for t, kind, keys in events:
        if kind == "put":
            _, _, ot_, _ = o.put(None, hash_rows(keys, d), k=len(keys))
            assert ot_ == t
        else:
            ost, oslots, _, ou, ot_ = o.sample_batch(32)
            assert ost == OT_OK and ot_ == t
            s, u = by_ticket[t]
            assert np.array_equal(s, np.array(oslots))
            assert np.array_equal(u, ou)
    compare_meta(g, o, 64)
    g.close()


@pytest.mark.parametrize("policy,C,T,d,seed,ops", [
    ("fifo", 64, 0, 256, 3, 150),
    ("fifo", 97, 0, 1003, 4, 150),      # prime capacity, ragged rows: the slot ring wraps many times
    ("firo", 64, 20, 256, 5, 150),
    ("firo", 300, 50, 4099, 6, 120),    # rows longer than one copy segment
])
def test_list_policy_sequence_bit_exact(policy, C, T, d, seed, ops):
    """FIFO / FIRO (evict on read) against the oracle's buffers: statuses,
    tickets, accepted counts, taken slots, gathered rows, per-slot metadata
    and counters bit-exact over puts and batches that cycle the slots, then
    the drain after end_reception."""
    from paper_2309_16743_amd import OT_NOT_READY, OT_OK, OT_POLICY_FIFO, OT_POLICY_FIRO, Reservoir
    from oracle import buffers as obf
    print(f"{policy} sequence C={C} T={T} d={d} seed={seed}", flush=True)
    rng = np.random.default_rng(seed)
    g = Reservoir(C, T, 6, d, seed, policy=OT_POLICY_FIFO if policy == "fifo" else OT_POLICY_FIRO)
    o = (obf.FIFOBuffer if policy == "fifo" else obf.FIROBuffer)(C, T, 6, d, seed)
    key = 0
    acc = torch.zeros(1, dtype=torch.int64, device=DEV)
    batches = 0
    for step in range(ops):
        if rng.random() < 0.5:
            k = int(rng.integers(0, 50))
            keys = np.arange(key, key + k)
            u, x = hash_rows(keys, d), hash_inputs(keys)
            ud, xd = padded(k, d), padded(k, 6)
            if k:
                ud.copy_(torch.from_numpy(u))
                xd.copy_(torch.from_numpy(x))
            t = g.put(xd if k else None, ud if k else None, accepted=acc)
            _, a, ot_, _ = o.put(x, u, k=k)
            assert t == ot_
            torch.cuda.synchronize()
            assert int(acc.item()) == a
            key += a
        else:
            b = int(rng.integers(1, 40))
            slots = torch.empty(b, dtype=torch.int32, device=DEV)
            ub, xb = padded(b, d), padded(b, 6)
            st, n, t = g.sample_batch(b, slots, x_out=xb, u_out=ub)
            ost, oslots, ox, ou, ot_ = o.sample_batch(b)
            assert st == ost
            if st == OT_OK:
                batches += 1
                assert t == ot_ and n == b
                torch.cuda.synchronize()
                assert np.array_equal(slots.cpu().numpy(), np.array(oslots))
                assert np.array_equal(ub.cpu().numpy(), ou)
                assert np.array_equal(xb.cpu().numpy(), ox)
            else:
                assert st == OT_NOT_READY
        if step % 10 == 9:
            compare_meta(g, o, 64)
    compare_meta(g, o, 64)
    assert batches > 10 and o.total_put > 2 * C
    g.end_reception()
    o.end_reception()
    while True:
        b = int(rng.integers(1, 40))
        slots = torch.empty(b, dtype=torch.int32, device=DEV)
        ub = padded(b, d)
        st, n, t = g.sample_batch(b, slots, u_out=ub)
        ost, oslots, _, ou, _ = o.sample_batch(b)
        assert st == ost
        if st != OT_OK:
            break
        torch.cuda.synchronize()
        assert n == len(oslots)
        assert np.array_equal(slots[:n].cpu().numpy(), np.array(oslots))
        assert np.array_equal(ub[:n].cpu().numpy(), ou)
        compare_meta(g, o, 64)
    assert o.N == 0 and g.stats()["policy"] == (1 if policy == "fifo" else 2)
    g.close()


@pytest.mark.parametrize("policy", [0, 2])
def test_largest_put_and_take(policy):
    """A put of the largest chunk (4096 rows) into a full buffer whose every
    sample is seen (4096 evictions for the Reservoir), and a 4096-row batch
    (drain for the Reservoir, random take for FIRO): bit-exact against the
    oracle (these calls use the most LDS of the assignment and take kernels)."""
    from paper_2309_16743_amd import OT_OK, Reservoir
    from oracle import buffers as obf
    C, d, k = 8192, 64, 4096
    g = Reservoir(C, 0, 6, d, 21, policy=policy)
    o = (orv.Reservoir if policy == 0 else obf.FIROBuffer)(C, 0, 6, d, 21)
    key = 0
    for _ in range(3):
        keys = np.arange(key, key + k)
        ud, xd = padded(k, d), padded(k, 6)
        ud.copy_(torch.from_numpy(hash_rows(keys, d)))
        xd.copy_(torch.from_numpy(hash_inputs(keys)))
        g.put(xd, ud)
        _, a, _, _ = o.put(hash_inputs(keys), hash_rows(keys, d), k=k)
        key += a
        if policy == 0:          # draw every sample at least once before the next put
            for _ in range(8):
                slots = torch.empty(k, dtype=torch.int32, device=DEV)
                assert g.sample_batch(k, slots)[0] == OT_OK
                st, oslots, _, _, _ = o.sample_batch(k)
                torch.cuda.synchronize()
                assert np.array_equal(slots.cpu().numpy(), np.array(oslots))
    compare_meta(g, o, 64)
    g.end_reception()
    o.end_reception()
    slots = torch.empty(k, dtype=torch.int32, device=DEV)
    ub = padded(k, d)
    st, n, _ = g.sample_batch(k, slots, u_out=ub)
    ost, oslots, _, ou, _ = o.sample_batch(k)
    torch.cuda.synchronize()
    assert st == ost == OT_OK and n == k
    assert np.array_equal(slots.cpu().numpy(), np.array(oslots)) and np.array_equal(ub.cpu().numpy(), ou)
    compare_meta(g, o, 64)
    g.close()


@pytest.mark.parametrize("C,k_evict", [
    (262144, 100),     # the largest reservoir whose put decisions run in one launch (1024 chunks of 256 slots)
    (262145, 100),     # one slot more: the tile-count / assign / victim kernels
    (5000, 1024),      # the largest put that runs in one launch
    (5000, 1025),      # one row more
])
def test_eviction_index_on_both_sides_of_the_one_launch_limits(C, k_evict):
    """Puts that replace seen samples pick the same victims (slots, seen counts,
    sample ids, eviction histogram bit-exact against the oracle) whether their
    decisions run in the single-launch kernel (reservoirs of up to 262,144
    slots, puts of up to 1024 rows) or in the three-kernel path."""
    from paper_2309_16743_amd import OT_OK, Reservoir
    print(f"eviction index C={C} k={k_evict}", flush=True)
    d = 1
    g = Reservoir(C, 0, 6, d, 11)
    o = orv.Reservoir(C, 0, 6, d, 11)
    key = 0

    def put(k):
        nonlocal key
        keys = np.arange(key, key + k)
        ud = padded(k, d)
        ud.copy_(torch.from_numpy(hash_rows(keys, d)))
        acc = torch.zeros(1, dtype=torch.int64, device=DEV)
        t = g.put(None, ud, accepted=acc)
        _, a, ot_, _ = o.put(None, hash_rows(keys, d), k=k)
        assert t == ot_
        torch.cuda.synchronize()
        assert int(acc.item()) == a
        key += a

    def draw(b):
        slots = torch.empty(b, dtype=torch.int32, device=DEV)
        st, n, t = g.sample_batch(b, slots)
        ost, oslots, _, _, ot_ = o.sample_batch(b)
        assert st == ost == OT_OK and t == ot_
        torch.cuda.synchronize()
        assert np.array_equal(slots.cpu().numpy(), np.array(oslots))

    while o.N < C:
        put(min(4096, C - o.N))
    for _ in range(3):
        draw(8192)
    compare_meta(g, o, 64)
    for i in range(4):
        put(k_evict)
        draw(4096)
    compare_meta(g, o, 64)
    assert o.total_evicted >= 4 * k_evict
    g.close()
