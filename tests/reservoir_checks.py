"""Comparison of a GPU reservoir's metadata with the oracle reservoir's."""
import numpy as np


def compare_meta(gres, ores, hist_len):
    """Seen counts, sample ids, eviction histogram (last bin collects the tail)
    and counters of the GPU reservoir `gres` equal those of oracle `ores`."""
    seen, ids, hist = gres.read_meta()
    o_seen = np.where(ores.occupied, ores.seen_count, -1)
    o_ids = np.where(ores.occupied, ores.sample_id, -1)
    assert np.array_equal(seen, o_seen)
    assert np.array_equal(ids, o_ids)
    oh = np.zeros(hist_len, np.int64)
    for k, c in ores.evict_hist.items():
        oh[min(k, hist_len - 1)] += c
    assert np.array_equal(hist, oh)
    st = gres.stats()
    assert (st["n"], st["unseen"], st["seen"]) == (ores.N, ores.U, ores.S)
    assert st["total_put"] == ores.total_put and st["total_evicted"] == ores.total_evicted
    assert st["total_draws"] == ores.total_draws and st["next_ticket"] == ores.next_ticket
    assert st["total_deleted"] == ores.total_deleted
