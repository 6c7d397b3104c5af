"""Host logic of the online loop that runs without a GPU: the log of received
messages (Sec. 3.1: after a client restart, messages already received are
discarded) and the learning-rate halving schedule (Sec. 4.4-4.5)."""
import torch

from paper_2309_16743_amd.online import HalvingLR, ReceptionLog


def _put(log, keys, accepted):
    """One put of `keys` whose device count reports `accepted` rows."""
    slot = log.count_slot()
    log.record(keys, log.next_count - 1)
    slot.fill_(accepted)


def test_received_messages_are_dropped_and_refused_rows_readmitted():
    log = ReceptionLog(torch.device("cpu"))
    first = [(0, 1), (1, 1), (2, 1)]
    assert log.new_rows(first).tolist() == [True, True, True]
    _put(log, first, 2)                           # the buffer accepted the prefix of two rows
    # client 0 resends step 1 after a restart; client 2's refused row comes again
    again = [(2, 1), (0, 1), (3, 1)]
    assert log.new_rows(again).tolist() == [True, False, True]
    _put(log, [(2, 1), (3, 1)], 2)
    assert log.keys().tolist() == [[0, 1], [1, 1], [2, 1], [3, 1]]
    assert log.new_rows([(1, 1), (3, 1), (4, 1)]).tolist() == [False, False, True]


def test_new_keys_never_wait_for_pending_counts():
    log = ReceptionLog(torch.device("cpu"))
    _put(log, [(0, 1)], 1)
    assert log.pending                             # not resolved: the keys below were never offered
    assert log.new_rows([(0, 2), (1, 2)]).tolist() == [True, True]
    assert log.pending
    assert log.new_rows([(0, 1)]).tolist() == [False]
    assert not log.pending


def test_count_words_are_recycled_after_resolving():
    log = ReceptionLog(torch.device("cpu"))
    n = len(log.counts) + 5
    for i in range(n):
        _put(log, [(i, 0)], 1)
    assert log.keys().shape == (n, 2)


def test_halving_schedule_blocks_and_floor():
    lr = HalvingLR(lr0=1e-3, every_samples=10_000, lr_min=2.5e-4)
    assert [lr(n) for n in (0, 9_999, 10_000, 19_999, 20_000, 10 ** 7)] == [1e-3, 1e-3, 5e-4, 5e-4, 2.5e-4, 2.5e-4]
