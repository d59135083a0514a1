"""Pins for the token-level model of asynchronous state reconciliation.

Algorithm 1 is a state machine; what the paper fixes about its result is the
construction in the proof of Theorem 4: once reconciled, the new primary holds
E(T_t) (+) dX_{t_evict:T}, the evicted state followed by every chunk that
arrived since the eviction, and the primary keeps serving throughout.  The
tests derive that sequence independently (from the chunk history alone) and
check the model against it for many completion schedules, plus a worked
example traced by hand.
"""
import random

import pytest

from oracle.asr_model import AsrModel, evict_oldest_half, flat


def chunk(i, size):
    return list(range(1000 + i * size, 1000 + (i + 1) * size))


def test_worked_example_by_hand():
    # X_pre = [0, 1]; chunks of two ids; tau = 8 tokens; catch-up threshold 2 tokens.
    m = AsrModel([0, 1], tau_mem=8, n_catchup=2)
    assert m.increment([10, 11]) == [10, 11]
    assert m.increment([12, 13]) == [12, 13]
    assert not m.reconciling
    # third chunk: |X_static| = 2 + 6 = 8 >= 8 -> evict the oldest 1 of 3 chunks
    assert m.increment([14, 15]) == [14, 15]
    assert m.reconciling and m.phase == "warmup"
    assert m.x_e() == [0, 1, 12, 13, 14, 15]
    # two chunks arrive during the warm-up and are buffered
    m.increment([16, 17])
    m.increment([18, 19])
    assert flat(m.buffer) == [16, 17, 18, 19]
    # warm-up done: 4 buffered tokens > 2 -> one catch-up round absorbs them
    m.secondary_done()
    assert m.phase == "catchup" and m.x_e() == [0, 1, 12, 13, 14, 15, 16, 17, 18, 19]
    # one more chunk during the catch-up
    assert m.increment([20, 21]) == [20, 21]   # still served by the old primary
    # catch-up done: 2 tokens <= 2 -> swap; the remainder [20, 21] is the new primary's next work
    m.secondary_done()
    assert not m.reconciling and m.swaps == 1
    assert m.primary_cached == [0, 1, 12, 13, 14, 15, 16, 17, 18, 19]
    assert m.primary_pending == [20, 21]
    # the next task on the new primary computes the remainder and its own chunk
    assert m.increment([22, 23]) == [20, 21, 22, 23]
    assert m.x_static() == [0, 1, 12, 13, 14, 15, 16, 17, 18, 19, 20, 21, 22, 23]
    # the reconciled state (14 tokens) is still above this tiny threshold, so the
    # same increment starts the next reconciliation
    assert [e[0] for e in m.log] == ["warmup", "catchup", "swap", "warmup"]
    assert m.x_e() == [0, 1, 18, 19, 20, 21, 22, 23]  # six chunks, oldest three dropped


def test_eviction_rule_keeps_prefix_and_newest_half():
    chunks = [[1], [2], [3], [4], [5]]
    assert evict_oldest_half(chunks) == [[3], [4], [5]]
    assert evict_oldest_half([[1], [2]]) == [[2]]
    assert evict_oldest_half([[1]]) == [[1]]


@pytest.mark.parametrize("seed", range(20))
def test_reconciled_state_is_evicted_state_plus_every_later_chunk(seed):
    """Theorem 4's construction, for random completion schedules and sizes."""
    rng = random.Random(seed)
    size = rng.choice([1, 3, 100])
    pre = list(range(rng.randint(1, 50)))
    tau = len(pre) + size * rng.randint(4, 12)
    n_catchup = size * rng.randint(1, 3)
    m = AsrModel(pre, tau_mem=tau, n_catchup=n_catchup)
    history = []          # every chunk, in arrival order
    trigger_at = None     # index into history of the chunk that triggered the eviction
    cycles = 0
    for i in range(400):
        c = chunk(i, size)
        was = m.reconciling
        served = m.increment(c)
        history.append(c)
        # every increment is served immediately, on whichever resource is primary
        assert served[-len(c):] == c
        if m.reconciling and not was:
            trigger_at = i
            static_at_trigger = [list(x) for x in m.chunks]
        if m.secondary_busy and rng.random() < 0.4:
            swaps = m.swaps
            m.secondary_done()
            if m.swaps > swaps:
                cycles += 1
                expected_chunks = evict_oldest_half(static_at_trigger) + history[trigger_at + 1:]
                assert m.x_static() == pre + flat(expected_chunks)
                assert m.primary_cached + m.primary_pending == m.x_static()
                assert len(m.primary_pending) <= n_catchup
                assert m.buffer == [] and not m.reconciling
        # the primary's cache plus its pending ids always spell its logical state
        assert m.primary_cached + m.primary_pending == m.x_static()
    assert cycles >= 2


def test_memory_stays_bounded_over_many_cycles():
    """A viable schedule (Theorem 4's inequality holds): each warm-up lasts 30
    tasks and each catch-up finishes before the next chunk arrives."""
    size, pre = 100, list(range(2048))
    m = AsrModel(pre, tau_mem=110_000, n_catchup=100)
    peak, warm_left = 0, None
    for i in range(6000):
        m.increment(chunk(i, size))
        peak = max(peak, m.static_len)
        if m.phase == "warmup":
            warm_left = 30 if warm_left is None else warm_left - 1
            if warm_left == 0:
                m.secondary_done()
                warm_left = None
        elif m.secondary_busy:
            m.secondary_done()
    assert m.evictions >= 5 and m.swaps >= 5
    # growth past tau is only what arrives while one reconciliation runs
    assert peak <= 110_000 + 32 * size
    assert m.static_len == len(m.x_static())


def test_catchup_that_never_converges_never_swaps():
    """Completions slower than arrivals: the catch-up loop keeps absorbing and
    the swap never happens (the non-viable side of Theorem 4's inequality)."""
    m = AsrModel(list(range(10)), tau_mem=10 + 5 * 4, n_catchup=4)
    for i in range(200):
        m.increment(chunk(i, 4))
        if m.secondary_busy and i % 3 == 0:
            m.secondary_done()
    assert m.evictions == 1 and m.swaps == 0 and m.reconciling
