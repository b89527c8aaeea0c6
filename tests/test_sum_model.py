"""The plain SUM-manager model (oracle/sum_model.py) against Algorithm 1
worked by hand and against invariants the algorithm's states imply."""
import random

import pytest

from oracle.sum_model import (AVAIL, BACKED, FREE, FULL, MODE_FAST, MODE_FULL, RESTORING,
                              NoSpace, SumModel)


def test_hand_worked_sequence():
    """3 units of 4 blocks; residuals 0 and 1 in units 0 and 1; unit 2 FREE.
    Each step worked by hand from the pseudocode of Algorithm 1."""
    m = SumModel(3, 4, 2)
    assert m.sets[FREE] == {2} and m.sets[BACKED] == {0, 1} and m.mode == MODE_FULL
    # AVAIL empty -> pop FREE unit 2; three blocks from it; unit 2 has room -> AVAIL
    assert m.alloc(3) == [8, 9, 10]
    assert m.sets[AVAIL] == {2} and m.sets[FREE] == set()
    # one block left in unit 2 -> FULL; AVAIL and FREE empty -> pop BACKED unit 0:
    # fast mode, residual 0 stale and evicted; block 0 from unit 0
    assert m.alloc(2) == [11, 0]
    assert m.sets[FULL] == {2} and m.sets[AVAIL] == {0} and m.sets[BACKED] == {1}
    assert m.mode == MODE_FAST and m.STALE == {0} and m.EVICTED == {0}
    # more than the room left (3 in unit 0 + 4 in BACKED unit 1 = 7): nothing taken
    with pytest.raises(NoSpace):
        m.alloc(8)
    assert m.counts()["free_blocks"] == 3 and m.sets[BACKED] == {1}
    # freeing one block of the FULL unit moves it to AVAIL; no unit empties
    assert m.free([9]) is False
    assert m.sets[AVAIL] == {0, 2} and m.sets[FULL] == set()
    # emptying unit 2 makes it FREE while residual 0 is evicted -> wake restore
    assert m.free([8, 10, 11]) is True
    assert m.sets[FREE] == {2}
    # the worker binds stale residual 0 to FREE unit 2 and copies it back
    assert m.restore_begin() == (0, 2)
    assert m.sets[RESTORING] == {2} and m.mode == MODE_FAST
    m.restore_done(0)
    assert m.sets[BACKED] == {1, 2} and m.mode == MODE_FULL and m.unit_of(0) == 2
    # unit 0 still holds block 0 as KV; freeing it returns the unit to FREE, no wake
    assert m.free([0]) is False
    assert m.sets[FREE] == {0} and m.restore_begin() is None


def check_invariants(m):
    units = [u for s in m.sets.values() for u in s]
    assert sorted(units) == list(range(m.n_units)), "each unit in exactly one set"
    for u in range(m.n_units):
        st = m.state_of(u)
        n = len(m.allocated[u])
        assert (st in (AVAIL, FULL)) == (n > 0)
        if st == FULL:
            assert n == m.B
        if st == AVAIL:
            assert 0 < n < m.B
        if st in (FREE, BACKED, RESTORING):
            assert n == 0
    bound = {u: r for r, u in m.binding.items()}
    assert len(bound) == len(m.binding), "one residual per unit"
    assert set(bound) == m.sets[BACKED] | m.sets[RESTORING]
    assert m.STALE <= m.EVICTED
    assert all(r not in m.binding for r in m.STALE)
    assert (m.mode == MODE_FAST) == bool(m.EVICTED)


@pytest.mark.parametrize("seed", range(6))
def test_random_operations_keep_invariants(seed):
    rng = random.Random(seed)
    n_units = rng.randint(1, 10)
    m = SumModel(n_units, rng.randint(1, 6), rng.randint(0, n_units))
    held = []
    for _ in range(300):
        op = rng.random()
        if op < 0.45:
            try:
                held += m.alloc(rng.randint(0, 2 * m.B))
            except NoSpace:
                pass
        elif op < 0.8 and held:
            rng.shuffle(held)
            k = rng.randint(1, len(held))
            m.free(held[:k])
            held = held[k:]
        elif op < 0.9:
            m.restore_begin()
        elif m.sets[RESTORING]:
            u = min(m.sets[RESTORING])
            m.restore_done([r for r, unit in m.binding.items() if unit == u][0])
        check_invariants(m)


def test_pressure_forces_fast_mode_and_release_restores_full():
    """Allocate until FREE is empty: BACKED units are evicted and the mode turns
    fast.  Freeing every block wakes the restore; restoring every evicted
    residual returns the mode to full with all residuals bound again."""
    m = SumModel(8, 16, 5)
    held = m.alloc(3 * 16)              # the three FREE units
    assert m.mode == MODE_FULL and not m.sets[FREE]
    held += m.alloc(20)                 # two more units, both taken from BACKED
    assert m.mode == MODE_FAST and m.EVICTED == {0, 1}
    wakes = [m.free([b]) for b in held]
    assert any(wakes)
    while True:
        step = m.restore_begin()
        if step is None:
            break
        m.restore_done(step[0])
    assert m.mode == MODE_FULL and not m.EVICTED and sorted(m.binding) == list(range(5))
    check_invariants(m)
