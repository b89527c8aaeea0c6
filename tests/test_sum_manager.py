"""The library's native SUM manager (dps_sum_*) against the plain model in
oracle/sum_model.py: the same operations, every observable compared after
each one.  Host-only; no GPU."""
import random

import pytest

from oracle.sum_model import AVAIL, BACKED, FREE, FULL, RESTORING, NoSpace, SumModel
from paper_2609_34380_amd import dps

STATE = {FREE: dps.UNIT_FREE, BACKED: dps.UNIT_BACKED, AVAIL: dps.UNIT_AVAIL,
         FULL: dps.UNIT_FULL, RESTORING: dps.UNIT_RESTORING}


def same(native, model):
    assert native.counts() == model.counts()
    assert native.mode == model.mode
    for u in range(model.n_units):
        assert native.unit_state(u) == STATE[model.state_of(u)], u
    for r in range(native.n_res):
        assert native.unit_of(r) == model.unit_of(r), r


@pytest.mark.parametrize("seed", range(12))
def test_native_matches_model(seed):
    rng = random.Random(100 + seed)
    n_units = rng.randint(1, 12)
    geom = (n_units, rng.randint(1, 8), rng.randint(0, n_units))
    native, model = dps.SumManager(*geom), SumModel(*geom)
    same(native, model)
    held = []
    for _ in range(400):
        op = rng.random()
        if op < 0.45:
            n = rng.randint(0, 3 * geom[1])
            got = native.alloc(n)
            try:
                want = model.alloc(n)
            except NoSpace:
                want = None
            assert got == want
            held += got or []
        elif op < 0.8 and held:
            rng.shuffle(held)
            k = rng.randint(1, len(held))
            assert native.free(held[:k]) == model.free(held[:k])
            held = held[k:]
        elif op < 0.9:
            assert native.restore_begin() == model.restore_begin()
        else:
            waiting = sorted(r for r, u in model.binding.items()
                             if u in model.sets[RESTORING])
            if waiting:
                native.restore_done(waiting[0])
                model.restore_done(waiting[0])
        same(native, model)


def test_rejected_calls_change_nothing():
    s = dps.SumManager(4, 4, 2)
    blocks = s.alloc(6)
    before = s.counts()
    for bad in ([blocks[0], blocks[0]], [99], [-1], [1]):   # twice, out of range, never given
        with pytest.raises(dps.DpsError):
            s.free(bad)
        assert s.counts() == before
    assert s.alloc(1000) is None and s.counts() == before
    with pytest.raises(dps.DpsError):
        s.restore_done(0)                                   # residual 0 is not restoring
    with pytest.raises(dps.DpsError):
        dps.SumManager(0, 4, 0)
    with pytest.raises(dps.DpsError):
        dps.SumManager(2, 4, 3)


def test_slots_follow_the_binding():
    s = dps.SumManager(5, 2, 3)
    assert s.slots(1, 8, 5).tolist() == [8, 9, 10, 11, 12]
    s.alloc(2 * 2 + 2)                   # units 3, 4, then BACKED unit 0
    with pytest.raises(dps.DpsError):
        s.slots(0, 8, 5)                 # residual 0 is evicted
    s.free(list(range(6, 10)))           # units 3 and 4 empty -> FREE
    assert s.restore_begin() == (0, 3)
    assert s.slots(0, 8, 5).tolist() == [24, 25, 26, 27, 28]
    with pytest.raises(dps.DpsError):
        s.slots(0, 8, 9)                 # more chunks than a unit holds


def test_concurrent_callers_keep_the_bookkeeping_whole():
    """The native manager locks every call: two host threads allocating and
    freeing KV blocks (the calls release the GIL) while a third reads the
    counts leave it exactly where it started, with every block handed out
    to one caller at a time."""
    import threading

    sm = dps.SumManager(8, 64, 2)
    start = sm.counts()
    seen = set()
    seen_lock = threading.Lock()
    errors = []

    def churn(seed):
        rnd = random.Random(seed)
        try:
            for _ in range(1500):
                blocks = sm.alloc(rnd.randint(1, 40))
                if blocks is None:
                    continue
                with seen_lock:
                    assert not seen.intersection(blocks)
                    seen.update(blocks)
                with seen_lock:
                    seen.difference_update(blocks)
                sm.free(blocks)
        except Exception as e:  # surfaced below
            errors.append(e)

    def read():
        try:
            for _ in range(3000):
                c = sm.counts()
                assert sum(c[k] for k in ("free", "backed", "avail", "full", "restoring")) == 8
        except Exception as e:  # surfaced below
            errors.append(e)

    threads = [threading.Thread(target=churn, args=(s,)) for s in (1, 2)]
    threads.append(threading.Thread(target=read))
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    end = sm.counts()
    assert end["free_blocks"] == end["avail"] * 64 and end["full"] == 0
    assert end["backed"] + end["evicted"] == start["backed"] == 2
    sm.close()
