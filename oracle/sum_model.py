"""Plain model of the SUM manager's unit bookkeeping (Sec. IV-B "SUM manager";
Sec. IV-D, Algorithm 1).

TEST INFRASTRUCTURE: only tests/ use it.  It shares no code with the
library's native manager (paper_2609_34380_amd/csrc/dps_sum.cpp); tests drive
both with the same operations and compare every observable.

The algorithm's steps in the paper's order and names; where the paper leaves
a choice open, the readings below (the same ones the library documents):
  - a "pop" takes the unit with the lowest id; a unit hands out its lowest
    free block indices first;
  - a request that does not fit in AVAIL, FREE and BACKED units together takes
    nothing (the loop would otherwise fail after taking what it found);
  - evicting a BACKED unit marks its residual both STALE (the mapping) and
    EVICTED (the data is on the host only); the restore worker binds the
    lowest stale residual to the lowest FREE unit (held as RESTORING), and the
    residual leaves EVICTED when its copy completes;
  - the mode is fast exactly while EVICTED is non-empty.
"""

FREE, BACKED, AVAIL, FULL, RESTORING = "FREE", "BACKED", "AVAIL", "FULL", "RESTORING"
MODE_FULL, MODE_FAST = 0, 1


class NoSpace(Exception):
    pass


class SumModel:
    def __init__(self, n_units, blocks_per_unit, n_res):
        assert 1 <= n_units and 1 <= blocks_per_unit and 0 <= n_res <= n_units
        self.B = blocks_per_unit
        self.n_units = n_units
        # the five unit sets and the two residual sets of Algorithm 1
        self.sets = {FREE: set(range(n_res, n_units)), BACKED: set(range(n_res)),
                     AVAIL: set(), FULL: set(), RESTORING: set()}
        self.STALE = set()
        self.EVICTED = set()
        self.allocated = {u: set() for u in range(n_units)}   # block indices in use
        self.binding = {r: r for r in range(n_res)}            # residual -> unit
        self.mode = MODE_FULL

    # -- helpers ------------------------------------------------------------
    def state_of(self, u):
        for name, units in self.sets.items():
            if u in units:
                return name
        raise AssertionError("unit %d in no set" % u)

    def _pop(self, name):
        u = min(self.sets[name])
        self.sets[name].remove(u)
        return u

    def _room(self):
        room = (len(self.sets[FREE]) + len(self.sets[BACKED])) * self.B
        return room + sum(self.B - len(self.allocated[u]) for u in self.sets[AVAIL])

    # -- AllocKVBlock(n) ----------------------------------------------------
    def alloc(self, n):
        if n > self._room():
            raise NoSpace()
        result = []
        while len(result) < n:
            if not self.sets[AVAIL]:
                if self.sets[FREE]:
                    u = self._pop(FREE)
                else:
                    u = self._pop(BACKED)
                    self.mode = MODE_FAST                  # activate lower-precision mode
                    r = [r for r, unit in self.binding.items() if unit == u][0]
                    del self.binding[r]
                    self.STALE.add(r)                      # mapping is stale
                    self.EVICTED.add(r)                    # data on the host only
                self.sets[AVAIL].add(u)
            u = self._pop(AVAIL)
            for i in range(self.B):
                if len(result) == n:
                    break
                if i not in self.allocated[u]:
                    self.allocated[u].add(i)
                    result.append(u * self.B + i)
            if len(self.allocated[u]) == self.B:
                self.sets[FULL].add(u)
            else:
                self.sets[AVAIL].add(u)
        return result

    # -- FreeKVBlock(blocks) ------------------------------------------------
    def free(self, blocks):
        assert len(set(blocks)) == len(blocks)
        for b in blocks:
            u, i = divmod(b, self.B)
            assert i in self.allocated[u] and self.state_of(u) in (AVAIL, FULL)
        wake = False
        for b in blocks:
            u, i = divmod(b, self.B)
            self.allocated[u].remove(i)                    # mark the block free
            if u in self.sets[FULL]:
                self.sets[FULL].remove(u)
                self.sets[AVAIL].add(u)
            if not self.allocated[u]:
                self.sets[AVAIL].remove(u)
                self.sets[FREE].add(u)
                if self.EVICTED:
                    wake = True                            # wake RestoreWeights
        return wake

    # -- restore worker -----------------------------------------------------
    def restore_begin(self):
        if not self.STALE or not self.sets[FREE]:
            return None
        r = min(self.STALE)
        self.STALE.remove(r)
        u = self._pop(FREE)
        self.sets[RESTORING].add(u)
        self.binding[r] = u
        return r, u

    def restore_done(self, r):
        u = self.binding[r]
        assert u in self.sets[RESTORING] and r in self.EVICTED
        self.sets[RESTORING].remove(u)
        self.sets[BACKED].add(u)
        self.EVICTED.remove(r)
        if not self.EVICTED:
            self.mode = MODE_FULL

    # -- observables --------------------------------------------------------
    def counts(self):
        return {"free": len(self.sets[FREE]), "backed": len(self.sets[BACKED]),
                "avail": len(self.sets[AVAIL]), "full": len(self.sets[FULL]),
                "restoring": len(self.sets[RESTORING]), "stale": len(self.STALE),
                "evicted": len(self.EVICTED),
                "free_blocks": sum(self.B - len(self.allocated[u]) for u in self.sets[AVAIL])}

    def unit_of(self, r):
        return self.binding.get(r, -1)
