"""CPU model of the wave hand-out protocol of the resident-tile pointwise kernel
(``pw_tile_f32`` in ``paper_2105_14713_amd/csrc/conv_pw_tile.hip``).

One workgroup: a loader wave copies pixel tiles into two LDS buffers, compute
waves take the units of each tile from an LDS counter; LDS flags order the two
sides (``sSetup``, ``sReady``, ``sLanded``, ``sDone``, ``sNext``).  The model
follows the kernel's code step by step as Python generators that yield at
every access to shared state, and runs them under random interleavings, with
the loader's copies completing in issue order at random times (as a wave's
vector loads do).  It checks that:

* every wave terminates (no spin-wait is left waiting);
* every unit of every tile of the workgroup's range is taken exactly once;
* every X read of tile k sees buffer k % 2 holding all of tile k's copies
  and no copy of another tile landing in it meanwhile;
* the loader does not leave copies outstanding at its end.

The tests that plant mistakes (a mutated protocol in the model) show that the
checks catch them.  No GPU is used.
"""
import random

import pytest

K_EARLY = 32   # copies of the second tile issued before the first is published (kTileEarly)


class Deadlock(Exception):
    pass


class Violation(Exception):
    pass


class Model:
    def __init__(self, rng, nc, ntiles, u0, u1, units, loads, tfirst_differs, mutant=None):
        self.rng = rng
        self.nc = nc                     # compute waves (kTileCompute)
        self.ntiles = ntiles
        self.units = units               # units per tile
        self.u0, self.u1 = u0, u1        # first unit of tile 0, end unit of the last tile
        self.loads = loads               # copies (load instructions) per tile, by tile index k
        self.tfirst_differs = tfirst_differs
        self.mutant = mutant
        # Chance per scheduling step that the oldest outstanding load lands:
        # slow memory lets many loads pile up behind a copy.
        self.mem_rate = rng.choice([0.005, 0.02, 0.1, 0.3])
        self.sNext = [0, 0]
        self.sReady = [0, 0]
        self.sLanded = [0, 0]
        self.sDone = [0, 0]
        self.sSetup = 0
        self.pending = []                # outstanding loads of the loader: (tile key, buffer)
        self.holds = [(None, 0), (None, 0)]   # per buffer: (tile key, completed loads of it)
        self.taken = {}
        self.empty = {(k, u) for k in range(ntiles) for u in range(units) if rng.random() < 0.2}

    def unit_begin(self, k):
        return self.u0 if k == 0 else 0

    def unit_end(self, k):
        return self.u1 if k == self.ntiles - 1 else self.units

    # ---- memory: loads complete in issue order
    def complete_one(self):
        key, b = self.pending.pop(0)
        t, n = self.holds[b]
        self.holds[b] = (key, n + 1) if t == key else (key, 1)

    def full(self, b, key):
        return self.holds[b] == (key, self.loads_of(key))

    def loads_of(self, key):
        return self.loads[key] if isinstance(key, int) else self.loads_first

    # ---- the loader wave
    def copy_tile(self, key, b, early):
        """Issues the tile's loads; with `early`, publishes the first tile as
        landed once K_EARLY of them are issued (all earlier loads are then
        complete).  Returns whether it did."""
        issued = 0
        for _ in range(self.loads_of(key)):
            self.pending.append((key, b))
            issued += 1
            yield
            if early and issued == K_EARLY:
                limit = K_EARLY if self.mutant != "early_publish_too_soon" else K_EARLY + 8
                while len(self.pending) > limit:          # wait_vmem<kTileEarly>
                    yield
                self.sLanded[0] = 1                       # land_first()
                yield
        return issued >= K_EARLY

    def loader(self):
        # Set-up: the first tile of the cost range (Tfirst) is copied at once.
        first_key = "Tfirst" if (self.tfirst_differs or not self.ntiles) else 0
        self.loads_first = self.rng.randint(1, 60)
        yield from self.copy_tile(first_key, 0, False)
        while self.sSetup < self.nc:
            yield
        early = self.ntiles > 1
        for k in range(self.ntiles):
            b = k & 1
            if k >= 2 and self.mutant != "no_done_wait":
                while self.sDone[b] < self.nc * (k // 2):
                    yield
            if k > 0 and not (k == 1 and early):
                self.sNext[b] = self.unit_begin(k)
                yield
                self.sReady[b] = k + 1
                yield
            if (k > 0 and not (k == 1 and early)) or (k == 0 and self.tfirst_differs):
                yield from self.copy_tile(k, b, False)
            if k == 0 and early:
                self.sNext[1] = self.unit_begin(1)
                yield
                self.sReady[1] = 2
                yield
                published = yield from self.copy_tile(1, 1, True)
                if published:
                    continue
            while self.pending:                            # wait_vmem<0>
                yield
            self.sLanded[b] = k + 1
            yield
        while self.pending:
            yield

    # ---- a compute wave
    def compute(self, w):
        self.sSetup += 1                                   # after its share of the set-up
        yield
        while self.sSetup < self.nc:
            yield
        if w == 0 and self.ntiles > 0:
            self.sNext[0] = self.unit_begin(0)
            yield
            self.sReady[0] = 1
            yield
        for k in range(self.ntiles):
            b = k & 1
            ue = self.unit_end(k)
            if self.mutant != "no_ready_wait":
                while self.sReady[b] < k + 1:
                    yield
            claimed = []

            def next_unit():
                # atomicAdd on the tile's counter until a unit with kept blocks
                # (units without any are stored as zeros right away)
                while True:
                    u = self.sNext[b]
                    self.sNext[b] = u + 1
                    if u >= ue:
                        return None
                    if (k, u) in self.taken:
                        raise Violation(f"unit {u} of tile {k} taken twice")
                    if not (0 <= u < self.units) or u < self.unit_begin(k):
                        raise Violation(f"unit {u} outside tile {k}'s range")
                    self.taken[(k, u)] = w
                    if (k, u) not in self.empty:
                        return u

            u = next_unit()
            yield
            if u is not None:
                claimed.append(u)
                for _ in range(3):                          # blocks j+1 .. j+3 planned ahead
                    nu = next_unit()
                    yield
                    if nu is None:
                        break
                    claimed.append(nu)
                while self.sLanded[b] < k + 1:
                    yield
                more = len(claimed) == 4
                while claimed:
                    claimed.pop(0)
                    if not self.full(b, k) or any(pb == b for _, pb in self.pending):
                        raise Violation(f"wave {w} read tile {k} from buffer {b} holding "
                                        f"{self.holds[b]} with {len(self.pending)} loads pending")
                    yield
                    if more:
                        nu = next_unit()
                        yield
                        if nu is None:
                            more = False
                        else:
                            claimed.append(nu)
            self.sDone[b] += 1                             # atomicAdd(&sDone[b], 1)
            yield

    def run(self, max_steps=400000):
        procs = {"loader": self.loader()}
        for w in range(self.nc):
            procs[w] = self.compute(w)
        steps = 0
        while procs:
            steps += 1
            if steps > max_steps:
                raise Deadlock(f"still running: {sorted(map(str, procs))}, pending {len(self.pending)}, "
                               f"ready {self.sReady} landed {self.sLanded} done {self.sDone}")
            if self.pending and self.rng.random() < self.mem_rate:
                self.complete_one()
                continue
            name = self.rng.choice(list(procs))
            try:
                next(procs[name])
            except StopIteration:
                del procs[name]
        if self.pending:
            raise Violation("loads outstanding after the loader ended")
        for k in range(self.ntiles):
            for u in range(self.unit_begin(k), self.unit_end(k)):
                if (k, u) not in self.taken:
                    raise Violation(f"unit {u} of tile {k} never taken")


def random_case(rng, mutant=None):
    nc = rng.choice([2, 3, 5, 15])
    units = rng.randint(1, 40)
    ntiles = rng.choice([0, 1, 1, 2, 2, 3, 4, 5])
    u0 = rng.randint(0, units - 1) if ntiles else 0
    u1 = rng.randint(1, units) if ntiles else 0
    if ntiles == 1:
        u1 = rng.randint(u0 + 1, units) if u0 + 1 <= units else units
    loads = [rng.choice([1, 5, K_EARLY - 1, K_EARLY, K_EARLY + 1, 80]) for _ in range(max(ntiles, 1))]
    return Model(rng, nc, ntiles, u0, u1, units, loads, rng.random() < 0.25, mutant)


@pytest.mark.parametrize("seed", range(300))
def test_pw_tile_protocol_random_interleavings(seed):
    random_case(random.Random(seed)).run()


def test_early_publish_path_is_exercised():
    """The early-publish branch (second tile copied right behind the first,
    the first published from inside that copy) runs in the random cases."""
    hits = 0
    for seed in range(300):
        m = random_case(random.Random(seed))
        if m.ntiles > 1 and m.loads[1] >= K_EARLY:
            hits += 1
    assert hits >= 30


@pytest.mark.parametrize("mutant", ["no_done_wait", "early_publish_too_soon", "no_ready_wait"])
def test_model_catches_planted_protocol_mistakes(mutant):
    """Each mutant drops one ordering of the protocol; some interleaving must
    expose it (a read of a buffer not holding its tile, a unit taken twice or
    never, or a wave left waiting)."""
    caught = 0
    for seed in range(400):
        try:
            random_case(random.Random(seed), mutant).run(max_steps=100000)
        except (Violation, Deadlock):
            caught += 1
    assert caught > 0, mutant
