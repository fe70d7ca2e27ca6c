"""The one-launch LSTM recurrence's step protocol, modelled on the CPU under adversarial schedules.

The kernel (one block per tile of a batch group; tiles of different groups never interact) is
a set of concurrent programs sharing three kinds of state: the h of each (step, tile), visible
to others some time after it is stored; a claim word per (step, tile); and the cell state a
helper leaves for the tile's next step.  This model runs the same decisions as the kernel:

* a block first claims every step of its own tile that nobody has claimed;
* for each step it owns, it polls h_{t-1} of the group; after a grace period it walks the group
  from the last step it has seen complete, and at the first step with h still missing it claims
  a missing, unclaimed tile and computes it (a helper), else polls again;
* after its last step it walks to the end of the sequence the same way.

Blocks may never start, start late, or be delayed at any point, and a stored h becomes visible
to each block after a delay of its own (caches of different dies see a store at different
times; a helper's cell state, stored and completed before its h, is visible at once).  Every
schedule must end with every (step, tile) computed exactly once, each by a block that itself
sees all of h_{t-1} and with the right cell state, and no block may wait forever.
"""
import heapq
import random

import pytest

pytestmark = pytest.mark.filterwarnings("ignore")


class Group:
    def __init__(self, ng, T, rng, max_delay):
        self.ng, self.T, self.rng, self.max_delay = ng, T, rng, max_delay
        # seen[b][t][m]: block b sees the h of (step t, tile m)
        self.seen = [[[False] * ng for _ in range(T)] for _ in range(ng)]
        self.pending = []                                   # (time it shows, observer, step, tile)
        self.claim = [[0] * ng for _ in range(T)]
        self.c_step = [-1] * ng                             # step of the cell state in memory
        self.computed = [[0] * ng for _ in range(T)]
        self.now = 0

    def tick(self):
        self.now += 1
        while self.pending and self.pending[0][0] <= self.now:
            _, b, t, m = heapq.heappop(self.pending)
            self.seen[b][t][m] = True

    def complete(self, b, t):
        return all(self.seen[b][t])

    def compute(self, b, t, m, cvalid_step, helper):
        # the input of (t, m) as block b reads it: all of h_{t-1}, and c_{t-1} of tile m
        assert t == 0 or self.complete(b, t - 1), f"({t}, {m}) computed from an incomplete h_{t - 1}"
        if t > 0:
            c = cvalid_step if cvalid_step is not None else self.c_step[m]
            assert c == t - 1, f"({t}, {m}) computed with the cell state of step {c}"
        self.computed[t][m] += 1
        if helper and t + 1 < self.T:
            self.c_step[m] = t                              # stored and completed before its h
        for o in range(self.ng):
            heapq.heappush(self.pending, (self.now + self.rng.randint(0, self.max_delay), o, t, m))


def block(g, own, grace):
    """One block's program: a generator that yields at every point where others may run."""
    T = g.T
    mine = set()
    for t in g.rng.sample(range(T), T):                     # claims, in any order (one thread per step)
        if g.claim[t][own] == 0:
            g.claim[t][own] = 1
            mine.add(t)
        yield
    v = -1
    c_own = None                                            # step of c this block holds in registers

    def help_until(target):
        nonlocal v
        while v < target:
            f = v + 1
            yield
            missing = [m for m in range(g.ng) if not g.seen[own][f][m]]
            if not missing:
                v = f
                continue
            pick = next((m for m in missing if g.claim[f][m] == 0), None)
            if pick is None:
                continue                                    # all claimed: poll again
            g.claim[f][pick] = 1
            yield
            g.compute(own, f, pick, None, helper=True)
            yield

    for t in range(T):
        if t not in mine:
            c_own = None
            continue
        while True:
            polls = 0
            while t > 0 and not g.complete(own, t - 1) and polls < grace:
                polls += 1
                yield
            if t == 0 or g.complete(own, t - 1):
                break
            yield from help_until(t - 1)
        g.compute(own, t, own, c_own, helper=False)
        c_own = t
        if v < t - 1:
            v = t - 1
        yield
    yield from help_until(T - 1)


def run(seed, ng, T, absent_frac, late_max, max_delay, grace, program=block):
    rng = random.Random(seed)
    g = Group(ng, T, rng, max_delay)
    start = {}
    for m in range(ng):
        if rng.random() < absent_frac:
            continue
        start[m] = rng.randint(0, late_max)
    if not start:
        start[rng.randrange(ng)] = 0                        # at least one block runs
    live = {m: program(g, m, grace) for m in start}
    for _ in range(200000):
        if not live:
            break
        g.tick()
        ready = [m for m in live if start[m] <= g.now]
        if not ready:
            continue
        m = rng.choice(ready)
        try:
            next(live[m])
        except StopIteration:
            del live[m]
    assert not live, f"seed {seed}: blocks still waiting after 200000 ticks"
    while g.pending:
        g.tick()
    for t in range(T):
        for m in range(ng):
            assert g.computed[t][m] == 1, f"seed {seed}: ({t}, {m}) computed {g.computed[t][m]} times"
    return g


@pytest.mark.parametrize("ng,T", [(1, 3), (2, 5), (3, 7), (5, 4)])
def test_every_schedule_finishes_each_tile_once_from_complete_inputs(ng, T):
    for seed in range(150):
        run(seed, ng, T, absent_frac=0.4, late_max=60, max_delay=6, grace=4)


def test_all_owners_present_need_no_helper():
    # with every block running and a grace longer than any wait, owners compute their own tiles
    for seed in range(50):
        g = run(seed, 4, 6, absent_frac=0.0, late_max=0, max_delay=3, grace=10 ** 6)
        assert all(c == 1 for row in g.computed for c in row)


def test_the_model_catches_a_helper_that_has_not_seen_its_input_complete():
    # planted mistake, the kernel's earlier form: a block waits only before the steps it owns
    # and, when that wait runs long, helps at the step it waits for.  An owner that starts late,
    # after helpers took its first steps, has not itself seen the step before that one complete
    # (others have), so sooner or later it computes a tile from an h it does not yet see.
    def old_block(g, own, grace):
        T = g.T
        mine = set()
        for t in g.rng.sample(range(T), T):
            if g.claim[t][own] == 0:
                g.claim[t][own] = 1
                mine.add(t)
            yield

        def await_step(s):
            polls = 0
            while not g.complete(own, s):
                polls += 1
                if polls > grace:
                    free = [m for m in range(g.ng) if not g.seen[own][s][m] and g.claim[s][m] == 0]
                    if free:
                        g.claim[s][free[0]] = 1
                        yield
                        g.compute(own, s, free[0], None, helper=True)
                yield

        c_own = None
        for t in range(T):
            if t not in mine:
                c_own = None
                continue
            if t > 0:
                yield from await_step(t - 1)
            g.compute(own, t, own, c_own, helper=False)
            c_own = t
            yield
        yield from await_step(T - 1)

    # the window is narrow (a late owner has to arrive while a step it does not yet see complete
    # still has a free tile), so the schedules are many and the delays long
    sched = dict(absent_frac=0.5, late_max=200, max_delay=200, grace=1)
    caught = 0
    for seed in range(600):
        try:
            run(seed, 8, 5, program=old_block, **sched)
        except AssertionError:
            caught += 1
    assert caught > 0
    # ... while the kernel's protocol passes the same schedules
    for seed in range(600):
        run(seed, 8, 5, **sched)
