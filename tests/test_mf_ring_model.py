"""A CPU model of the one-compute-unit matrix-completion epoch's protocol
(the Read Protocol of Sec. 5 at row grain, every rating on one block).

Actors, each taking one small step at a time:
  * the producer stages ratings into a ring of RING slots, PB at a time, after
    checking that no worker may still read the slots it reuses: it reads the
    ticket counter first, then every worker's bound, and reuses the slots of
    ratings below min(bound, T * counter) only; then it publishes `ready`;
  * a worker publishes a bound (T times the counter as it reads now), takes a
    ticket of T consecutive ratings from the counter, publishes the ticket's
    first rating as its bound, waits for `ready`, reads the ticket's ring
    slots, clears its bound, then runs each rating as soon as both of its
    rows carry the rating's previous writers as tags, and publishes both rows
    tagged with the rating.

The model runs under random and adversarial schedulers and checks that (a)
no worker ever reads a ring slot the producer has reused, (b) the run never
deadlocks while work remains, and (c) the rows end as running the ratings
one after another gives.  Planted mistakes (a producer that ignores the
counter or reads it after the bounds, a worker that clears its bound before
reading its slots) must be caught.  Plain Python: no kernel code is run and
none is shared."""
import random

import pytest

INF = float("inf")


def make_ratings(rng, n, nu, ni, hot=0.5):
    """(user, item) per rating; a few hot rows make long chains."""
    out = []
    for _ in range(n):
        u = 0 if rng.random() < hot / 2 else rng.randrange(nu)
        i = 0 if rng.random() < hot / 2 else rng.randrange(ni)
        out.append((u, nu + i))  # rows: users, then items
    return out


def previous(ratings):
    last, prev = {}, []
    for q, (a, b) in enumerate(ratings):
        prev.append((last.get(a, -1), last.get(b, -1)))
        last[a] = q
        last[b] = q
    return prev


def step_values(va, vb, q):
    """A rating's new row values from both old ones (order matters)."""
    return ((va * 31 + vb * 17 + q + 1) % 1000003, (vb * 29 + va * 13 + q + 3) % 1000003)


def sequential(ratings, rows):
    val = [0] * rows
    for q, (a, b) in enumerate(ratings):
        val[a], val[b] = step_values(val[a], val[b], q)
    return val


class SlotReused(AssertionError):
    pass


class Deadlock(AssertionError):
    pass


def run(ratings, rows, workers, T, RING, PB, pick, plant=None, max_steps=200000):
    n = len(ratings)
    prev = previous(ratings)
    n_tk = (n + T - 1) // T
    tag = [-1] * rows
    val = [0] * rows
    ring = [None] * RING  # the rating a slot holds
    sh = {"ready": 0, "next": 0}
    prog = [INF] * workers

    def producer():
        q0 = 0
        while q0 < n:
            # ring space: the counter first, then every worker's bound
            if plant == "ignore_counter":
                cnt = INF
            elif plant == "counter_last":
                cnt = None
            else:
                cnt = T * sh["next"]
                yield
            mn = INF
            for w in range(workers):
                mn = min(mn, prog[w])
                yield
            if plant == "counter_last":
                cnt = T * sh["next"]
                yield
            mn = min(mn, cnt)
            if mn + RING < q0 + PB:
                continue  # no space yet: check again
            for q in range(q0, min(q0 + PB, n)):
                ring[q % RING] = q
                yield
            sh["ready"] = min(q0 + PB, n)
            yield
            q0 += PB

    def worker(w):
        while True:
            prog[w] = T * sh["next"]
            yield
            k = sh["next"]
            sh["next"] += 1  # the atomic take
            yield
            if k >= n_tk:
                prog[w] = INF
                return
            q0 = T * k
            prog[w] = q0
            yield
            qs = list(range(q0, min(q0 + T, n)))
            while sh["ready"] < qs[-1] + 1:
                yield
            if plant == "clear_early":
                prog[w] = INF
                yield
            for q in qs:
                if ring[q % RING] != q:
                    raise SlotReused("worker %d read slot of rating %d: holds %r" % (w, q, ring[q % RING]))
                yield
            prog[w] = INF
            yield
            pending = list(qs)
            while pending:
                for q in list(pending):
                    a, b = ratings[q]
                    pa, pb = prev[q]
                    if tag[a] == pa and tag[b] == pb:
                        va, vb = val[a], val[b]
                        yield
                        na, nb = step_values(va, vb, q)
                        val[a], tag[a] = na, q
                        yield
                        val[b], tag[b] = nb, q
                        pending.remove(q)
                        yield
                if pending:
                    yield  # a poll round with nothing ready

    actors = [producer()] + [worker(w) for w in range(workers)]
    alive = list(range(len(actors)))
    stalled = 0
    for steps in range(max_steps):
        if not alive:
            return val
        before = (sh["ready"], sh["next"], tuple(tag), tuple(prog), tuple(ring))
        i = pick(alive, steps)
        try:
            next(actors[i])
        except StopIteration:
            alive.remove(i)
        after = (sh["ready"], sh["next"], tuple(tag), tuple(prog), tuple(ring))
        stalled = 0 if after != before else stalled + 1
        if stalled > 50 * len(actors) * (RING + workers + 4):
            raise Deadlock("no progress: ready %d, next %d, alive %r" % (sh["ready"], sh["next"], alive))
    raise Deadlock("step limit")


def random_pick(rng):
    return lambda alive, step: rng.choice(alive)


def bursty_pick(rng):
    """Runs one actor for a while, then another: long stretches in which the
    producer or a worker races ahead of the others."""
    state = {"cur": None, "left": 0}

    def pick(alive, step):
        if state["cur"] not in alive or state["left"] == 0:
            state["cur"] = rng.choice(alive)
            state["left"] = rng.randint(1, 40)
        state["left"] -= 1
        return state["cur"]

    return pick


def starve_pick(rng, victim):
    """The victim actor runs only rarely."""
    return lambda alive, step: (victim if victim in alive and rng.random() < 0.02
                                else rng.choice([a for a in alive if a != victim] or alive))


CASES = [  # (seed, ratings, users, items, workers, RING, PB)
    (1, 24, 3, 2, 2, 8, 2),
    (2, 40, 4, 3, 3, 8, 4),
    (3, 60, 5, 5, 4, 16, 4),
    (4, 33, 2, 2, 3, 8, 2),
    (5, 80, 8, 3, 4, 16, 8),
]


@pytest.mark.parametrize("case", CASES)
def test_ring_protocol_sequential_result(case):
    seed, n, nu, ni, workers, RING, PB = case
    rng = random.Random(seed)
    ratings = make_ratings(rng, n, nu, ni)
    want = sequential(ratings, nu + ni)
    for trial in range(20):
        srng = random.Random(seed * 1000 + trial)
        picks = [random_pick(srng), bursty_pick(srng)] + [starve_pick(srng, v) for v in range(workers + 1)]
        for pick in picks:
            assert run(ratings, nu + ni, workers, 2, RING, PB, pick) == want


@pytest.mark.parametrize("plant", ["ignore_counter", "counter_last", "clear_early"])
def test_ring_protocol_planted_mistakes_caught(plant):
    caught = 0
    for seed in range(40):
        rng = random.Random(seed)
        ratings = make_ratings(rng, 40, 3, 3)
        srng = random.Random(7 * seed + 1)
        for pick in (bursty_pick(srng), random_pick(srng), starve_pick(srng, 1)):
            try:
                run(ratings, 6, 3, 2, 8, 2, pick, plant=plant)
            except SlotReused:
                caught += 1
    assert caught > 0, "a planted mistake in the ring protocol went unnoticed"


def test_sequential_reference_is_order_sensitive():
    """The model's check has teeth: two ratings on one row give a different
    result when swapped."""
    r = [(0, 2), (0, 3)]
    assert sequential(r, 4) != sequential(list(reversed(r)), 4)
