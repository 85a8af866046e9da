"""A CPU model of the sync-free mini-batch epoch's hand-over protocol (the
Read Protocol of Sec. 5 with a batch as the iteration): every feature's
weight shares one word with the tag of the union entry that wrote it last;
blocks take batches in index order from a shared ticket counter; a batch
reads each of its features once and polls those whose word does not yet
carry the feature's previous union entry, computes, and publishes its words
one by one (the features the next batch needs first).

The model runs the protocol under every interleaving of the blocks' single
steps (exhaustively for tiny inputs, under random and adversarial schedulers
for larger ones), with blocks that start late (a launch that is not
cooperative) and checks that (a) it never deadlocks while the earliest
unfinished batch can step, and (b) the final words are those of running the
batches one after another.  A planted mistake (a batch that reads without
checking the tag) must be caught.  The model is plain Python: no kernel code
is executed, and none is shared."""
import random

import pytest


def make_batches(rng, nb, d, width):
    """Each batch's union of features, ascending, at least one feature."""
    return [sorted(rng.sample(range(d), rng.randint(1, width))) for _ in range(nb)]


def prev_entries(batches):
    """For batch b and its k-th feature: the previous batch that touches the
    feature (-1 if none), the tag the word must carry before b may read it."""
    last = {}
    prev = []
    for b, feats in enumerate(batches):
        prev.append([last.get(f, -1) for f in feats])
        for f in feats:
            last[f] = b
    return prev


def next_entries(batches):
    """For batch b's k-th feature: is the next batch touching it b + 1."""
    nxt = []
    for b, feats in enumerate(batches):
        later = set(batches[b + 1]) if b + 1 < len(batches) else set()
        nxt.append([f in later for f in feats])
    return nxt


def update(old, b, f):
    """A batch's new value of a feature: depends on the old value, so a lost
    or reordered update changes the result."""
    return (old * 1000003 + 7 * b + f + 1) % (1 << 31)


def sequential(batches, d):
    w = [0] * d
    for b, feats in enumerate(batches):
        for f in feats:
            w[f] = update(w[f], b, f)
    return w


class Block:
    """One block's state: idle (take a ticket), reading (feature k of its
    batch: one poll per step), publishing (one word per step)."""

    def __init__(self, start):
        self.start = start       # scheduler step before which the block is not resident
        self.state = "idle"
        self.b = -1
        self.k = 0
        self.vals = []
        self.order = []


def run(batches, d, n_blocks, pick, check_tag=True, max_steps=10 ** 6, starts=None):
    """Runs the protocol; pick(runnable, blocks, step) chooses the block that
    takes the next step.  Returns the final values, or raises on deadlock."""
    nb = len(batches)
    prev = prev_entries(batches)
    urgent = next_entries(batches)
    words = [(0, -1)] * d        # (value, tag of the last writer)
    ticket = 0
    blocks = [Block(0 if starts is None else starts[i]) for i in range(n_blocks)]
    done = 0
    for step in range(max_steps):
        runnable = []
        for i, blk in enumerate(blocks):
            if blk.state == "exit" or step < blk.start:
                continue
            if blk.state == "reading":
                f = batches[blk.b][blk.k]
                if check_tag and words[f][1] != prev[blk.b][blk.k]:
                    # a poll that would fail: the block can step (spin) but
                    # makes no progress; only count it runnable if nothing
                    # else is, to tell deadlock from waiting
                    continue
            runnable.append(i)
        if not runnable:
            live = [blk for blk in blocks if blk.state != "exit"]
            if not live:
                break
            if any(step < blk.start for blk in live):
                continue  # a block not yet resident: time passes
            raise RuntimeError("deadlock: every live block waits")
        blk = blocks[pick(runnable, blocks, step)]
        if blk.state == "idle":
            blk.b = ticket
            ticket += 1
            if blk.b >= nb:
                blk.state = "exit"
                continue
            blk.state, blk.k, blk.vals = "reading", 0, []
        elif blk.state == "reading":
            f = batches[blk.b][blk.k]
            blk.vals.append(update(words[f][0], blk.b, f))
            blk.k += 1
            if blk.k == len(batches[blk.b]):
                ks = range(len(batches[blk.b]))
                # publish the features the next batch needs first
                blk.order = [k for k in ks if urgent[blk.b][k]] + \
                            [k for k in ks if not urgent[blk.b][k]]
                blk.state = "publishing"
        elif blk.state == "publishing":
            k = blk.order.pop(0)
            words[batches[blk.b][k]] = (blk.vals[k], blk.b)
            if not blk.order:
                blk.state = "idle"
                done += 1
    else:
        raise RuntimeError("no end within the step bound")
    assert done == nb
    return [v for v, _ in words]


def uniform_pick(rng):
    return lambda runnable, blocks, step: rng.choice(runnable)


def latest_first(runnable, blocks, step):
    """Adversarial: always step the block holding the latest batch (idle
    blocks count as latest), so early batches advance only when forced."""
    return max(runnable, key=lambda i: (blocks[i].state == "idle", blocks[i].b))


def earliest_last_publish(runnable, blocks, step):
    """Adversarial: delay every publish as long as anything else can step."""
    others = [i for i in runnable if blocks[i].state != "publishing"]
    return (others or runnable)[0]


def all_schedules(batches, d, n_blocks):
    """Results over every interleaving of single steps: the choice sequences
    are enumerated like an odometer (a run replays a prefix of choices and
    takes the first runnable block after it)."""
    results = set()
    path = []  # (choice, number of runnable blocks) at each step of the last run
    runs = 0
    while True:
        record = []

        def pick(runnable, blocks, step):
            i = len(record)
            c = path[i][0] if i < len(path) else 0
            record.append((c, len(runnable)))
            return runnable[c]

        results.add(tuple(run(batches, d, n_blocks, pick)))
        runs += 1
        path = record
        while path and path[-1][0] + 1 >= path[-1][1]:
            path.pop()
        if not path:
            return results, runs
        c, k = path[-1]
        path[-1] = (c + 1, k)


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("nb,d,n_blocks", [(3, 2, 2), (4, 3, 2), (3, 3, 3)])
def test_every_interleaving_of_tiny_inputs(seed, nb, d, n_blocks):
    rng = random.Random(seed)
    batches = make_batches(rng, nb, d, 2)
    got, runs = all_schedules(batches, d, n_blocks)
    assert runs > 1
    assert got == {tuple(sequential(batches, d))}


@pytest.mark.parametrize("seed", range(20))
@pytest.mark.parametrize("n_blocks", [2, 5, 32])
def test_random_and_adversarial_schedulers(seed, n_blocks):
    rng = random.Random(1000 + seed)
    nb = rng.randint(20, 80)
    d = rng.randint(3, 40)
    batches = make_batches(rng, nb, d, min(d, 8))
    ref = sequential(batches, d)
    for pick in (uniform_pick(rng), latest_first, earliest_last_publish):
        # blocks become resident at random times (a launch that is not cooperative)
        starts = [rng.randint(0, 200) for _ in range(n_blocks)]
        assert run(batches, d, n_blocks, pick, starts=starts) == ref


def test_a_chain_of_batches_sharing_one_feature():
    """Every batch touches feature 0 (the configs' hot feature): the batches
    form one chain and the blocks hand the word on in ticket order."""
    batches = [[0] + ([1 + b % 5] if b % 2 else []) for b in range(60)]
    ref = sequential(batches, 6)
    for n_blocks in (1, 2, 7, 32):
        assert run(batches, 6, n_blocks, latest_first) == ref


def test_reading_without_the_tag_check_is_caught():
    """The planted mistake: a batch that reads a word without waiting for its
    previous writer.  Some schedule then differs from the sequential result."""
    rng = random.Random(5)
    batches = make_batches(rng, 30, 6, 3)
    ref = sequential(batches, 6)
    wrong = 0
    for s in range(20):
        r = random.Random(s)
        got = run(batches, 6, 4, uniform_pick(r), check_tag=False)
        wrong += got != ref
    assert wrong > 0
