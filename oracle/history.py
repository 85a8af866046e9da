"""Execution-history predicates of Sec. 4 -- TEST INFRASTRUCTURE ONLY.

A history is a sequence of operations (kind, worker, partition, iteration):
kind 'r' reads a partition, 'w' writes it (Definition 3).  The predicates are
the paper's:

* ``sequential``  -- Definition 4: operations of different iterations do not
  interleave, and within an iteration every read precedes every write.
* ``bsp``         -- Sec. 4.3: Read Barrier (every write of iteration a
  precedes every read of iteration a+1) and Write Barrier (every read of
  iteration a precedes every write of iteration a).
* ``rcwc``        -- Sec. 4.4: Read Constraint (the write of partition p in
  iteration a precedes every read of p in iteration a+1) and Write Constraint
  (every read of p in iteration a precedes the write of p in iteration a).
* ``partition_serial`` -- the three per-partition conditions that the proof of
  Theorem 2 establishes: restricted to one partition, the operations of
  different iterations do not interleave, come in increasing iteration order,
  and reads precede the write inside an iteration.  Unlike ``rcwc`` it also
  covers histories in which an iteration touches only some partitions (one
  sparse SGD example touches only its own features).

``parse`` reads the notation of the paper's figures, e.g.
``r_1[\\pi_1][1]w[\\pi_2][1]``; a missing worker subscript means worker 0.
"""
from __future__ import annotations

import re
from collections import defaultdict

_OP = re.compile(r"([rw])(?:_\{?(\d+)\}?)?\[\\pi_\{?(\d+)\}?\]\[(\d+)\]")


def parse(text: str):
    ops = [(m.group(1), int(m.group(2) or 0), int(m.group(3)), int(m.group(4)))
           for m in _OP.finditer(text)]
    if not ops:
        raise ValueError("no operations in %r" % text)
    return ops


def sequential(h) -> bool:
    last_iter = None
    wrote = False
    seen = set()
    for kind, _, _, it in h:
        if it != last_iter:
            if it in seen:
                return False          # iteration resumed after another one ran
            seen.add(it)
            last_iter, wrote = it, False
        if kind == "w":
            wrote = True
        elif wrote:
            return False              # read after a write in the same iteration
    return sorted(seen) == [it for it in dict.fromkeys(op[3] for op in h)]


def bsp(h) -> bool:
    pos = defaultdict(list)
    for t, (kind, _, _, it) in enumerate(h):
        pos[(kind, it)].append(t)
    for it in {op[3] for op in h}:
        writes, reads_next = pos[("w", it)], pos[("r", it + 1)]
        if writes and reads_next and max(writes) > min(reads_next):
            return False
        reads, writes = pos[("r", it)], pos[("w", it)]
        if reads and writes and max(reads) > min(writes):
            return False
    return True


def rcwc(h) -> bool:
    pos = defaultdict(list)
    for t, (kind, _, part, it) in enumerate(h):
        pos[(kind, part, it)].append(t)
    for (kind, part, it), ts in list(pos.items()):
        if kind != "w":
            continue
        reads_next = pos.get(("r", part, it + 1), [])
        if reads_next and max(ts) > min(reads_next):
            return False
        reads_same = pos.get(("r", part, it), [])
        if reads_same and max(reads_same) > min(ts):
            return False
    return True


def partition_serial(h) -> bool:
    per_part = defaultdict(list)
    for kind, _, part, it in h:
        per_part[part].append((kind, it))
    for ops in per_part.values():
        cur, wrote, done = None, False, set()
        for kind, it in ops:
            if it != cur:
                if it in done or (cur is not None and it < cur):
                    return False
                if cur is not None:
                    done.add(cur)
                cur, wrote = it, False
            if kind == "w":
                wrote = True
            elif wrote:
                return False
    return True


def level_history(row_ptr, col, level, within=None):
    """History of a level-by-level execution of one SGD epoch.

    Example i is iteration i; it reads every feature it touches, then writes
    them.  Levels run in increasing order; inside a level all reads of all its
    examples come first (in the order given by ``within``, default ascending
    index), then all writes.  This is what a concurrent execution of one level
    may look like in the worst case: any interleaving of a level's examples
    that keeps each example's reads before its writes is covered by it."""
    import numpy as np

    level = np.asarray(level)
    h = []
    for lv in sorted(set(level.tolist())):
        members = [int(i) for i in np.nonzero(level == lv)[0]]
        if within is not None:
            members = within(members)
        for i in members:
            for p in range(row_ptr[i], row_ptr[i + 1]):
                h.append(("r", 0, int(col[p]), i))
        for i in members:
            for p in range(row_ptr[i], row_ptr[i + 1]):
                h.append(("w", 0, int(col[p]), i))
    return h
