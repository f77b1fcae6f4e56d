"""Reference enumeration of the paper's dQ-reduction schedules, and its DAG model.

TEST INFRASTRUCTURE ONLY: imported by the test suite, never by the product
path.  It shares no code with the closed-form schedule functions in the HIP
library; the tests compare the two tables entry by entry.

A schedule says, for one attention head, (a) which KV tiles each workgroup
owns and in which order it visits the Q tiles of each (a "chain" of tasks),
and (b) the order in which the dQ partials of each Q tile are summed.  Both
are written here as plain enumerations, straight from the paper's words, and
the accumulation order is *derived* by sorting rather than by a formula:

* NAIVE -- the deterministic baseline of the Background section and of the
  schedule analysis (Section 3.2): every KV tile visits its Q tiles in
  ascending order; each dQ tile is accumulated in ascending KV order.
* DESCENDING -- Descending Q-Tile Iteration (Section 3.3): same work, Q tiles
  visited last-to-first; the accumulation order is unchanged (ascending KV).
* SHIFT -- Shift Scheduling, full mask (Section 3.4, "Optimal Schedule for
  Full Masks"): workgroup j starts at a cyclically shifted Q tile; the dQ
  order follows the visiting timestamps (Fig. 6 caption: distinct timestamps
  per dQ row induce the reduction sequence).  With T_r = g*T_c Q tiles the
  shift is g tiles per workgroup (reading for unequal tile sizes).  When the
  workgroups of one head cannot all run at once (the "refine or aggregate
  heads" case of Section 3.1), the KV tiles are cut into groups of `group`
  consecutive tiles: each dQ tile sums group 0's partials in visiting order,
  then group 1's, and so on.
* SYMSHIFT -- Symmetric Shift, causal mask (Section 3.4, "Symmetric Shift
  Scheduling for Causal Masks"): workgroup p owns KV tiles p and T-1-p; phase 1
  is a cyclic shift over the dense lower-left rectangle, phase 2 walks the
  upper-left triangle top-down from the diagonal and then the lower-right
  triangle bottom-up, ending on the diagonal; the dQ order follows the
  visiting timestamps.

Q tile i (rows [i*Br, (i+1)*Br)) and KV tile j (rows [j*Bc, (j+1)*Bc)) interact
under a causal mask iff the last query row of the Q tile reaches the first key
of the KV tile: (i+1)*Br - 1 >= j*Bc.
"""
from __future__ import annotations

import heapq
from dataclasses import dataclass

NAIVE, DESCENDING, SHIFT, SYMSHIFT = "naive", "descending", "shift", "symshift"
SCHEDULES = (NAIVE, DESCENDING, SHIFT, SYMSHIFT)


def interacts(i: int, j: int, br: int, bc: int, causal: bool) -> bool:
    """Does Q tile i see any key of KV tile j?"""
    return (not causal) or ((i + 1) * br - 1 >= j * bc)


@dataclass
class Schedule:
    """One head's schedule.

    chains[w] = list of (kv_tile, q_tile) in the order workgroup w runs them.
    order[i]  = KV tiles contributing to Q tile i, in accumulation order.
    """
    chains: list
    order: dict

    def rank(self, i: int, j: int) -> int:
        return self.order[i].index(j)

    def step_of(self):
        """(i, j) -> (workgroup, position in its chain)."""
        out = {}
        for w, ch in enumerate(self.chains):
            for t, (j, i) in enumerate(ch):
                out[(i, j)] = (w, t)
        return out


def build(kind: str, t_r: int, t_c: int, causal: bool, br: int, bc: int, group: int | None = None) -> Schedule:
    """Enumerate one head's schedule for t_r Q tiles and t_c KV tiles
    (`group`: SHIFT only, KV tiles per group; None = one group)."""
    valid_q = {j: [i for i in range(t_r) if interacts(i, j, br, bc, causal)] for j in range(t_c)}
    if kind == NAIVE:
        chains = [[(j, i) for i in valid_q[j]] for j in range(t_c)]
        by_timestamp = False
    elif kind == DESCENDING:
        chains = [[(j, i) for i in reversed(valid_q[j])] for j in range(t_c)]
        by_timestamp = False
    elif kind == SHIFT:
        if causal:
            raise ValueError("shift is the full-mask schedule; symshift is its causal form")
        if t_r % t_c:
            raise ValueError("shift needs a whole number of Q tiles per KV tile")
        g = t_r // t_c
        chains = [[(j, (j * g + t) % t_r) for t in range(t_r)] for j in range(t_c)]
        by_timestamp = True
    elif kind == SYMSHIFT:
        if not causal or t_r != t_c or t_r % 2:
            raise ValueError("symshift needs a causal mask, equal tile counts and an even count")
        n, h = t_r, t_r // 2
        chains = []
        for p in range(h):
            ch = []
            # phase 1: cyclic shift over the dense rectangle Q tiles [h, n) x KV tiles [0, h)
            for t in range(h):
                ch.append((p, h + (p + t) % h))
            # phase 2, upper-left triangle: KV p, top-down from its diagonal tile
            for i in range(p, h):
                ch.append((p, i))
            # phase 2, lower-right triangle: KV n-1-p, bottom-up, ending on its diagonal
            for i in range(n - 1, n - 2 - p, -1):
                ch.append((n - 1 - p, i))
            chains.append(ch)
        by_timestamp = True
    else:
        raise ValueError(kind)

    contributors = {i: [] for i in range(t_r)}
    for w, ch in enumerate(chains):
        for t, (j, i) in enumerate(ch):
            contributors[i].append((t, j))
    if by_timestamp:
        gsize = group if (kind == SHIFT and group) else t_c
        order = {i: [j for (_, t, j) in sorted((j // gsize, t, j) for (t, j) in c)]
                 for i, c in contributors.items()}
    else:
        order = {i: sorted(j for (t, j) in c) for i, c in contributors.items()}
    return Schedule(chains, order)


def check(s: Schedule, t_r: int, t_c: int, causal: bool, br: int, bc: int, group: int | None = None) -> dict:
    """Structural properties the paper asks of a schedule.

    coverage     -- every interacting (Q tile, KV tile) pair runs exactly once
    contiguous   -- each KV tile's tasks are consecutive within one chain
                    (register-resident dK/dV; Section 3.1, optimization constraint)
    conflict_free-- no two chains reduce into the same dQ tile at the same step
                    (Section 3.4, the resource conflict the lemma rules out)
    monotone     -- along each dQ tile's accumulation order the step strictly
                    increases, i.e. every ordering edge goes from the end of a
                    reduction to the start of a deeper one (Lemma 1's condition
                    depth(u) <= depth(v) on the chain DAG); with groups, within
                    each group's part of the order (later groups run after
                    earlier ones, so no edge between groups can close a cycle)
    """
    pairs = [(i, j) for ch in s.chains for (j, i) in ch]
    want = {(i, j) for i in range(t_r) for j in range(t_c) if interacts(i, j, br, bc, causal)}
    coverage = len(pairs) == len(set(pairs)) and set(pairs) == want
    contiguous = True
    owner = {}
    for w, ch in enumerate(s.chains):
        seen = []
        for (j, _) in ch:
            if not seen or seen[-1] != j:
                if j in seen or j in owner:
                    contiguous = False
                seen.append(j)
        for j in seen:
            owner[j] = w
    step = s.step_of()
    per_step = {}
    for (i, j), (w, t) in step.items():
        per_step.setdefault(t, []).append(i)
    conflict_free = all(len(v) == len(set(v)) for v in per_step.values())
    monotone = True
    gsize = group or t_c
    for i, js in s.order.items():
        for g0 in range(0, t_c, gsize):
            ts = [step[(i, j)][1] for j in js if g0 <= j < g0 + gsize]
            if any(b <= a for a, b in zip(ts, ts[1:])):
                monotone = False
    return dict(coverage=coverage, contiguous=contiguous, conflict_free=conflict_free,
                monotone=monotone)


class Deadlock(RuntimeError):
    pass


def simulate(schedules, n_workers: int, c, r, chain_major: bool = False):
    """Critical path of the DAG model of Section 3.1, by list scheduling.

    schedules: one Schedule per head, dispatched to n_workers identical SMs
    head-major (all chains of head 0, then head 1, ...) or, with chain_major,
    chain w of every head before chain w+1; a free SM takes the next chain.
    Every task is a compute phase of length c followed by a reduction phase of
    length r; a chain runs its tasks back to back.  A reduction into dQ tile i
    of a head may start only after the reduction of the previous KV tile in
    that tile's accumulation order (a zero-weight dependency edge).  Returns
    the makespan.
    """
    queue = []  # chains in dispatch order: (head, chain)
    if chain_major:
        for w in range(max(len(s.chains) for s in schedules)):
            for h, s in enumerate(schedules):
                if w < len(s.chains):
                    queue.append((h, w))
    else:
        for h, s in enumerate(schedules):
            for w in range(len(s.chains)):
                queue.append((h, w))
    pred = {}  # (h, i, j) -> (h, i, j_prev) or None
    for h, s in enumerate(schedules):
        for i, js in s.order.items():
            for k, j in enumerate(js):
                pred[(h, i, j)] = (h, i, js[k - 1]) if k else None
    done = {}      # (h, i, j) -> reduction end time
    waiting = {}   # (h, i, j) awaited predecessor -> (chain key, task index)
    events = []    # (time, seq, kind, payload)
    seq = 0
    next_chain = 0
    finished = 0
    makespan = 0

    def push(t, kind, payload):
        nonlocal seq
        heapq.heappush(events, (t, seq, kind, payload))
        seq += 1

    def start_chain(t):
        nonlocal next_chain
        if next_chain < len(queue):
            key = queue[next_chain]
            next_chain += 1
            push(t + c, "computed", (key, 0))

    for _ in range(min(n_workers, len(queue))):
        start_chain(0)
    while events:
        t, _, kind, (key, k) = heapq.heappop(events)
        h, w = key
        j, i = schedules[h].chains[w][k]
        if kind == "computed":
            p = pred[(h, i, j)]
            if p is None or p in done:
                push(t, "reduced_start", (key, k))
            else:
                waiting[p] = (key, k)
        elif kind == "reduced_start":
            push(t + r, "reduced", (key, k))
        else:  # reduced
            done[(h, i, j)] = t
            makespan = max(makespan, t)
            if (h, i, j) in waiting:
                push(t, "reduced_start", waiting.pop((h, i, j)))
            if k + 1 < len(schedules[h].chains[w]):
                push(t + c, "computed", (key, k + 1))
            else:
                finished += 1
                start_chain(t)
    if finished != len(queue):
        raise Deadlock(f"{len(queue) - finished} chains never finished")
    return makespan
