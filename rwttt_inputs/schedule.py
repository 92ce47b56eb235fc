"""Per-step role schedules: which owner exposes which transition at each step.

A schedule lists, for every decode step t, the owners that expose a transition
(READ or WRITE), the WRITE chunk rank C, whether that WRITE is an injected
failure, and whether the step emits a token.  The list order is the order in
which the serving loop presents events to the planner (shuffled where the
workload says so).  Nothing here plans, applies or commits anything.
"""

from dataclasses import dataclass

import numpy as np

from .workloads import READ, WRITE

SCHED_KEY = 6


@dataclass(frozen=True)
class StepItem:
    owner: int
    effect: int          # READ or WRITE
    chunk: int = 0       # C for a WRITE
    fail: bool = False   # injected failure of this WRITE
    emit: bool = True    # the step produces a decode token


def _rng(wl, *key):
    ss = np.random.SeedSequence(entropy=wl.seed, spawn_key=(SCHED_KEY,) + tuple(key))
    return np.random.Generator(np.random.PCG64(ss))


def _tiny(wl):
    # WRITEs at 0-indexed steps 3, 7, 11, 15 for both owners; the chunk is the
    # four steps 4k..4k+3 (the WRITE step's own input included).  Owner 1's
    # third WRITE (step 11) is the forced failure.
    out = []
    writes = {0: 0, 1: 0}
    for t in range(wl.n_steps):
        items = []
        for r in range(wl.n_owners):
            if t % 4 == 3:
                writes[r] += 1
                items.append(StepItem(r, WRITE, wl.chunk, fail=(r == 1 and writes[r] == 3)))
            else:
                items.append(StepItem(r, READ))
        out.append(items)
    return out


def _read_only(wl):
    return [[StepItem(r, READ) for r in range(wl.n_owners)] for _ in range(wl.n_steps)]


def _staggered(wl):
    # Owner s sits at phase (t + stagger*s) mod period and WRITEs at the last
    # phase: every owner does period-1 READs, then one WRITE.
    out = []
    for t in range(wl.n_steps):
        items = []
        for s in range(wl.n_owners):
            ph = (t + wl.stagger * s) % wl.period
            if ph == wl.period - 1:
                items.append(StepItem(s, WRITE, wl.chunk))
            else:
                items.append(StepItem(s, READ))
        out.append(items)
    return out


def _ragged(wl):
    # Per step: a permutation of the owners; the first half READ, the next
    # quarter WRITE (C uniform over chunk_choices, Bernoulli(fail_rate)
    # injected failure), the rest idle.  Events are then shuffled.
    out = []
    n = wl.n_owners
    nr, nw = n // 2, n // 4
    for t in range(wl.n_steps):
        g = _rng(wl, t)
        perm = g.permutation(n)
        items = [StepItem(int(r), READ) for r in perm[:nr]]
        for r in perm[nr:nr + nw]:
            c = int(wl.chunk_choices[int(g.integers(len(wl.chunk_choices)))])
            f = bool(g.random() < wl.fail_rate)
            items.append(StepItem(int(r), WRITE, c, fail=f))
        order = g.permutation(len(items))
        out.append([items[int(i)] for i in order])
    return out


def _prefill_decode(wl):
    # Prefill: n_prefill chunk WRITEs for every owner, outside the decode
    # window (they emit no token).  Then READ decode steps.
    out = []
    for t in range(wl.n_steps):
        if t < wl.n_prefill:
            out.append([StepItem(r, WRITE, wl.chunk, emit=False) for r in range(wl.n_owners)])
        else:
            out.append([StepItem(r, READ) for r in range(wl.n_owners)])
    return out


_BUILDERS = {
    "tiny": _tiny,
    "read_only": _read_only,
    "staggered": _staggered,
    "ragged": _ragged,
    "prefill_decode": _prefill_decode,
}


def build_trace(wl, n_steps=None):
    """Return ``trace[t] -> list[StepItem]`` for t < n_steps (default: all)."""
    trace = _BUILDERS[wl.schedule](wl)
    if n_steps is not None:
        trace = trace[:n_steps]
    return trace


def step_items(wl, t):
    """Role list of an arbitrary step t, also past the workload's length.

    The staggered and read-only schedules are periodic; the benchmark uses this
    to run warm-up steps ahead of the timed window without running out of
    schedule.
    """
    if wl.schedule == "staggered":
        items = []
        for s in range(wl.n_owners):
            ph = (t + wl.stagger * s) % wl.period
            items.append(StepItem(s, WRITE, wl.chunk) if ph == wl.period - 1 else StepItem(s, READ))
        return items
    if wl.schedule == "read_only":
        return [StepItem(r, READ) for r in range(wl.n_owners)]
    return build_trace(wl)[t]
