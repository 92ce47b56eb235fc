"""CPU oracle of RW-TTT's owner-scoped fast-weight READ/WRITE path.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import or run this module.  It shares no
code with the HIP/C++ path; the two meet only in the seeded input generators
of ``rwttt_inputs``.

What it computes (Yang et al., "RW-TTT: Batched Serving for Request-Owned
Test-Time Training State"):

* READ  (Section 3, Ownership; Section 4.2 primitives table, ApplyState):
      y_r = x_r W0 + x_r dW_r         version v unchanged
* WRITE (Section 3, Ownership; Section 4.2 "WRITE" and BoundaryUpdate):
      candidate dW_r' = dW_r + eta * Z_r^T G_r, invisible until commit.
  The paper leaves the update formula to the backend; this synthetic rule is
  the one the workloads state.  The WRITE step also emits y_r, read at v.
* Commit / Rollback (Section 4.2 "CONTROL"; Section 4.1 snapshot
  c_r^v <- s_r^v): commit publishes the candidate as v+1, rollback keeps v.
* Planner (Section 3 eqs. event / compatibility / wait-budget, Section 4.3):
  legal groups share (effect, backend type, shape class, placement), every
  member is at its committed version, the owner map is injective, and no
  event waits more than w steps.
* Serving loop: Algorithm 1, with its failure branch (rollback of a failed
  WRITE group's owners) taken as intended behaviour.

Precision: all floating point is float64.  The paper fixes bf16 decode I/O
(Section 5.1), so y is rounded to the io dtype (bf16 by round-to-nearest-even,
or fp32) and a WRITE candidate is rounded to the state dtype; nothing else is
rounded.  bf16 values arrive as uint16 bit patterns and are widened exactly.

Planner readings where the paper is silent (the order of emitted groups, the
"current legal prefix"): events are checked first (alias, then dirty, then
stale version), valid events are bucketed by the key
(effect, backend type, shape class, placement) compared as integers, each
bucket is ordered by (ready step, owner), full groups of the target size B are
emitted in that order, and the remainder is emitted only when w == 0 or its
oldest event has waited w steps; otherwise it is deferred.  B == 0 means no
size target.
"""

from dataclasses import dataclass, field

import numpy as np

READ, WRITE = 0, 1
# backend state types tau (Section 4.1 payloads; Section 4.4 backend instantiations)
FAST_WEIGHT, DELTA_ADAPTER = 0, 1

OK = 0
DEFERRED = 1
E_INVALID = -1
E_STALE_VERSION = -2
E_OWNER_ALIAS = -3
E_KEY_MISMATCH = -4
E_NOT_DIRTY = -5
E_DIRTY = -6
E_CAPACITY = -7


# --------------------------------------------------------------------------
# Number formats
# --------------------------------------------------------------------------

def widen(a, dtype):
    """Exact float64 value of an io/state tensor (bf16 as uint16 bits)."""
    if dtype == "bf16":
        u = np.asarray(a, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
        return u.view(np.float32).astype(np.float64)
    return np.asarray(a, dtype=np.float32).astype(np.float64)


def bf16_round(a):
    """Round float64 values to the nearest bf16 value, ties to even.

    bf16 keeps 8 significant bits.  For |a| in [2^(e-1), 2^e) the spacing of
    bf16 values is 2^(e-8); below the smallest normal (2^-126) the spacing is
    fixed at 2^-133.  Division and multiplication by a power of two are exact
    in float64, and ``np.rint`` rounds halves to even.
    """
    a = np.asarray(a, dtype=np.float64)
    _, e = np.frexp(a)
    e = np.maximum(e, -125)
    q = np.ldexp(1.0, e - 8)
    with np.errstate(over="ignore", invalid="ignore"):
        r = np.rint(a / q) * q
    r = np.where(np.abs(r) >= 2.0 ** 128, np.copysign(np.inf, a), r)
    return np.where(a == 0, a, r)


def bf16_bits(a):
    """bf16 bit patterns of values that are already bf16-representable."""
    return (np.asarray(a, dtype=np.float64).astype(np.float32).view(np.uint32)
            >> np.uint32(16)).astype(np.uint16)


def round_to(a, dtype):
    """Round exact float64 results to the paper-fixed storage precision."""
    if dtype == "bf16":
        return bf16_round(a)
    return np.asarray(a, dtype=np.float64).astype(np.float32).astype(np.float64)


# --------------------------------------------------------------------------
# READ and WRITE arithmetic (one owner at a time)
# --------------------------------------------------------------------------

def read_apply(x, W0, D):
    """y = x W0 + x dW for one owner (Section 3, Read; ApplyState).

    x: [d_ff] or [n, d_ff]; W0, D: [d_ff, d_model]; all float64.  Unrounded.
    """
    return x @ W0 + x @ D


def write_candidate(D, Z, G, eta):
    """dW + eta Z^T G for one owner (Section 3, Write; BoundaryUpdate).

    D: [d_ff, d_model]; Z: [C, d_ff]; G: [C, d_model]; float64.  Unrounded.
    """
    return D + eta * (Z.T @ G)


def adapter_read(x, W0, A, B):
    """y = x W0 + (x A) B for one owner of the DeltaAdapterState backend
    (Section 4.4; Appendix D).  A: [d_ff, r]; B: [r, d_model]; float64."""
    return x @ W0 + (x @ A) @ B


def adapter_write(A, B, Z, G, eta):
    """Candidate (A', B') of an adapter WRITE with evidence Z [C, d_ff], G [C, d_model].

    The fast-weight rule moves dW by eta Z^T G.  For dW = A B the same evidence
    moves each factor along the matching direction, both taken from the live
    factors: A' = A + eta (Z^T G) B^T = A + eta Z^T (G B^T) and
    B' = B + eta A^T (Z^T G) = B + eta (Z A)^T G.  Unrounded float64.
    """
    M = Z.T @ G
    return A + eta * (M @ B.T), B + eta * (A.T @ M)


# --------------------------------------------------------------------------
# Planner (Section 3 eqs. event, compatibility, wait-budget; Section 4.3)
# --------------------------------------------------------------------------

@dataclass(frozen=True)
class Event:
    owner: int
    backend_type: int
    shape_class: int
    placement: int
    effect: int
    expected_version: int
    ready_step: int

    @property
    def key(self):
        # kappa = (rho, tau, sigma, pi)
        return (self.effect, self.backend_type, self.shape_class, self.placement)


@dataclass
class Group:
    key: tuple
    owners: list

    @property
    def effect(self):
        return self.key[0]


@dataclass
class Plan:
    status: int
    groups: list = field(default_factory=list)
    deferred: list = field(default_factory=list)    # event indices
    ev_status: list = field(default_factory=list)


def plan(events, V, dirty, n_owners, step, B=0, w=0):
    """Legal groups of the ready events at decode step ``step``.

    V[r]: committed version of owner r; dirty[r]: owner r holds an
    uncommitted candidate.  Returns a Plan; ``ev_status[i]`` is OK (issued),
    DEFERRED, or a negative rejection code.
    """
    n = len(events)
    st = [OK] * n
    seen = set()
    for e in events:
        if 0 <= e.owner < n_owners:
            if e.owner in seen:
                return Plan(E_OWNER_ALIAS, ev_status=[E_OWNER_ALIAS] * n)
            seen.add(e.owner)
    valid = []
    for i, e in enumerate(events):
        if e.effect not in (READ, WRITE) or not (0 <= e.owner < n_owners) or e.ready_step > step:
            st[i] = E_INVALID
        elif dirty[e.owner]:
            st[i] = E_DIRTY
        elif e.expected_version != V[e.owner]:
            st[i] = E_STALE_VERSION
        else:
            valid.append(i)

    buckets = {}
    for i in valid:
        buckets.setdefault(events[i].key, []).append(i)

    groups, deferred = [], []
    for key in sorted(buckets):
        idx = sorted(buckets[key], key=lambda i: (events[i].ready_step, events[i].owner))
        if B > 0:
            n_full = len(idx) // B
            for g in range(n_full):
                members = idx[g * B:(g + 1) * B]
                groups.append(Group(key, [events[i].owner for i in members]))
            rest = idx[n_full * B:]
        else:
            rest = idx
        if not rest:
            continue
        oldest = min(events[i].ready_step for i in rest)
        if w == 0 or step - oldest >= w:
            groups.append(Group(key, [events[i].owner for i in rest]))
        else:
            for i in rest:
                st[i] = DEFERRED
                deferred.append(i)
    return Plan(OK, groups, deferred, st)


# --------------------------------------------------------------------------
# Owner state table and the serving loop (Algorithm 1)
# --------------------------------------------------------------------------

def _copy_state(v):
    """A fast-weight array or an adapter (A, B) pair, copied."""
    return tuple(a.copy() for a in v) if isinstance(v, tuple) else v.copy()


class OwnerTable:
    """Committed fast weights, versions and pending candidates per owner.

    Values are float64 arrays holding state-dtype-representable numbers.
    """

    def __init__(self, n_owners, layers):
        self.n_owners = n_owners
        self.layers = list(layers)
        self.D = {}                      # (r, l) -> committed dW (version V[r])
        self.V = [0] * n_owners
        self.cand = {}                   # (r, l) -> candidate of version V[r]+1
        self.dirty = [False] * n_owners

    def commit(self, r):
        """Publish the candidate of owner r as version V[r]+1 (CONTROL)."""
        if not self.dirty[r]:
            return E_NOT_DIRTY
        for l in self.layers:
            if (r, l) in self.cand:
                self.D[(r, l)] = self.cand.pop((r, l))
        self.V[r] += 1
        self.dirty[r] = False
        return OK

    def rollback(self, r):
        """Drop owner r's candidate; the committed state and V[r] stay."""
        if not self.dirty[r]:
            return E_NOT_DIRTY
        for l in self.layers:
            self.cand.pop((r, l), None)
        self.dirty[r] = False
        return OK

    def fork(self, src, dst):
        """Owner dst starts a new lineage from src's committed state and
        version (Section 4.2 CONTROL, fork); src's open candidate stays its own."""
        if src == dst:
            return E_OWNER_ALIAS
        if self.dirty[dst]:
            return E_DIRTY
        for l in self.layers:
            self.D[(dst, l)] = _copy_state(self.D[(src, l)])
        self.V[dst] = self.V[src]
        return OK

    def checkpoint(self, r):
        """Owner r's committed state and version (the snapshot of Section 4.1)."""
        return {l: _copy_state(self.D[(r, l)]) for l in self.layers}, self.V[r]

    def resume(self, r, snap):
        """Restore a checkpoint taken by checkpoint() into owner r."""
        if self.dirty[r]:
            return E_DIRTY
        state, v = snap
        for l in self.layers:
            self.D[(r, l)] = _copy_state(state[l])
        self.V[r] = v
        return OK


@dataclass
class StepRecord:
    step: int
    plan: Plan
    versions: list
    y: dict             # (owner, layer) -> float64 values in the io dtype


def run_trace(wl, trace, src, steps=None, layers=None, cols=None,
              B=0, w=0, sigma=None, keep_y=True, table=None, on_step=None, rank=0):
    """Sequential semantics of a workload trace, one owner at a time.

    ``cols`` restricts every d_model-indexed tensor (W0, dW, G, y) to a column
    subset.  Both the READ output and the WRITE update of column n only involve
    column n of W0, dW and G, so the restricted run computes exactly those
    columns of the full run.

    ``rank`` > 0 runs the DeltaAdapterState backend instead: each state is the
    pair (A, B) of that rank, read with adapter_read and updated with
    adapter_write (no column restriction: an adapter update mixes columns).
    """
    from rwttt_inputs import shape_class
    steps = range(len(trace)) if steps is None else steps
    layers = list(range(wl.n_layers)) if layers is None else list(layers)
    sigma = shape_class if sigma is None else sigma
    if rank and cols is not None:
        raise ValueError("an adapter run has no column restriction")
    sel = (lambda a: a) if cols is None else (lambda a: a[..., cols])

    if table is None:
        table = OwnerTable(wl.n_owners, layers)
        for r in range(wl.n_owners):
            for l in layers:
                if rank:
                    a, b = src.adapter_init(r, l, rank)
                    table.D[(r, l)] = (widen(a, wl.state_dtype), widen(b, wl.state_dtype))
                else:
                    table.D[(r, l)] = sel(widen(src.dw_init(r, l), wl.state_dtype))
    W0 = {l: sel(widen(src.w0(l), wl.io_dtype)) for l in layers}

    records = []
    for t in steps:
        items = trace[t]
        by_owner = {it.owner: it for it in items}
        # tau is the owners' state type: every owner of a run holds the same kind
        tau = DELTA_ADAPTER if rank else FAST_WEIGHT
        events = [Event(it.owner, tau, sigma(wl, it.effect, it.chunk), 0, it.effect,
                        table.V[it.owner], t) for it in items]
        p = plan(events, table.V, table.dirty, wl.n_owners, t, B, w)
        ys = {}
        for g in p.groups:
            for r in g.owners:
                it = by_owner[r]
                if g.effect == WRITE:
                    table.dirty[r] = True
                for l in layers:
                    D = table.D[(r, l)]
                    if it.emit:
                        x = widen(src.x(t, r, l), wl.io_dtype)
                        y = adapter_read(x, W0[l], *D) if rank else read_apply(x, W0[l], D)
                        ys[(r, l)] = round_to(y, wl.io_dtype)
                    if g.effect == WRITE:
                        Z, G = src.zg(t, r, l, it.chunk)
                        Z, G = widen(Z, wl.io_dtype), sel(widen(G, wl.io_dtype))
                        if rank:
                            table.cand[(r, l)] = tuple(round_to(v, wl.state_dtype)
                                                       for v in adapter_write(*D, Z, G, wl.eta))
                        else:
                            table.cand[(r, l)] = round_to(write_candidate(D, Z, G, wl.eta),
                                                          wl.state_dtype)
            if g.effect == WRITE:
                for r in g.owners:
                    if by_owner[r].fail:
                        table.rollback(r)
                    else:
                        table.commit(r)
        rec = StepRecord(t, p, list(table.V), ys if keep_y else {})
        records.append(rec)
        if on_step is not None:
            on_step(rec, table)
    return records, table


# --------------------------------------------------------------------------
# Tolerance metrics used by the parity tests
# --------------------------------------------------------------------------

def rel_frobenius(a, ref):
    """||a - ref||_F / ||ref||_F over all elements, in float64; the absolute
    error norm when the reference is all zero."""
    a = np.asarray(a, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref)
    num = np.linalg.norm(a - ref)
    return float(num / den) if den > 0 else float(num)


def max_rel_floor(a, ref, floor_frac=1e-2):
    """max_i |a_i - b_i| / max(|b_i|, floor_frac * rms(b)) over all elements.

    The floor keeps an element that nearly cancels from dominating a relative
    measure; an all-zero reference (rms 0) gives the absolute error, and an
    empty one 0.
    """
    a = np.asarray(a, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    if ref.size == 0:
        return 0.0
    rms = float(np.sqrt(np.mean(ref * ref)))
    den = np.maximum(np.abs(ref), floor_frac * rms)
    den = np.where(den == 0, 1.0, den)
    return float(np.max(np.abs(a - ref) / den))
