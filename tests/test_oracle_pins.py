"""Pins of the CPU oracle against facts other than itself.

Each test checks the oracle against something it does not compute the same
way: pure-Python brute force with exactly rounded sums, closed forms, a
different library routine, or counts the paper prints.  A plausible mistake
in the oracle (a dropped term, a flipped sign, a transposed operand, a wrong
version rule, a planner that mixes keys) fails at least one of them.
"""

import itertools
import json
import math
import os
import random

import numpy as np
import pytest
import torch

import oracle as O
from rwttt_inputs import (READ, WRITE, TensorSource, build_trace, workload, draw,
                          f32_to_bf16_bits, bf16_bits_to_f32, shape_class)

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# --------------------------------------------------------------------------
# bf16 rounding
# --------------------------------------------------------------------------

def test_bf16_round_matches_torch_on_float32_values():
    rng = np.random.default_rng(0)
    a = np.concatenate([
        rng.standard_normal(20000).astype(np.float32),
        (rng.standard_normal(2000) * 1e-38).astype(np.float32),   # subnormal range
        (rng.standard_normal(2000) * 1e30).astype(np.float32),
        np.array([0.0, -0.0, 1.0, -1.0, 3.0e38, -3.0e38], dtype=np.float32),
    ])
    ref = torch.from_numpy(a).to(torch.bfloat16).to(torch.float64).numpy()
    got = O.bf16_round(a.astype(np.float64))
    assert np.array_equal(got, ref)


def test_bf16_round_ties_to_even_by_hand():
    # spacing of bf16 in [1, 2) is 2^-7; in the subnormal range 2^-133
    cases = [
        (1 + 2.0 ** -8, 1.0),                       # tie, lower mantissa even
        (1 + 3 * 2.0 ** -8, 1 + 2.0 ** -6),         # tie, upper mantissa even
        (1 + 2.0 ** -8 + 2.0 ** -30, 1 + 2.0 ** -7),  # just above the tie
        (-(1 + 3 * 2.0 ** -8), -(1 + 2.0 ** -6)),
        (2.0 ** -134, 0.0),                         # subnormal tie to even (0)
        (3 * 2.0 ** -134, 2.0 ** -132),             # subnormal tie to even
        (2.0 ** 128, math.inf),
    ]
    for v, want in cases:
        assert O.bf16_round(np.array([v]))[0] == want, v


def test_input_bf16_narrowing_matches_torch():
    rng = np.random.default_rng(1)
    a = rng.standard_normal(50000).astype(np.float32) * np.float32(3.7)
    bits = f32_to_bf16_bits(a)
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(bits, ref)
    assert np.array_equal(bf16_bits_to_f32(bits).astype(np.float64), O.widen(bits, "bf16"))


# --------------------------------------------------------------------------
# READ: y = x W0 + x dW
# --------------------------------------------------------------------------

def _brute_read(x, W0, D):
    K, N = W0.shape
    return np.array([math.fsum(x[k] * W0[k, n] for k in range(K)) +
                     math.fsum(x[k] * D[k, n] for k in range(K)) for n in range(N)])


def test_read_matches_exact_brute_force():
    rng = np.random.default_rng(2)
    K, N = 37, 11
    x, W0, D = rng.standard_normal(K), rng.standard_normal((K, N)), rng.standard_normal((K, N))
    got = O.read_apply(x, W0, D)
    ref = _brute_read(x, W0, D)
    assert np.max(np.abs(got - ref)) <= 1e-12 * np.max(np.abs(ref))


def test_read_unit_input_selects_rows():
    # x = e_k selects row k of both matrices; a transposed operand would not.
    rng = np.random.default_rng(3)
    for K, N in [(9, 5), (6, 6)]:
        W0, D = rng.standard_normal((K, N)), rng.standard_normal((K, N))
        for k in range(K):
            x = np.zeros(K)
            x[k] = 1.0
            assert np.array_equal(O.read_apply(x, W0, D), W0[k] + D[k])


def test_read_zero_state_is_the_plain_projection_and_batch_rows_independent():
    rng = np.random.default_rng(4)
    K, N = 16, 7
    X, W0 = rng.standard_normal((3, K)), rng.standard_normal((K, N))
    Y = O.read_apply(X, W0, np.zeros((K, N)))
    for i in range(3):
        assert np.allclose(Y[i], _brute_read(X[i], W0, np.zeros((K, N))), rtol=0, atol=1e-12)


# --------------------------------------------------------------------------
# WRITE: dW + eta Z^T G
# --------------------------------------------------------------------------

def _brute_write(D, Z, G, eta):
    C, K = Z.shape
    N = G.shape[1]
    out = np.empty_like(D)
    for k in range(K):
        for n in range(N):
            out[k, n] = D[k, n] + eta * math.fsum(Z[c, k] * G[c, n] for c in range(C))
    return out


def test_write_matches_exact_brute_force():
    rng = np.random.default_rng(5)
    C, K, N = 5, 13, 6
    D, Z, G = rng.standard_normal((K, N)), rng.standard_normal((C, K)), rng.standard_normal((C, N))
    got = O.write_candidate(D, Z, G, 0.37)
    assert np.max(np.abs(got - _brute_write(D, Z, G, 0.37))) < 1e-13


def test_write_rank_one_is_outer_product():
    rng = np.random.default_rng(6)
    K, N = 12, 8
    D, z, g = rng.standard_normal((K, N)), rng.standard_normal(K), rng.standard_normal(N)
    got = O.write_candidate(D, z[None, :], g[None, :], 0.5)
    assert np.allclose(got, D + 0.5 * np.outer(z, g), rtol=0, atol=1e-14)


def test_write_unit_evidence_touches_one_row_with_plus_sign():
    rng = np.random.default_rng(7)
    K, N = 10, 4
    D, G = rng.standard_normal((K, N)), rng.standard_normal((1, N))
    Z = np.zeros((1, K))
    Z[0, 3] = 1.0
    got = O.write_candidate(D, Z, G, 0.25)
    expect = D.copy()
    expect[3] += 0.25 * G[0]
    assert np.array_equal(got, expect)


def test_write_eta_zero_is_identity_and_chunks_concatenate():
    rng = np.random.default_rng(8)
    K, N = 11, 9
    D = rng.standard_normal((K, N))
    Z1, G1 = rng.standard_normal((3, K)), rng.standard_normal((3, N))
    Z2, G2 = rng.standard_normal((4, K)), rng.standard_normal((4, N))
    assert np.array_equal(O.write_candidate(D, Z1, G1, 0.0), D)
    two = O.write_candidate(O.write_candidate(D, Z1, G1, 0.1), Z2, G2, 0.1)
    one = O.write_candidate(D, np.vstack([Z1, Z2]), np.vstack([G1, G2]), 0.1)
    assert np.allclose(two, one, rtol=0, atol=1e-13)


# --------------------------------------------------------------------------
# Planner
# --------------------------------------------------------------------------

def _ev(owner, effect=READ, sigma=0, v=0, ready=0, tau=0, pi=0):
    return O.Event(owner, tau, sigma, pi, effect, v, ready)


def _check_plan_properties(events, V, dirty, n_owners, step, B, w, p):
    """Legality, injectivity, wait bound and maximality of a plan."""
    issued = set()
    for g in p.groups:
        assert len(g.owners) > 0
        if B > 0:
            assert len(g.owners) <= B
        evs = [next(e for e in events if e.owner == r) for r in g.owners]
        # eq. compatibility: one key per group, every member at V(r)
        assert len({e.key for e in evs}) == 1 and evs[0].key == g.key
        assert all(e.expected_version == V[e.owner] for e in evs)
        # injective owner map
        assert len(set(g.owners)) == len(g.owners)
        for r in g.owners:
            assert r not in issued
            issued.add(r)
    for i, e in enumerate(events):
        s = p.ev_status[i]
        if s == O.OK:
            assert e.owner in issued
        elif s == O.DEFERRED:
            # eq. wait-budget: a deferred event has not yet waited w steps
            assert step - e.ready_step < w
        else:
            assert e.owner not in issued
    # maximality: two emitted groups of one key can only coexist when the
    # earlier ones are full
    by_key = {}
    for g in p.groups:
        by_key.setdefault(g.key, []).append(len(g.owners))
    for sizes in by_key.values():
        if B == 0:
            assert len(sizes) == 1
        else:
            assert all(s == B for s in sizes[:-1])
    # no deferred event could have joined an emitted partial group of its key
    for i in p.deferred:
        k = events[i].key
        assert all(len(g.owners) == B for g in p.groups if g.key == k) or B == 0


def test_plan_brute_force_small_event_sets():
    rng = random.Random(0)
    n_owners = 5
    for trial in range(3000):
        n = rng.randint(0, n_owners)
        owners = rng.sample(range(n_owners), n)
        V = [rng.randint(0, 2) for _ in range(n_owners)]
        dirty = [rng.random() < 0.15 for _ in range(n_owners)]
        step = rng.randint(0, 4)
        B = rng.choice([0, 1, 2, 3])
        w = rng.choice([0, 1, 2])
        events = []
        for r in owners:
            v = V[r] if rng.random() < 0.8 else V[r] + 1
            events.append(_ev(r, rng.choice([READ, WRITE]), rng.choice([0, 7]), v,
                              rng.randint(0, step)))
        p = O.plan(events, V, dirty, n_owners, step, B, w)
        assert p.status == O.OK
        _check_plan_properties(events, V, dirty, n_owners, step, B, w, p)
        for i, e in enumerate(events):
            if dirty[e.owner]:
                assert p.ev_status[i] == O.E_DIRTY
            elif e.expected_version != V[e.owner]:
                assert p.ev_status[i] == O.E_STALE_VERSION
            else:
                assert p.ev_status[i] in (O.OK, O.DEFERRED)
        # permutation invariance of groups and owner maps
        perm = events[:]
        rng.shuffle(perm)
        q = O.plan(perm, V, dirty, n_owners, step, B, w)
        assert [(g.key, g.owners) for g in q.groups] == [(g.key, g.owners) for g in p.groups]
        assert sorted(perm[i].owner for i in q.deferred) == sorted(events[i].owner for i in p.deferred)


def test_plan_greedy_unbounded_is_one_group_per_key():
    # B = infinity, w = 0: exactly one group per distinct key, READ before WRITE
    events = [_ev(4, WRITE, 64), _ev(0, READ), _ev(2, WRITE, 16), _ev(1, READ),
              _ev(3, WRITE, 64), _ev(5, WRITE, 16)]
    p = O.plan(events, [0] * 6, [False] * 6, 6, 0, 0, 0)
    assert [(g.effect, g.key[2], g.owners) for g in p.groups] == [
        (READ, 0, [0, 1]), (WRITE, 16, [2, 5]), (WRITE, 64, [3, 4])]
    assert p.deferred == []


def test_plan_rejections_and_alias():
    V, dirty = [3, 0, 1], [False, True, False]
    p = O.plan([_ev(0, v=2), _ev(1, v=0), _ev(2, v=1)], V, dirty, 3, 0)
    assert p.ev_status == [O.E_STALE_VERSION, O.E_DIRTY, O.OK]
    assert [g.owners for g in p.groups] == [[2]]
    p = O.plan([_ev(0), _ev(0, WRITE)], [0], [False], 1, 0)
    assert p.status == O.E_OWNER_ALIAS and p.groups == []
    p = O.plan([_ev(7), _ev(0, effect=5), _ev(1, ready=3)], [0, 0], [False, False], 2, 1)
    assert p.ev_status == [O.E_INVALID] * 3


def test_plan_wait_budget_defers_then_issues():
    # B=4, w=2: three compatible events ready at step 0 wait until step 2
    events = [_ev(r, ready=0) for r in range(3)]
    for step, issued in [(0, False), (1, False), (2, True)]:
        p = O.plan(events, [0] * 3, [False] * 3, 3, step, 4, 2)
        assert bool(p.groups) == issued
        assert len(p.deferred) == (0 if issued else 3)
    # a full group never waits
    events = [_ev(r, ready=0) for r in range(4)]
    p = O.plan(events, [0] * 4, [False] * 4, 4, 0, 4, 2)
    assert [g.owners for g in p.groups] == [[0, 1, 2, 3]]


def test_plan_wait_bound_holds_over_time():
    # eq. wait-budget: called every step, no event waits more than w steps
    rng = random.Random(1)
    for w in (0, 1, 2, 4):
        for B in (0, 2, 3):
            n_owners = 6
            V, dirty = [0] * n_owners, [False] * n_owners
            pending = {}
            waits = []
            for step in range(60):
                for r in range(n_owners):
                    if r not in pending and rng.random() < 0.4:
                        eff = rng.choice([READ, WRITE])
                        pending[r] = _ev(r, eff, 0, V[r], step)
                evs = list(pending.values())
                p = O.plan(evs, V, dirty, n_owners, step, B, w)
                for g in p.groups:
                    for r in g.owners:
                        waits.append(step - pending.pop(r).ready_step)
                        if g.effect == WRITE:
                            V[r] += 1
            assert waits and max(waits) <= w


def test_plan_bounded_groups_with_mixed_ready_steps_by_hand():
    """B = 2, w = 3, events of one READ key that became ready at different steps,
    plus two WRITE keys.  Members are taken in (ready step, owner) order, so the
    oldest events fill the full groups first (eq. wait-budget: the oldest is the
    one closest to its bound) and ties in ready step go by owner id; the
    remainder waits until its oldest member has waited w steps."""
    events = [_ev(1, ready=5), _ev(0, ready=3), _ev(4, ready=1), _ev(2, ready=3), _ev(3, ready=2),
              _ev(6, WRITE, 16, ready=4), _ev(5, WRITE, 16, ready=4), _ev(7, WRITE, 64, ready=0),
              _ev(8, WRITE, 16, ready=5)]
    V, dirty = [0] * 9, [False] * 9
    p = O.plan(events, V, dirty, 9, 5, 2, 3)
    assert [(g.effect, g.key[2], g.owners) for g in p.groups] == [
        (READ, 0, [4, 3]), (READ, 0, [0, 2]),     # ready 1, 2 | ready 3, 3 (owner order)
        (WRITE, 16, [5, 6]),                      # ready 4, 4: owner order
        (WRITE, 64, [7]),                         # alone, but waited 5 >= 3 steps
    ]
    # owner 1 (READ, ready 5) and owner 8 (WRITE C=16, ready 5) have waited 0 steps
    assert sorted(events[i].owner for i in p.deferred) == [1, 8]
    assert [p.ev_status[i] for i in range(9)] == [O.DEFERRED, O.OK, O.OK, O.OK, O.OK,
                                                  O.OK, O.OK, O.OK, O.DEFERRED]
    # three steps later the two remainders have waited w steps and are issued
    q = O.plan([events[0], events[8]], V, dirty, 9, 8, 2, 3)
    assert [(g.effect, g.key[2], g.owners) for g in q.groups] == [(READ, 0, [1]), (WRITE, 16, [8])]
    assert q.deferred == []
    # one step earlier they are still deferred
    q = O.plan([events[0], events[8]], V, dirty, 9, 7, 2, 3)
    assert q.groups == [] and sorted(q.deferred) == [0, 1]
    # B = 3: the remainder [2] keeps its own oldest ready step (3): at step 5 it
    # has waited 2 < 3 steps and is deferred, although owner 4 (ready 1) waited 4
    p = O.plan(events[:5], V, dirty, 9, 5, 3, 3)
    assert [g.owners for g in p.groups] == [[4, 3, 0]]
    assert sorted(events[i].owner for i in p.deferred) == [1, 2]


def test_uniform_trace_counts_match_paper():
    g = json.load(open(os.path.join(GOLDEN, "uniform_trace.json")))
    S, T, C = g["streams"], g["decode_tokens"], g["ttt_chunk"]
    V, dirty = [0] * S, [False] * S
    reads = writes = tokens = 0
    for t in range(T):
        # stream s reaches its TTT boundary at its own phase s*16
        events = [_ev(s, WRITE if (t + 16 * s) % C == C - 1 else READ,
                      C if (t + 16 * s) % C == C - 1 else 0, V[s], t) for s in range(S)]
        p = O.plan(events, V, dirty, S, t)
        for grp in p.groups:
            tokens += len(grp.owners)
            if grp.effect == READ:
                reads += len(grp.owners)
            else:
                writes += len(grp.owners)
                for r in grp.owners:
                    V[r] += 1
    assert (reads, writes, tokens) == (g["read_owner_steps"], g["update_owner_steps"], g["generated_tokens"])
    assert V == [T // C] * S


# --------------------------------------------------------------------------
# Whole traces: versions, rollback, sequential brute force, closed forms
# --------------------------------------------------------------------------

def _tiny_run():
    wl = workload(0)
    trace = build_trace(wl)
    src = TensorSource(wl)
    return wl, trace, src, O.run_trace(wl, trace, src)


def test_tiny_trace_versions_and_rollback():
    wl, trace, src, (records, table) = _tiny_run()
    # 4 WRITEs per owner, owner 1's third fails: V = (4, 3)
    assert records[-1].versions == [4, 3]
    assert [r.versions for r in records if r.step in (3, 7, 11, 15)] == [[1, 1], [2, 2], [3, 2], [4, 3]]
    # every step: one READ group then one WRITE group at t % 4 == 3
    for rec in records:
        eff = [g.effect for g in rec.plan.groups]
        assert eff == ([WRITE] if rec.step % 4 == 3 else [READ])
        assert sorted(r for g in rec.plan.groups for r in g.owners) == [0, 1]


def test_tiny_trace_equals_per_request_sequential_brute_force():
    """Batched execution through the planner equals sequential execution.

    The brute force walks each request alone through its own steps in order,
    with exactly rounded sums (math.fsum) and no planner, groups or table.
    """
    wl, trace, src, (records, table) = _tiny_run()
    W0 = O.widen(src.w0(0), "f32")
    K, N = W0.shape
    for r in range(wl.n_owners):
        D = np.zeros((K, N))
        for t in range(wl.n_steps):
            it = next(i for i in trace[t] if i.owner == r)
            x = O.widen(src.x(t, r, 0), "f32")
            y = np.array([math.fsum(np.concatenate([x * W0[:, n], x * D[:, n]])) for n in range(N)])
            y = y.astype(np.float32).astype(np.float64)
            assert np.max(np.abs(records[t].y[(r, 0)] - y)) <= 2 ** -22 * np.max(np.abs(y))
            if it.effect == WRITE and not it.fail:
                Z, G = src.zg(t, r, 0, it.chunk)
                Z, G = O.widen(Z, "f32"), O.widen(G, "f32")
                upd = np.array([[math.fsum(Z[:, k] * G[:, n]) for n in range(N)] for k in range(K)])
                D = (D + wl.eta * upd).astype(np.float32).astype(np.float64)
        assert O.rel_frobenius(table.D[(r, 0)], D) < 1e-6


def test_zero_init_closed_form_after_committed_writes():
    """Zero-initialised state: dW_v = eta * sum_j Z_j^T G_j over committed j,
    and y_t = x_t W0 + eta * sum_j (x_t Z_j^T) G_j -- a different association
    of the same products."""
    wl, trace, src, (records, table) = _tiny_run()
    W0 = O.widen(src.w0(0), "f32")
    for r in range(wl.n_owners):
        committed = []
        for t in range(wl.n_steps):
            x = O.widen(src.x(t, r, 0), "f32")
            y = x @ W0
            for Z, G in committed:
                y = y + wl.eta * ((x @ Z.T) @ G)
            assert O.max_rel_floor(records[t].y[(r, 0)], y) < 1e-4
            it = next(i for i in trace[t] if i.owner == r)
            if it.effect == WRITE and not it.fail:
                Z, G = src.zg(t, r, 0, it.chunk)
                committed.append((O.widen(Z, "f32"), O.widen(G, "f32")))
        closed = sum(wl.eta * (Z.T @ G) for Z, G in committed)
        assert O.rel_frobenius(table.D[(r, 0)], closed) < 1e-5


def test_rollback_restores_version_and_state_exactly():
    wl = workload(0)
    trace = build_trace(wl)
    src = TensorSource(wl)
    snaps = {}

    def on_step(rec, table):
        snaps[rec.step] = {k: v.copy() for k, v in table.D.items()}

    records, table = O.run_trace(wl, trace, src, on_step=on_step)
    # owner 1's failed WRITE at step 11: state and version equal those after step 10
    assert np.array_equal(snaps[11][(1, 0)], snaps[10][(1, 0)])
    assert records[11].versions[1] == records[10].versions[1]
    # owner 0 committed at step 11
    assert not np.array_equal(snaps[11][(0, 0)], snaps[10][(0, 0)])


def test_reads_leave_state_and_versions_unchanged_and_writes_stay_owner_local():
    wl, trace, src = workload(0), build_trace(workload(0)), TensorSource(workload(0))
    snaps = {}

    def on_step(rec, table):
        snaps[rec.step] = ({k: v.copy() for k, v in table.D.items()}, list(table.V))

    O.run_trace(wl, trace, src, on_step=on_step)
    for t in range(1, wl.n_steps):
        prev, cur = snaps[t - 1], snaps[t]
        for it in trace[t]:
            same = np.array_equal(prev[0][(it.owner, 0)], cur[0][(it.owner, 0)])
            if it.effect == READ or it.fail:
                assert same and prev[1][it.owner] == cur[1][it.owner]
            else:
                assert not same and cur[1][it.owner] == prev[1][it.owner] + 1


def test_event_order_does_not_change_results():
    wl = workload(0)
    trace = build_trace(wl)
    src = TensorSource(wl)
    rec_a, tab_a = O.run_trace(wl, trace, src)
    rev = [list(reversed(items)) for items in trace]
    rec_b, tab_b = O.run_trace(wl, rev, src)
    for a, b in zip(rec_a, rec_b):
        assert [(g.key, g.owners) for g in a.plan.groups] == [(g.key, g.owners) for g in b.plan.groups]
        assert a.versions == b.versions
        for k in a.y:
            assert np.array_equal(a.y[k], b.y[k])
    for k in tab_a.D:
        assert np.array_equal(tab_a.D[k], tab_b.D[k])


def test_state_contract_stress_five_injected_failures():
    g = json.load(open(os.path.join(GOLDEN, "state_contract_stress.json")))
    wl = workload(0)
    base = build_trace(wl)
    # inject 5 failures over both owners' WRITEs and check each restores v
    fails = {(3, 0), (7, 1), (11, 0), (11, 1), (15, 0)}
    assert len(fails) == g["injected_failures"]
    trace = [[type(it)(it.owner, it.effect, it.chunk, (t, it.owner) in fails, it.emit)
              for it in items] for t, items in enumerate(base)]
    src = TensorSource(wl)
    snaps = {}
    records, table = O.run_trace(wl, trace, src,
                                 on_step=lambda rec, tb: snaps.__setitem__(rec.step, (
                                     {k: v.copy() for k, v in tb.D.items()}, list(tb.V))))
    passed = 0
    for (t, r) in sorted(fails):
        prev = snaps[t - 1] if t > 0 else None
        if prev is not None and np.array_equal(prev[0][(r, 0)], snaps[t][0][(r, 0)]) \
                and prev[1][r] == snaps[t][1][r]:
            passed += 1
    assert passed == g["passed"]
    assert records[-1].versions == [4 - 3, 4 - 2]


def test_column_restricted_run_equals_full_run():
    wl = workload(0)
    trace = build_trace(wl)
    src = TensorSource(wl)
    full, tf = O.run_trace(wl, trace, src)
    cols = np.array([0, 5, 17, 63])
    part, tp = O.run_trace(wl, trace, src, cols=cols)
    for a, b in zip(full, part):
        for k in a.y:
            assert np.array_equal(a.y[k][cols], b.y[k])
    for k in tf.D:
        assert np.array_equal(tf.D[k][:, cols], tp.D[k])


def test_inputs_are_seeded_and_blockwise_reproducible():
    wl = workload(3)
    a = draw((4, 5), 0.5, "bf16", wl.seed, (99, 1))
    b = draw((4, 5), 0.5, "bf16", wl.seed, (99, 1))
    c = draw((4, 5), 0.5, "bf16", wl.seed, (99, 2))
    assert np.array_equal(a, b) and not np.array_equal(a, c)
    t3 = build_trace(wl, 3)
    assert [len(items) for items in t3] == [24, 24, 24]
    for items in t3:
        assert sum(i.effect == WRITE for i in items) == 8
        assert len({i.owner for i in items}) == 24
        assert all(i.chunk in (16, 32, 64) for i in items if i.effect == WRITE)


def test_fork_checkpoint_resume_are_independent_copies():
    """Fork starts a separate lineage (Section 4.2 CONTROL): the child equals the
    parent at the fork, and later commits on either side stay on that side.
    A checkpoint restores state and version exactly (Section 4.1 snapshot)."""
    wl = workload(0)
    trace, src = build_trace(wl), TensorSource(wl)
    records, table = O.run_trace(wl, trace, src, steps=range(8))
    assert table.V == [2, 2]
    W0 = O.widen(src.w0(0), "f32")
    x = O.widen(src.x(8, 0, 0), "f32")
    before1 = table.D[(1, 0)].copy()
    assert table.fork(0, 0) == O.E_OWNER_ALIAS
    snap = table.checkpoint(0)
    assert table.fork(0, 1) == O.OK
    assert table.V[1] == table.V[0] and np.array_equal(table.D[(1, 0)], table.D[(0, 0)])
    assert not np.array_equal(table.D[(1, 0)], before1)
    assert np.array_equal(O.read_apply(x, W0, table.D[(1, 0)]), O.read_apply(x, W0, table.D[(0, 0)]))
    # a commit on the parent leaves the child at the fork point
    child = table.D[(1, 0)].copy()
    Z, G = src.zg(11, 0, 0, 4)
    table.cand[(0, 0)] = O.write_candidate(table.D[(0, 0)], O.widen(Z, "f32"), O.widen(G, "f32"), wl.eta)
    table.dirty[0] = True
    assert table.fork(1, 0) == O.E_DIRTY
    assert table.resume(0, snap) == O.E_DIRTY
    assert table.commit(0) == O.OK
    assert table.V == [3, 2]
    assert np.array_equal(table.D[(1, 0)], child)
    assert not np.array_equal(table.D[(0, 0)], child)
    # resume returns the parent to its checkpoint, exactly
    assert table.resume(0, snap) == O.OK
    assert table.V[0] == 2 and np.array_equal(table.D[(0, 0)], child)


# --------------------------------------------------------------------------
# DeltaAdapterState backend (Section 4.4; Appendix D)
# --------------------------------------------------------------------------

def _adapter_case(K=24, N=16, r=3, C=5, seed=4):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal(K), rng.standard_normal((K, N)), rng.standard_normal((K, r)),
            rng.standard_normal((r, N)), np.abs(rng.standard_normal((C, K))),
            rng.standard_normal((C, N)))


def test_adapter_read_equals_fast_weight_read_of_the_materialised_delta():
    """Exact apply equivalence: x W0 + (x A) B == x W0 + x (A B)."""
    x, W0, A, B, _, _ = _adapter_case()
    got = O.adapter_read(x, W0, A, B)
    assert np.allclose(got, O.read_apply(x, W0, A @ B), rtol=1e-12, atol=1e-12)
    K, N = W0.shape
    brute = [math.fsum([x[k] * W0[k, n] for k in range(K)] +
                       [x[k] * A[k, j] * B[j, n] for k in range(K) for j in range(A.shape[1])])
             for n in range(N)]
    assert np.allclose(got, brute, rtol=1e-12, atol=1e-12)


def test_adapter_write_moves_each_factor_along_the_evidence_gradient():
    """(A' - A) / eta and (B' - B) / eta equal the finite-difference derivatives of
    <Z^T G, A B> (the quantity the fast-weight rule increases), each factor
    taken at the live value."""
    _, _, A, B, Z, G = _adapter_case()
    eta = 0.37
    A1, B1 = O.adapter_write(A, B, Z, G, eta)
    M = Z.T @ G

    def f(a, b):
        return float(np.sum(M * (a @ b)))

    h = 1e-6
    for (i, j) in [(0, 0), (7, 2), (23, 1)]:
        d = np.zeros_like(A)
        d[i, j] = h
        fd = (f(A + d, B) - f(A - d, B)) / (2 * h)
        assert abs((A1[i, j] - A[i, j]) / eta - fd) < 1e-6 * max(1.0, abs(fd))
    for (i, j) in [(0, 0), (2, 15), (1, 7)]:
        d = np.zeros_like(B)
        d[i, j] = h
        fd = (f(A, B + d) - f(A, B - d)) / (2 * h)
        assert abs((B1[i, j] - B[i, j]) / eta - fd) < 1e-6 * max(1.0, abs(fd))


def test_adapter_write_special_cases():
    _, _, A, B, Z, G = _adapter_case()
    eta = 0.1
    # zero B: A is unchanged and B' = eta (Z A)^T G
    A1, B1 = O.adapter_write(A, np.zeros_like(B), Z, G, eta)
    assert np.array_equal(A1, A)
    assert np.allclose(B1, eta * (Z @ A).T @ G, rtol=1e-12)
    # zero A: B is unchanged
    A1, B1 = O.adapter_write(np.zeros_like(A), B, Z, G, eta)
    assert np.array_equal(B1, B)
    # one evidence row: A' = A + eta outer(z, B g)
    A1, B1 = O.adapter_write(A, B, Z[:1], G[:1], eta)
    assert np.allclose(A1, A + eta * np.outer(Z[0], B @ G[0]), rtol=1e-12)
    assert np.allclose(B1, B + eta * np.outer(A.T @ Z[0], G[0]), rtol=1e-12)
    # eta = 0 is the identity
    A1, B1 = O.adapter_write(A, B, Z, G, 0.0)
    assert np.array_equal(A1, A) and np.array_equal(B1, B)


def test_adapter_write_first_order_moves_the_product_like_the_fast_weight_rule():
    """A' B' - A B = eta (M B^T B + A A^T M) + O(eta^2), M = Z^T G."""
    _, _, A, B, Z, G = _adapter_case()
    M = Z.T @ G
    lin = M @ B.T @ B + A @ A.T @ M
    for eta in (1e-4, 1e-5):
        A1, B1 = O.adapter_write(A, B, Z, G, eta)
        err = (A1 @ B1 - A @ B) / eta - lin
        assert np.max(np.abs(err)) <= 50 * eta * np.max(np.abs(M)) ** 2 * max(1.0, np.max(np.abs(A)) * np.max(np.abs(B)))


def test_adapter_trace_equals_per_request_sequential_application():
    """The adapter run plans and versions exactly like the fast-weight run (the
    plan never looks at the payload; only the backend type in the key differs),
    and its outputs equal each request walked alone through adapter_read /
    adapter_write in order."""
    wl, rank = workload(0), 3
    trace, src = build_trace(wl), TensorSource(wl)
    fw, _ = O.run_trace(wl, trace, src)
    ad, table = O.run_trace(wl, trace, src, rank=rank)
    assert [r.versions for r in ad] == [r.versions for r in fw]
    assert all(g.key[1] == O.DELTA_ADAPTER for r in ad for g in r.plan.groups)
    assert all(g.key[1] == O.FAST_WEIGHT for r in fw for g in r.plan.groups)
    drop_tau = lambda k: (k[0],) + tuple(k[2:])
    assert [[(drop_tau(g.key), g.owners) for g in r.plan.groups] for r in ad] == \
           [[(drop_tau(g.key), g.owners) for g in r.plan.groups] for r in fw]
    W0 = O.widen(src.w0(0), "f32")
    for r in range(wl.n_owners):
        a, b = src.adapter_init(r, 0, rank)
        A, B = O.widen(a, "f32"), O.widen(b, "f32")
        for t in range(wl.n_steps):
            it = next(i for i in trace[t] if i.owner == r)
            x = O.widen(src.x(t, r, 0), "f32")
            y = (x @ A) @ B + x @ W0
            assert O.max_rel_floor(ad[t].y[(r, 0)], y) <= 1e-6
            if it.effect == WRITE and not it.fail:
                Z, G = src.zg(t, r, 0, it.chunk)
                Z, G = O.widen(Z, "f32"), O.widen(G, "f32")
                A, B = A + wl.eta * (Z.T @ (G @ B.T)), B + wl.eta * ((Z @ A).T @ G)
                A, B = A.astype(np.float32).astype(np.float64), B.astype(np.float32).astype(np.float64)
        assert O.rel_frobenius(table.D[(r, 0)][0], A) < 1e-6
        assert O.rel_frobenius(table.D[(r, 0)][1], B) < 1e-6


# --------------------------------------------------------------------------
# The tolerance metrics every parity verdict rests on, by hand
# --------------------------------------------------------------------------

def test_rel_frobenius_by_hand():
    # ||(0, 0.5)|| / ||(3, 4)|| = 0.5 / 5
    assert O.rel_frobenius([3.0, 4.5], [3.0, 4.0]) == pytest.approx(0.1, rel=1e-15)
    # the norm is over every element of a matrix, not a row or a column:
    # error (1, 2, 2) against reference (2, 0, 0, 4, 4) -> 3 / 6
    a = np.array([[3.0, 2.0, 0.0], [6.0, 4.0, 0.0]])
    ref = np.array([[2.0, 0.0, 0.0], [4.0, 4.0, 0.0]])
    assert O.rel_frobenius(a, ref) == pytest.approx(0.5, rel=1e-15)
    # the error's sign does not matter, and equal arrays give exactly 0
    assert O.rel_frobenius([-1.0, 0.0], [1.0, 0.0]) == pytest.approx(2.0, rel=1e-15)
    assert O.rel_frobenius(ref, ref) == 0.0
    # an all-zero reference falls back to the absolute error norm
    assert O.rel_frobenius([0.0, 3.0, 4.0], [0.0, 0.0, 0.0]) == pytest.approx(5.0, rel=1e-15)


def test_max_rel_floor_by_hand():
    ref = np.array([1.0, -2.0, 1e-3, 4.0])
    rms = math.sqrt((1.0 + 4.0 + 1e-6 + 16.0) / 4.0)           # 2.29128...
    floor = 1e-2 * rms
    # one element off: |0.01| / |1|
    assert O.max_rel_floor(ref + [0.01, 0, 0, 0], ref) == pytest.approx(0.01, rel=1e-12)
    # an element below the floor is judged against the floor (0.0005 / 0.0229),
    # not against its own magnitude (0.0005 / 0.001 = 0.5)
    got = O.max_rel_floor(ref + [0, 0, 5e-4, 0], ref)
    assert got == pytest.approx(5e-4 / floor, rel=1e-12)
    assert got < 0.05
    # the worst element decides, not the mean: errors 0.01/1 and 0.08/2 -> 0.04
    assert O.max_rel_floor(ref + [0.01, 0.08, 0, 0], ref) == pytest.approx(0.04, rel=1e-12)
    # a 2-D array is judged over all its elements with one rms
    m = np.array([[1.0, 0.0], [0.0, -1.0]])                     # rms 1/sqrt(2)
    err = np.array([[0.0, 1e-3], [0.0, 0.0]])                   # at a zero reference element
    assert O.max_rel_floor(m + err, m) == pytest.approx(1e-3 / (1e-2 / math.sqrt(2.0)), rel=1e-12)
    # an all-zero reference: rms 0, so the error is absolute; empty arrays give 0
    assert O.max_rel_floor([0.0, 1e-3], [0.0, 0.0]) == pytest.approx(1e-3, rel=1e-15)
    assert O.max_rel_floor([0.0, 0.0], [0.0, 0.0]) == 0.0
    assert O.max_rel_floor(np.zeros(0), np.zeros(0)) == 0.0
    # an explicit floor fraction is honoured
    assert O.max_rel_floor(ref + [0, 0, 5e-4, 0], ref, floor_frac=0.1) == \
        pytest.approx(5e-4 / (0.1 * rms), rel=1e-12)
