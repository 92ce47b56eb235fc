"""The bounded-wait scheduling simulator over the library's planner (CPU only).

Every simulated issue is checked against the wait bound (Section 3, eq.
wait-budget), group legality and injectivity (eq. compatibility; Section 4.3),
and per-request update counts and versions; these tests require zero
violations and check the sweep's expected monotone trends.
"""

import pytest

R = pytest.importorskip("paper_2605_28053_amd._rwttt",
                        reason="librwttt.so not built (python -m paper_2605_28053_amd.build)")
from paper_2605_28053_amd.scheduler_sim import ServiceModel, make_requests, simulate, sweep


def model():
    # per-layer microseconds, affine in the group size like the measured kernels
    return ServiceModel(4, [30.0 + 13.0 * b for b in range(8)],
                        {64: [55.0 + 45.0 * b for b in range(8)],
                         128: [80.0 + 75.0 * b for b in range(8)]}, 10.0, "synthetic")


def test_service_model_lookup_and_extension():
    m = model()
    assert m.read(1) == 30.0 and m.read(8) == 30.0 + 13.0 * 7
    assert m.read(10) == pytest.approx(30.0 + 13.0 * 9)         # linear past the table
    assert m.write(3, 100) == m.write(3, 128)                    # next larger chunk
    assert m.write(3, 512) == m.write(3, 128)                    # largest chunk
    assert m.group_us(R.RWTTT_READ, 2, 0) == 4 * m.read(2)


@pytest.mark.parametrize("kind", ["uniform", "phase_skew", "poisson", "heterogeneous"])
@pytest.mark.parametrize("B,w", [(8, 0), (8, 4), (4, 0), (4, 2), (2, 8), (0, 3)])
def test_no_violations_and_every_request_completes(kind, B, w):
    reqs = make_requests(kind, n_streams=8, n_tokens=96, chunk=32, seed=3)
    res = simulate(reqs, model(), chunk=32, B=B, w=w)
    assert res.violations == 0
    assert res.max_wait_steps <= w
    assert res.tok_s > 0


def test_greedy_uniform_trace_forms_full_groups():
    reqs = make_requests("uniform", n_streams=8, n_tokens=64, chunk=16)
    res = simulate(reqs, model(), chunk=16, B=8, w=0)
    assert res.mean_group == {"READ": 8.0, "WRITE": 8.0}
    assert res.max_wait_steps == 0
    # 64 steps, one group each, 4 layers per group
    assert res.steps == 64 and res.launches == 64 * 4


def test_phase_skew_splits_write_groups_and_costs_throughput():
    m = model()
    step_s = 1e-6 * m.tick_us(8)
    uni = simulate(make_requests("uniform", 8, 128, 32), m, chunk=32, B=8, w=0)
    skew = simulate(make_requests("phase_skew", 8, 128, 32, step_s=step_s), m, chunk=32, B=8, w=0)
    assert skew.mean_group["WRITE"] == 1.0
    assert skew.tok_s < uni.tok_s


def test_a_step_where_everything_waits_costs_a_tick():
    """Two streams, B = 2, w = 3: stream 1 is ready one tick after stream 0, so
    stream 0's first READ waits one step (one full-batch tick) for its partner."""
    m = model()
    tick = m.tick_us(2)
    assert tick == 10.0 + 4 * (30.0 + 13.0)
    reqs = make_requests("phase_skew", 2, 4, 1000, step_s=1e-6 * tick)
    res = simulate(reqs, m, chunk=1000, B=2, w=3)
    assert res.violations == 0 and res.max_wait_steps == 1
    # stream 0 waits one tick, then both take 4 full steps
    full = 10.0 + 4 * (30.0 + 13.0)
    assert res.makespan_s == pytest.approx(1e-6 * (tick + 4 * full))
    # greedy: no wait, stream 0 runs alone for the first step
    res0 = simulate(reqs, m, chunk=1000, B=2, w=0)
    assert res0.max_wait_steps == 0 and res0.first_token_p95_ms < res.first_token_p95_ms


def test_wait_budget_sweep_on_phase_skew_trades_first_token_latency_for_full_groups():
    """The shape of the paper's wait-budget sweep (Appendix B): on the phase-skew
    trace with B = 8, first-token p95 rises with w until the start-up skew of
    seven steps is absorbed (w = 8 and 16 alike), throughput stays within a few
    percent, WRITE groups fill up, and no run breaks a contract check."""
    rows = sweep(model(), "phase_skew", waits=(0, 1, 2, 4, 8, 16), seeds=range(2), n_streams=8,
                 n_tokens=512, chunk=128, B=8)
    p95 = [r["first_token_p95_ms"] for r in rows]
    assert all(a < b for a, b in zip(p95[:5], p95[1:5]))
    assert p95[5] == p95[4]
    tok = [r["tok_s"] for r in rows]
    assert max(tok) / min(tok) < 1.08
    assert rows[0]["mean_write_group"] == 1.0 and rows[4]["mean_write_group"] == 8.0
    assert all(r["violations"] == 0 for r in rows)
    assert [r["max_wait_steps"] for r in rows] == [0, 1, 2, 4, 7, 7]


def test_wait_budget_trades_latency_for_denser_write_groups():
    rows = sweep(model(), "poisson", waits=(0, 16), seeds=range(3), n_streams=8, n_tokens=128,
                 chunk=32, B=2)
    assert all(r["violations"] == 0 for r in rows)
    assert rows[1]["mean_write_group"] > rows[0]["mean_write_group"]
    assert rows[1]["first_token_p95_ms"] >= rows[0]["first_token_p95_ms"]
    assert rows[1]["max_wait_steps"] <= 16


def test_simulation_is_deterministic():
    a = simulate(make_requests("poisson", 8, 64, 16, seed=5), model(), 16, 4, 2)
    b = simulate(make_requests("poisson", 8, 64, 16, seed=5), model(), 16, 4, 2)
    assert a == b
