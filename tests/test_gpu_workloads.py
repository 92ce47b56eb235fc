"""Full-shape workloads through the serving loop, against the oracle.

The GPU runs every column at the real shapes and in the launch configuration
the benchmark times; the oracle follows the same trace on a seeded sample of
d_model columns (READ output and WRITE update of column n only involve column
n of W0, dW and G, so the restricted oracle computes those columns exactly).

Tolerances: plans, owner maps and versions bit-exact; bf16 outputs
max |a-b| / max(|b|, 1e-2 rms(b)) <= 2e-2; state (fp32 or bf16) relative
Frobenius error <= 1e-3.  A recursively updated bf16 state is compared by the
Frobenius norm only: a one-ulp difference of an element that a later WRITE
cancels towards zero is large relative to that element but not to the state.
"""

import numpy as np
import pytest
import torch

import oracle as O
from rwttt_inputs import TensorSource, build_trace, workload
from tests.gpu_util import R, host_f64, plan_tuples, run_gpu_trace, say

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

BF16_OUT_TOL = 2e-2
STATE_TOL = 1e-3


def sample_cols(wl, n=64, seed=5):
    rng = np.random.default_rng(seed)
    inner = rng.choice(np.arange(1, wl.d_model - 1), n - 2, replace=False)
    return np.sort(np.concatenate([[0, wl.d_model - 1], inner]))


def check_trace(wl, steps, layers, n_cols=64, threads=16, snap_version=None):
    """With ``snap_version`` = k, every owner's state is also compared when its
    committed version first reaches k (returns how many owners were)."""
    src = TensorSource(wl, memo=True)
    src.prefetch(range(wl.n_owners), layers, threads)
    trace = build_trace(wl, max(steps) + 1)
    cols = sample_cols(wl, n_cols)
    ref_snap, gpu_snap = {}, {}

    def oracle_snap(rec, table):
        for r in range(wl.n_owners):
            if table.V[r] == snap_version and r not in ref_snap:
                ref_snap[r] = (rec.step, [table.D[(r, l)].copy() for l in layers])

    def gpu_snap_at(sess, t):
        for r, v in enumerate(sess.versions()):
            if v == snap_version and r not in gpu_snap:
                gpu_snap[r] = (t, [host_f64(sess.live(r, i), wl.state_dtype)[:, cols]
                                   for i in range(len(layers))])

    ref, table = O.run_trace(wl, trace, src, steps=steps, layers=layers, cols=cols,
                             on_step=oracle_snap if snap_version else None)
    say("oracle done", wl.name)
    sess, got = run_gpu_trace(wl, trace, src, steps, layers=layers, cols=cols,
                              on_step=gpu_snap_at if snap_version else None)
    assert set(gpu_snap) == set(ref_snap)
    for r, (t, states) in ref_snap.items():
        assert gpu_snap[r][0] == t, r
        for i, l in enumerate(layers):
            err = O.rel_frobenius(gpu_snap[r][1][i], states[i])
            assert err <= STATE_TOL, (r, l, t, err)
    n_writes = n_fail = 0
    for rec, (res, versions, ys) in zip(ref, got):
        assert plan_tuples(res) == [(g.key, g.owners) for g in rec.plan.groups], rec.step
        assert versions == rec.versions, rec.step
        assert res.plan.ev_status == rec.plan.ev_status
        assert set(ys) == set(rec.y)
        for k, v in rec.y.items():
            err = O.max_rel_floor(ys[k], v)
            assert err <= BF16_OUT_TOL, (rec.step, k, err)
        n_writes += len(res.committed) + len(res.rolled_back)
        n_fail += len(res.rolled_back)
    worst = 0.0
    for r in range(wl.n_owners):
        for i, l in enumerate(layers):
            live = host_f64(sess.live(r, i), wl.state_dtype)[:, cols]
            err = O.rel_frobenius(live, table.D[(r, l)])
            worst = max(worst, err)
            assert err <= STATE_TOL, (r, l, err)
    say(wl.name, "writes", n_writes, "rolled back", n_fail, "worst state error", worst)
    sess.close()
    return n_writes, n_fail, table, len(ref_snap)


def test_mixed36_bench_workload_sampled():
    """The bench workload: 8 streams, C=64 WRITEs at steps 8 and 16; first and last layer."""
    wl = workload(2)
    n_writes, n_fail, table, _ = check_trace(wl, range(18), layers=[0, 35])
    assert n_writes == 2 and n_fail == 0
    assert table.V == [0, 0, 0, 0, 0, 0, 1, 1]


def test_ragged32_sampled():
    """32 owners, shuffled events, C in {16,32,64}, injected failures rolled back.
    Every owner is also checked at the step its 16th WRITE commits (fp32 state
    within 1e-3 relative Frobenius after 16 writes): 20 owners get there within
    72 steps."""
    wl = workload(3)
    n_writes, n_fail, table, n16 = check_trace(wl, range(72), layers=[0], snap_version=16)
    assert n_writes == 72 * 8 and n_fail > 0
    assert sum(table.V) == n_writes - n_fail
    assert n16 == 20


def test_prefill8b_bf16_state_sampled():
    """8B-class shape, bf16 state from zero: 8 prefill C=512 WRITE groups, then decode."""
    wl = workload(4)
    n_writes, n_fail, table, _ = check_trace(wl, range(12), layers=[0])
    assert n_writes == 64 and n_fail == 0
    assert table.V == [8] * 8


@pytest.mark.parametrize("rank", [0, 8])
def test_two_stream_serving_is_bit_identical_to_one_stream(rank):
    """READ and WRITE groups on two joined streams give the same bits as one
    stream, with fast-weight state (rank 0) and with rank-8 adapter state."""
    from paper_2605_28053_amd.serving import StreamPair
    wl = workload(3)
    src = TensorSource(wl, memo=True)
    if not rank:
        src.prefetch(range(wl.n_owners), [0], 16)
    trace = build_trace(wl, 12)
    backend = R.RWTTT_DELTA_ADAPTER if rank else R.RWTTT_FAST_WEIGHT
    one, out1 = run_gpu_trace(wl, trace, src, range(12), backend=backend, rank=rank)
    pair = StreamPair()
    pair.wait_for_current()
    two, out2 = run_gpu_trace(wl, trace, src, range(12), stream=pair, backend=backend, rank=rank)
    for (r1, v1, y1), (r2, v2, y2) in zip(out1, out2):
        assert plan_tuples(r1) == plan_tuples(r2) and v1 == v2
        assert set(y1) == set(y2)
        for k in y1:
            assert np.array_equal(y1[k], y2[k]), k
    for r in range(wl.n_owners):
        assert torch.equal(one.live(r, 0), two.live(r, 0)), r
