"""GPU parity of the HIP path against the CPU oracle, through the C ABI.

Tolerances (written where they are used):
  * plans, owner maps, versions: bit-exact;
  * fp32 state: relative Frobenius error <= 1e-3 (after up to 16 WRITEs);
  * bf16 outputs: max_i |a-b| / max(|b|, 1e-2 rms(b)) <= 2e-2;
  * fp32 outputs (tiny fp32 workload): the same metric <= 1e-4.
"""

import numpy as np
import pytest
import torch

import oracle as O
from rwttt_inputs import READ, WRITE, TensorSource, build_trace, workload, draw
from tests.gpu_util import (R, Session, all_slot_hashes, host_f64, plan_tuples, read_group,
                            run_gpu_trace, say, slot_hash, small_workload, to_device, to_host,
                            write_group)

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

BF16_OUT_TOL = 2e-2
F32_OUT_TOL = 1e-4
STATE_TOL = 1e-3


def out_tol(dtype):
    return BF16_OUT_TOL if dtype == "bf16" else F32_OUT_TOL


# --------------------------------------------------------------------------
# whole tiny trace
# --------------------------------------------------------------------------

def test_tiny_trace_matches_oracle():
    wl = workload(0)
    trace, src = build_trace(wl), TensorSource(wl)
    say("tiny trace", wl.name)
    snaps = {}
    ref, table = O.run_trace(wl, trace, src,
                             on_step=lambda rec, tb: snaps.__setitem__(rec.step, None))
    sess, got = run_gpu_trace(wl, trace, src, range(wl.n_steps))
    for rec, (res, versions, ys) in zip(ref, got):
        assert plan_tuples(res) == [(g.key, g.owners) for g in rec.plan.groups]
        assert versions == rec.versions
        for k, v in rec.y.items():
            assert O.max_rel_floor(ys[k], v) <= F32_OUT_TOL, (rec.step, k)
    for r in range(wl.n_owners):
        live = host_f64(sess.live(r, 0), wl.state_dtype)
        assert O.rel_frobenius(live, table.D[(r, 0)]) <= STATE_TOL
    assert sess.versions() == [4, 3]


# --------------------------------------------------------------------------
# READ at small and ragged shapes
# --------------------------------------------------------------------------

READ_CASES = [
    # d_ff, d_model, io, state, n_owners, group
    (8, 8, "bf16", "f32", 3, [2, 0]),                  # smallest shape
    (256, 64, "f32", "f32", 2, [1, 0]),
    (1000, 264, "bf16", "f32", 12, [3, 0, 7, 11, 5]),
    (1000, 264, "bf16", "bf16", 12, [2, 9, 4, 0, 1, 6, 8, 10, 11]),
    (520, 1032, "bf16", "f32", 20, list(range(19, -1, -1))[:17]),
    (264, 520, "f32", "bf16", 3, [2]),
    (9728, 2560, "bf16", "f32", 8, list(range(8))),
    (264, 136, "bf16", "f32", 64, list(range(63, -1, -1))),   # the largest group
]


@pytest.mark.parametrize("d_ff,d_model,io,state,n_owners,group", READ_CASES)
def test_read_matches_oracle(d_ff, d_model, io, state, n_owners, group):
    wl = small_workload(d_ff, d_model, io, state, n_owners)
    say("read", d_ff, d_model, io, state, group)
    src = TensorSource(wl)
    sess = Session(wl, src)
    X = draw((n_owners, d_ff), 1.0, io, wl.seed, (77, 1))
    xd = to_device(X, io)
    tdt = torch.float32 if io == "f32" else torch.bfloat16
    before = all_slot_hashes(sess)
    y = torch.zeros((n_owners, d_model), dtype=tdt, device="cuda")
    read_group(sess, group, 0, xd, y)
    torch.cuda.synchronize()
    W0 = O.widen(src.w0(0), io)
    for r in group:
        ref = O.round_to(O.read_apply(O.widen(X[r], io), W0, O.widen(src.dw_init(r, 0), state)), io)
        assert O.max_rel_floor(host_f64(y[r], io), ref) <= out_tol(io), r
    # READ leaves every slot and version untouched
    assert all_slot_hashes(sess) == before
    assert sess.versions() == [0] * n_owners
    # rows outside the group are not written
    others = [r for r in range(n_owners) if r not in group]
    if others:
        assert torch.count_nonzero(y[others].float()).item() == 0
    # batched == sequential and owner order: bit-identical rows
    y1 = torch.zeros_like(y)
    for r in group:
        read_group(sess, [r], 0, xd, y1)
    y2 = torch.zeros_like(y)
    read_group(sess, list(reversed(group)), 0, xd, y2)
    torch.cuda.synchronize()
    assert torch.equal(y[group].view(torch.int16 if io == "bf16" else torch.int32),
                       y1[group].view(torch.int16 if io == "bf16" else torch.int32))
    assert torch.equal(y[group], y2[group])


# --------------------------------------------------------------------------
# WRITE, commit, rollback at small and ragged shapes
# --------------------------------------------------------------------------

WRITE_CASES = [
    # d_ff, d_model, io, state, chunk, group
    (8, 8, "bf16", "f32", 1, [1]),                     # smallest shape
    (8, 8, "bf16", "bf16", 70, [2, 0]),                # smallest shape, GEMM path
    (256, 64, "f32", "f32", 4, [0, 1]),
    (1000, 264, "bf16", "f32", 1, [2]),
    (1000, 264, "bf16", "f32", 17, [0, 3, 1]),
    (1000, 264, "bf16", "bf16", 64, [1, 2]),
    (520, 1032, "bf16", "f32", 100, [3, 0]),
    (264, 136, "bf16", "bf16", 150, [0, 2]),           # GEMM with 5 rank stages (last stage index 1 of 3)
    (520, 264, "bf16", "f32", 150, [1]),
    (128, 64, "bf16", "f32", 32, [0, 1, 2, 3]),
    (9728, 2560, "bf16", "f32", 64, [1]),
    (264, 136, "bf16", "f32", 33, [11, 4, 0, 7, 2, 9, 5, 1, 10, 3, 8, 6]),   # 12 owners, stream path
    (264, 136, "bf16", "bf16", 130, [9, 2, 5, 0, 7, 3, 8, 1, 6, 4]),        # 10 owners, GEMM path
    (264, 520, "f32", "bf16", 5, [1, 0]),              # fp32 evidence into bf16 state (VALU path)
    (2056, 264, "bf16", "bf16", 64, [2, 0]),           # 65 row tiles over 33 partitions of 2 and 1 items
    (3080, 264, "bf16", "f32", 48, [0, 2, 1]),         # 97 row tiles over 49 partitions of 2 and 1 items
]


@pytest.mark.parametrize("d_ff,d_model,io,state,chunk,group", WRITE_CASES)
def test_write_commit_rollback_match_oracle(d_ff, d_model, io, state, chunk, group):
    n_owners = max(4, max(group) + 1)
    wl = small_workload(d_ff, d_model, io, state, n_owners, eta=0.05)
    say("write", d_ff, d_model, io, state, chunk, group)
    src = TensorSource(wl)
    sess = Session(wl, src)
    zs, gs, ref = [], [], {}
    for r in group:
        Z = draw((chunk, d_ff), 1.0, io, wl.seed, (78, r), absval=True)
        G = draw((chunk, d_model), 1.0, io, wl.seed, (79, r))
        zs.append(to_device(Z, io))
        gs.append(to_device(G, io))
        ref[r] = O.round_to(O.write_candidate(O.widen(src.dw_init(r, 0), state), O.widen(Z, io),
                                              O.widen(G, io), wl.eta), state)
    before = all_slot_hashes(sess)
    st = write_group(sess, group, 0, chunk, zs, gs)
    assert st == R.RWTTT_OK, R.rwttt_strerror(st)
    torch.cuda.synchronize()
    after = all_slot_hashes(sess)
    # only the group's shadow slots changed
    for key in before:
        r, i, s = key
        if r in group and s == 1:
            continue
        assert after[key] == before[key], key
    for r in group:
        shadow = host_f64(sess.shadow(r, 0), state)
        if state == "f32":
            assert O.rel_frobenius(shadow, ref[r]) <= STATE_TOL
        else:
            assert O.max_rel_floor(shadow, ref[r]) <= BF16_OUT_TOL
        assert sess.version(r) == (0, True)
    # roll back the first owner, commit the rest
    keep_live = slot_hash(sess.live(group[0], 0))
    assert R.rwttt_rollback(sess.ctx, [group[0]]) == R.RWTTT_OK
    assert slot_hash(sess.live(group[0], 0)) == keep_live
    assert sess.version(group[0]) == (0, False)
    if len(group) > 1:
        shadow_hash = {r: slot_hash(sess.shadow(r, 0)) for r in group[1:]}
        assert R.rwttt_commit(sess.ctx, group[1:]) == R.RWTTT_OK
        for r in group[1:]:
            assert sess.version(r) == (1, False)
            assert slot_hash(sess.live(r, 0)) == shadow_hash[r]


# --------------------------------------------------------------------------
# WRITE with its token (the step's output at version v)
# --------------------------------------------------------------------------

TOKEN_CASES = [
    # d_ff, d_model, io, state, chunk, group, n_owners
    (40, 24, "bf16", "f32", 1, [2], 3),               # one row tile, one partition
    (1000, 264, "bf16", "f32", 17, [0, 3, 1], 4),     # ragged rows and columns
    (1000, 264, "bf16", "bf16", 64, [1, 2], 4),
    (1576, 520, "bf16", "f32", 64, [4, 0, 2], 5),     # 50 row tiles, one per partition
    (2056, 264, "bf16", "bf16", 64, [2, 0, 3], 4),    # bf16 state, partitions of 2 and 1 items
    (3080, 264, "bf16", "f32", 48, [1, 0], 3),        # fp32 state, partitions of 2 and 1 items
    (264, 520, "f32", "bf16", 5, [1, 0], 2),          # fp32 evidence, bf16 state: READ, then VALU
    (520, 1032, "bf16", "f32", 100, [3, 0], 4),       # large chunk: READ, then the GEMM
    (256, 64, "f32", "f32", 4, [0, 1], 2),            # fp32 evidence
    (9728, 2560, "bf16", "f32", 64, [5, 1, 7], 8),    # full 4B-layer shape
]


@pytest.mark.parametrize("d_ff,d_model,io,state,chunk,group,n_owners", TOKEN_CASES)
def test_write_token_matches_oracle(d_ff, d_model, io, state, chunk, group, n_owners):
    wl = small_workload(d_ff, d_model, io, state, n_owners, eta=0.05)
    say("write+token", d_ff, d_model, io, state, chunk, group)
    src = TensorSource(wl)
    sess = Session(wl, src)
    X = draw((n_owners, d_ff), 1.0, io, wl.seed, (77, 2))
    xd = to_device(X, io)
    tdt = torch.float32 if io == "f32" else torch.bfloat16
    zs, gs = [], []
    for r in group:
        zs.append(to_device(draw((chunk, d_ff), 1.0, io, wl.seed, (78, r), absval=True), io))
        gs.append(to_device(draw((chunk, d_model), 1.0, io, wl.seed, (79, r)), io))
    sentinel = torch.full((n_owners, d_model), 7.0, dtype=tdt, device="cuda")
    y = sentinel.clone()
    st = write_group(sess, group, 0, chunk, zs, gs, x_dev=xd, y_dev=y)
    assert st == R.RWTTT_OK, R.rwttt_strerror(st)
    torch.cuda.synchronize()
    W0 = O.widen(src.w0(0), io)
    for r in group:
        # the token reads version v: the candidate in the shadow slot is not visible
        ref = O.round_to(O.read_apply(O.widen(X[r], io), W0, O.widen(src.dw_init(r, 0), state)), io)
        assert O.max_rel_floor(host_f64(y[r], io), ref) <= out_tol(io), r
    others = [r for r in range(n_owners) if r not in group]
    if others:
        assert torch.equal(y[others], sentinel[others])
    shadow_tok = {r: slot_hash(sess.shadow(r, 0)) for r in group}
    # the candidate does not depend on whether the token was asked for
    assert R.rwttt_rollback(sess.ctx, group) == R.RWTTT_OK
    assert write_group(sess, group, 0, chunk, zs, gs) == R.RWTTT_OK
    torch.cuda.synchronize()
    assert {r: slot_hash(sess.shadow(r, 0)) for r in group} == shadow_tok
    # an owner's token is bit-identical alone and in any group order
    assert R.rwttt_rollback(sess.ctx, group) == R.RWTTT_OK
    y1 = sentinel.clone()
    for i, r in enumerate(group):
        assert write_group(sess, [r], 0, chunk, [zs[i]], [gs[i]], x_dev=xd, y_dev=y1) == R.RWTTT_OK
        assert R.rwttt_rollback(sess.ctx, [r]) == R.RWTTT_OK
    rev = list(reversed(range(len(group))))
    y2 = sentinel.clone()
    assert write_group(sess, [group[i] for i in rev], 0, chunk, [zs[i] for i in rev],
                       [gs[i] for i in rev], x_dev=xd, y_dev=y2) == R.RWTTT_OK
    torch.cuda.synchronize()
    assert torch.equal(y[group], y1[group])
    assert torch.equal(y[group], y2[group])
    assert {r: slot_hash(sess.shadow(r, 0)) for r in group} == shadow_tok
    # the token equals a READ of the same owners up to fp32 summation order
    y3 = torch.zeros_like(y)
    read_group(sess, group, 0, xd, y3)
    torch.cuda.synchronize()
    for r in group:
        assert O.max_rel_floor(host_f64(y[r], io), host_f64(y3[r], io)) <= out_tol(io), r


def test_write_token_argument_errors():
    wl = small_workload(256, 64, "bf16", "f32", 2)
    sess = Session(wl, TensorSource(wl))
    z = torch.zeros((4, 256), dtype=torch.bfloat16, device="cuda")
    gg = torch.zeros((4, 64), dtype=torch.bfloat16, device="cuda")
    x = torch.zeros((2, 256), dtype=torch.bfloat16, device="cuda")
    g = R.make_group(WRITE, 0, 1)
    # x without y (or y without x) is rejected before anything is marked dirty
    st = R.rwttt_write(sess.ctx, g, R.u32_array([0]), 0, 4, [z.data_ptr()], [gg.data_ptr()],
                       0.1, x.data_ptr(), 0)
    assert st == R.RWTTT_E_INVALID
    assert sess.version(0) == (0, False)


# --------------------------------------------------------------------------
# TailBufferUpdate: READ steps append x; a WRITE takes its chunk from the tail
# --------------------------------------------------------------------------

TAIL_CASES = [
    # io, state, chunk
    ("bf16", "f32", 4),
    ("bf16", "bf16", 17),
    ("bf16", "f32", 70),      # large chunk: READ for the token, then the GEMM
    ("f32", "f32", 4),        # fp32 evidence
]


@pytest.mark.parametrize("io,state,chunk", TAIL_CASES)
def test_tail_append_then_write_from_tail(io, state, chunk):
    d_ff, d_model, n_owners = 1000, 264, 4
    wl = small_workload(d_ff, d_model, io, state, n_owners, eta=0.05)
    say("tail", io, state, chunk)
    src = TensorSource(wl)
    sess = Session(wl, src, tail_rows=chunk + 2)
    tdt = torch.float32 if io == "f32" else torch.bfloat16
    readers = [0, 2, 3]
    writers = [2, 0]
    X = [draw((n_owners, d_ff), 1.0, io, wl.seed, (80, t)) for t in range(chunk)]
    W0 = O.widen(src.w0(0), io)
    for t in range(chunk - 1):
        xd = to_device(X[t], io)
        y = torch.zeros((n_owners, d_model), dtype=tdt, device="cuda")
        g = R.make_group(READ, 0, len(readers))
        assert R.rwttt_read_append(sess.ctx, g, R.u32_array(readers), 0, xd.data_ptr(),
                                   y.data_ptr()) == R.RWTTT_OK
        torch.cuda.synchronize()
        if t == 0:
            for r in readers:
                ref = O.round_to(O.read_apply(O.widen(X[t][r], io), W0,
                                              O.widen(src.dw_init(r, 0), state)), io)
                assert O.max_rel_floor(host_f64(y[r], io), ref) <= out_tol(io)
    for r in range(n_owners):
        assert R.rwttt_tail_len(sess.ctx, r, 0) == (chunk - 1 if r in readers else 0)
        # the tail holds the appended rows bit for bit
        got = to_host(sess.tails[r][0][:chunk - 1], io)
        if r in readers:
            assert np.array_equal(got, np.stack([X[t][r] for t in range(chunk - 1)]))
    assert sess.versions() == [0] * n_owners
    # the WRITE step: Z = the tail rows, then this step's own x
    xd = to_device(X[chunk - 1], io)
    y = torch.zeros((n_owners, d_model), dtype=tdt, device="cuda")
    Gs = {r: draw((chunk, d_model), 1.0, io, wl.seed, (81, r)) for r in writers}
    gds = [to_device(Gs[r], io) for r in writers]
    wg = R.make_group(WRITE, 0, len(writers))
    assert R.rwttt_write(sess.ctx, wg, R.u32_array(writers), 0, chunk, None,
                         [g.data_ptr() for g in gds], wl.eta, xd.data_ptr(), y.data_ptr(),
                         stream=torch.cuda.current_stream().cuda_stream) == R.RWTTT_OK
    torch.cuda.synchronize()
    for r in writers:
        Z = np.stack([X[t][r] for t in range(chunk)])
        D0 = O.widen(src.dw_init(r, 0), state)
        cand = O.round_to(O.write_candidate(D0, O.widen(Z, io), O.widen(Gs[r], io), wl.eta), state)
        shadow = host_f64(sess.shadow(r, 0), state)
        if state == "f32":
            assert O.rel_frobenius(shadow, cand) <= STATE_TOL
        else:
            assert O.max_rel_floor(shadow, cand) <= BF16_OUT_TOL
        ref = O.round_to(O.read_apply(O.widen(X[chunk - 1][r], io), W0, D0), io)
        assert O.max_rel_floor(host_f64(y[r], io), ref) <= out_tol(io)
        assert R.rwttt_tail_len(sess.ctx, r, 0) == chunk
        assert np.array_equal(to_host(sess.tails[r][0][chunk - 1], io), X[chunk - 1][r])
    # the boundary closes on commit and on rollback; other owners keep their tails
    assert R.rwttt_commit(sess.ctx, [2]) == R.RWTTT_OK
    assert R.rwttt_rollback(sess.ctx, [0]) == R.RWTTT_OK
    assert [R.rwttt_tail_len(sess.ctx, r, 0) for r in range(n_owners)] == [0, 0, 0, chunk - 1]
    assert sess.versions() == [0, 0, 1, 0]


# --------------------------------------------------------------------------
# Fork, checkpoint and resume (Section 4.2 CONTROL; Section 4.1 snapshot)
# --------------------------------------------------------------------------

@pytest.mark.parametrize("state", ["f32", "bf16"])
def test_fork_checkpoint_resume_match_oracle(state):
    d_ff, d_model, n_owners, L = 1000, 264, 4, 2
    base = small_workload(d_ff, d_model, "bf16", state, n_owners, eta=0.05)
    import dataclasses
    wl = dataclasses.replace(base, n_layers=L)
    say("fork/checkpoint", state)
    src = TensorSource(wl)
    sess = Session(wl, src)
    table = O.OwnerTable(n_owners, range(L))
    for r in range(n_owners):
        for l in range(L):
            table.D[(r, l)] = O.widen(src.dw_init(r, l), state)
    chunk = 16

    def write_commit(owners, key):
        zs = {l: [] for l in range(L)}
        gs = {l: [] for l in range(L)}
        for r in owners:
            for l in range(L):
                Z = draw((chunk, d_ff), 1.0, "bf16", wl.seed, (key, r, l), absval=True)
                G = draw((chunk, d_model), 1.0, "bf16", wl.seed, (key + 1, r, l))
                zs[l].append(to_device(Z, "bf16"))
                gs[l].append(to_device(G, "bf16"))
                table.cand[(r, l)] = O.round_to(O.write_candidate(
                    table.D[(r, l)], O.widen(Z, "bf16"), O.widen(G, "bf16"), wl.eta), state)
            table.dirty[r] = True
        for l in range(L):
            assert write_group(sess, owners, l, chunk, zs[l], gs[l]) == R.RWTTT_OK
        assert R.rwttt_commit(sess.ctx, owners) == R.RWTTT_OK
        for r in owners:
            assert table.commit(r) == O.OK
        torch.cuda.synchronize()

    def check_state(r):
        for l in range(L):
            got = host_f64(sess.live(r, l), state)
            assert O.rel_frobenius(got, table.D[(r, l)]) <= STATE_TOL, (r, l)

    write_commit([0, 1], 90)
    # fork 0 -> 2: live slots bit-identical, versions equal, READs bit-identical
    assert R.rwttt_fork(sess.ctx, 0, 2, torch.cuda.current_stream().cuda_stream) == R.RWTTT_OK
    assert table.fork(0, 2) == O.OK
    torch.cuda.synchronize()
    assert sess.versions() == table.V == [1, 1, 1, 0]
    for l in range(L):
        assert slot_hash(sess.live(2, l)) == slot_hash(sess.live(0, l))
    x = to_device(draw((n_owners, d_ff), 1.0, "bf16", wl.seed, (92,)), "bf16")
    y = torch.zeros((n_owners, d_model), dtype=torch.bfloat16, device="cuda")
    X = draw((n_owners, d_ff), 1.0, "bf16", wl.seed, (92,))
    x[2] = x[0]
    read_group(sess, [0, 2], 1, x, y)
    torch.cuda.synchronize()
    assert torch.equal(y[0], y[2])
    # checkpoint owner 1 to pinned host memory, then move it on and resume
    nbytes = sess.live(1, 0).numel() * sess.live(1, 0).element_size()
    host = [torch.empty(nbytes, dtype=torch.uint8, pin_memory=True) for _ in range(L)]
    st, v = R.rwttt_checkpoint(sess.ctx, 1, [h.data_ptr() for h in host],
                               torch.cuda.current_stream().cuda_stream)
    assert st == R.RWTTT_OK and v == 1
    snap = table.checkpoint(1)
    torch.cuda.synchronize()
    hashes = [slot_hash(sess.live(1, l)) for l in range(L)]
    # the lineages are separate: writes to the child and the parent stay local
    write_commit([2], 94)
    write_commit([0, 1], 96)
    assert sess.versions() == table.V == [2, 2, 2, 0]
    for r in range(n_owners):
        check_state(r)
    assert R.rwttt_resume(sess.ctx, 1, [h.data_ptr() for h in host], v,
                          torch.cuda.current_stream().cuda_stream) == R.RWTTT_OK
    assert table.resume(1, snap) == O.OK
    torch.cuda.synchronize()
    assert sess.versions() == table.V == [2, 1, 2, 0]
    assert [slot_hash(sess.live(1, l)) for l in range(L)] == hashes
    check_state(1)
    # READ outputs of every owner against the oracle
    xd = to_device(X, "bf16")
    y = torch.zeros((n_owners, d_model), dtype=torch.bfloat16, device="cuda")
    for l in range(L):
        read_group(sess, list(range(n_owners)), l, xd, y)
        torch.cuda.synchronize()
        W0 = O.widen(src.w0(l), "bf16")
        for r in range(n_owners):
            ref = O.round_to(O.read_apply(O.widen(X[r], "bf16"), W0, table.D[(r, l)]), "bf16")
            assert O.max_rel_floor(host_f64(y[r], "bf16"), ref) <= BF16_OUT_TOL, (r, l)


@pytest.mark.parametrize("chunk", [16, 80])
def test_largest_group_read_and_write_with_token(chunk):
    """RWTTT_MAX_GROUP owners in one READ and one WRITE group (kernel argument
    arrays full), against the oracle; the group is a permutation."""
    n, d_ff, d_model = R.RWTTT_MAX_GROUP, 264, 136
    wl = small_workload(d_ff, d_model, "bf16", "f32", n, eta=0.05)
    say("max group", chunk)
    src = TensorSource(wl)
    sess = Session(wl, src)
    group = list(np.random.default_rng(5).permutation(n))
    X = draw((n, d_ff), 1.0, "bf16", wl.seed, (93,))
    xd = to_device(X, "bf16")
    y = torch.zeros((n, d_model), dtype=torch.bfloat16, device="cuda")
    read_group(sess, group, 0, xd, y)
    torch.cuda.synchronize()
    W0 = O.widen(src.w0(0), "bf16")
    for r in range(n):
        ref = O.round_to(O.read_apply(O.widen(X[r], "bf16"), W0, O.widen(src.dw_init(r, 0), "f32")), "bf16")
        assert O.max_rel_floor(host_f64(y[r], "bf16"), ref) <= BF16_OUT_TOL, r
    zs = [to_device(draw((chunk, d_ff), 1.0, "bf16", wl.seed, (94, r), absval=True), "bf16") for r in group]
    gs = [to_device(draw((chunk, d_model), 1.0, "bf16", wl.seed, (95, r)), "bf16") for r in group]
    y2 = torch.zeros_like(y)
    assert write_group(sess, group, 0, chunk, zs, gs, x_dev=xd, y_dev=y2) == R.RWTTT_OK
    assert R.rwttt_commit(sess.ctx, group) == R.RWTTT_OK
    torch.cuda.synchronize()
    if chunk > 64:
        assert torch.equal(y2, y)              # this token is a READ at version v, bit for bit
    else:
        for r in range(n):                     # the fused token sums in another order
            assert O.max_rel_floor(host_f64(y2[r], "bf16"), host_f64(y[r], "bf16")) <= BF16_OUT_TOL, r
    for i, r in enumerate(group):
        cand = O.round_to(O.write_candidate(O.widen(src.dw_init(r, 0), "f32"), host_f64(zs[i], "bf16"),
                                            host_f64(gs[i], "bf16"), wl.eta), "f32")
        assert O.rel_frobenius(host_f64(sess.live(r, 0), "f32"), cand) <= STATE_TOL, r
    assert sess.versions() == [1] * n


def test_injected_write_failure_rolls_back_exactly():
    wl = small_workload(520, 264, "bf16", "f32", 3)
    src = TensorSource(wl)
    sess = Session(wl, src)
    say("inject failure")
    z = [to_device(draw((16, 520), 1.0, "bf16", 1, (1,)), "bf16")]
    g = [to_device(draw((16, 264), 1.0, "bf16", 1, (2,)), "bf16")]
    live = slot_hash(sess.live(1, 0))
    assert R.rwttt_inject_write_failures(sess.ctx, 1) == R.RWTTT_OK
    assert write_group(sess, [1], 0, 16, z, g) == R.RWTTT_E_WRITE_FAILED
    assert R.rwttt_commit(sess.ctx, [1]) == R.RWTTT_E_WRITE_FAILED
    assert R.rwttt_rollback(sess.ctx, [1]) == R.RWTTT_OK
    torch.cuda.synchronize()
    assert slot_hash(sess.live(1, 0)) == live and sess.version(1) == (0, False)
    # the owner writes normally afterwards
    assert write_group(sess, [1], 0, 16, z, g) == R.RWTTT_OK
    assert R.rwttt_commit(sess.ctx, [1]) == R.RWTTT_OK
    assert sess.version(1) == (1, False)


# --------------------------------------------------------------------------
# full shapes, in the launch configuration of the benchmark
# --------------------------------------------------------------------------

def test_sixteen_writes_fp32_state_full_shape():
    """16 consecutive WRITE+commit of one owner at d_ff 9728, d_model 2560, C 64."""
    import dataclasses
    wl = dataclasses.replace(workload(2), n_owners=1, n_layers=1)
    src = TensorSource(wl)
    say("16 writes full shape")
    sess = Session(wl, src)
    D = O.widen(src.dw_init(0, 0), "f32")
    for t in range(16):
        Z, G = src.zg(t, 0, 0, 64)
        st = write_group(sess, [0], 0, 64, [to_device(Z, "bf16")], [to_device(G, "bf16")])
        assert st == R.RWTTT_OK
        assert R.rwttt_commit(sess.ctx, [0]) == R.RWTTT_OK
        D = O.round_to(O.write_candidate(D, O.widen(Z, "bf16"), O.widen(G, "bf16"), wl.eta), "f32")
    torch.cuda.synchronize()
    err = O.rel_frobenius(host_f64(sess.live(0, 0), "f32"), D)
    say("rel frobenius after 16 writes", err)
    assert err <= STATE_TOL
    assert sess.version(0) == (16, False)


def test_read8_full_shape_matches_oracle():
    """Eight owners at d_ff 9728, d_model 2560: bf16 io, fp32 state."""
    wl = workload(1)
    src = TensorSource(wl)
    say("read8 full shape")
    sess = Session(wl, src)
    W0 = O.widen(src.w0(0), "bf16")
    D = [O.widen(src.dw_init(r, 0), "f32") for r in range(8)]
    y = torch.zeros((8, wl.d_model), dtype=torch.bfloat16, device="cuda")
    for t in range(2):
        X = src.x_step(t)[:, 0]
        read_group(sess, list(range(8)), 0, to_device(X, "bf16"), y)
        torch.cuda.synchronize()
        for r in range(8):
            ref = O.round_to(O.read_apply(O.widen(X[r], "bf16"), W0, D[r]), "bf16")
            err = O.max_rel_floor(host_f64(y[r], "bf16"), ref)
            assert err <= BF16_OUT_TOL, (t, r, err)


# --------------------------------------------------------------------------
# exact bf16 rounding (round to nearest even, ties included)
# --------------------------------------------------------------------------

def test_read_bf16_output_rounding_is_exact():
    """y = e_0 W0 + e_0 dW with W0 = 0 is exactly dW[0] in fp32; its bf16 bits must be RNE."""
    d_ff, d_model, n = 256, 512, 2
    wl = small_workload(d_ff, d_model, "bf16", "f32", n)
    sess = Session(wl, None)
    rng = np.random.default_rng(11)
    base = (O.bf16_bits(O.bf16_round(rng.standard_normal(d_model))).astype(np.uint32) << 16)
    row = np.where(rng.random(d_model) < 0.5, base | 0x8000, base | rng.integers(0, 0x10000, d_model))
    row = row.astype(np.uint32).view(np.float32)
    for r in range(n):
        sess.slots[r][0][0].zero_()
        sess.slots[r][0][0][0] = torch.from_numpy(row * (r + 1)).cuda()
    sess.w0[0].zero_()
    x = np.zeros((n, d_ff), dtype=np.uint16)
    x[:, 0] = 0x3F80
    y = torch.zeros((n, d_model), dtype=torch.bfloat16, device="cuda")
    read_group(sess, [0, 1], 0, to_device(x, "bf16"), y)
    torch.cuda.synchronize()
    for r in range(n):
        want = O.bf16_bits(O.round_to((row * (r + 1)).astype(np.float64), "bf16"))
        assert np.array_equal(to_host(y[r], "bf16"), want), r


@pytest.mark.parametrize("chunk", [1, 128, 150, 170])
def test_write_bf16_state_rounding_is_exact(chunk):
    """live + 1.0 * Z^T G with one unit rank is an exact fp32 sum; the bf16 shadow must be RNE.

    chunk 1 takes the streaming WRITE kernel, the others the GEMM kernel, whose last rank stage
    then sits in each of its three LDS stages in turn (4, 5 and 6 stages of 32 ranks).
    """
    d_ff, d_model = 256, 512
    wl = small_workload(d_ff, d_model, "bf16", "bf16", 1, eta=1.0)
    src = TensorSource(wl)
    sess = Session(wl, src)
    L = draw((d_ff, d_model), 1.0, "bf16", 3, (1,))
    to_device(L, "bf16", out=sess.slots[0][0][0])
    Z = np.zeros((chunk, d_ff), dtype=np.uint16)
    Z[chunk - 1, :] = 0x3F80                     # rank chunk-1 is all ones
    G = draw((chunk, d_model), 1.0, "bf16", 3, (2,))
    st = write_group(sess, [0], 0, chunk, [to_device(Z, "bf16")], [to_device(G, "bf16")], eta=1.0)
    assert st == R.RWTTT_OK
    torch.cuda.synchronize()
    want = O.bf16_bits(O.round_to(O.write_candidate(O.widen(L, "bf16"), O.widen(Z, "bf16"),
                                                    O.widen(G, "bf16"), 1.0), "bf16"))
    got = to_host(sess.shadow(0, 0), "bf16")
    ties = np.mean((O.widen(L, "bf16") + O.widen(G[chunk - 1], "bf16")[None, :]) !=
                   O.bf16_round(O.widen(L, "bf16") + O.widen(G[chunk - 1], "bf16")[None, :]))
    say("inexact sums (rounded):", ties)
    assert np.array_equal(got, want)


# --------------------------------------------------------------------------
# degenerate updates: eta = 0 or Z = 0 leave the candidate equal to live, bit for bit
# --------------------------------------------------------------------------

DEGENERATE_CASES = [
    # d_ff, d_model, io, state, chunk: the streaming kernel, the GEMM, the fp32-evidence kernel
    (1000, 264, "bf16", "f32", 17),
    (1000, 264, "bf16", "bf16", 64),
    (520, 264, "bf16", "bf16", 150),
    (520, 264, "bf16", "f32", 100),
    (256, 64, "f32", "f32", 4),
    (264, 520, "f32", "bf16", 5),
]


@pytest.mark.parametrize("d_ff,d_model,io,state,chunk", DEGENERATE_CASES)
def test_zero_step_or_zero_evidence_gives_a_candidate_equal_to_live(d_ff, d_model, io, state, chunk):
    """With eta = 0 (and random evidence), or with Z = 0 (and eta = 1), the
    candidate dW + eta Z^T G is exactly the live state (Section 3, Write with
    a null update), in both state dtypes and on every WRITE kernel; the token is
    still the READ at version v."""
    wl = small_workload(d_ff, d_model, io, state, 3)
    say("degenerate write", d_ff, d_model, io, state, chunk)
    src = TensorSource(wl)
    sess = Session(wl, src)
    Z = to_device(draw((chunk, d_ff), 1.0, io, wl.seed, (96, 1), absval=True), io)
    G = to_device(draw((chunk, d_model), 1.0, io, wl.seed, (97, 1)), io)
    Z0 = torch.zeros_like(Z)
    live = slot_hash(sess.live(1, 0))
    for zz, eta in ((Z, 0.0), (Z0, 1.0)):
        assert write_group(sess, [1], 0, chunk, [zz], [G], eta=eta) == R.RWTTT_OK
        torch.cuda.synchronize()
        assert slot_hash(sess.shadow(1, 0)) == live, eta
        assert R.rwttt_commit(sess.ctx, [1]) == R.RWTTT_OK
        torch.cuda.synchronize()
        assert slot_hash(sess.live(1, 0)) == live
    assert sess.version(1) == (2, False)
    # with a token the step's output is the READ of the unchanged state
    X = draw((3, d_ff), 1.0, io, wl.seed, (98,))
    xd = to_device(X, io)
    tdt = torch.float32 if io == "f32" else torch.bfloat16
    y = torch.zeros((3, d_model), dtype=tdt, device="cuda")
    assert write_group(sess, [1], 0, chunk, [Z0], [G], eta=1.0, x_dev=xd, y_dev=y) == R.RWTTT_OK
    torch.cuda.synchronize()
    ref = O.round_to(O.read_apply(O.widen(X[1], io), O.widen(src.w0(0), io),
                                  O.widen(src.dw_init(1, 0), state)), io)
    assert O.max_rel_floor(host_f64(y[1], io), ref) <= out_tol(io)
    assert slot_hash(sess.shadow(1, 0)) == live
