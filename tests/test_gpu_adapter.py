"""GPU parity of the DeltaAdapterState backend (Section 4.4; Appendix D)
against the oracle, through the C ABI.

Tolerances as for the fast-weight backend: bf16 outputs max relative error
(floored at 1e-2 rms) <= 2e-2, fp32 outputs <= 1e-4, fp32 state relative
Frobenius <= 1e-3 (after up to 16 WRITEs); owner maps, versions, slot hashes,
and batched-versus-sequential results exact.
"""

import dataclasses

import numpy as np
import pytest
import torch

import oracle as O
from rwttt_inputs import READ, WRITE, TensorSource, build_trace, draw, workload
from tests.gpu_util import (R, Session, all_slot_hashes, host_f64, plan_tuples, read_group,
                            run_gpu_trace, say, slot_hash, small_workload, to_device, write_group)

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

BF16_OUT_TOL = 2e-2
F32_OUT_TOL = 1e-4
STATE_TOL = 1e-3
ADA = R.RWTTT_DELTA_ADAPTER


def out_tol(dtype):
    return BF16_OUT_TOL if dtype == "bf16" else F32_OUT_TOL


def factors_f64(sess, slot, state):
    a, b = sess.factors(slot)
    return host_f64(a, state), host_f64(b, state)


def oracle_factors(src, r, rank, state):
    a, b = src.adapter_init(r, 0, rank)
    return O.widen(a, state), O.widen(b, state)


READ_CASES = [
    # d_ff, d_model, io, state, rank, n_owners, group
    (256, 64, "f32", "f32", 4, 2, [1, 0]),
    (1000, 264, "bf16", "f32", 8, 6, [3, 0, 5]),
    (1000, 264, "bf16", "bf16", 1, 4, [2, 1]),
    (520, 1032, "bf16", "f32", 32, 5, [4, 2, 0, 1]),
    (9728, 2560, "bf16", "f32", 8, 8, list(range(8))),
    # rank above 8 (a second u-share pass) that is not a power of two
    (3000, 2600, "bf16", "f32", 12, 9, [7, 2, 8, 0, 5, 1, 3, 4, 6]),
    (520, 264, "f32", "bf16", 4, 3, [2, 0]),          # fp32 io, bf16 factors
]


@pytest.mark.parametrize("d_ff,d_model,io,state,rank,n_owners,group", READ_CASES)
def test_adapter_read_matches_oracle(d_ff, d_model, io, state, rank, n_owners, group):
    wl = small_workload(d_ff, d_model, io, state, n_owners)
    say("adapter read", d_ff, d_model, io, state, rank, group)
    src = TensorSource(wl)
    sess = Session(wl, src, backend=ADA, rank=rank)
    X = draw((n_owners, d_ff), 1.0, io, wl.seed, (85, rank))
    xd = to_device(X, io)
    tdt = torch.float32 if io == "f32" else torch.bfloat16
    before = all_slot_hashes(sess)
    y = torch.zeros((n_owners, d_model), dtype=tdt, device="cuda")
    read_group(sess, group, 0, xd, y)
    torch.cuda.synchronize()
    W0 = O.widen(src.w0(0), io)
    for r in group:
        A, B = oracle_factors(src, r, rank, state)
        ref = O.round_to(O.adapter_read(O.widen(X[r], io), W0, A, B), io)
        assert O.max_rel_floor(host_f64(y[r], io), ref) <= out_tol(io), r
    assert all_slot_hashes(sess) == before
    assert sess.versions() == [0] * n_owners
    others = [r for r in range(n_owners) if r not in group]
    if others:
        assert torch.count_nonzero(y[others].float()).item() == 0
    # batched == one owner at a time == reversed order, bit for bit
    y1 = torch.zeros_like(y)
    for r in group:
        read_group(sess, [r], 0, xd, y1)
    y2 = torch.zeros_like(y)
    read_group(sess, list(reversed(group)), 0, xd, y2)
    torch.cuda.synchronize()
    assert torch.equal(y[group], y1[group])
    assert torch.equal(y[group], y2[group])


WRITE_CASES = [
    # d_ff, d_model, io, state, rank, chunk, group
    (256, 64, "f32", "f32", 4, 4, [0, 1]),
    (1000, 264, "bf16", "f32", 8, 17, [2, 0]),
    (1000, 264, "bf16", "bf16", 8, 64, [1]),
    (520, 1032, "bf16", "f32", 32, 130, [3, 1, 0]),
    (9728, 2560, "bf16", "f32", 8, 64, [1, 3]),
    # ranks that are not powers of two (Q through the per-row path) in the
    # 8- and 16-wide rank classes of the update, and a chunk of two passes
    (2104, 1096, "bf16", "f32", 5, 33, [2, 0]),
    (2104, 1096, "bf16", "bf16", 12, 70, [3]),
    (1000, 264, "f32", "f32", 16, 20, [1, 2]),
    (520, 264, "f32", "bf16", 4, 6, [1, 2]),          # fp32 evidence into bf16 factors
]


@pytest.mark.parametrize("d_ff,d_model,io,state,rank,chunk,group", WRITE_CASES)
def test_adapter_write_token_commit_rollback_match_oracle(d_ff, d_model, io, state, rank, chunk,
                                                          group):
    n_owners = 4
    wl = small_workload(d_ff, d_model, io, state, n_owners, eta=0.01)
    say("adapter write", d_ff, d_model, io, state, rank, chunk, group)
    src = TensorSource(wl)
    sess = Session(wl, src, backend=ADA, rank=rank)
    tdt = torch.float32 if io == "f32" else torch.bfloat16
    X = draw((n_owners, d_ff), 1.0, io, wl.seed, (86, rank))
    xd = to_device(X, io)
    zs, gs, ref = [], [], {}
    for r in group:
        Z = draw((chunk, d_ff), 1.0, io, wl.seed, (87, r), absval=True)
        G = draw((chunk, d_model), 1.0, io, wl.seed, (88, r))
        zs.append(to_device(Z, io))
        gs.append(to_device(G, io))
        A, B = oracle_factors(src, r, rank, state)
        A1, B1 = O.adapter_write(A, B, O.widen(Z, io), O.widen(G, io), wl.eta)
        ref[r] = (O.round_to(A1, state), O.round_to(B1, state), A, B)
    before = all_slot_hashes(sess)
    y = torch.zeros((n_owners, d_model), dtype=tdt, device="cuda")
    st = write_group(sess, group, 0, chunk, zs, gs, x_dev=xd, y_dev=y)
    assert st == R.RWTTT_OK, R.rwttt_strerror(st)
    torch.cuda.synchronize()
    after = all_slot_hashes(sess)
    for key in before:
        r, i, s = key
        if r in group and s == 1:
            continue
        assert after[key] == before[key], key
    W0 = O.widen(src.w0(0), io)
    for r in group:
        A1, B1, A, B = ref[r]
        gA, gB = factors_f64(sess, sess.shadow(r, 0), state)
        if state == "f32":
            assert O.rel_frobenius(gA, A1) <= STATE_TOL and O.rel_frobenius(gB, B1) <= STATE_TOL
        else:
            assert O.max_rel_floor(gA, A1) <= BF16_OUT_TOL and O.max_rel_floor(gB, B1) <= BF16_OUT_TOL
        tok = O.round_to(O.adapter_read(O.widen(X[r], io), W0, A, B), io)
        assert O.max_rel_floor(host_f64(y[r], io), tok) <= out_tol(io), r
    # rollback the first owner, commit the rest
    keep = slot_hash(sess.live(group[0], 0))
    assert R.rwttt_rollback(sess.ctx, [group[0]]) == R.RWTTT_OK
    assert slot_hash(sess.live(group[0], 0)) == keep and sess.version(group[0]) == (0, False)
    if len(group) > 1:
        sh = {r: slot_hash(sess.shadow(r, 0)) for r in group[1:]}
        assert R.rwttt_commit(sess.ctx, group[1:]) == R.RWTTT_OK
        for r in group[1:]:
            assert sess.version(r) == (1, False) and slot_hash(sess.live(r, 0)) == sh[r]
    # the candidate does not depend on the group or on the token being asked for
    if len(group) > 1:
        r, i = group[1], 1
        solo = Session(wl, src, backend=ADA, rank=rank)
        assert write_group(solo, [r], 0, chunk, [zs[i]], [gs[i]]) == R.RWTTT_OK
        torch.cuda.synchronize()
        assert slot_hash(solo.shadow(r, 0)) == sh[r]
        solo.close()


@pytest.mark.parametrize("rank", [3, 4])
def test_adapter_tiny_trace_matches_oracle(rank):
    """The tiny fp32 trace (a WRITE every 4 steps, the 3rd write of owner 1
    forced to fail) through the serving loop with rank-r adapter state: plans,
    versions and every token against the oracle's sequential run, and the final
    factors."""
    wl = workload(0)
    trace, src = build_trace(wl), TensorSource(wl)
    say("adapter tiny trace", wl.name, rank)
    ref, table = O.run_trace(wl, trace, src, rank=rank)
    sess, got = run_gpu_trace(wl, trace, src, range(wl.n_steps), backend=ADA, rank=rank)
    for rec, (res, versions, ys) in zip(ref, got):
        assert plan_tuples(res) == [(g.key, g.owners) for g in rec.plan.groups]
        assert versions == rec.versions
        for k, v in rec.y.items():
            assert O.max_rel_floor(ys[k], v) <= out_tol(wl.io_dtype), (rec.step, k)
    for r in range(wl.n_owners):
        gA, gB = factors_f64(sess, sess.live(r, 0), wl.state_dtype)
        A, B = table.D[(r, 0)]
        assert O.rel_frobenius(gA, A) <= STATE_TOL and O.rel_frobenius(gB, B) <= STATE_TOL
    assert sess.versions() == [4, 3]


def test_adapter_sixteen_writes_full_shape():
    d_ff, d_model, rank = 9728, 2560, 8
    wl = small_workload(d_ff, d_model, "bf16", "f32", 2, eta=1e-3)
    say("adapter 16 writes")
    src = TensorSource(wl)
    sess = Session(wl, src, backend=ADA, rank=rank)
    A, B = oracle_factors(src, 1, rank, "f32")
    for k in range(16):
        Z = draw((64, d_ff), 1.0, "bf16", wl.seed, (89, k), absval=True)
        G = draw((64, d_model), 1.0, "bf16", wl.seed, (90, k))
        A, B = O.adapter_write(A, B, O.widen(Z, "bf16"), O.widen(G, "bf16"), wl.eta)
        A, B = O.round_to(A, "f32"), O.round_to(B, "f32")
        assert write_group(sess, [1], 0, 64, [to_device(Z, "bf16")], [to_device(G, "bf16")]) == R.RWTTT_OK
        assert R.rwttt_commit(sess.ctx, [1]) == R.RWTTT_OK
    torch.cuda.synchronize()
    gA, gB = factors_f64(sess, sess.live(1, 0), "f32")
    assert sess.versions() == [0, 16]
    assert O.rel_frobenius(gA, A) <= STATE_TOL and O.rel_frobenius(gB, B) <= STATE_TOL


def test_adapter_tail_and_fork():
    d_ff, d_model, rank, chunk, n_owners = 1000, 264, 8, 5, 3
    wl = small_workload(d_ff, d_model, "bf16", "f32", n_owners, eta=0.01)
    src = TensorSource(wl)
    sess = Session(wl, src, backend=ADA, rank=rank, tail_rows=chunk)
    X = [draw((n_owners, d_ff), 1.0, "bf16", wl.seed, (91, t)) for t in range(chunk)]
    y = torch.zeros((n_owners, d_model), dtype=torch.bfloat16, device="cuda")
    for t in range(chunk - 1):
        g = R.make_group(READ, 0, 2)
        assert R.rwttt_read_append(sess.ctx, g, R.u32_array([0, 2]), 0, to_device(X[t], "bf16").data_ptr(),
                                   y.data_ptr()) == R.RWTTT_OK
    G = draw((chunk, d_model), 1.0, "bf16", wl.seed, (92,))
    gd = to_device(G, "bf16")
    xd = to_device(X[chunk - 1], "bf16")
    wg = R.make_group(WRITE, 0, 1)
    assert R.rwttt_write(sess.ctx, wg, R.u32_array([2]), 0, chunk, None, [gd.data_ptr()], wl.eta,
                         xd.data_ptr(), y.data_ptr()) == R.RWTTT_OK
    assert R.rwttt_commit(sess.ctx, [2]) == R.RWTTT_OK
    torch.cuda.synchronize()
    Z = np.stack([X[t][2] for t in range(chunk)])
    A, B = oracle_factors(src, 2, rank, "f32")
    A1, B1 = O.adapter_write(A, B, O.widen(Z, "bf16"), O.widen(G, "bf16"), wl.eta)
    gA, gB = factors_f64(sess, sess.live(2, 0), "f32")
    assert O.rel_frobenius(gA, A1) <= STATE_TOL and O.rel_frobenius(gB, B1) <= STATE_TOL
    assert R.rwttt_tail_len(sess.ctx, 2, 0) == 0 and R.rwttt_tail_len(sess.ctx, 0, 0) == chunk - 1
    # fork the updated owner: the child's adapter slot is a bit copy, version and all
    assert R.rwttt_fork(sess.ctx, 2, 1) == R.RWTTT_OK
    torch.cuda.synchronize()
    assert slot_hash(sess.live(1, 0)) == slot_hash(sess.live(2, 0))
    assert sess.versions() == [0, 1, 1]
    # checkpoint owner 2's committed factors to pinned host memory, move the owner
    # on by another committed write, then resume: factors and version come back exactly
    nbytes = sess.live(2, 0).numel() * sess.live(2, 0).element_size()
    host = torch.empty(nbytes, dtype=torch.uint8, pin_memory=True)
    st, v = R.rwttt_checkpoint(sess.ctx, 2, [host.data_ptr()], torch.cuda.current_stream().cuda_stream)
    assert st == R.RWTTT_OK and v == 1
    torch.cuda.synchronize()
    saved = slot_hash(sess.live(2, 0))
    Z2 = to_device(draw((chunk, d_ff), 1.0, "bf16", wl.seed, (93,), absval=True), "bf16")
    assert write_group(sess, [2], 0, chunk, [Z2], [gd]) == R.RWTTT_OK
    assert R.rwttt_commit(sess.ctx, [2]) == R.RWTTT_OK
    torch.cuda.synchronize()
    assert sess.versions() == [0, 1, 2] and slot_hash(sess.live(2, 0)) != saved
    assert R.rwttt_resume(sess.ctx, 2, [host.data_ptr()], v,
                          torch.cuda.current_stream().cuda_stream) == R.RWTTT_OK
    torch.cuda.synchronize()
    assert sess.versions() == [0, 1, 1] and slot_hash(sess.live(2, 0)) == saved
    # the forked child kept its own copy throughout
    assert slot_hash(sess.live(1, 0)) == saved
