"""rwttt_read_noalloc, the READ for callers that cannot allocate device memory,
against rwttt_read and the oracle, through the C ABI.

Both entry points run the same kernels in the same summation order, so their
outputs must be bit-identical; each is also within the bf16 output tolerance
(max |a-b| / max(|b|, 1e-2 rms(b)) <= 2e-2) of the oracle.  The no-alloc calls
run on a host-only context (no workspace) over the same slots.
"""

import numpy as np
import pytest
import torch

import oracle as O
from rwttt_inputs import READ, TensorSource, draw
from tests.gpu_util import R, Session, host_f64, read_group, say, small_workload, to_device

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

BF16_OUT_TOL = 2e-2


def host_only_ctx(sess):
    """A context over the session's W0 and slots with no workspace."""
    wl = sess.wl
    slots = [p for r in range(wl.n_owners) for i in range(sess.L)
             for p in (sess.slots[r][i][0].data_ptr(), sess.slots[r][i][1].data_ptr())]
    cfg = R.make_config(wl.n_owners, sess.L, wl.d_ff, wl.d_model,
                        R.RWTTT_BF16 if wl.io_dtype == "bf16" else R.RWTTT_F32,
                        R.RWTTT_BF16 if wl.state_dtype == "bf16" else R.RWTTT_F32,
                        sess.max_group, [w.data_ptr() for w in sess.w0], slots)
    return R.rwttt_create(cfg), cfg


def noalloc_read(ctx, owners, x, y):
    g = R.make_group(READ, 0, len(owners))
    st = R.rwttt_read_noalloc(ctx, g, R.u32_array(owners), 0, x.data_ptr(), y.data_ptr(),
                              torch.cuda.current_stream().cuda_stream, expected=[0] * len(owners))
    assert st == R.RWTTT_OK, R.rwttt_strerror(st)


def check_pair(sess, ctx, src, owners, key, oracle_owners):
    wl = sess.wl
    n = wl.n_owners
    X = draw((n, wl.d_ff), 1.0, wl.io_dtype, wl.seed, key)
    xd = to_device(X, wl.io_dtype)
    ref_y = torch.full((n, wl.d_model), 3.0, dtype=torch.bfloat16, device="cuda")
    got_y = ref_y.clone()
    read_group(sess, owners, 0, xd, ref_y)
    noalloc_read(ctx, owners, xd, got_y)
    torch.cuda.synchronize()
    assert torch.equal(got_y.view(torch.int16), ref_y.view(torch.int16))
    others = [r for r in range(n) if r not in owners]
    if others:
        assert torch.all(got_y[others] == 3.0)
    W0 = O.widen(src.w0(0), wl.io_dtype)
    for r in oracle_owners:
        ref = O.round_to(O.read_apply(O.widen(X[r], wl.io_dtype), W0,
                                      O.widen(src.dw_init(r, 0), wl.state_dtype)), wl.io_dtype)
        err = O.max_rel_floor(host_f64(got_y[r], wl.io_dtype), ref)
        assert err <= BF16_OUT_TOL, (r, err)


@pytest.mark.parametrize("state", ["f32", "bf16"])
def test_noalloc_read_equals_read_on_two_calls_second_smaller(state):
    wl = small_workload(9728, 2560, "bf16", state, 8)
    say("noalloc read", state)
    src = TensorSource(wl)
    sess = Session(wl, src)
    ctx, cfg = host_only_ctx(sess)
    try:
        # every owner at the 4B-layer shape, then a smaller group in another order
        check_pair(sess, ctx, src, list(range(8)), (95, 1), [0, 7])
        check_pair(sess, ctx, src, [5, 2, 7], (95, 2), [2])
        assert R.rwttt_version(ctx, 0) == (0, False)
    finally:
        R.rwttt_destroy(ctx)
        sess.close()
    # a smaller shape with ragged tiles after the large one: the array keeps the
    # previous call's partial sums, which this call must overwrite, not add to
    wl2 = small_workload(1000, 264, "bf16", state, 3)
    src2 = TensorSource(wl2)
    sess2 = Session(wl2, src2)
    ctx2, cfg2 = host_only_ctx(sess2)
    try:
        check_pair(sess2, ctx2, src2, [2, 0], (95, 3), [0, 2])
    finally:
        R.rwttt_destroy(ctx2)
        sess2.close()


def test_noalloc_read_rejects_a_group_above_the_array_and_a_stale_version():
    wl = small_workload(1000, 264, "bf16", "f32", 2)
    sess = Session(wl, TensorSource(wl))
    ctx, cfg = host_only_ctx(sess)
    x = torch.zeros((2, 1000), dtype=torch.bfloat16, device="cuda")
    y = torch.zeros((2, 264), dtype=torch.bfloat16, device="cuda")
    g = R.make_group(READ, 0, 2)
    st = R.rwttt_read_noalloc(ctx, g, R.u32_array([0, 1]), 0, x.data_ptr(), y.data_ptr(),
                              torch.cuda.current_stream().cuda_stream, expected=[0, 1])
    assert st == R.RWTTT_E_STALE_VERSION
    R.rwttt_destroy(ctx)
    sess.close()
