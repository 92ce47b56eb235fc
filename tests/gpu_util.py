"""Helpers shared by the GPU tests: device inputs, slot hashes, oracle views."""

import dataclasses
import hashlib
import sys

import numpy as np
import torch

import oracle as O
from rwttt_inputs import READ, WRITE, TensorSource, draw, workload
from paper_2605_28053_amd import _rwttt as R
from paper_2605_28053_amd.serving import Session, to_device, to_host


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def small_workload(d_ff, d_model, io, state, n_owners, seed=123, eta=0.01, dw_std=0.05):
    base = workload(3)
    return dataclasses.replace(base, name=f"t{d_ff}x{d_model}", n_owners=n_owners, n_layers=1,
                               d_ff=d_ff, d_model=d_model, io_dtype=io, state_dtype=state,
                               seed=seed, eta=eta, dw_std=dw_std,
                               w0_std=float(1.0 / np.sqrt(d_ff)))


def slot_hash(t):
    return hashlib.sha1(t.detach().contiguous().view(torch.uint8).cpu().numpy().tobytes()).hexdigest()


def all_slot_hashes(sess):
    return {(r, i, s): slot_hash(sess.slots[r][i][s])
            for r in range(sess.wl.n_owners) for i in range(sess.L) for s in range(2)}


def read_group(sess, owners, li, x_dev, y_dev, effect=READ):
    g = R.make_group(effect, 0, len(owners))
    st = R.rwttt_read(sess.ctx, g, R.u32_array(owners), li, x_dev.data_ptr(), y_dev.data_ptr(),
                      torch.cuda.current_stream().cuda_stream)
    assert st == R.RWTTT_OK, R.rwttt_strerror(st)


def write_group(sess, owners, li, chunk, zs, gs, eta=None, x_dev=None, y_dev=None):
    """One WRITE group; with x_dev/y_dev the step's token is returned in y_dev."""
    g = R.make_group(WRITE, 0, len(owners))
    st = R.rwttt_write(sess.ctx, g, R.u32_array(owners), li, chunk,
                       [z.data_ptr() for z in zs], [x.data_ptr() for x in gs],
                       sess.wl.eta if eta is None else eta,
                       0 if x_dev is None else x_dev.data_ptr(),
                       0 if y_dev is None else y_dev.data_ptr(),
                       stream=torch.cuda.current_stream().cuda_stream)
    return st


def host_f64(t, dtype):
    return O.widen(to_host(t, dtype), dtype)


def run_gpu_trace(wl, trace, src, steps, layers=None, cols=None, fail_hook=None, stream=None,
                  backend=0, rank=0, on_step=None):
    """Run steps of a trace through Session.step (the serving loop) and collect
    (StepResult, versions after the step, {(owner, layer): y row}) per step.
    ``on_step(sess, t)`` runs after each step, once the device is idle."""
    layers = list(range(wl.n_layers)) if layers is None else list(layers)
    sess = Session(wl, src, layers, backend=backend, rank=rank)
    out = []
    tdt = torch.float32 if wl.io_dtype == "f32" else torch.bfloat16
    for t in steps:
        items = trace[t]
        X = [to_device(src.x_step(t)[:, l], wl.io_dtype) for l in layers]
        Y = [torch.zeros((wl.n_owners, wl.d_model), dtype=tdt, device="cuda") for _ in layers]
        keep, zg = [], {}
        for it in items:
            if it.effect == WRITE:
                zd, gd = [], []
                for l in layers:
                    Z, G = src.zg(t, it.owner, l, it.chunk)
                    zd.append(to_device(Z, wl.io_dtype))
                    gd.append(to_device(G, wl.io_dtype))
                keep += zd + gd
                zg[it.owner] = ([z.data_ptr() for z in zd], [g.data_ptr() for g in gd])
        if stream is not None:
            stream.wait_for_current()
        res = sess.step(t, items, [x.data_ptr() for x in X], [y.data_ptr() for y in Y], zg,
                        torch.cuda.current_stream().cuda_stream if stream is None else stream,
                        fail_hook)
        torch.cuda.synchronize()
        ys = {}
        for it in items:
            if it.emit:
                for i, l in enumerate(layers):
                    row = host_f64(Y[i][it.owner], wl.io_dtype)
                    ys[(it.owner, l)] = row if cols is None else row[cols]
        out.append((res, sess.versions(), ys))
        if on_step is not None:
            on_step(sess, t)
    return sess, out


def plan_tuples(res):
    p = res.plan
    return [((p.group(i).effect, p.group(i).backend_type, p.group(i).shape_class,
              p.group(i).placement), p.owners(i)) for i in range(p.n_groups)]


