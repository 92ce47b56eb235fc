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


def write_group(sess, owners, li, chunk, zs, gs, eta=None):
    g = R.make_group(WRITE, 0, len(owners))
    st = R.rwttt_write(sess.ctx, g, R.u32_array(owners), li, chunk,
                       [z.data_ptr() for z in zs], [x.data_ptr() for x in gs],
                       sess.wl.eta if eta is None else eta,
                       torch.cuda.current_stream().cuda_stream)
    return st


def host_f64(t, dtype):
    return O.widen(to_host(t, dtype), dtype)
