"""Serving loop of Algorithm 1 on top of the C ABI, with torch as the allocator.

``Session`` owns the device memory of one workload -- W0 per layer, two state
slots per (owner, layer) and the library workspace -- and runs decode steps:
View (committed versions) -> events -> rwttt_plan -> per layer, per group:
rwttt_read for READ groups, rwttt_write (update plus the step's token) for
WRITE groups -> commit or rollback of the WRITE owners.  When a workload's
update evidence is the chunk's own activations, the session attaches tail
buffers: READ steps append x to them (rwttt_read_append) and a WRITE takes its
chunk from the tail.  Host code here only marshals arguments; every number is
computed by the library's kernels.
"""

from dataclasses import dataclass

import numpy as np
import torch

from . import _rwttt as R
from rwttt_inputs import READ, WRITE, shape_class

TORCH_DTYPE = {"f32": torch.float32, "bf16": torch.bfloat16}
CODE = {"f32": R.RWTTT_F32, "bf16": R.RWTTT_BF16}


def to_device(a, dtype, device="cuda", out=None):
    """Copy a host array (float32, or bf16 bit patterns as uint16) to the device."""
    if dtype == "bf16":
        host = torch.from_numpy(np.ascontiguousarray(a).view(np.int16))
        if out is None:
            out = torch.empty(host.shape, dtype=torch.bfloat16, device=device)
        out.view(torch.int16).copy_(host)
        return out
    host = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    if out is None:
        out = torch.empty(host.shape, dtype=torch.float32, device=device)
    out.copy_(host)
    return out


def to_host(t, dtype):
    """Device tensor -> host array in the input module's representation."""
    if dtype == "bf16":
        return t.detach().view(torch.int16).cpu().numpy().view(np.uint16)
    return t.detach().float().cpu().numpy()


class StreamPair:
    """Two torch streams (default priority) for READ and WRITE groups.

    join() makes each stream wait for the other's work so far: the next
    step's reads see this step's committed candidates, and the next step's
    WRITEs overwrite a shadow slot only after the reads that used it.
    """

    def __init__(self, device="cuda"):
        self.read_stream = torch.cuda.Stream(device=device)
        self.write_stream = torch.cuda.Stream(device=device)
        self.read = self.read_stream.cuda_stream
        self.write = self.write_stream.cuda_stream

    def join(self):
        e_r = torch.cuda.Event()
        e_w = torch.cuda.Event()
        e_r.record(self.read_stream)
        e_w.record(self.write_stream)
        self.read_stream.wait_event(e_w)
        self.write_stream.wait_event(e_r)

    def wait_for_current(self):
        """Order both streams after the work already on torch's current stream."""
        cur = torch.cuda.current_stream()
        self.read_stream.wait_stream(cur)
        self.write_stream.wait_stream(cur)


@dataclass
class StepResult:
    plan: R.PlanResult
    committed: list
    rolled_back: list
    statuses: list


class Session:
    """Device-resident state of one workload plus the serving loop."""

    def __init__(self, wl, src=None, layers=None, max_group=None, device="cuda",
                 init_state=True, init_w0=True, tail_rows=None, backend=R.RWTTT_FAST_WEIGHT,
                 rank=0):
        self.wl = wl
        self.device = device
        self.backend, self.rank = backend, rank
        self.layers = list(range(wl.n_layers)) if layers is None else list(layers)
        self.L = len(self.layers)
        sdt, iodt = TORCH_DTYPE[wl.state_dtype], TORCH_DTYPE[wl.io_dtype]
        K, N = wl.d_ff, wl.d_model
        # a fast-weight slot is dW [K, N]; an adapter slot is A [K, r] then B [r, N]
        shape = (K, N) if backend == R.RWTTT_FAST_WEIGHT else ((K + N) * rank,)
        self.w0 = [torch.empty((K, N), dtype=iodt, device=device) for _ in self.layers]
        self.slots = [[[torch.empty(shape, dtype=sdt, device=device) for _ in range(2)]
                       for _ in self.layers] for _ in range(wl.n_owners)]
        if src is not None and init_w0:
            for i, l in enumerate(self.layers):
                to_device(src.w0(l), wl.io_dtype, device, out=self.w0[i])
        if src is not None and init_state:
            for r in range(wl.n_owners):
                for i, l in enumerate(self.layers):
                    if backend == R.RWTTT_FAST_WEIGHT:
                        to_device(src.dw_init(r, l), wl.state_dtype, device, out=self.slots[r][i][0])
                    else:
                        a, b = src.adapter_init(r, l, rank)
                        to_device(np.concatenate([a.reshape(-1), b.reshape(-1)]), wl.state_dtype,
                                  device, out=self.slots[r][i][0])
        self.max_group = max_group or min(R.RWTTT_MAX_GROUP, wl.n_owners)
        slot_ptrs = []
        for r in range(wl.n_owners):
            for i in range(self.L):
                slot_ptrs += [self.slots[r][i][0].data_ptr(), self.slots[r][i][1].data_ptr()]
        cfg = R.make_config(wl.n_owners, self.L, K, N, CODE[wl.io_dtype], CODE[wl.state_dtype],
                            self.max_group, [w.data_ptr() for w in self.w0], slot_ptrs,
                            backend=backend, rank=rank)
        ws_bytes = R.rwttt_workspace_bytes(cfg)
        self.workspace = torch.empty(ws_bytes, dtype=torch.uint8, device=device)
        cfg.workspace = self.workspace.data_ptr()
        cfg.workspace_bytes = ws_bytes
        self.cfg = cfg
        self.ctx = R.rwttt_create(cfg)
        # tail buffers (TailBufferState) when Z is the chunk's own inputs
        if tail_rows is None:
            tail_rows = 0 if wl.z_abs else max((wl.chunk,) + tuple(wl.chunk_choices))
        self.tail_rows = tail_rows
        self.tails = []
        if tail_rows:
            self.tails = [[torch.zeros((tail_rows, K), dtype=iodt, device=device)
                           for _ in self.layers] for _ in range(wl.n_owners)]
            st = R.rwttt_attach_tail(self.ctx, [t.data_ptr() for row in self.tails for t in row],
                                     tail_rows)
            if st != R.RWTTT_OK:
                raise R.RwtttError(st, "rwttt_attach_tail")

    def close(self):
        if self.ctx:
            R.rwttt_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---- owner table views -------------------------------------------------
    def version(self, r):
        return R.rwttt_version(self.ctx, r)

    def versions(self):
        return [R.rwttt_version(self.ctx, r)[0] for r in range(self.wl.n_owners)]

    def live(self, r, li):
        """Live slot tensor of owner r at local layer index li."""
        ptr = R.rwttt_slot(self.ctx, r, li, 0)
        a, b = self.slots[r][li]
        return a if a.data_ptr() == ptr else b

    def shadow(self, r, li):
        ptr = R.rwttt_slot(self.ctx, r, li, 1)
        a, b = self.slots[r][li]
        return a if a.data_ptr() == ptr else b

    def factors(self, slot):
        """(A [d_ff, r], B [r, d_model]) views of an adapter slot tensor."""
        K, N, r = self.wl.d_ff, self.wl.d_model, self.rank
        return slot[:K * r].view(K, r), slot[K * r:].view(r, N)

    # ---- one decode step (Algorithm 1) ------------------------------------
    def events(self, t, items):
        evs = []
        for it in items:
            v, _ = R.rwttt_version(self.ctx, it.owner)
            evs.append((it.owner, self.backend, shape_class(self.wl, it.effect, it.chunk), 0,
                        it.effect, v, t))
        return evs

    def step(self, t, items, x_ptrs, y_ptrs, zg_ptrs, stream=0, fail_hook=None, timer=None):
        """Run one step.

        x_ptrs[i], y_ptrs[i]: device addresses of [n_owners, d_ff] inputs and
        [n_owners, d_model] outputs of local layer i.  zg_ptrs[r] =
        (z_ptrs_per_layer, g_ptrs_per_layer) for each WRITE owner r (with tail
        buffers attached the z pointers are not used).

        ``stream`` is one HIP stream handle for every launch, or a
        ``StreamPair``: READ groups then go on its read stream and WRITE groups
        (update with its token) on its write stream, so groups of disjoint
        owners overlap on the device; the pair is joined both ways at the end
        of the step.  ``timer``, if given, has launch(kind, count, chunk,
        stream) called before every library call and close() after every
        group.
        """
        pair = stream if isinstance(stream, StreamPair) else None
        s_read = pair.read if pair else stream
        s_write = pair.write if pair else stream
        wl = self.wl
        by_owner = {it.owner: it for it in items}
        evs = self.events(t, items)
        plan = R.rwttt_plan(self.ctx, evs, t)
        if plan.status != R.RWTTT_OK:
            raise R.RwtttError(plan.status, "rwttt_plan")
        # the version each member was planned at, indexed like the owner map:
        # every read and write re-checks it against the owner table
        planned = {e[0]: e[5] for e in evs}
        expected = R.u64_array(planned[plan.owner_map_c[i]] for i in range(plan.n_mapped))
        statuses = []
        write_groups = []
        for gi in range(plan.n_groups):
            g = plan.group(gi)
            owners = plan.owners(gi)
            emit = any(by_owner[r].emit for r in owners)
            is_write = g.effect == WRITE
            chunk = by_owner[owners[0]].chunk if is_write else 0
            stream = s_write if is_write else s_read
            failed = False
            for i in range(self.L):
                need_token = emit
                if is_write and not failed:
                    # the WRITE transition returns the step's token with the candidate
                    zs = None if self.tails else [zg_ptrs[r][0][i] for r in owners]
                    gs = [zg_ptrs[r][1][i] for r in owners]
                    tok = emit or bool(self.tails)
                    if timer is not None:
                        timer.launch("write_token" if tok else "write", g.count, chunk, stream)
                    st = R.rwttt_write(self.ctx, g, plan.owner_map_c, i, chunk, zs, gs, wl.eta,
                                       x_ptrs[i] if tok else 0, y_ptrs[i] if tok else 0,
                                       stream, expected)
                    statuses.append(st)
                    if st == R.RWTTT_OK:
                        need_token = False
                    else:
                        failed = True
                if need_token:
                    # READ groups, and the layers of a WRITE group whose update failed:
                    # the token at the unchanged version v (a READ step also appends
                    # its input to the owner's tail)
                    if timer is not None:
                        timer.launch("read", g.count, 0, stream)
                    fn = R.rwttt_read_append if self.tails and not is_write else R.rwttt_read
                    st = fn(self.ctx, g, plan.owner_map_c, i, x_ptrs[i], y_ptrs[i], stream, expected)
                    if st != R.RWTTT_OK:
                        raise R.RwtttError(st, "rwttt_read")
            if is_write:
                write_groups.append((owners, failed))
            if timer is not None:
                timer.close()
        if pair is not None:
            pair.join()
        committed, rolled = [], []
        for owners, failed in write_groups:
            # the failure branch of Algorithm 1 rolls a failed group back;
            # otherwise each owner commits unless its WRITE is declared failed
            bad = owners if failed else [r for r in owners if by_owner[r].fail or
                                         (fail_hook is not None and fail_hook(t, r))]
            good = [r for r in owners if r not in bad]
            if good:
                st = R.rwttt_commit(self.ctx, good)
                if st != R.RWTTT_OK:
                    raise R.RwtttError(st, "rwttt_commit")
            if bad:
                st = R.rwttt_rollback(self.ctx, bad)
                if st != R.RWTTT_OK:
                    raise R.RwtttError(st, "rwttt_rollback")
            committed += good
            rolled += bad
        return StepResult(plan, committed, rolled, statuses)
