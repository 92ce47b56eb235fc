#!/usr/bin/env python3
"""Aggregate decode throughput of the owner-scoped fast-weight READ/WRITE path.

Workload: 8 request streams at 4B-class shape (d_model 2560, d_ff 9728), 36
fast-weight layers, bf16 activations, fp32 fast-weight state; each stream does
64 READ decode steps then one C=64 WRITE, phases staggered by 8 steps so most
steps mix READ owners and a WRITE owner.  One benchmark step is one decode
step of all 8 streams through every layer: rwttt_plan, the READ group's
launches, the WRITE group's token launches and update launches, and the
commits -- the whole hot path.  Every WRITE step also emits its token, so a
step yields 8 tokens.

Inputs are seeded synthetic tensors, resident in HBM before timing starts.
The timed region is bracketed by torch.cuda.synchronize().  Runs of launches
are also bracketed by HIP events on the launch stream; the READ kernel's
average bandwidth over the timed region gives the roofline fraction.  The CPU
oracle is then timed on a bounded sample of the same trace.  Finally a few
steps of the other three workloads (8-owner READ-only, 32-owner ragged, 8B
prefill then decode) are measured the same way and reported as compact
records in the same line; the prefill workload's decode throughput is timed
apart from its prefill WRITEs.
"""

import argparse
import json
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "aggregate decode tok/s (8 TTT streams, 1 GPU); % HBM peak READ, % MFMA WRITE"
HBM_PEAK_GBS = 8000.0
BF16_MFMA_PEAK_TFLOPS = 2500.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


KERNEL_SOURCES = ("rwttt_kernels.hip", "rwttt_device.h", "rwttt_kernels.h")


def code_lines(text):
    """The lines of a C/HIP source with // comments, blank lines and indentation removed."""
    out = []
    for line in text.splitlines():
        code = line.split("//", 1)[0].strip()
        if code:
            out.append(code)
    return out


def kernel_source_sha():
    """SHA-256 over the code (comments dropped) of the fast-weight kernel sources, in a fixed order."""
    import hashlib
    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        text = open(os.path.join(ROOT, "paper_2605_28053_amd", "csrc", name), encoding="utf-8").read()
        h.update("\n".join(code_lines(text)).encode())
        h.update(b"\0")
    return h.hexdigest()


def measured_traffic(records, wl):
    """Mean HBM bytes per READ call from the committed rocprofv3 PMC summary.

    The summary holds FETCH_SIZE and WRITE_SIZE per dispatch, scaled by what
    the same counters read for a plain 1 GiB device copy, per READ group size
    at one shape.  It is used only if the kernel source is the one the
    counters were taken on and the workload's READ has that shape and every
    group size in the table; else None.
    """
    path = os.path.join(ROOT, "profiles", "hbm_traffic__mixed8-4b-36L.json")
    try:
        summ = json.load(open(path))
        sha = kernel_source_sha()
    except OSError:
        return None
    if summ.get("kernel_source_sha256") != sha:
        return None
    shape = {"d_model": wl.d_model, "d_ff": wl.d_ff, "io": wl.io_dtype, "state": wl.state_dtype}
    if summ.get("read_shape") != shape:
        return None
    table = summ["read_call_bytes_by_group_size"]
    tot, calls = 0.0, 0
    for _, b, _, _, _, n in records:
        e = table.get(str(b))
        if e is None:
            return None
        tot += n * (e["fetch"] + e["write"])
        calls += n
    return tot / calls


class LaunchTimer:
    """HIP events around runs of launches of one kind.

    ``launch(kind, count, chunk, stream)`` is called before every library
    call; consecutive calls of the same kind, group size and chunk on one
    stream form one span between two events recorded on that stream, and
    ``close()`` ends the open spans.  An event pair per call would put a
    marker between every two kernels; a span per run of calls keeps the
    stream as the serving loop issues it.  The average call duration of a
    span is its elapsed time over its number of calls (inter-call gaps
    included, so the figure is conservative).
    """

    def __init__(self, torch, streams=()):
        self.torch = torch
        self.records = []            # (kind, count, chunk, start event, end event, calls)
        self._open = {}
        self._streams = {s.cuda_stream: s for s in streams}

    def launch(self, kind, count, chunk, stream):
        cur = self._open.get(stream)
        if cur is not None and cur[:3] == [kind, count, chunk]:
            cur[5] += 1
            return
        if cur is not None:
            self._close(stream)
        st = self._stream(stream)
        e = self.torch.cuda.Event(enable_timing=True)
        e.record(st)
        self._open[stream] = [kind, count, chunk, e, st, 1]

    def close(self):
        for stream in list(self._open):
            self._close(stream)

    def _close(self, stream):
        kind, count, chunk, e0, st, n = self._open.pop(stream)
        e1 = self.torch.cuda.Event(enable_timing=True)
        e1.record(st)
        self.records.append((kind, count, chunk, e0, e1, n))

    def _stream(self, handle):
        if handle in self._streams:
            return self._streams[handle]
        return self.torch.cuda.current_stream()

    def summary(self, wl, rank=0):
        """Per call kind: launches, HIP-event time, algorithmic bytes and flops.

        Algorithmic work follows the measurement plan: a READ of B owners moves
        W0 once, each live state once, x and y; a WRITE of one owner reads its
        live state, writes its shadow and reads Z and G, and does 2 C d_ff d_model
        flops.  A WRITE step's token adds its x and y; its second read of W0
        (and, where the token is not fused, of the live state) is reported as
        ``token_extra_bytes``, not counted.
        """
        K, N = wl.d_ff, wl.d_model
        io, st = wl.io_bytes, (4 if wl.state_dtype == "f32" else 2)
        out = {}
        for kind in ("read", "write", "write_token"):
            recs = [r for r in self.records if r[0] == kind]
            if not recs:
                continue
            ms = sum(s.elapsed_time(e) for _, _, _, s, e, _ in recs)
            calls = sum(n for *_, n in recs)
            extra = 0
            if rank:
                # adapter: W0 once, each owner's A and B, x and y; WRITE reads the live
                # factors, writes the shadow and reads Z and G
                tok = kind != "write"
                rb = sum(n * (K * N * io + b * (K + N) * (rank * st + io)) for _, b, _, _, _, n in recs)
                rf = sum(n * b * (2.0 * K * N + 2.0 * rank * (K + N)) for _, b, _, _, _, n in recs)
                wb = sum(n * b * (2 * (K + N) * rank * st + io * c * (K + N)) for _, b, c, _, _, n in recs)
                wf = sum(n * 4.0 * b * c * rank * (K + N) for _, b, c, _, _, n in recs)
                byt = (rb if tok else 0) + (wb if kind != "read" else 0)
                flop = (rf if tok else 0) + (wf if kind != "read" else 0)
            elif kind == "read":
                byt = sum(n * (K * N * (io + b * st) + b * io * (K + N)) for _, b, _, _, _, n in recs)
                flop = sum(n * 4.0 * b * K * N for _, b, _, _, _, n in recs)
            else:
                tok = kind == "write_token"
                byt = sum(n * b * (2 * st * K * N + io * c * (K + N) + (io * (K + N) if tok else 0))
                          for _, b, c, _, _, n in recs)
                flop = sum(n * 2.0 * b * c * K * N for _, b, c, _, _, n in recs)
                if tok:
                    extra = sum(n * (K * N * io + (0 if fused_token(wl, c) else b * st * K * N))
                                for _, b, c, _, _, n in recs)
            by_chunk = {}
            if kind != "read":
                for c in sorted({r[2] for r in recs}):
                    sub = [r for r in recs if r[2] == c]
                    cms = sum(s.elapsed_time(e) for _, _, _, s, e, _ in sub)
                    cn = sum(r[5] for r in sub)
                    by_chunk[c] = dict(launches=cn, avg_us=1e3 * cms / cn,
                                       owners=sum(r[1] * r[5] for r in sub) / cn)
            out[kind] = dict(launches=calls, total_ms=ms, avg_us=1e3 * ms / calls,
                             bytes=byt, flops=flop, records=recs, token_extra_bytes=extra,
                             by_chunk=by_chunk,
                             gbs=byt / (ms * 1e-3) / 1e9, tflops=flop / (ms * 1e-3) / 1e12)
        return out


def fused_token(wl, chunk):
    """Whether a WRITE with its token runs as one fused kernel (bf16 evidence, C <= 64)."""
    return wl.io_dtype == "bf16" and chunk <= 64


def write_kernel_name(wl, chunk, rank=0):
    if rank:
        return "adapter_pq_kernel+adapter_update_kernel"
    if wl.io_dtype != "bf16":
        return "write_valu_kernel"
    return "write_stream_kernel" if chunk <= 64 else "write_gemm_kernel"


def items_fn(wl):
    """t -> the step's StepItems; a finite trace is built once."""
    from rwttt_inputs import build_trace
    from rwttt_inputs.schedule import step_items
    if wl.schedule in ("staggered", "read_only"):
        return lambda t: step_items(wl, t)
    trace = build_trace(wl)
    return lambda t: trace[t]


def prepare(wl, layers, n_steps, threads, keep_layers, rank=0):
    """Device-resident state and inputs for steps [0, n_steps)."""
    import torch
    from rwttt_inputs import TensorSource, WRITE
    from paper_2605_28053_amd.serving import Session, to_device

    src = TensorSource(wl, cache_steps=False)
    backend = 1 if rank else 0
    sess = Session(wl, None, layers, init_state=False, init_w0=False, backend=backend, rank=rank)

    def init(j):
        if not rank:
            return src.dw_init(j[0], j[2])
        a, b = src.adapter_init(j[0], j[2], rank)
        return np.concatenate([a.reshape(-1), b.reshape(-1)])

    kept = {}
    with ThreadPoolExecutor(threads) as ex:
        for i, arr in enumerate(ex.map(src.w0, layers)):
            to_device(arr, wl.io_dtype, out=sess.w0[i])
        jobs = [(r, i, l) for r in range(wl.n_owners) for i, l in enumerate(layers)]
        for lo in range(0, len(jobs), 2 * threads):
            part = jobs[lo:lo + 2 * threads]
            for (r, i, l), arr in zip(part, ex.map(init, part)):
                to_device(arr, wl.state_dtype, out=sess.slots[r][i][0])
                if l in keep_layers:
                    kept[(r, l)] = arr
        log(f"state resident: {len(jobs)} slots of {sess.slots[0][0][0].numel() * sess.slots[0][0][0].element_size() / 1e6:.2f} MB")

        L, Rn = len(layers), wl.n_owners
        X = torch.empty((n_steps, L, Rn, wl.d_ff), dtype=torch.bfloat16, device="cuda")
        lidx = np.array(layers)

        def xs(t):
            return np.ascontiguousarray(src.x_step(t)[:, lidx].transpose(1, 0, 2))

        for t, arr in enumerate(ex.map(xs, range(n_steps))):
            to_device(arr, wl.io_dtype, out=X[t])
        items_at = items_fn(wl)
        writes = [(t, it.owner, it.chunk) for t in range(n_steps)
                  for it in items_at(t) if it.effect == WRITE]

        def zg(w):
            Z, G = src.zg_owner(*w)
            return Z[lidx], G[lidx]

        ZG = {}
        for (t, r, c), (Z, G) in zip(writes, ex.map(zg, writes)):
            zd, gd = to_device(Z, wl.io_dtype), to_device(G, wl.io_dtype)
            ZG[(t, r)] = (zd, gd, [zd[i].data_ptr() for i in range(L)],
                          [gd[i].data_ptr() for i in range(L)])
    Y = torch.empty((L, Rn, wl.d_model), dtype=torch.bfloat16, device="cuda")
    torch.cuda.synchronize()
    return sess, X, Y, ZG, kept


def run_gpu(args, wl, layers, warmup, steps, keep=()):
    """Run the workload's trace through the serving loop and time its windows.

    A periodic schedule (READ-only, staggered) runs ``warmup`` untimed steps,
    then one timed "decode" window of ``steps`` steps.  The ragged trace does
    the same on its first warmup + steps steps.  The prefill-then-decode trace
    runs once untimed, then again as two timed windows: "prefill" (the chunk
    WRITEs, which emit no token) and "decode" (the READ steps), so decode
    throughput never includes prefill time.  Each window is bracketed by
    torch.cuda.synchronize() and has its own HIP-event launch timer.
    """
    import torch

    if wl.schedule in ("staggered", "read_only", "ragged"):
        if wl.schedule == "ragged":
            steps = max(1, min(steps, wl.n_steps - warmup))
        n = warmup + steps
        warm = range(warmup)
        windows = [("decode", range(warmup, n))]
    else:
        n = wl.n_steps
        warm = range(n)
        windows = [("prefill", range(0, wl.n_prefill)), ("decode", range(wl.n_prefill, n))]
    t0 = time.time()
    sess, X, Y, ZG, kept = prepare(wl, layers, n, args.threads, set(keep), args.rank)
    log(f"{wl.name}: setup {time.time() - t0:.1f} s")
    from paper_2605_28053_amd.serving import StreamPair
    if args.streams == 2:
        pair = StreamPair()
        pair.wait_for_current()
        sp, tstreams = pair, (pair.read_stream, pair.write_stream)
    else:
        sp, tstreams = torch.cuda.current_stream().cuda_stream, ()
    y_ptrs = [Y[i].data_ptr() for i in range(len(layers))]

    items_at = items_fn(wl)

    def one(t, timer=None):
        items = items_at(t)
        x_ptrs = [X[t, i].data_ptr() for i in range(len(layers))]
        zg = {r: (ZG[(t, r)][2], ZG[(t, r)][3]) for r in [it.owner for it in items] if (t, r) in ZG}
        res = sess.step(t, items, x_ptrs, y_ptrs, zg, sp, timer=timer)
        return sum(1 for it in items if it.emit), res

    for t in warm:
        one(t)
    torch.cuda.synchronize()
    out = {}
    for label, rng in windows:
        timer = LaunchTimer(torch, tstreams) if args.kernel_events == "on" else None
        tokens = writes = 0
        torch.cuda.synchronize()
        t_start = time.perf_counter()
        for t in rng:
            k, res = one(t, timer)
            tokens += k
            writes += len(res.committed) + len(res.rolled_back)
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t_start
        out[label] = dict(tokens=tokens, elapsed=elapsed, writes=writes, steps=len(rng),
                          kernels=timer.summary(wl, args.rank) if timer is not None else {})
    versions = sess.versions()
    sess.close()
    return dict(windows=out, versions=versions, kept=kept, warmup=len(warm))


def host_info():
    """The host the oracle ran on: logical CPUs, CPU model and memory."""
    info = {"nproc": os.cpu_count()}
    try:
        # a virtualised host may name only the family: keep the family,
        # model and stepping numbers and the clock beside the name
        keys = {"model name": "cpu", "cpu family": "cpu_family", "model": "cpu_model",
                "stepping": "cpu_stepping", "cpu MHz": "cpu_mhz"}
        for line in open("/proc/cpuinfo"):
            k, _, v = line.partition(":")
            k = k.strip()
            if k in keys and keys[k] not in info:
                info[keys[k]] = v.strip()
            if not line.strip() and "cpu" in info:
                break
        for line in open("/proc/meminfo"):
            if line.startswith("MemTotal"):
                info["ram_gb"] = round(int(line.split()[1]) / 1024 ** 2, 1)
                break
    except OSError:
        pass
    return info


def run_cpu_baseline(args, wl, kept):
    """The oracle as it stands, on steps [0, S) of the same trace, a layer subset,
    with every BLAS thread the host gives it; then a shorter sample on one thread."""
    import oracle as O
    from rwttt_inputs import TensorSource, build_trace
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()
                            if i.get("user_api") == "blas"] or [1])
    except Exception:
        threadpool_limits = None
        blas_threads = os.cpu_count()
    layers = [l for l in args.cpu_layers if l < wl.n_layers] or [0]
    steps = range(min(args.cpu_steps, wl.n_steps))
    trace = build_trace(wl, len(steps))
    src = TensorSource(wl)

    def timed(steps, layers):
        table = None
        if not args.rank:
            table = O.OwnerTable(wl.n_owners, layers)
            for r in range(wl.n_owners):
                for l in layers:
                    arr = kept.get((r, l))
                    table.D[(r, l)] = O.widen(arr if arr is not None else src.dw_init(r, l),
                                              wl.state_dtype)
        for t in steps:                   # draw the inputs outside the timed window
            src.x_step(t)
        t0 = time.perf_counter()
        records, _ = O.run_trace(wl, trace, src, steps=steps, layers=layers, table=table,
                                 rank=args.rank)
        dt = time.perf_counter() - t0
        tokens = sum(len(rec.y) for rec in records) / len(layers)
        return tokens / (dt * wl.n_layers / len(layers)), dt

    value, dt = timed(steps, layers)
    out = dict(value=value, unit="tok/s", cores=int(blas_threads), kind="oracle",
               sample=(f"float64 numpy oracle on decode steps 0-{len(steps) - 1} of the same "
                       f"trace, layers {layers} of {wl.n_layers}, all {wl.n_owners} owners; "
                       f"{dt:.2f} s measured, scaled x{wl.n_layers / len(layers):g} to all layers"))
    out["host"] = host_info()
    if threadpool_limits is not None:
        steps1 = range(min(len(steps), 30))
        with threadpool_limits(limits=1):
            v1, dt1 = timed(steps1, layers[:1])
        out["single_thread"] = dict(value=v1, unit="tok/s", cores=1,
                                    sample=f"decode steps 0-{len(steps1) - 1}, layer {layers[0]}; "
                                           f"{dt1:.2f} s measured")
    return out


def time_library_write(torch, wl, wr, calls=20):
    """The same update as the commonest WRITE call, shadow = live + eta * Z^T G, as one
    torch.baddbmm over the call's owners (bf16 operands and state, fp32 accumulate in
    the library), on fresh seeded tensors of the workload's distributions.  Context
    for the WRITE kernel's figure only: no step of the measured path runs here."""
    if wl.state_dtype != "bf16":
        return {"skipped": "the library update needs one dtype for state and operands; "
                           f"this workload's state is {wl.state_dtype}"}
    counts = {}
    for _, b, c, _, _, n in wr["records"]:
        counts[(b, c)] = counts.get((b, c), 0) + n
    (b, c), _ = max(counts.items(), key=lambda kv: kv[1])
    K, N = wl.d_ff, wl.d_model
    gen = torch.Generator(device="cuda").manual_seed(0)
    bf = torch.bfloat16
    zt = torch.randn(b, c, K, device="cuda", dtype=bf, generator=gen).abs_().transpose(1, 2).contiguous()
    g = torch.randn(b, c, N, device="cuda", dtype=bf, generator=gen)
    live = torch.randn(b, K, N, device="cuda", dtype=bf, generator=gen).mul_(0.02)
    out = torch.empty_like(live)
    for _ in range(3):
        torch.baddbmm(live, zt, g, alpha=wl.eta, out=out)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(calls):
        torch.baddbmm(live, zt, g, alpha=wl.eta, out=out)
    e1.record()
    torch.cuda.synchronize()
    us = 1e3 * e0.elapsed_time(e1) / calls
    # the bare product with a bf16 result: no live term, the same bytes written
    for _ in range(3):
        torch.bmm(zt, g, out=out)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(calls):
        torch.bmm(zt, g, out=out)
    e1.record()
    torch.cuda.synchronize()
    us_bmm = 1e3 * e0.elapsed_time(e1) / calls
    flop = 2.0 * b * c * K * N
    return {"op": "torch.baddbmm(live, Z^T, G, alpha=eta), bf16, out of place",
            "owners": b, "chunk": c, "calls": calls, "avg_us": round(us, 2),
            "tflops": round(flop / us / 1e6, 1),
            "mfma_frac": round(flop / us / 1e6 / BF16_MFMA_PEAK_TFLOPS, 4),
            "bmm_without_live_avg_us": round(us_bmm, 2),
            "this_write_avg_us": round(wr["avg_us"], 2)}


def pmc_summary(dirs):
    """Per-dispatch HBM bytes of the READ and fused-WRITE calls from rocprofv3 PMC
    databases, as the table measured_traffic() reads.  `dirs` holds the
    directories of four runs: the plain 1 GiB copy and the bench, each once with
    FETCH_SIZE and once with WRITE_SIZE (see profiles/hbm_traffic__mixed8-4b-36L.md).
    Each counter is scaled by what it reads for the copy of known size."""
    import glob
    import re
    import sqlite3
    from collections import defaultdict
    from rwttt_inputs import workload

    def rows(d):
        (db,) = glob.glob(os.path.join(d, "*_results.db"))
        q = ("select p.name, p.counter_value, k.grid_x, k.grid_y from pmc_events p "
             "join kernels k on k.dispatch_id = p.dispatch_id")
        return sqlite3.connect(db).execute(q).fetchall()

    scale, per = {}, {}
    for cn in ("FETCH_SIZE", "WRITE_SIZE"):
        copy = [v for n, v, _, _ in rows(dirs[f"copy_{cn}"]) if "copy" in n.lower()]
        scale[cn] = (1 << 30) / (max(copy) * 1024.0)
        agg = defaultdict(list)
        for n, v, gx, gy in rows(dirs[f"bench_{cn}"]):
            m = re.search(r"(\w+_kernel)\b", n)
            agg[(m.group(1) if m else n, gx, gy)].append(v * 1024.0 * scale[cn])
        per[cn] = agg
    wl = workload(2)
    pairs = ((wl.d_ff + 255) // 256) * ((wl.d_model + 255) // 256)
    pairs8 = (pairs + 7) // 8 * 8
    # a READ call of B owners = one read_partial_kernel launch (grid of B slots)
    # + one read_reduce_kernel launch (grid_y = B); a reduce of grid_y 1 with no
    # READ partner is the fused WRITE token's
    table = {}
    for cn in per:
        for (name, gx, gy), vs in per[cn].items():
            if name == "read_partial_kernel":
                e = table.setdefault(str(gx // 256 // pairs8), {"fetch": 0.0, "write": 0.0})
                e["fetch" if cn == "FETCH_SIZE" else "write"] += sum(vs) / len(vs)
    for cn in per:
        for (name, gx, gy), vs in per[cn].items():
            if name == "read_reduce_kernel" and str(gy) in table:
                table[str(gy)]["fetch" if cn == "FETCH_SIZE" else "write"] += sum(vs) / len(vs)
    wr = {cn: [sum(vs) / len(vs) for (name, _, _), vs in per[cn].items()
               if name == "write_stream_kernel"] for cn in per}
    return {"kernel_source_sha256": kernel_source_sha(), "workload": wl.name,
            "read_shape": {"d_model": wl.d_model, "d_ff": wl.d_ff, "io": wl.io_dtype,
                           "state": wl.state_dtype},
            "calibration": {"copy_bytes": 1 << 30, "fetch_scale": scale["FETCH_SIZE"],
                            "write_scale": scale["WRITE_SIZE"]},
            "read_call_bytes_by_group_size": table,
            "write_call_bytes": {"fetch": max(wr["FETCH_SIZE"]), "write": max(wr["WRITE_SIZE"])}}


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=260)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--layers", type=int, default=None, help="fast-weight layers (default 36)")
    ap.add_argument("--threads", type=int, default=16, help="host threads for input generation")
    ap.add_argument("--cpu-baseline", choices=["on", "off"], default=None,
                    help="time the oracle on a sample of the workload (default: on for workload 2)")
    ap.add_argument("--cpu-steps", type=int, default=100)
    ap.add_argument("--cpu-layers", type=int, nargs="+", default=[0, 1])
    ap.add_argument("--kernel-events", choices=["on", "off"], default="on")
    ap.add_argument("--streams", type=int, choices=[1, 2], default=1,
                    help="2: READ and WRITE groups on two streams, joined every step")
    ap.add_argument("--workload", type=int, choices=[1, 2, 3, 4], default=2,
                    help="2 (default): mixed8-4b-36L; 1 read8-4b; 3 ragged32-4b; 4 prefill8-8b")
    ap.add_argument("--rank", type=int, default=0,
                    help="0: fast-weight state (default); r > 0: the rank-r adapter backend")
    ap.add_argument("--sub-workloads", choices=["on", "off"], default=None,
                    help="also measure a few steps of workloads 1, 3 and 4 as compact records "
                         "in the same line (default: on for workload 2)")
    ap.add_argument("--library-write", choices=["on", "off"], default="off",
                    help="also time torch.baddbmm (the vendor GEMM library) on the same "
                         "update as one WRITE call, for a bf16 state (context, not the value)")
    ap.add_argument("--pmc-summary", metavar="DIR",
                    help="only summarise the PMC runs under DIR (pmc_copy_FETCH_SIZE, "
                         "pmc_bench_FETCH_SIZE, ... subdirectories) into the traffic table JSON")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="BYTES",
                    help="only run 5 plain device copies of BYTES each (HBM counter calibration)")
    args = ap.parse_args()

    if args.pmc_summary:
        dirs = {f"{k}_{cn}": os.path.join(args.pmc_summary, f"pmc_{k}_{cn}")
                for k in ("copy", "bench") for cn in ("FETCH_SIZE", "WRITE_SIZE")}
        print(json.dumps(pmc_summary(dirs), indent=1))
        return

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path "
              "(owners would shard across GPUs with no exchange); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    if args.calibrate_copy:
        # A plain copy of known size: reads and writes exactly BYTES per launch.
        a = torch.ones(args.calibrate_copy // 4, dtype=torch.float32, device="cuda")
        b = torch.empty_like(a)
        for _ in range(5):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": args.calibrate_copy, "launches": 5}))
        return
    from rwttt_inputs import workload
    if args.cpu_baseline is None:
        args.cpu_baseline = "on" if args.workload == 2 else "off"
    if args.sub_workloads is None:
        args.sub_workloads = "on" if args.workload == 2 and not args.rank else "off"
    wl = workload(args.workload)
    layers = list(range(wl.n_layers if args.layers is None else args.layers))

    g = run_gpu(args, wl, layers, args.warmup, args.steps,
                keep=args.cpu_layers if args.cpu_baseline == "on" else ())
    dec = g["windows"]["decode"]
    tok_s = dec["tokens"] / dec["elapsed"]
    kern = dec["kernels"]
    line = {
        "metric": METRIC,
        "value": round(tok_s, 2),
        "unit": "tok/s",
        "n_gpus": 1,
        "steps": dec["steps"],
        "warmup": g["warmup"],
        "ms_per_step": round(1e3 * dec["elapsed"] / dec["steps"], 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": f"{wl.name}: {wl.n_owners} streams, {len(layers)} fast-weight layers, "
                        f"d_model {wl.d_model}, d_ff {wl.d_ff}, {wl.io_dtype} io, "
                        f"{wl.state_dtype} state"
                        + (f" as rank-{args.rank} adapters (A, B)" if args.rank else "")
                        + f"; {wl.description}",
            "backend": f"delta_adapter rank {args.rank}" if args.rank else "fast_weight",
            "owners": wl.n_owners, "layers": len(layers), "d_model": wl.d_model, "d_ff": wl.d_ff,
            "io": wl.io_dtype, "state": wl.state_dtype, "accumulate": "f32",
            "write_chunk": wl.chunk or list(wl.chunk_choices),
            "tokens_timed": dec["tokens"], "writes_timed": dec["writes"],
            "parallelism": "single-gpu",
            "streams": args.streams,
        },
    }
    if "read" in kern:
        rd = kern["read"]
        traffic = None if args.rank else measured_traffic(rd["records"], wl)
        line["roofline"] = {"bound": "hbm",
                            "kernel": ("adapter_read_partial_kernel+adapter_read_reduce_kernel"
                                       if args.rank else "read_partial_kernel+read_reduce_kernel"),
                            "achieved": round(rd["gbs"], 1), "peak": HBM_PEAK_GBS,
                            "unit": "GB/s", "frac": round(rd["gbs"] / HBM_PEAK_GBS, 4),
                            "traffic": None if traffic is None else round(traffic),
                            "algorithmic_bytes_per_launch": round(rd["bytes"] / rd["launches"]),
                            "avg_launch_us": round(rd["avg_us"], 2),
                            "launches": rd["launches"]}
    wk = write_record(wl, kern, args.rank)
    if wk:
        line["write_kernel"] = wk
    if "prefill" in g["windows"]:
        line["prefill"] = prefill_record(wl, g["windows"]["prefill"], args.rank)
    wkind = "write_token" if "write_token" in kern else "write"
    if args.library_write == "on":
        pk = g["windows"].get("prefill", dec)["kernels"]
        pkind = "write" if "write" in pk else "write_token"
        if pkind in pk:
            line["library_write"] = time_library_write(torch, wl, pk[pkind])
    if args.cpu_baseline == "on":
        line["cpu_baseline"] = run_cpu_baseline(args, wl, g["kept"])
    del g
    if args.sub_workloads == "on":
        line["workloads"] = {}
        for wid, warm, steps in ((1, 3, 20), (3, 8, 40), (4, 0, 0)):
            torch.cuda.empty_cache()
            line["workloads"][workload(wid).name] = sub_record(args, workload(wid), warm, steps)
    line["paper_context"] = ("274.61 tok/s, 9.31x over sequential serving: full Qwen3-4B "
                             "In-Place-TTT model, 8 streams, one unnamed GPU (not this metric)")
    print(json.dumps(line), flush=True)


def write_record(wl, kern, rank=0):
    """The WRITE calls of a window: HBM fraction on algorithmic bytes (live read,
    shadow write, Z, G, and a token's x and y), MFMA fraction on the update's
    flops, and the token's second W0 read (plus its live read where not fused)
    reported beside them."""
    wkind = "write_token" if "write_token" in kern else "write"
    if wkind not in kern:
        return None
    wr = kern[wkind]
    chunks = sorted(wr["by_chunk"])
    names = sorted({write_kernel_name(wl, c, rank) for c in chunks})
    if wkind == "write_token" and not rank:
        names.append("read_reduce_kernel (token)" if all(fused_token(wl, c) for c in chunks)
                     else "READ launch (token)")
    return {"kernel": "+".join(names),
            "achieved_gbs": round(wr["gbs"], 1),
            "hbm_frac": round(wr["gbs"] / HBM_PEAK_GBS, 4),
            "achieved_tflops": round(wr["tflops"], 2),
            "mfma_frac": round(wr["tflops"] / BF16_MFMA_PEAK_TFLOPS, 5),
            "algorithmic_bytes_per_launch": round(wr["bytes"] / wr["launches"]),
            "token_extra_bytes_per_launch": round(wr["token_extra_bytes"] / wr["launches"]),
            "avg_launch_us": round(wr["avg_us"], 2), "launches": wr["launches"],
            "by_chunk": {str(c): {"launches": v["launches"], "avg_us": round(v["avg_us"], 2),
                                  "owners": round(v["owners"], 2)}
                         for c, v in wr["by_chunk"].items()}}


def prefill_record(wl, win, rank=0):
    """The prefill window of a prefill-then-decode trace: chunk WRITEs with no token."""
    rec = {"ms": round(1e3 * win["elapsed"], 3), "steps": win["steps"], "writes": win["writes"]}
    wk = write_record(wl, win["kernels"], rank)
    if wk:
        rec["write_kernel"] = wk
    return rec


def sub_record(args, wl, warmup, steps):
    """A compact record of one more workload: decode tok/s, READ and WRITE
    fractions, and the prefill window where the workload has one."""
    g = run_gpu(args, wl, list(range(wl.n_layers)), warmup, steps)
    dec = g["windows"]["decode"]
    rec = {"tok_s": round(dec["tokens"] / dec["elapsed"], 1), "steps": dec["steps"],
           "warmup": g["warmup"], "tokens": dec["tokens"],
           "ms_per_step": round(1e3 * dec["elapsed"] / dec["steps"], 4)}
    kern = dec["kernels"]
    if "read" in kern:
        rd = kern["read"]
        rec["read"] = {"frac": round(rd["gbs"] / HBM_PEAK_GBS, 4), "avg_us": round(rd["avg_us"], 2),
                       "launches": rd["launches"],
                       "owners": round(sum(r[1] * r[5] for r in rd["records"]) / rd["launches"], 2)}
    wk = write_record(wl, kern, args.rank)
    if wk:
        rec["write"] = {k: wk[k] for k in ("kernel", "hbm_frac", "mfma_frac", "avg_launch_us",
                                            "launches", "by_chunk")}
    if "prefill" in g["windows"]:
        pr = prefill_record(wl, g["windows"]["prefill"], args.rank)
        rec["prefill"] = {"ms": pr["ms"], "writes": pr["writes"]}
        if "write_kernel" in pr:
            rec["prefill"].update({k: pr["write_kernel"][k] for k in
                                   ("kernel", "mfma_frac", "hbm_frac", "avg_launch_us", "launches")})
    return rec


if __name__ == "__main__":
    main()
