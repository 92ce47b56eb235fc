"""Bounded-wait scheduling simulator over the library's planner.

The planner (``rwttt_plan``) decides, at every decode step, which ready
transitions are issued together and which wait (Section 3, eqs. compatibility
and wait-budget; Section 4.3).  A wait budget ``w`` lets a partial group wait up
to ``w`` steps for compatible partners: denser groups, fewer launches, at the
cost of latency.  This module replays request traces through the real C
planner, charges every issued group the GPU time measured for the library's
own kernels at that group size (a ``ServiceModel``), and reports throughput,
decode-ready-to-first-token and completion latencies, and every contract
violation it can check (the shape of the paper's wait-budget sweep, Appendix
B, and its dynamic-traffic study, Section 5.3).

Trace kinds (one decode stream per request, fixed prefill):
  uniform        all streams ready at t = 0, update boundaries aligned;
  phase_skew     streams out of phase: stream s becomes decode-ready one
                 full-batch decode step after stream s - 1 (its fixed prefill
                 ends later), update boundaries counted from each stream's
                 own decode start, so unless the start-up skew is absorbed by
                 waiting the streams reach their boundaries on different steps;
  poisson        decode-ready times from a Poisson process, boundaries aligned
                 to each stream's own start;
  heterogeneous  ready at t = 0, decode lengths drawn from [n/4, 2n].

Time model: every decode step takes time, issued or not.  A step that issues
groups costs their measured service times (plus a fixed per-step overhead);
a step in which every ready event is deferred by the wait budget still costs
one idle tick, by default a full-batch decode step (a READ group of the target
size B, or of every stream when B = 0, through every layer): the loop's
cadence, so that waiting is paid for in latency.

A request's i-th decode token (1-based, counted from its chunk phase) is a
WRITE step when (phase + i) is a multiple of the chunk size C, else a READ.
Versions: each issued WRITE commits (no injected failures here), so an owner's
version after the trace is its number of boundaries.

CLI (GPU needed for ``calibrate`` only):
  python -m paper_2605_28053_amd.scheduler_sim calibrate --out FILE
  python -m paper_2605_28053_amd.scheduler_sim sweep --model FILE [--kind phase_skew]
"""

import argparse
import json
import math
from dataclasses import dataclass, field

import numpy as np

from . import _rwttt as R

READ, WRITE = R.RWTTT_READ, R.RWTTT_WRITE


# ---------------------------------------------------------------------------
# Service times
# ---------------------------------------------------------------------------

@dataclass
class ServiceModel:
    """GPU time of one group launch per layer, in microseconds.

    read_us[B-1]: one READ call for a group of B owners; write_us[C][B-1]: one
    WRITE call (update plus the step's token) for B owners at chunk C.  Group
    sizes beyond the table extend the last two points linearly; a chunk not in
    the table uses the next larger one.
    """
    layers: int
    read_us: list
    write_us: dict
    step_overhead_us: float = 0.0
    source: str = ""
    idle_step_us: float = None      # a step with nothing issued; None: a full-batch READ step

    @staticmethod
    def _at(table, b):
        if b <= len(table):
            return float(table[b - 1])
        if len(table) == 1:
            return float(table[0]) * b
        slope = table[-1] - table[-2]
        return float(table[-1] + slope * (b - len(table)))

    def read(self, b):
        return self._at(self.read_us, b)

    def write(self, b, chunk):
        keys = sorted(int(c) for c in self.write_us)
        c = next((k for k in keys if k >= chunk), keys[-1])
        return self._at(self.write_us[c], b)

    def group_us(self, effect, b, chunk):
        per_layer = self.read(b) if effect == READ else self.write(b, chunk)
        return self.layers * per_layer

    def tick_us(self, batch):
        """Time of a decode step in which every ready event waits: the fixed
        idle step if set, else one READ step of ``batch`` owners."""
        if self.idle_step_us is not None:
            return float(self.idle_step_us)
        return self.step_overhead_us + self.group_us(READ, batch, 0)

    def to_json(self, path):
        json.dump({"layers": self.layers, "read_us": self.read_us,
                   "write_us": {str(k): v for k, v in self.write_us.items()},
                   "step_overhead_us": self.step_overhead_us, "source": self.source,
                   "idle_step_us": self.idle_step_us},
                  open(path, "w"), indent=1)

    @classmethod
    def from_json(cls, path):
        d = json.load(open(path))
        return cls(d["layers"], d["read_us"], {int(k): v for k, v in d["write_us"].items()},
                   d.get("step_overhead_us", 0.0), d.get("source", ""), d.get("idle_step_us"))


# ---------------------------------------------------------------------------
# Traces
# ---------------------------------------------------------------------------

@dataclass
class Request:
    rid: int
    ready_s: float          # decode-ready time (prefill done)
    n_tokens: int           # decode tokens to generate
    phase: int              # tokens of the current chunk already seen at decode start


def make_requests(kind, n_streams=8, n_tokens=512, chunk=128, seed=0, mean_gap_ms=50.0,
                  step_s=0.0):
    """``step_s``: one full-batch decode step in seconds, the phase-skew
    trace's spacing of decode-ready times."""
    rng = np.random.default_rng(seed)
    reqs = []
    t = 0.0
    for s in range(n_streams):
        ready, n, phase = 0.0, n_tokens, 0
        if kind == "phase_skew":
            ready = s * step_s
        elif kind == "poisson":
            if s:
                t += float(rng.exponential(mean_gap_ms * 1e-3))
            ready = t
        elif kind == "heterogeneous":
            n = int(rng.integers(max(1, n_tokens // 4), 2 * n_tokens + 1))
        elif kind != "uniform":
            raise ValueError(kind)
        reqs.append(Request(s, ready, n, phase))
    return reqs


# ---------------------------------------------------------------------------
# Simulation
# ---------------------------------------------------------------------------

@dataclass
class SimResult:
    tok_s: float
    first_token_p95_ms: float
    completion_p95_s: float
    violations: int
    steps: int
    launches: int
    mean_group: dict = field(default_factory=dict)
    max_wait_steps: int = 0
    makespan_s: float = 0.0


def _shape(effect, chunk):
    # sigma: the chunk size separates WRITE shapes; all READs share one shape
    return (chunk << 1) | 1 if effect == WRITE else 0


def decode_tick_us(model, B, n_streams):
    """The idle-step tick of a run with target group size B over n streams."""
    return model.tick_us(B if B > 0 else n_streams)


def simulate(reqs, model, chunk=128, B=0, w=0, max_steps=1_000_000):
    """Replay requests through rwttt_plan with target group size B and wait budget w."""
    n = len(reqs)
    tick = decode_tick_us(model, B, n)
    fake = [0x1000 * (i + 1) for i in range(2 * n + 1)]
    cfg = R.make_config(n, 1, 8, 8, R.RWTTT_BF16, R.RWTTT_F32, min(n, R.RWTTT_MAX_GROUP),
                        fake[:1], fake[1:])          # host-only context: planning only
    ctx = R.rwttt_create(cfg)
    try:
        produced = [0] * n
        ready_step = [None] * n
        version = [0] * n
        first_tok, done_at = [None] * n, [None] * n
        writes = [0] * n
        clock, step, launches, violations, max_wait = 0.0, 0, 0, 0, 0
        sizes = {READ: [], WRITE: []}
        while step < max_steps:
            live = [r for r in range(n) if produced[r] < reqs[r].n_tokens]
            if not live:
                break
            active = [r for r in live if reqs[r].ready_s <= clock + 1e-12]
            if not active:
                clock = min(reqs[r].ready_s for r in live)
                continue
            events = []
            for r in active:
                if ready_step[r] is None:
                    ready_step[r] = step
                eff = WRITE if (reqs[r].phase + produced[r] + 1) % chunk == 0 else READ
                v, _ = R.rwttt_version(ctx, r)      # the context's V(r): planning only
                events.append((r, 0, _shape(eff, chunk), 0, eff, v, ready_step[r]))
            plan = R.rwttt_plan(ctx, events, step, B, w)
            if plan.status != R.RWTTT_OK:
                raise R.RwtttError(plan.status, "rwttt_plan")
            issued = []
            # a step in which everything waits still takes one decode-step tick
            t_step = model.step_overhead_us if plan.n_groups else tick
            for gi in range(plan.n_groups):
                g = plan.group(gi)
                owners = plan.owners(gi)
                effs = {events[active.index(r)][4] for r in owners}
                if len(effs) != 1 or len(set(owners)) != len(owners) or g.effect not in effs:
                    violations += 1                  # mixed keys or a repeated owner
                t_step += model.group_us(g.effect, g.count, chunk)
                launches += model.layers
                sizes[g.effect].append(g.count)
                issued += [(r, g.effect) for r in owners]
            clock += t_step * 1e-6
            for r, eff in issued:
                wait = step - ready_step[r]
                max_wait = max(max_wait, wait)
                if wait < 0 or (w > 0 and wait > w) or (w == 0 and wait != 0):
                    violations += 1                  # eq. wait-budget
                produced[r] += 1
                if eff == WRITE:
                    version[r] += 1
                    writes[r] += 1
                if first_tok[r] is None:
                    first_tok[r] = clock - reqs[r].ready_s
                if produced[r] == reqs[r].n_tokens:
                    done_at[r] = clock - reqs[r].ready_s
                ready_step[r] = step + 1
            step += 1
        for r in range(n):
            q = reqs[r]
            expect = (q.phase + q.n_tokens) // chunk - q.phase // chunk
            if done_at[r] is None or writes[r] != expect or version[r] != expect:
                violations += 1                      # starvation or a lost/extra update
        total = sum(q.n_tokens for q in reqs)
        makespan = max(done_at[r] + reqs[r].ready_s for r in range(n) if done_at[r] is not None)
        return SimResult(
            tok_s=total / makespan if makespan > 0 else float("inf"),
            first_token_p95_ms=1e3 * float(np.percentile([x for x in first_tok if x is not None], 95)),
            completion_p95_s=float(np.percentile([x for x in done_at if x is not None], 95)),
            violations=violations, steps=step, launches=launches,
            mean_group={("READ" if k == READ else "WRITE"): (float(np.mean(v)) if v else 0.0)
                        for k, v in sizes.items()},
            max_wait_steps=max_wait, makespan_s=makespan)
    finally:
        R.rwttt_destroy(ctx)


def sweep(model, kind="phase_skew", waits=(0, 1, 2, 4, 8, 16), seeds=range(5), n_streams=8,
          n_tokens=512, chunk=128, B=None):
    """Average simulate() over seeds for each wait budget; B defaults to n_streams."""
    B = n_streams if B is None else B
    rows = []
    for w in waits:
        step_s = 1e-6 * decode_tick_us(model, B, n_streams)
        res = [simulate(make_requests(kind, n_streams, n_tokens, chunk, seed, step_s=step_s),
                        model, chunk, B, w)
               for seed in seeds]
        rows.append(dict(w=w, tok_s=float(np.mean([r.tok_s for r in res])),
                         first_token_p95_ms=float(np.mean([r.first_token_p95_ms for r in res])),
                         completion_p95_s=float(np.mean([r.completion_p95_s for r in res])),
                         violations=int(sum(r.violations for r in res)),
                         launches=float(np.mean([r.launches for r in res])),
                         mean_read_group=float(np.mean([r.mean_group["READ"] for r in res])),
                         mean_write_group=float(np.mean([r.mean_group["WRITE"] for r in res])),
                         max_wait_steps=max(r.max_wait_steps for r in res)))
    return rows


# ---------------------------------------------------------------------------
# Calibration on the GPU: per-layer call times of the library's kernels
# ---------------------------------------------------------------------------

def calibrate(layers=36, max_b=8, chunks=(64, 128), reps=20, d_ff=9728, d_model=2560):
    """Time rwttt_read and rwttt_write (with its token) for B = 1..max_b owners at
    the 4B-class shape (bf16 io, fp32 state, one layer, HIP events)."""
    import dataclasses
    import torch
    from rwttt_inputs import workload
    from .serving import Session

    wl = dataclasses.replace(workload(1), n_owners=max_b, n_layers=1, d_ff=d_ff, d_model=d_model)
    sess = Session(wl, None, init_state=False, init_w0=False)
    for r in range(max_b):
        for s in range(2):
            sess.slots[r][0][s].normal_(0.0, math.sqrt(1e-3))
    sess.w0[0].normal_(0.0, 1.0 / math.sqrt(d_ff))
    x = torch.randn((max_b, d_ff), device="cuda").to(torch.bfloat16)
    y = torch.empty((max_b, d_model), dtype=torch.bfloat16, device="cuda")
    stream = torch.cuda.current_stream()

    def timed(fn):
        for _ in range(3):
            fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            fn()
        e1.record(stream)
        e1.synchronize()
        return 1e3 * e0.elapsed_time(e1) / reps

    read_us, write_us = [], {c: [] for c in chunks}
    for b in range(1, max_b + 1):
        owners = list(range(b))
        g = R.make_group(READ, 0, b)
        om = R.u32_array(owners)
        def rd():
            st = R.rwttt_read(sess.ctx, g, om, 0, x.data_ptr(), y.data_ptr(), stream.cuda_stream)
            if st != R.RWTTT_OK:
                raise R.RwtttError(st, f"rwttt_read (hip {R.rwttt_last_hip_error(sess.ctx)})")
        read_us.append(timed(rd))
        for c in chunks:
            Z = torch.rand((b, c, d_ff), device="cuda").to(torch.bfloat16)
            G = torch.randn((b, c, d_model), device="cuda").to(torch.bfloat16)
            wg = R.make_group(WRITE, 0, b)

            def one():
                st = R.rwttt_write(sess.ctx, wg, om, 0, c, [Z[i].data_ptr() for i in range(b)],
                                   [G[i].data_ptr() for i in range(b)], 1e-3, x.data_ptr(),
                                   y.data_ptr(), stream=stream.cuda_stream)
                if st != R.RWTTT_OK:
                    raise R.RwtttError(st, f"rwttt_write (hip {R.rwttt_last_hip_error(sess.ctx)})")
                R.rwttt_rollback(sess.ctx, owners)   # keep the owners writable
            write_us[c].append(timed(one))
    torch.cuda.synchronize()
    sess.close()
    name = torch.cuda.get_device_properties(0).gcnArchName
    return ServiceModel(layers, read_us, write_us, 0.0,
                        source=f"rwttt_read / rwttt_write(+token) per layer on {name}, "
                               f"d_ff {d_ff}, d_model {d_model}, bf16 io, fp32 state, "
                               f"HIP events over {reps} calls")


def main():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    sub = ap.add_subparsers(dest="cmd", required=True)
    c = sub.add_parser("calibrate")
    c.add_argument("--out", required=True)
    c.add_argument("--layers", type=int, default=36)
    s = sub.add_parser("sweep")
    s.add_argument("--model", required=True)
    s.add_argument("--kind", default="phase_skew")
    s.add_argument("--waits", type=int, nargs="+", default=[0, 1, 2, 4, 8, 16])
    s.add_argument("--chunk", type=int, default=128)
    s.add_argument("--tokens", type=int, default=512)
    s.add_argument("--B", type=int, default=None)
    a = ap.parse_args()
    if a.cmd == "calibrate":
        m = calibrate(layers=a.layers)
        m.to_json(a.out)
        print(json.dumps({"read_us": m.read_us, "write_us": m.write_us}))
    else:
        m = ServiceModel.from_json(a.model)
        for row in sweep(m, a.kind, a.waits, chunk=a.chunk, n_tokens=a.tokens, B=a.B):
            print(json.dumps(row))


if __name__ == "__main__":
    main()
