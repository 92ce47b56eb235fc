"""Host-side checks of the C ABI that need no GPU.

The library loads on a machine without a GPU; planning, the owner table and
every validation path run on the host.  A context without workspace never
touches the device, and the fake slot addresses below are never dereferenced.
"""

import os
import random
import re
import subprocess
import sys

import pytest

import oracle as O

R = pytest.importorskip("paper_2605_28053_amd._rwttt",
                        reason="librwttt.so not built (python -m paper_2605_28053_amd.build)")

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "rwttt.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(rwttt_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = declared_functions()
    assert len(names) == 21
    out = subprocess.run(["nm", "-D", "--defined-only", R.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (rwttt_\w+)", out))
    for n in names:
        assert n in exported, n
        assert hasattr(R.lib(), n)


def host_ctx(n_owners=6, n_layers=2, d_ff=64, d_model=32, max_group=8):
    w0 = [0x10000 * (i + 1) for i in range(n_layers)]
    slots = [0x1000000 + 0x1000 * i for i in range(n_owners * n_layers * 2)]
    cfg = R.make_config(n_owners, n_layers, d_ff, d_model, R.RWTTT_BF16, R.RWTTT_F32,
                        max_group, w0, slots)
    return R.rwttt_create(cfg), cfg


def make_dirty(ctx, owners, layer=0):
    """Open a (failed) candidate for owners without touching the device."""
    g = R.make_group(R.RWTTT_WRITE, 0, len(owners))
    assert R.rwttt_inject_write_failures(ctx, 1) == R.RWTTT_OK
    st = R.rwttt_write(ctx, g, R.u32_array(owners), layer, 4, [0x100] * len(owners),
                       [0x200] * len(owners), 1.0)
    assert st == R.RWTTT_E_WRITE_FAILED


def test_plan_matches_oracle_planner_bit_exactly():
    rng = random.Random(11)
    for trial in range(400):
        n_owners = rng.randint(1, 12)
        ctx, _ = host_ctx(n_owners=n_owners)
        dirty = [rng.random() < 0.2 for _ in range(n_owners)]
        d_owners = [r for r in range(n_owners) if dirty[r]]
        if d_owners:
            make_dirty(ctx, d_owners)
        step = rng.randint(0, 6)
        B = rng.choice([0, 0, 1, 2, 3, 5])
        w = rng.choice([0, 0, 1, 2, 4])
        owners = rng.sample(range(n_owners + 2), rng.randint(0, n_owners))
        events = []
        for r in owners:
            events.append((r, rng.choice([0, 1]), rng.choice([0, 3, 9]), rng.choice([0, 1]),
                           rng.choice([0, 1, 1, 1, 2]), rng.choice([0, 0, 0, 1]),
                           rng.randint(0, step + 1)))
        if owners and rng.random() < 0.05:
            events.append(events[0])          # alias
        p = R.rwttt_plan(ctx, events, step, B, w)
        oe = [O.Event(r, tau, sig, pi, eff, v, rd) for (r, tau, sig, pi, eff, v, rd) in events]
        q = O.plan(oe, [0] * n_owners, dirty, n_owners, step, B, w)
        assert p.status == q.status
        assert p.ev_status == q.ev_status
        if q.status == O.OK:
            got = [((p.group(i).effect, p.group(i).backend_type, p.group(i).shape_class,
                     p.group(i).placement), p.owners(i)) for i in range(p.n_groups)]
            assert got == [(g.key, g.owners) for g in q.groups]
            assert p.deferred == q.deferred
        R.rwttt_destroy(ctx)


def test_plan_capacity_reports_needed_sizes():
    ctx, _ = host_ctx()
    events = [(r, 0, 0, 0, r % 2, 0, 0) for r in range(6)]
    p = R.rwttt_plan(ctx, events, 0, cap=1)
    assert p.status == R.RWTTT_E_CAPACITY
    assert (p.n_groups, p.n_mapped) == (2, 6)
    p = R.rwttt_plan(ctx, events, 0)
    assert p.status == R.RWTTT_OK and [p.owners(i) for i in range(2)] == [[0, 2, 4], [1, 3, 5]]


def test_owner_table_state_machine_and_error_codes():
    ctx, _ = host_ctx(n_owners=4)
    # commit / rollback of a clean owner
    assert R.rwttt_commit(ctx, [0]) == R.RWTTT_E_NOT_DIRTY
    assert R.rwttt_rollback(ctx, [0]) == R.RWTTT_E_NOT_DIRTY
    assert R.rwttt_commit(ctx, [9]) == R.RWTTT_E_INVALID
    # a WRITE needs a WRITE group
    rg = R.make_group(R.RWTTT_READ, 0, 1)
    assert R.rwttt_write(ctx, rg, R.u32_array([1]), 0, 4, [0x100], [0x200], 1.0) == R.RWTTT_E_KEY_MISMATCH
    # failed WRITE: dirty, cannot commit, plan rejects, rollback restores
    live0 = R.rwttt_slot(ctx, 1, 0, 0)
    make_dirty(ctx, [1, 2])
    assert R.rwttt_version(ctx, 1) == (0, True)
    assert R.rwttt_commit(ctx, [1]) == R.RWTTT_E_WRITE_FAILED
    p = R.rwttt_plan(ctx, [(1, 0, 0, 0, 0, 0, 0), (3, 0, 0, 0, 0, 0, 0)], 0)
    assert p.ev_status == [R.RWTTT_E_DIRTY, R.RWTTT_OK]
    # aliasing is checked before anything changes
    assert R.rwttt_rollback(ctx, [1, 1]) == R.RWTTT_E_OWNER_ALIAS
    assert R.rwttt_rollback(ctx, [1, 3]) == R.RWTTT_E_NOT_DIRTY
    assert R.rwttt_version(ctx, 1) == (0, True)
    assert R.rwttt_rollback(ctx, [1, 2]) == R.RWTTT_OK
    assert R.rwttt_version(ctx, 1) == (0, False)
    assert R.rwttt_slot(ctx, 1, 0, 0) == live0
    # the same layer cannot be written twice in one open transition
    make_dirty(ctx, [0], layer=1)
    wg = R.make_group(R.RWTTT_WRITE, 0, 1)
    assert R.rwttt_write(ctx, wg, R.u32_array([0]), 1, 4, [0x100], [0x200], 1.0) == R.RWTTT_E_WRITE_FAILED
    assert R.rwttt_rollback(ctx, [0]) == R.RWTTT_OK
    # no workspace: device calls are refused, nothing is launched
    assert R.rwttt_read(ctx, rg, R.u32_array([0]), 0, 0x1000, 0x2000) == R.RWTTT_E_INVALID
    assert R.rwttt_write(ctx, wg, R.u32_array([3]), 0, 4, [0x100], [0x200], 1.0) == R.RWTTT_E_INVALID
    assert R.rwttt_version(ctx, 3) == (0, False)
    empty = R.make_group(R.RWTTT_READ, 0, 0)
    assert R.rwttt_read(ctx, empty, R.u32_array([]), 0, 0x1000, 0x2000) == R.RWTTT_OK
    # bad layer, alias inside a group
    assert R.rwttt_read(ctx, rg, R.u32_array([0]), 5, 0x1000, 0x2000) == R.RWTTT_E_INVALID
    ag = R.make_group(R.RWTTT_READ, 0, 2)
    assert R.rwttt_read(ctx, ag, R.u32_array([2, 2]), 0, 0x1000, 0x2000) == R.RWTTT_E_OWNER_ALIAS


def test_read_and_write_recheck_planned_versions():
    """Each member's planned version is checked against V(r) before anything
    changes (Section 3, eq. compatibility); `expected` is indexed like the owner
    map, so a group in the middle of the map reads its own entries."""
    ctx, _ = host_ctx(n_owners=4)                          # every V(r) is 0
    omap = R.u32_array([3, 2, 0])
    rg = R.make_group(R.RWTTT_READ, 1, 2)                  # members 2, 0
    stale = [9, 1, 0]                                       # owner 2 is at 0, not 1
    assert R.rwttt_read(ctx, rg, omap, 0, 0x1000, 0x2000, expected=stale) == R.RWTTT_E_STALE_VERSION
    assert R.rwttt_read_append(ctx, rg, omap, 0, 0x1000, 0x2000, expected=stale) == \
        R.RWTTT_E_STALE_VERSION
    wg = R.make_group(R.RWTTT_WRITE, 1, 2)
    assert R.rwttt_write(ctx, wg, omap, 0, 4, [0x100] * 2, [0x200] * 2, 1.0,
                         expected=stale) == R.RWTTT_E_STALE_VERSION
    assert [R.rwttt_version(ctx, r) for r in range(4)] == [(0, False)] * 4
    # entry 0 belongs to owner 3, which is not in the group: its value is not read
    ok = [9, 0, 0]
    assert R.rwttt_read(ctx, rg, omap, 0, 0x1000, 0x2000, expected=ok) == R.RWTTT_E_INVALID  # host-only
    assert R.rwttt_inject_write_failures(ctx, 1) == R.RWTTT_OK
    assert R.rwttt_write(ctx, wg, omap, 0, 4, [0x100] * 2, [0x200] * 2, 1.0,
                         expected=ok) == R.RWTTT_E_WRITE_FAILED
    assert R.rwttt_version(ctx, 2) == (0, True) and R.rwttt_version(ctx, 0) == (0, True)


def test_tail_state_machine_and_errors_before_any_launch():
    """Tail validation paths that return before the device is touched: the
    workspace address below is never dereferenced."""
    n_owners, n_layers, d_ff, d_model = 3, 2, 64, 32
    w0 = [0x10000 * (i + 1) for i in range(n_layers)]
    slots = [0x1000000 + 0x1000 * i for i in range(n_owners * n_layers * 2)]
    cfg = R.make_config(n_owners, n_layers, d_ff, d_model, R.RWTTT_BF16, R.RWTTT_F32, 4, w0, slots)
    ws = R.rwttt_workspace_bytes(cfg)
    cfg = R.make_config(n_owners, n_layers, d_ff, d_model, R.RWTTT_BF16, R.RWTTT_F32, 4, w0, slots,
                        workspace=0x40000000, workspace_bytes=ws)
    ctx = R.rwttt_create(cfg)
    rg = R.make_group(R.RWTTT_READ, 0, 1)
    wg = R.make_group(R.RWTTT_WRITE, 0, 1)
    one = R.u32_array([1])
    # no tail attached
    assert R.rwttt_read_append(ctx, rg, one, 0, 0x2000, 0x3000) == R.RWTTT_E_INVALID
    assert R.rwttt_write(ctx, wg, one, 0, 1, None, [0x200], 1.0, 0x2000, 0x3000) == R.RWTTT_E_INVALID
    assert R.rwttt_tail_len(ctx, 1, 0) == 0
    tails = [0x2000000 + 0x1000 * i for i in range(n_owners * n_layers)]
    assert R.rwttt_attach_tail(ctx, tails, 0) == R.RWTTT_E_INVALID
    assert R.rwttt_attach_tail(ctx, tails[:-1] + [tails[-1] + 8], 4) == R.RWTTT_E_INVALID
    assert R.rwttt_attach_tail(ctx, tails, 4) == R.RWTTT_OK
    # a tail WRITE needs chunk == tail_len + 1, a token, and fits the tail
    assert R.rwttt_write(ctx, wg, one, 0, 2, None, [0x200], 1.0, 0x2000, 0x3000) == R.RWTTT_E_INVALID
    assert R.rwttt_write(ctx, wg, one, 0, 5, None, [0x200], 1.0, 0x2000, 0x3000) == R.RWTTT_E_INVALID
    assert R.rwttt_write(ctx, wg, one, 0, 1, None, [0x200], 1.0) == R.RWTTT_E_INVALID
    assert R.rwttt_version(ctx, 1) == (0, False)
    # an injected failure opens the candidate without launching; rollback closes it
    assert R.rwttt_inject_write_failures(ctx, 1) == R.RWTTT_OK
    assert R.rwttt_write(ctx, wg, one, 0, 1, None, [0x200], 1.0, 0x2000, 0x3000) == R.RWTTT_E_WRITE_FAILED
    assert R.rwttt_version(ctx, 1) == (0, True)
    assert R.rwttt_rollback(ctx, [1]) == R.RWTTT_OK
    assert R.rwttt_tail_len(ctx, 1, 0) == 0
    with pytest.raises(R.RwtttError):
        R.rwttt_tail_len(ctx, 3, 0)
    R.rwttt_destroy(ctx)


def test_fork_checkpoint_resume_validation():
    ctx, _ = host_ctx(n_owners=4, n_layers=2)
    assert R.rwttt_fork(ctx, 1, 1) == R.RWTTT_E_OWNER_ALIAS
    assert R.rwttt_fork(ctx, 1, 7) == R.RWTTT_E_INVALID
    make_dirty(ctx, [2])
    assert R.rwttt_fork(ctx, 1, 2) == R.RWTTT_E_DIRTY
    assert R.rwttt_resume(ctx, 2, [0x5000, 0x6000], 3) == R.RWTTT_E_DIRTY
    # no workspace: a host-only context refuses the device copy
    assert R.rwttt_fork(ctx, 1, 3) == R.RWTTT_E_INVALID
    assert R.rwttt_checkpoint(ctx, 9, [0x5000, 0x6000])[0] == R.RWTTT_E_INVALID
    assert R.rwttt_checkpoint(ctx, 1, [0x5000, 0])[0] == R.RWTTT_E_INVALID
    assert R.rwttt_checkpoint(ctx, 1, [0x5000, 0x6000])[0] == R.RWTTT_E_INVALID
    assert R.rwttt_resume(ctx, 1, [0x5000, 0x6000], 3) == R.RWTTT_E_INVALID
    assert R.rwttt_resume(ctx, 1, [0, 0x6000], 3) == R.RWTTT_E_INVALID
    assert R.rwttt_version(ctx, 1) == (0, False)
    assert R.rwttt_rollback(ctx, [2]) == R.RWTTT_OK
    R.rwttt_destroy(ctx)


def test_slots_are_live_and_shadow_of_each_owner_layer():
    ctx, cfg = host_ctx(n_owners=3, n_layers=2)
    for r in range(3):
        for l in range(2):
            base = 0x1000000 + 0x1000 * ((r * 2 + l) * 2)
            assert R.rwttt_slot(ctx, r, l, 0) == base
            assert R.rwttt_slot(ctx, r, l, 1) == base + 0x1000


def test_create_rejects_bad_configs():
    ok = dict(n_owners=2, n_layers=1, d_ff=64, d_model=32, io_dtype=1, state_dtype=0, max_group=2)

    def make(**kw):
        a = dict(ok)
        a.update(kw)
        slots = kw.pop("_slots", None) or [0x1000000 + 0x1000 * i for i in range(a["n_owners"] * a["n_layers"] * 2)]
        cfg = R.make_config(a["n_owners"], a["n_layers"], a["d_ff"], a["d_model"], a["io_dtype"],
                            a["state_dtype"], a["max_group"], [0x10000] * a["n_layers"], slots)
        return cfg

    for bad in [dict(d_ff=60), dict(d_model=12), dict(max_group=0), dict(max_group=65),
                dict(io_dtype=3), dict(n_owners=0)]:
        with pytest.raises(R.RwtttError) as e:
            R.rwttt_create(make(**bad))
        assert e.value.status == R.RWTTT_E_INVALID
    dup = make()
    dup.slots[1] = dup.slots[0]
    with pytest.raises(R.RwtttError) as e:
        R.rwttt_create(dup)
    assert e.value.status == R.RWTTT_E_OWNER_ALIAS
    small = make()
    small.workspace = 0x100000000
    small.workspace_bytes = 16
    with pytest.raises(R.RwtttError) as e:
        R.rwttt_create(small)
    assert e.value.status == R.RWTTT_E_CAPACITY


def test_strerror_covers_every_code():
    for code in range(-9, 2):
        assert R.rwttt_strerror(code) != "unknown status"
    assert R.rwttt_strerror(-42) == "unknown status"


def test_bench_refuses_more_than_one_gpu():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_bench_traffic_applies_only_to_its_shape_and_source(tmp_path, monkeypatch):
    """The PMC traffic table is reported only for the READ shape, group sizes and
    kernel source it was measured on (a table written here, keyed like the
    committed one)."""
    import json
    import bench
    from rwttt_inputs import workload
    mixed, prefill, ragged = workload(2), workload(4), workload(3)
    table = {"kernel_source_sha256": bench.kernel_source_sha(), "workload": mixed.name,
             "read_shape": {"d_model": mixed.d_model, "d_ff": mixed.d_ff,
                            "io": mixed.io_dtype, "state": mixed.state_dtype},
             "read_call_bytes_by_group_size": {"8": {"fetch": 800.0, "write": 3.0},
                                               "7": {"fetch": 700.0, "write": 2.0}}}
    (tmp_path / "profiles").mkdir()
    (tmp_path / "profiles" / "hbm_traffic__mixed8-4b-36L.json").write_text(json.dumps(table))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "kernel_source_sha", lambda: table["kernel_source_sha256"])
    rec = lambda b, n: ("read", b, 0, None, None, n)
    assert bench.measured_traffic([rec(8, 3), rec(7, 1)], mixed) == (3 * 803.0 + 702.0) / 4
    assert bench.measured_traffic([rec(8, 1)], prefill) is None      # another shape
    assert bench.measured_traffic([rec(16, 1)], ragged) is None      # a group size not measured
    monkeypatch.setattr(bench, "kernel_source_sha", lambda: "0" * 64)
    assert bench.measured_traffic([rec(8, 1)], mixed) is None        # other kernel code
    # comments and indentation do not change the key, code does
    code = "int a; // x\n  int b;\n\n"
    assert bench.code_lines(code) == ["int a;", "int b;"]
    assert bench.code_lines("int a; // y\nint b;") == bench.code_lines(code)


def test_bench_pmc_summary_scales_and_groups_by_call(tmp_path):
    """The PMC summariser scales each counter by the copy calibration and sums a
    READ call's partial and reduce launches per group size (synthetic databases
    with the rocpd columns it reads)."""
    import sqlite3
    import bench
    ns = "void rwttt::(anonymous namespace)::"
    part = ns + "read_partial_kernel<unsigned short, float>(rwttt::(anonymous namespace)::ReadParams)"
    red = ns + "read_reduce_kernel<unsigned short>(rwttt::(anonymous namespace)::ReadParams)"
    wst = ns + "write_stream_kernel<float, true>(rwttt::(anonymous namespace)::WriteParams)"
    copy = "__amd_rocclr_copyBuffer"

    def db(path, rows):
        path.mkdir()
        c = sqlite3.connect(str(path / "x_results.db"))
        c.execute("create table pmc_events (dispatch_id int, name text, counter_value real)")
        c.execute("create table kernels (dispatch_id int, grid_x int, grid_y int)")
        for i, (name, v, gx, gy) in enumerate(rows):
            c.execute("insert into pmc_events values (?, ?, ?)", (i, name, v))
            c.execute("insert into kernels values (?, ?, ?)", (i, gx, gy))
        c.commit()

    kib = (1 << 30) / 1024
    db(tmp_path / "pmc_copy_FETCH_SIZE", [(copy, kib / 2, 1, 1)])    # reads half: scale 2
    db(tmp_path / "pmc_copy_WRITE_SIZE", [(copy, kib, 1, 1)])
    blocks8 = 384 * 8 * 256
    db(tmp_path / "pmc_bench_FETCH_SIZE", [(part, 100.0, blocks8, 1), (part, 300.0, blocks8, 1),
                                           (red, 10.0, 10240, 8), (red, 1.0, 10240, 1),
                                           (wst, 50.0, 122880, 1)])
    db(tmp_path / "pmc_bench_WRITE_SIZE", [(part, 4.0, blocks8, 1), (red, 2.0, 10240, 8),
                                           (red, 7.0, 10240, 1), (wst, 60.0, 122880, 1)])
    dirs = {f"{k}_{cn}": str(tmp_path / f"pmc_{k}_{cn}")
            for k in ("copy", "bench") for cn in ("FETCH_SIZE", "WRITE_SIZE")}
    out = bench.pmc_summary(dirs)
    assert out["calibration"]["fetch_scale"] == 2.0 and out["calibration"]["write_scale"] == 1.0
    assert out["read_call_bytes_by_group_size"] == {"8": {"fetch": (200.0 + 10.0) * 2 * 1024,
                                                          "write": (4.0 + 2.0) * 1024}}
    assert out["write_call_bytes"] == {"fetch": 50.0 * 2 * 1024, "write": 60.0 * 1024}
    assert out["kernel_source_sha256"] == bench.kernel_source_sha()


def test_plain_c_client_builds_against_the_header_and_runs(tmp_path):
    """The header is C (not only C++): a C11 client compiles with gcc, links the
    library and drives planning and the owner table on a host-only context."""
    exe = str(tmp_path / "abi_host_check")
    libdir = os.path.dirname(R.LIB_PATH)
    subprocess.run(["gcc", "-std=c11", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "tests", "c", "abi_host_check.c"), "-L", libdir, "-lrwttt",
                    f"-Wl,-rpath,{libdir}", "-o", exe], check=True, capture_output=True, text=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip() == "ok"


def test_noalloc_read_validates_before_touching_the_device():
    """rwttt_read_noalloc refuses, on the host, what it cannot run: a group whose
    partial sums exceed the static array (d_ff 14336, d_model 4096, fp32 state:
    56 x 4096 fp32 values = 917,504 bytes per owner, so 18 owners fit in 16 MiB
    and 19 do not), an adapter context, a stale planned version, an alias."""
    assert R.RWTTT_NOALLOC_SCRATCH_BYTES == 16 << 20
    assert 18 * 56 * 4096 * 4 <= R.RWTTT_NOALLOC_SCRATCH_BYTES < 19 * 56 * 4096 * 4
    ctx, _ = host_ctx(n_owners=20, n_layers=1, d_ff=14336, d_model=4096, max_group=20)
    g19 = R.make_group(R.RWTTT_READ, 0, 19)
    assert R.rwttt_read_noalloc(ctx, g19, R.u32_array(range(19)), 0, 0x1000, 0x2000) == R.RWTTT_E_CAPACITY
    g2 = R.make_group(R.RWTTT_READ, 0, 2)
    assert R.rwttt_read_noalloc(ctx, g2, R.u32_array([3, 3]), 0, 0x1000, 0x2000) == R.RWTTT_E_OWNER_ALIAS
    assert R.rwttt_read_noalloc(ctx, g2, R.u32_array([3, 4]), 0, 0x1000, 0x2000,
                                expected=[0, 2]) == R.RWTTT_E_STALE_VERSION
    assert R.rwttt_read_noalloc(ctx, g2, R.u32_array([3, 4]), 1, 0x1000, 0x2000) == R.RWTTT_E_INVALID
    empty = R.make_group(R.RWTTT_READ, 0, 0)
    assert R.rwttt_read_noalloc(ctx, empty, R.u32_array([]), 0, 0x1000, 0x2000) == R.RWTTT_OK
    R.rwttt_destroy(ctx)
    w0 = [0x10000]
    slots = [0x1000000 + 0x1000 * i for i in range(4)]
    cfg = R.make_config(2, 1, 64, 32, R.RWTTT_BF16, R.RWTTT_F32, 2, w0, slots,
                        backend=R.RWTTT_DELTA_ADAPTER, rank=4)
    actx = R.rwttt_create(cfg)
    g1 = R.make_group(R.RWTTT_READ, 0, 1)
    assert R.rwttt_read_noalloc(actx, g1, R.u32_array([0]), 0, 0x1000, 0x2000) == R.RWTTT_E_INVALID
    R.rwttt_destroy(actx)


class _Ev:
    """Stand-in for a pair of HIP events: elapsed_time(end) gives the span in ms."""

    def __init__(self, ms):
        self.ms = ms

    def elapsed_time(self, end):
        return end.ms - self.ms


def test_bench_counts_algorithmic_bytes_and_flops_per_call():
    """The bench's per-call accounting: a READ of B owners moves W0 once, each
    live state, x and y; a WRITE moves live, shadow, Z and G per owner and does
    2 C d_ff d_model flops; a WRITE step's token adds x and y, and its second
    W0 pass (plus the live state when not fused) is reported, not counted."""
    sys.path.insert(0, ROOT)
    import bench
    from rwttt_inputs import workload
    wl = workload(2)                          # bf16 io, fp32 state, 9728 x 2560
    K, N, io, st = wl.d_ff, wl.d_model, 2, 4
    t = bench.LaunchTimer(None)
    t.records = [("read", 8, 0, _Ev(0.0), _Ev(1.0), 10), ("read", 7, 0, _Ev(1.0), _Ev(1.5), 4),
                 ("write_token", 1, 64, _Ev(0.0), _Ev(0.5), 10)]
    s = t.summary(wl)
    rd = K * N * (io + 8 * st) + 8 * io * (K + N)
    rd7 = K * N * (io + 7 * st) + 7 * io * (K + N)
    assert s["read"]["bytes"] == 10 * rd + 4 * rd7
    assert s["read"]["launches"] == 14 and s["read"]["total_ms"] == pytest.approx(1.5)
    assert s["read"]["gbs"] == pytest.approx((10 * rd + 4 * rd7) / 1.5e-3 / 1e9)
    w = s["write_token"]
    assert w["bytes"] == 10 * (2 * st * K * N + io * 64 * (K + N) + io * (K + N))
    assert w["bytes"] // 10 == 200826880                      # 200.8 MB per one-owner call
    assert w["flops"] == 10 * 2.0 * 64 * K * N
    assert w["token_extra_bytes"] == 10 * K * N * io          # W0 once per call, fused token
    rec = bench.write_record(wl, s)
    assert rec["hbm_frac"] == pytest.approx(w["bytes"] / 0.5e-3 / 1e9 / 8000.0, rel=1e-3)
    assert rec["token_extra_bytes_per_launch"] == K * N * io
    assert rec["kernel"].startswith("write_stream_kernel")
    # C = 512 with a token: a READ of the group first (W0 and the live state again)
    w4 = workload(4)
    K4, N4 = w4.d_ff, w4.d_model
    t.records = [("write_token", 8, 512, _Ev(0.0), _Ev(0.6), 1), ("write", 8, 512, _Ev(0.0), _Ev(0.6), 1)]
    s4 = t.summary(w4)
    assert s4["write_token"]["token_extra_bytes"] == K4 * N4 * 2 + 8 * 2 * K4 * N4
    assert s4["write"]["token_extra_bytes"] == 0
    assert s4["write"]["bytes"] == 8 * (2 * 2 * K4 * N4 + 2 * 512 * (K4 + N4))
    assert bench.write_record(w4, {"write": s4["write"]})["kernel"] == "write_gemm_kernel"
