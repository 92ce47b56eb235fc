"""ctypes binding of ``include/rwttt.h`` (argument marshalling only).

Every function keeps its C name.  Device buffers are passed as integers
(``tensor.data_ptr()``) and streams as integers (``stream.cuda_stream``); the
library never sees a torch type.  Loading fails loudly if the HIP library has
not been built: there is no fallback.
"""

import ctypes as C
import os

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "librwttt.so")

RWTTT_OK = 0
RWTTT_DEFERRED = 1
RWTTT_E_INVALID = -1
RWTTT_E_STALE_VERSION = -2
RWTTT_E_OWNER_ALIAS = -3
RWTTT_E_KEY_MISMATCH = -4
RWTTT_E_NOT_DIRTY = -5
RWTTT_E_DIRTY = -6
RWTTT_E_CAPACITY = -7
RWTTT_E_HIP = -8
RWTTT_E_WRITE_FAILED = -9
RWTTT_READ = 0
RWTTT_WRITE = 1
RWTTT_F32 = 0
RWTTT_BF16 = 1
RWTTT_MAX_GROUP = 64
RWTTT_FAST_WEIGHT = 0
RWTTT_DELTA_ADAPTER = 1
RWTTT_MAX_RANK = 32
RWTTT_ADAPTER_MAX_CHUNK = 1024
RWTTT_NOALLOC_SCRATCH_BYTES = 16 << 20


class rwttt_event(C.Structure):
    _fields_ = [("owner", C.c_uint32), ("backend_type", C.c_uint32),
                ("shape_class", C.c_uint32), ("placement", C.c_uint32),
                ("effect", C.c_int32), ("reserved", C.c_uint32),
                ("expected_version", C.c_uint64), ("ready_step", C.c_uint64)]


class rwttt_group(C.Structure):
    _fields_ = [("effect", C.c_int32), ("backend_type", C.c_uint32),
                ("shape_class", C.c_uint32), ("placement", C.c_uint32),
                ("first", C.c_uint32), ("count", C.c_uint32)]


class rwttt_config(C.Structure):
    _fields_ = [("n_owners", C.c_uint32), ("n_layers", C.c_uint32),
                ("d_ff", C.c_uint32), ("d_model", C.c_uint32),
                ("io_dtype", C.c_int32), ("state_dtype", C.c_int32),
                ("max_group", C.c_uint32), ("backend", C.c_uint32),
                ("rank", C.c_uint32), ("reserved", C.c_uint32),
                ("w0", C.POINTER(C.c_void_p)), ("slots", C.POINTER(C.c_void_p)),
                ("workspace", C.c_void_p), ("workspace_bytes", C.c_size_t)]


class RwtttError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        super().__init__(f"{where}: {rwttt_strerror(status)} ({status})")


def _load():
    if not os.path.exists(_LIB_PATH):
        raise ImportError(
            f"{_LIB_PATH} is missing: build the HIP library first "
            "(python -m paper_2605_28053_amd.build)")
    # One HIP runtime per process: PyTorch-ROCm ships its own libamdhip64 under
    # the same soname as the system one.  Loading torch first makes the library
    # bind to torch's runtime, so device memory and streams from torch are
    # valid here; loaded the other way round the process would hold two
    # runtimes and the second one finds no device.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = C.CDLL(_LIB_PATH)
    P, U32, U64, I32, VP = C.POINTER, C.c_uint32, C.c_uint64, C.c_int32, C.c_void_p
    sig = {
        "rwttt_workspace_bytes": (I32, [P(rwttt_config), P(C.c_size_t)]),
        "rwttt_slot_bytes": (I32, [P(rwttt_config), P(C.c_size_t)]),
        "rwttt_create": (I32, [P(rwttt_config), P(VP)]),
        "rwttt_destroy": (I32, [VP]),
        "rwttt_plan": (I32, [VP, P(rwttt_event), U32, U64, U32, U32,
                             P(rwttt_group), U32, P(U32), P(U32), U32, P(U32),
                             P(U32), U32, P(U32), P(I32)]),
        "rwttt_read": (I32, [VP, P(rwttt_group), P(U32), P(U64), U32, VP, VP, VP]),
        "rwttt_read_append": (I32, [VP, P(rwttt_group), P(U32), P(U64), U32, VP, VP, VP]),
        "rwttt_read_noalloc": (I32, [VP, P(rwttt_group), P(U32), P(U64), U32, VP, VP, VP]),
        "rwttt_attach_tail": (I32, [VP, P(VP), U32]),
        "rwttt_tail_len": (I32, [VP, U32, U32, P(U32)]),
        "rwttt_write": (I32, [VP, P(rwttt_group), P(U32), P(U64), U32, U32, P(VP), P(VP),
                              C.c_float, VP, VP, VP]),
        "rwttt_commit": (I32, [VP, P(U32), U32]),
        "rwttt_rollback": (I32, [VP, P(U32), U32]),
        "rwttt_version": (I32, [VP, U32, P(U64), P(I32)]),
        "rwttt_slot": (I32, [VP, U32, U32, I32, P(VP)]),
        "rwttt_fork": (I32, [VP, U32, U32, VP]),
        "rwttt_checkpoint": (I32, [VP, U32, P(VP), P(U64), VP]),
        "rwttt_resume": (I32, [VP, U32, P(VP), U64, VP]),
        "rwttt_inject_write_failures": (I32, [VP, U32]),
        "rwttt_last_hip_error": (I32, [VP]),
        "rwttt_strerror": (C.c_char_p, [I32]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    return lib


_lib = _load()
LIB_PATH = _LIB_PATH


def lib():
    return _lib


def rwttt_strerror(status):
    return _lib.rwttt_strerror(int(status)).decode()


def _u32(seq):
    seq = list(seq)
    return (C.c_uint32 * max(1, len(seq)))(*seq), len(seq)


# ---------------------------------------------------------------------------
# Entry points, same names as the C ABI
# ---------------------------------------------------------------------------

def make_config(n_owners, n_layers, d_ff, d_model, io_dtype, state_dtype, max_group,
                w0_ptrs, slot_ptrs, workspace=0, workspace_bytes=0, backend=0, rank=0):
    """A ``rwttt_config`` plus the pointer arrays it references (kept alive)."""
    w0 = (C.c_void_p * len(w0_ptrs))(*[int(p) for p in w0_ptrs])
    slots = (C.c_void_p * len(slot_ptrs))(*[int(p) for p in slot_ptrs])
    cfg = rwttt_config(n_owners, n_layers, d_ff, d_model, io_dtype, state_dtype, max_group,
                       backend, rank, 0,
                       C.cast(w0, C.POINTER(C.c_void_p)), C.cast(slots, C.POINTER(C.c_void_p)),
                       int(workspace) or None, int(workspace_bytes))
    cfg._keep = (w0, slots)
    return cfg


def rwttt_workspace_bytes(cfg):
    out = C.c_size_t(0)
    st = _lib.rwttt_workspace_bytes(C.byref(cfg), C.byref(out))
    if st != RWTTT_OK:
        raise RwtttError(st, "rwttt_workspace_bytes")
    return out.value


def rwttt_slot_bytes(cfg):
    out = C.c_size_t(0)
    st = _lib.rwttt_slot_bytes(C.byref(cfg), C.byref(out))
    if st != RWTTT_OK:
        raise RwtttError(st, "rwttt_slot_bytes")
    return out.value


def rwttt_create(cfg):
    ctx = C.c_void_p(0)
    st = _lib.rwttt_create(C.byref(cfg), C.byref(ctx))
    if st != RWTTT_OK:
        raise RwtttError(st, "rwttt_create")
    return ctx


def rwttt_destroy(ctx):
    return _lib.rwttt_destroy(ctx)


class PlanResult:
    """Outputs of ``rwttt_plan`` held in ctypes arrays reusable by read/write."""

    def __init__(self, status, groups, n_groups, owner_map, n_mapped, deferred, n_deferred, ev_status):
        self.status = status
        self.groups_c = groups
        self.owner_map_c = owner_map
        self.n_groups = n_groups
        self.n_mapped = n_mapped
        self.deferred = list(deferred[:n_deferred])
        self.ev_status = list(ev_status)

    def group(self, i):
        return self.groups_c[i]

    def owners(self, i):
        g = self.groups_c[i]
        return list(self.owner_map_c[g.first:g.first + g.count])


def rwttt_plan(ctx, events, step, target_b=0, wait_budget=0, cap=None):
    """Plan ``events`` (iterable of 7-tuples or rwttt_event) at decode step."""
    evs = [e if isinstance(e, rwttt_event) else rwttt_event(
        e[0], e[1], e[2], e[3], e[4], 0, e[5], e[6]) for e in events]
    n = len(evs)
    cap = max(1, n) if cap is None else cap
    ev_arr = (rwttt_event * max(1, n))(*evs)
    groups = (rwttt_group * cap)()
    omap = (C.c_uint32 * cap)()
    defer = (C.c_uint32 * cap)()
    st_arr = (C.c_int32 * max(1, n))()
    ng, nm, nd = C.c_uint32(0), C.c_uint32(0), C.c_uint32(0)
    st = _lib.rwttt_plan(ctx, ev_arr, n, int(step), int(target_b), int(wait_budget),
                         groups, cap, C.byref(ng), omap, cap, C.byref(nm),
                         defer, cap, C.byref(nd), st_arr)
    return PlanResult(st, groups, ng.value, omap, nm.value, defer, nd.value, st_arr[:n])


def _u64_or_null(seq):
    if seq is None or isinstance(seq, C.Array):
        return seq
    seq = list(seq)
    return (C.c_uint64 * max(1, len(seq)))(*seq)


def rwttt_read(ctx, group, owner_map, layer, x_ptr, y_ptr, stream=0, expected=None):
    """``group``: rwttt_group (or pointer); ``owner_map``: ctypes uint32 array;
    ``expected``: None or the planned versions, indexed like ``owner_map``."""
    return _lib.rwttt_read(ctx, C.byref(group), owner_map, _u64_or_null(expected), int(layer),
                           int(x_ptr), int(y_ptr), int(stream) or None)


def rwttt_read_append(ctx, group, owner_map, layer, x_ptr, y_ptr, stream=0, expected=None):
    return _lib.rwttt_read_append(ctx, C.byref(group), owner_map, _u64_or_null(expected),
                                  int(layer), int(x_ptr), int(y_ptr), int(stream) or None)


def rwttt_read_noalloc(ctx, group, owner_map, layer, x_ptr, y_ptr, stream=0, expected=None):
    return _lib.rwttt_read_noalloc(ctx, C.byref(group), owner_map, _u64_or_null(expected),
                                   int(layer), int(x_ptr), int(y_ptr), int(stream) or None)


def rwttt_attach_tail(ctx, tail_ptrs, rows):
    arr = (C.c_void_p * max(1, len(tail_ptrs)))(*[int(p) for p in tail_ptrs])
    return _lib.rwttt_attach_tail(ctx, arr, int(rows))


def rwttt_tail_len(ctx, owner, layer):
    n = C.c_uint32(0)
    st = _lib.rwttt_tail_len(ctx, int(owner), int(layer), C.byref(n))
    if st != RWTTT_OK:
        raise RwtttError(st, "rwttt_tail_len")
    return n.value


def rwttt_write(ctx, group, owner_map, layer, chunk, z_ptrs, g_ptrs, eta, x_ptr=0, y_ptr=0,
                stream=0, expected=None):
    """x_ptr/y_ptr: the WRITE step's owner-indexed token input/output (0: no token).
    z_ptrs=None: the chunk is the owners' tails plus this step's x.
    expected: None or the planned versions, indexed like ``owner_map``."""
    n = len(g_ptrs)
    z = None if z_ptrs is None else (C.c_void_p * max(1, n))(*[int(p) for p in z_ptrs])
    g = (C.c_void_p * max(1, n))(*[int(p) for p in g_ptrs])
    return _lib.rwttt_write(ctx, C.byref(group), owner_map, _u64_or_null(expected), int(layer),
                            int(chunk), z, g, float(eta), int(x_ptr) or None, int(y_ptr) or None,
                            int(stream) or None)


def rwttt_commit(ctx, owners):
    arr, n = _u32(owners)
    return _lib.rwttt_commit(ctx, arr, n)


def rwttt_rollback(ctx, owners):
    arr, n = _u32(owners)
    return _lib.rwttt_rollback(ctx, arr, n)


def rwttt_version(ctx, owner):
    v, d = C.c_uint64(0), C.c_int32(0)
    st = _lib.rwttt_version(ctx, int(owner), C.byref(v), C.byref(d))
    if st != RWTTT_OK:
        raise RwtttError(st, "rwttt_version")
    return v.value, bool(d.value)


def rwttt_slot(ctx, owner, layer, which):
    p = C.c_void_p(0)
    st = _lib.rwttt_slot(ctx, int(owner), int(layer), int(which), C.byref(p))
    if st != RWTTT_OK:
        raise RwtttError(st, "rwttt_slot")
    return p.value


def rwttt_fork(ctx, src, dst, stream=0):
    return _lib.rwttt_fork(ctx, int(src), int(dst), int(stream) or None)


def rwttt_checkpoint(ctx, owner, dst_ptrs, stream=0):
    """Returns (status, version)."""
    arr = (C.c_void_p * max(1, len(dst_ptrs)))(*[int(p) for p in dst_ptrs])
    v = C.c_uint64(0)
    st = _lib.rwttt_checkpoint(ctx, int(owner), arr, C.byref(v), int(stream) or None)
    return st, v.value


def rwttt_resume(ctx, owner, src_ptrs, version, stream=0):
    arr = (C.c_void_p * max(1, len(src_ptrs)))(*[int(p) for p in src_ptrs])
    return _lib.rwttt_resume(ctx, int(owner), arr, int(version), int(stream) or None)


def rwttt_inject_write_failures(ctx, count):
    return _lib.rwttt_inject_write_failures(ctx, int(count))


def rwttt_last_hip_error(ctx):
    return _lib.rwttt_last_hip_error(ctx)


def make_group(effect, first, count, backend_type=0, shape_class=0, placement=0):
    return rwttt_group(effect, backend_type, shape_class, placement, first, count)


def u32_array(seq):
    return _u32(seq)[0]


def u64_array(seq):
    seq = list(seq)
    return (C.c_uint64 * max(1, len(seq)))(*seq)
