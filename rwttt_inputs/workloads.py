"""The five synthetic workloads of the fast-weight READ/WRITE path.

Shapes follow the paper's evaluated checkpoint class (a Qwen3-4B In-Place-TTT
model: fast weights live in the MLP down-projection, Section 1 and Section 5.1)
plus an 8B-class long-context case.  The paper leaves the update rule to the
backend (Section 4.2, "WRITE"); the synthetic rule used everywhere here is
    dW <- dW + eta * Z^T G
with Z the chunk's d_ff-side evidence and G a d_model-side signal.

Distributions are written N(0, a) with ``a`` the variance.
"""

from dataclasses import dataclass, field
import math

READ = 0     # version-preserving transition (Section 3, Ownership)
WRITE = 1    # version-creating transition (Section 3, Ownership)
IDLE = -1    # the owner exposes no transition this step

IO_F32, IO_BF16 = 0, 1
DTYPE_CODE = {"f32": 0, "bf16": 1}


@dataclass(frozen=True)
class Workload:
    name: str
    description: str
    n_owners: int
    n_layers: int
    d_model: int
    d_ff: int
    io_dtype: str          # x, W0, y, Z, G: "f32" | "bf16"
    state_dtype: str       # fast-weight slots: "f32" | "bf16"
    n_steps: int
    seed: int
    w0_std: float
    dw_std: float          # 0.0 means the fast weights start at zero
    eta: float
    schedule: str          # tiny | read_only | staggered | ragged | prefill_decode
    chunk: int = 0         # fixed WRITE chunk rank C (0: drawn per WRITE)
    chunk_choices: tuple = ()
    fail_rate: float = 0.0
    period: int = 0        # staggered: steps per READ...READ,WRITE cycle
    stagger: int = 0       # staggered: phase offset between owners
    n_prefill: int = 0     # prefill_decode: number of prefill chunks
    z_abs: bool = True     # Z ~ |N(0,1)| (else Z is assembled from x)
    extra: dict = field(default_factory=dict)

    @property
    def state_bytes(self):
        s = 4 if self.state_dtype == "f32" else 2
        return self.d_ff * self.d_model * s

    @property
    def io_bytes(self):
        return 4 if self.io_dtype == "f32" else 2


WORKLOADS = {
    0: Workload(
        name="tiny-f32",
        description="2 requests, 1 layer, d_model 64, d_ff 256, all fp32; "
                    "a C=4 WRITE every 4 steps, request 1's 3rd write fails",
        n_owners=2, n_layers=1, d_model=64, d_ff=256,
        io_dtype="f32", state_dtype="f32", n_steps=16, seed=0,
        w0_std=math.sqrt(1.0 / 256), dw_std=0.0, eta=1e-2,
        schedule="tiny", chunk=4, z_abs=False),
    1: Workload(
        name="read8-4b",
        description="8 streams READ-only decode, 1 layer, d_model 2560, "
                    "d_ff 9728, bf16 io, fp32 fast weights",
        n_owners=8, n_layers=1, d_model=2560, d_ff=9728,
        io_dtype="bf16", state_dtype="f32", n_steps=256, seed=1,
        w0_std=math.sqrt(1.0 / 9728), dw_std=math.sqrt(1e-3), eta=0.0,
        schedule="read_only"),
    2: Workload(
        name="mixed8-4b-36L",
        description="8 streams, 36 layers, d_model 2560, d_ff 9728; each "
                    "stream does 64 READs then one C=64 WRITE, phases staggered",
        n_owners=8, n_layers=36, d_model=2560, d_ff=9728,
        io_dtype="bf16", state_dtype="f32", n_steps=260, seed=2,
        w0_std=math.sqrt(1.0 / 9728), dw_std=math.sqrt(1e-3), eta=1e-3,
        schedule="staggered", chunk=64, period=65, stagger=8),
    3: Workload(
        name="ragged32-4b",
        description="32 requests, 1 layer, d_model 2560, d_ff 9728; per step "
                    "16 READ, 8 WRITE (C in {16,32,64}), 8 idle, shuffled; "
                    "5% of WRITEs fail",
        n_owners=32, n_layers=1, d_model=2560, d_ff=9728,
        io_dtype="bf16", state_dtype="f32", n_steps=512, seed=7,
        w0_std=math.sqrt(1.0 / 9728), dw_std=math.sqrt(1e-3), eta=1e-3,
        schedule="ragged", chunk_choices=(16, 32, 64), fail_rate=0.05),
    4: Workload(
        name="prefill8-8b",
        description="8 requests, 1 layer, d_model 4096, d_ff 14336, bf16 fast "
                    "weights from zero; 8 prefill WRITEs of C=512, then 128 "
                    "READ decode steps",
        n_owners=8, n_layers=1, d_model=4096, d_ff=14336,
        io_dtype="bf16", state_dtype="bf16", n_steps=8 + 128, seed=4,
        w0_std=math.sqrt(1.0 / 14336), dw_std=0.0, eta=5e-4,
        schedule="prefill_decode", chunk=512, n_prefill=8),
}


def workload(i):
    return WORKLOADS[int(i)]


def shape_class(wl, effect, chunk):
    """Opaque operator shape class sigma (Section 3, Legal batching).

    It packs the io and state dtypes and, for a WRITE, the chunk rank, so that
    WRITEs of different chunk sizes never share a group.  Only equality of the
    packed value matters to the planner.
    """
    c = int(chunk) if effect == WRITE else 0
    return (c << 8) | (DTYPE_CODE[wl.state_dtype] << 1) | DTYPE_CODE[wl.io_dtype]
