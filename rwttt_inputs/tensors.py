"""Seeded tensor draws for the synthetic workloads.

Every tensor block has its own numpy ``SeedSequence`` keyed by
(workload seed, kind, indices), so any block can be regenerated on its own and
in any order: the GPU harness draws everything, the oracle redraws only the
blocks it samples, and both see identical values.

Recipe: a block is drawn as float32 standard normals (numpy PCG64), scaled by
the float32 value of the standard deviation (absolute value for |N(0,1)|), and,
for a bf16 tensor, narrowed to bf16 by round-to-nearest-even on the float32
bits.  bf16 tensors are held as ``uint16`` bit patterns.
"""

import numpy as np

from .workloads import Workload

K_W0, K_DW, K_X, K_Z, K_G, K_ADA_A, K_ADA_B, K_TEST = 1, 2, 3, 4, 5, 6, 7, 9


def f32_to_bf16_bits(a):
    """Round float32 values to bf16 bit patterns, nearest-even (finite inputs)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b):
    """Widen bf16 bit patterns to float32 (exact)."""
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _gen(seed, key):
    ss = np.random.SeedSequence(entropy=int(seed), spawn_key=tuple(int(k) for k in key))
    return np.random.Generator(np.random.PCG64(ss))


def draw(shape, std, dtype, seed, key, absval=False):
    """One seeded block: N(0, std^2) (or |N(0,1)|*std) as float32 or bf16 bits."""
    g = _gen(seed, key)
    n = int(np.prod(shape)) if len(shape) else 1
    a = g.standard_normal(n, dtype=np.float32)
    if absval:
        np.abs(a, out=a)
    if std != 1.0:
        a *= np.float32(std)
    a = a.reshape(shape)
    if dtype == "bf16":
        return f32_to_bf16_bits(a)
    if dtype == "f32":
        return a
    raise ValueError(dtype)


class TensorSource:
    """Lazily drawn tensors of one workload.

    x(t, r, l)      [d_ff]               io dtype
    w0(l)           [d_ff, d_model]      io dtype
    dw_init(r, l)   [d_ff, d_model]      state dtype (zeros when dw_std == 0)
    adapter_init(r, l, rank)  ([d_ff, rank], [rank, d_model])  state dtype
    zg(t, r, l, C)  ([C, d_ff], [C, d_model])  io dtype
    """

    def __init__(self, wl: Workload, cache_steps=True, memo=False):
        self.wl = wl
        self._xcache = {}
        self._cache_steps = cache_steps
        self._memo = {} if memo else None

    def _remember(self, key, fn):
        if self._memo is None:
            return fn()
        if key not in self._memo:
            self._memo[key] = fn()
        return self._memo[key]

    def prefetch(self, owners, layers, threads=8):
        """Draw W0 and the initial state of (owners x layers) in parallel (memo only)."""
        from concurrent.futures import ThreadPoolExecutor
        assert self._memo is not None, "prefetch needs memo=True"
        jobs = [("w0", l) for l in layers] + [("dw", r, l) for r in owners for l in layers]
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(lambda j: self.w0(j[1]) if j[0] == "w0" else self.dw_init(j[1], j[2]), jobs))

    # ---- shared weights and initial state --------------------------------
    def w0(self, l):
        wl = self.wl
        return self._remember(("w0", l), lambda: draw(
            (wl.d_ff, wl.d_model), wl.w0_std, wl.io_dtype, wl.seed, (K_W0, l)))

    def dw_init(self, r, l):
        wl = self.wl
        if wl.dw_std == 0.0:
            dt = np.float32 if wl.state_dtype == "f32" else np.uint16
            return np.zeros((wl.d_ff, wl.d_model), dtype=dt)
        return self._remember(("dw", r, l), lambda: draw(
            (wl.d_ff, wl.d_model), wl.dw_std, wl.state_dtype, wl.seed, (K_DW, r, l)))

    def adapter_init(self, r, l, rank):
        """Initial low-rank factors of the adapter backend, state dtype:
        A [d_ff, rank] ~ N(0, 1/d_ff), B [rank, d_model] ~ N(0, 1/rank)."""
        wl = self.wl
        return self._remember(("ada", r, l, rank), lambda: (
            draw((wl.d_ff, rank), float(1.0 / np.sqrt(wl.d_ff)), wl.state_dtype, wl.seed,
                 (K_ADA_A, r, l, rank)),
            draw((rank, wl.d_model), float(1.0 / np.sqrt(rank)), wl.state_dtype, wl.seed,
                 (K_ADA_B, r, l, rank))))

    # ---- per-step activations --------------------------------------------
    def x_step(self, t):
        """All activations of step t: [n_owners, n_layers, d_ff]."""
        if t in self._xcache:
            return self._xcache[t]
        wl = self.wl
        a = draw((wl.n_owners, wl.n_layers, wl.d_ff), 1.0, wl.io_dtype, wl.seed, (K_X, t))
        if self._cache_steps:
            self._xcache[t] = a
        return a

    def x(self, t, r, l):
        return self.x_step(t)[r, l]

    # ---- WRITE evidence ----------------------------------------------------
    def zg_owner(self, t, r, C):
        """Z [n_layers, C, d_ff] and G [n_layers, C, d_model] of owner r's WRITE at t."""
        wl = self.wl
        if wl.z_abs:
            Z = draw((wl.n_layers, C, wl.d_ff), 1.0, wl.io_dtype, wl.seed, (K_Z, t, r), absval=True)
        else:
            # The chunk's own activations: the inputs of steps t-C+1 .. t.
            Z = np.stack([np.stack([self.x(s, r, l) for s in range(t - C + 1, t + 1)])
                          for l in range(wl.n_layers)])
        G = draw((wl.n_layers, C, wl.d_model), 1.0, wl.io_dtype, wl.seed, (K_G, t, r))
        return Z, G

    def zg(self, t, r, l, C):
        Z, G = self._remember(("zg", t, r, C), lambda: self.zg_owner(t, r, C))
        return Z[l], G[l]
