"""Seeded synthetic workloads for the expert-choice MoE layer.

This module only draws random numbers and stores them in the storage formats the
layer consumes (fp32, or bf16 by round-to-nearest-even).  It holds none of the
layer's arithmetic: no routing, no capacity rule, no FFN.  Both the HIP path and
the CPU oracle consume the exact arrays produced here.

Every tensor gets its own child of ``numpy.random.SeedSequence(seed)`` and is
filled in fixed-size chunks, chunk ``c`` from its own grand-child PCG64 stream,
so the values do not depend on the number of threads used to draw them.

Weight layouts (row-major):
  X  [N, d]      tokens, groups (sequences) contiguous
  Wg [E, d]      router projection, row j scores expert j
  W1 [E, h, d]   gate projection of expert j's SwiGLU FFN
  W3 [E, h, d]   up projection
  W2 [E, d, h]   down projection
  t  [G]         per-sequence mask ratio (only for time-dependent capacity)
  dY [N, d]      upstream gradient (training workload only)

The shapes follow the paper's 8B-A1B MoE block (hidden 2048, 64 fine-grained
experts, sequence length about 2048; Appendix E) and the capacity settings of
Section 4; the value distributions are normal because the trained activations
and routers of the paper are not available.
"""
from __future__ import annotations

import dataclasses
from concurrent.futures import ThreadPoolExecutor
from typing import Optional, Sequence

import numpy as np

_CHUNK = 1 << 22  # elements per independent PCG64 stream


def f32_to_bf16_bits(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (nearest, ties to even); return the uint16 bit patterns."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def _normal(ss: np.random.SeedSequence, shape, std: float, threads: int = 8) -> np.ndarray:
    n = int(np.prod(shape))
    out = np.empty(n, dtype=np.float32)
    nchunks = max(1, -(-n // _CHUNK))
    kids = ss.spawn(nchunks)

    def fill(c):
        lo, hi = c * _CHUNK, min(n, (c + 1) * _CHUNK)
        g = np.random.Generator(np.random.PCG64(kids[c]))
        g.standard_normal(hi - lo, dtype=np.float32, out=out[lo:hi])
        if std != 1.0:
            out[lo:hi] *= np.float32(std)

    if nchunks == 1:
        fill(0)
    else:
        with ThreadPoolExecutor(min(threads, nchunks)) as ex:
            list(ex.map(fill, range(nchunks)))
    return out.reshape(shape)


@dataclasses.dataclass(frozen=True)
class Workload:
    """Shapes, storage dtype and capacity rule of one synthetic layer invocation."""
    name: str
    group_lengths: tuple          # L_g for each routing group (sequence)
    d_model: int
    n_experts: int
    d_ff: int
    dtype: str                    # "f32" or "bf16"
    seed: int
    x_std: float = 1.0
    w_std: float = 0.02
    capacity_factor: Optional[float] = None   # fixed c (experts per token on average)
    c_min: Optional[float] = None             # time-dependent c(t) = c_min + (c_max-c_min)(1-t)
    c_max: Optional[float] = None
    inv_temperatures: tuple = (1.0,)
    backward: bool = False
    dy_seed: Optional[int] = None
    d_shared: int = 0             # hidden width of the shared experts side by side (0: none)

    @property
    def n_tokens(self) -> int:
        return int(sum(self.group_lengths))

    @property
    def n_groups(self) -> int:
        return len(self.group_lengths)

    @property
    def group_offsets(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.group_lengths)]).astype(np.int32)

    @property
    def time_dependent(self) -> bool:
        return self.capacity_factor is None


@dataclasses.dataclass
class Inputs:
    """Drawn arrays.  bf16 tensors are uint16 bit patterns, fp32 tensors are float32."""
    wl: Workload
    X: np.ndarray
    Wg: np.ndarray
    W1: np.ndarray
    W3: np.ndarray
    W2: np.ndarray
    t: Optional[np.ndarray]       # float64 [G] mask ratios, or None
    dY: Optional[np.ndarray] = None
    shared: Optional[tuple] = None   # (Ws1 [hs,d], Ws3 [hs,d], Ws2 [d,hs]) or None


def draw(wl: Workload, with_dy: Optional[bool] = None, threads: int = 8) -> Inputs:
    """Draw X, Wg, W1, W3, W2 (and t, dY) for a workload, in that order."""
    N, d, E, h = wl.n_tokens, wl.d_model, wl.n_experts, wl.d_ff
    kids = np.random.SeedSequence(wl.seed).spawn(6)
    raw = [
        _normal(kids[0], (N, d), wl.x_std, threads),
        _normal(kids[1], (E, d), wl.w_std, threads),
        _normal(kids[2], (E, h, d), wl.w_std, threads),
        _normal(kids[3], (E, h, d), wl.w_std, threads),
        _normal(kids[4], (E, d, h), wl.w_std, threads),
    ]
    t = None
    if wl.time_dependent:
        t = np.random.Generator(np.random.PCG64(kids[5])).uniform(0.0, 1.0, wl.n_groups)
    conv = f32_to_bf16_bits if wl.dtype == "bf16" else (lambda a: a)
    X, Wg, W1, W3, W2 = (conv(a) for a in raw)
    dY = None
    if with_dy if with_dy is not None else wl.backward:
        seed = wl.dy_seed if wl.dy_seed is not None else wl.seed + 1000
        dY = conv(_normal(np.random.SeedSequence(seed).spawn(1)[0], (N, d), 1.0, threads))
    shared = None
    if wl.d_shared:
        hs = wl.d_shared
        sk = np.random.SeedSequence([wl.seed, 2]).spawn(3)   # apart from the draws above
        shared = tuple(conv(_normal(k, shp, wl.w_std, threads))
                       for k, shp in zip(sk, ((hs, d), (hs, d), (d, hs))))
    return Inputs(wl, X, Wg, W1, W3, W2, t, dY, shared)


# The five workloads.  Sizes follow the paper's 8B-A1B block (Appendix E) and the
# capacity schedules of Section 4; seeds are fixed so every run sees the same bits.
TINY_F32 = Workload("tiny_f32_L128_d64_E8_h128_c2", (128,), 64, 8, 128, "f32", seed=0,
                    x_std=1.0, w_std=1.0 / 8.0, capacity_factor=2.0)
STATIC_BF16 = Workload("static_bf16_8x2048_d2048_E64_h1024_c8", (2048,) * 8, 2048, 64, 1024,
                       "bf16", seed=1, capacity_factor=8.0)
TIMESTEP_BF16 = Workload("timestep_bf16_8x2048_d2048_E64_h1024_c12-8t", (2048,) * 8, 2048, 64,
                         1024, "bf16", seed=2, c_min=4.0, c_max=12.0)
FINE_BF16 = Workload("fine_bf16_4x4096_d2048_E128_h768_c8", (4096,) * 4, 2048, 128, 768,
                     "bf16", seed=3, capacity_factor=8.0, inv_temperatures=(2.0, 1.0, 0.5))
TRAIN_BF16 = dataclasses.replace(TIMESTEP_BF16, name="train_bf16_8x2048_d2048_E64_h1024_c12-8t",
                                 backward=True, dy_seed=4)

# single-sample decoding (Section 5.2): one sequence of 2048 tokens, every expert
# choosing from that one pool, capacity c(t) = 12 - 8t at the sample's mask ratio
# (at most k_max = 2048 * 12 / 64 = 384 tokens per expert), forward only
DECODE_BF16 = Workload("decode_bf16_1x2048_d2048_E64_h1024_c12-8t", (2048,), 2048, 64, 1024,
                       "bf16", seed=5, c_min=4.0, c_max=12.0)

# the training workload with the 8B-A1B block's 2 shared experts (each of the
# routed experts' width) added to every token
TRAIN_SHARED_BF16 = dataclasses.replace(
    TRAIN_BF16, name="train_shared_bf16_8x2048_d2048_E64_h1024_s2x1024_c12-8t", d_shared=2048)

WORKLOADS = {w.name: w for w in (TINY_F32, STATIC_BF16, TIMESTEP_BF16, FINE_BF16, TRAIN_BF16,
                                 TRAIN_SHARED_BF16, DECODE_BF16)}


def small(name: str, group_lengths: Sequence[int], d: int, E: int, h: int, dtype: str = "bf16",
          seed: int = 7, capacity_factor: Optional[float] = None, c_min=None, c_max=None,
          inv_temperature: float = 1.0, backward: bool = False, d_shared: int = 0) -> Workload:
    """A reduced workload for parity tests (any shapes; weights std 1/sqrt(d))."""
    return Workload(name, tuple(int(x) for x in group_lengths), d, E, h, dtype, seed,
                    x_std=1.0, w_std=float(1.0 / np.sqrt(d)), capacity_factor=capacity_factor,
                    c_min=c_min, c_max=c_max, inv_temperatures=(inv_temperature,),
                    backward=backward, dy_seed=seed + 100, d_shared=d_shared)
