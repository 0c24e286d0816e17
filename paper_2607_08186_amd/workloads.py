"""Named workload shapes and useful-work accounting for the SFA hot path.

Shapes follow the paper's dense Qwen3-8B study (Sec. "Progressive expansion",
32 query / 8 key-value heads of width 128) and its 617B-like head layout
(Table "model_config": 96/8 heads, width 128, here one GPU's 64/8 share).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

INTRA, MIX, LOCAL = 0, 1, 2
MODE_NAMES = {INTRA: "intra", MIX: "mix", LOCAL: "local"}

# Window of the local cross-stream layers in these workloads, in expanded positions
# (p - w < p' <= p).  The paper names local layers (Fig. "masks" (b), cost O(nLw)) but
# gives no w; 4096 expanded positions is a 1024-token window of the base model at n=4.
LOCAL_WINDOW = 4096

# bf16 dense MFMA peak of one MI355X (256 CU x 2.4 GHz x 4096 flop/clk/CU)
MI355X_BF16_PEAK_TFLOPS = 2516.6
MI355X_HBM_PEAK_GBS = 8000.0


@dataclass(frozen=True)
class Shape:
    B: int
    L: int
    n: int
    Hq: int
    Hkv: int
    D: int

    @property
    def N(self) -> int:
        return self.n * self.L

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.D)


@dataclass(frozen=True)
class Workload:
    name: str
    shape: Shape
    dtype: str = "bf16"
    qkv_std: float = 1.0 / math.sqrt(2.0)
    dout_std: float = 1.0
    k_spike: tuple | None = None
    modes: tuple = (INTRA, MIX)
    extra: dict = field(default_factory=dict)


TINY = Workload("tiny-f32-L64-n2", Shape(1, 64, 2, 2, 1, 32), dtype="f32", qkv_std=1.0)
QWEN8B = Workload("qwen3-8b-like-L4096-n4", Shape(1, 4096, 4, 32, 8, 128))
SWEEP = tuple(Workload(f"sweep-B2-L2048-n{n}", Shape(2, 2048, n, 32, 8, 128)) for n in (1, 2, 4, 8))
FRONTIER = Workload("frontier-share-L8192-n4", Shape(1, 8192, 4, 64, 8, 128),
                    k_spike=(0.01, 8.0))

# 36-layer stack: mixing layers at these indices, intra-stream elsewhere, each layer at
# the Qwen3-8B-like shape; plus the stream expansion from n tables of V x Dm.
STACK_LAYERS = 36
STACK_MIX_LAYERS = (8, 17, 26, 35)
STACK_VOCAB = 151936
STACK_DMODEL = 4096
STACK_EMBED_STD = 0.02


def stack_modes():
    return [MIX if i in STACK_MIX_LAYERS else INTRA for i in range(STACK_LAYERS)]


def visible_pairs(s: Shape, mode: int, window: int = LOCAL_WINDOW) -> int:
    """Visible (query, key) pairs summed over batch and query heads (``window`` only
    matters for local layers: row p sees min(p + 1, w) keys)."""
    if mode == INTRA:
        return s.B * s.Hq * s.n * s.L * (s.L + 1) // 2
    if mode == LOCAL:
        w = min(window, s.N)
        return s.B * s.Hq * (w * (w + 1) // 2 + (s.N - w) * w)
    return s.B * s.Hq * s.N * (s.N + 1) // 2


def visible_pairs_final(s: Shape, window: int = 0) -> int:
    """Visible pairs of a final-stream layer (queries at t*n + n - 1 only, keys over all
    N rows): token t's query sees (t+1)*n keys, at most `window` of them when window > 0."""
    full = s.n * s.L * (s.L + 1) // 2
    if window <= 0:
        return s.B * s.Hq * full
    t0 = min(s.L, window // s.n)  # tokens whose whole prefix fits in the window
    return s.B * s.Hq * (s.n * t0 * (t0 + 1) // 2 + (s.L - t0) * window)


# useful flop per visible pair per head dim: fwd QK^T + PV; bwd recompute QK^T, dV, dP, dQ, dK
FWD_FLOP_PER_PAIR_D = 4
BWD_FLOP_PER_PAIR_D = 10


def useful_flop(s: Shape, mode: int, phase: str = "fwdbwd", window: int = LOCAL_WINDOW) -> int:
    c = {"fwd": FWD_FLOP_PER_PAIR_D, "bwd": BWD_FLOP_PER_PAIR_D,
         "fwdbwd": FWD_FLOP_PER_PAIR_D + BWD_FLOP_PER_PAIR_D}[phase]
    return c * s.D * visible_pairs(s, mode, window)


def stack_useful_flop(s: Shape = QWEN8B.shape) -> int:
    return sum(useful_flop(s, m) for m in stack_modes())


def embed_bytes(B: int, L: int, n: int, Dm: int, esize: int = 2) -> int:
    """Compulsory traffic of the expansion: read n*L rows, write n*L rows, read ids."""
    return 2 * B * n * L * Dm * esize + B * L * 4


def final_gather_bytes(B: int, L: int, n: int, Dm: int, backward: bool, esize: int = 2) -> int:
    """Compulsory traffic of the final-stream gather (read and write L rows) or of its
    adjoint (read L rows, write all n*L rows)."""
    row = B * Dm * esize
    return (L + n * L) * row if backward else 2 * L * row


def embed_bwd_bytes(B: int, L: int, n: int, Dm: int, n_distinct: int, esize: int = 2) -> int:
    """Compulsory traffic of the expansion's backward: read every upstream expanded row
    and the ids once, write one fp32 gradient row per (distinct id, stream) and the
    distinct ids (the sort of the B*L (id, token) pairs is not counted)."""
    return B * n * L * Dm * esize + B * L * 4 + n * n_distinct * Dm * 4 + n_distinct * 4
