"""The five synthetic workloads (self-attention and one cross non-local mean).

Sizes follow the paper's image setting (Section 2: n = H x W pixels, heads
independent) with d, iteration count T (Algorithm 1 default is 8) and window
side 2b + 1 (Algorithm 2) per workload.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field


@dataclass(frozen=True)
class Workload:
    name: str
    batch: int
    heads: int
    Hq: int
    Wq: int
    Hk: int
    Wk: int
    d: int
    dtype: str          # storage type of Q, K, V, output: "f32" or "bf16"
    sigma: float        # key blur (px)
    F: float            # max displacement |f| (px)
    iters: int          # PatchMatch iterations T
    window: int         # attend window side 2b + 1
    grid_scale: float = 1.0      # tau(p) = grid_scale * p + f(p)
    outlier_frac: float = 0.0    # fraction of queries with a random target
    data_seed: int = 1000
    pm_seed: int = 12345
    extra: dict = field(default_factory=dict)

    @property
    def S(self) -> int:
        return self.batch * self.heads

    @property
    def dv(self) -> int:
        return self.d

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.d)

    @property
    def nq(self) -> int:
        return self.S * self.Hq * self.Wq

    @property
    def elem_bytes(self) -> int:
        return 2 if self.dtype == "bf16" else 4

    @property
    def rs_steps(self) -> int:
        """Random-search steps per iteration: distances R, R/2, ..., 1."""
        R, k = max(self.Hk, self.Wk), 1
        while R > 1:
            R //= 2
            k += 1
        return k

    @property
    def candidates(self) -> int:
        """Nominal candidates per query-iteration: 16 propagation + random search."""
        return 16 + self.rs_steps

    def describe(self) -> str:
        grid = f"{self.Hq}x{self.Wq}" if (self.Hq, self.Wq) == (self.Hk, self.Wk) else \
            f"{self.Hq}x{self.Wq}->{self.Hk}x{self.Wk}"
        return (f"{self.name}: B{self.batch}xH{self.heads} {grid} d={self.d} {self.dtype} "
                f"T={self.iters} window={self.window}x{self.window}")


CONFIGS = [
    Workload("tiny32", 1, 1, 32, 32, 32, 32, 16, "f32", sigma=2, F=8, iters=4, window=3,
             data_seed=1000),
    Workload("self64", 4, 8, 64, 64, 64, 64, 64, "f32", sigma=3, F=16, iters=5, window=3,
             data_seed=1001),
    Workload("self128_bf16", 2, 8, 128, 128, 128, 128, 64, "bf16", sigma=4, F=32, iters=6, window=5,
             data_seed=1002),
    Workload("self256_bf16", 1, 4, 256, 256, 256, 256, 64, "bf16", sigma=6, F=64, iters=7, window=5,
             outlier_frac=0.05, data_seed=1003),
    Workload("cross128to192", 2, 4, 128, 128, 192, 192, 32, "f32", sigma=4, F=24, iters=6, window=3,
             grid_scale=1.5, data_seed=1004),
]

#: the headline workload (256x256 grid, d = 64, bf16 storage, 4 slices)
HEADLINE = 3

#: Measurement-only workloads (not parity cases): one 2048 x 2048 slice with the headline's
#: generator, d, storage, sweeps and window.  Q, K and V are 512 MiB each, so the working set
#: (1.5 GiB) is far past the 256 MB Infinity Cache and HBM serves the gathers.
EXTRA = [
    Workload("large2048_bf16", 1, 1, 2048, 2048, 2048, 2048, 64, "bf16", sigma=6, F=128, iters=7, window=5,
             outlier_frac=0.05, data_seed=1005),
]


def get(i) -> Workload:
    """A workload by index into CONFIGS, or by name (CONFIGS and EXTRA)."""
    if isinstance(i, str) and not i.isdigit():
        for w in CONFIGS + EXTRA:
            if w.name == i:
                return w
        raise KeyError(f"no workload named {i!r}")
    return CONFIGS[int(i)]
