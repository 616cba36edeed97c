"""Seeded synthetic workloads for the Polyglot window-LM step.

This module holds no arithmetic of the method: it only draws inputs
(parameters, word windows, corrupt centre ids, scatter-add operands) from
seeded generators and names the workload presets.  It is the one module that
both the oracle tests and the GPU path use, so both see identical inputs.

Stand-in for the Polyglot corpora (Wikipedia text in 100+ languages, §1
Introduction), which are not available: word ids are drawn i.i.d. from a
bounded Zipf law over a frequency-ranked vocabulary, id = rank - 1, which
gives the heavy duplicate rows that make the embedding scatter-add of §4.2
(Table 1) and §4.3 hard.  Corrupt centre ids are uniform over the vocabulary.
Parameters are N(0, 0.01^2) (standard deviation 0.01).

Every per-step batch uses ``numpy.random.default_rng([seed, step])`` so any
step can be regenerated on its own.
"""
from __future__ import annotations

from dataclasses import dataclass, replace
from functools import lru_cache

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    V: int          # vocabulary rows
    d: int          # embedding width
    win: int        # window length (odd; centre at win // 2)
    H: int          # hidden units
    B: int          # windows per step
    lr: float       # SGD learning rate
    steps: int      # steps the workload is specified for
    zipf_s: float   # Zipf exponent of the word ids
    seed: int
    init_std: float = 0.01

    @property
    def K(self) -> int:
        return self.win * self.d

    def with_batch(self, B: int) -> "Workload":
        return replace(self, B=B, name=f"{self.name.split('_B')[0]}_B{B}")


PRESETS = {
    "tiny": Workload("tiny", V=1000, d=16, win=5, H=8, B=32, lr=0.01, steps=100,
                     zipf_s=1.0, seed=1),
    "poly256": Workload("poly256", V=100_000, d=64, win=5, H=32, B=256, lr=0.01,
                        steps=1000, zipf_s=1.0, seed=2),
    "sweep_1024": Workload("sweep_1024", V=100_000, d=64, win=5, H=32, B=1024, lr=0.01,
                           steps=200, zipf_s=1.0, seed=3),
    "sweep_4096": Workload("sweep_4096", V=100_000, d=64, win=5, H=32, B=4096, lr=0.01,
                           steps=200, zipf_s=1.0, seed=3),
    "sweep_16384": Workload("sweep_16384", V=100_000, d=64, win=5, H=32, B=16384, lr=0.01,
                            steps=200, zipf_s=1.0, seed=3),
    "sweep_65536": Workload("sweep_65536", V=100_000, d=64, win=5, H=32, B=65536, lr=0.01,
                            steps=200, zipf_s=1.0, seed=3),
    "stress": Workload("stress", V=1_000_000, d=128, win=11, H=256, B=16384, lr=0.005,
                       steps=200, zipf_s=1.0, seed=5),
}


@dataclass(frozen=True)
class ScatterWorkload:
    name: str
    rows: int
    d: int
    N: int
    zipf_s: float
    y_std: float
    seed: int


SCATTER_ISO = ScatterWorkload("scatter_iso", rows=100_000, d=64, N=65_536 * 5, zipf_s=1.2,
                              y_std=1e-3, seed=4)


@lru_cache(maxsize=16)
def _zipf_cdf(V: int, s: float) -> np.ndarray:
    w = np.arange(1, V + 1, dtype=np.float64) ** (-s)
    cdf = np.cumsum(w)
    return cdf / cdf[-1]


def zipf_ids(rng: np.random.Generator, V: int, s: float, size) -> np.ndarray:
    """Bounded Zipf(s) ids over [0, V): P(id = r - 1) proportional to r^-s,
    drawn by inverse CDF (numpy's own zipf needs s > 1 and is unbounded)."""
    u = rng.random(size)
    ids = np.searchsorted(_zipf_cdf(V, float(s)), u, side="right")
    return np.minimum(ids, V - 1).astype(np.int32)


def init_params(w: Workload, seed: int | None = None, dtype=np.float32) -> dict:
    """E[V][d], W1[H][win*d], b1[H], w2[H], b2[1], all N(0, init_std^2)."""
    rng = np.random.default_rng([w.seed if seed is None else seed, 1 << 30])
    std = w.init_std

    def n(*shape):
        return (rng.standard_normal(shape, dtype=np.float32) * np.float32(std)).astype(dtype)

    return {"E": n(w.V, w.d), "W1": n(w.H, w.K), "b1": n(w.H), "w2": n(w.H), "b2": n(1)}


def batch(w: Workload, step: int, B: int | None = None):
    """Windows [B][win] (Zipf ids) and corrupt centre ids [B] (uniform) of one step."""
    B = w.B if B is None else B
    rng = np.random.default_rng([w.seed, step])
    windows = zipf_ids(rng, w.V, w.zipf_s, (B, w.win))
    corrupt = rng.integers(0, w.V, size=B, dtype=np.int64).astype(np.int32)
    return windows, corrupt


def scatter_inputs(sw: ScatterWorkload = SCATTER_ISO, N: int | None = None):
    """table[rows][d] ~ N(0, 0.01^2), idx[N] ~ Zipf(s), Y[N][d] ~ N(0, y_std^2)."""
    N = sw.N if N is None else N
    rng = np.random.default_rng([sw.seed, 0])
    table = rng.standard_normal((sw.rows, sw.d), dtype=np.float32) * np.float32(0.01)
    idx = zipf_ids(rng, sw.rows, sw.zipf_s, N)
    Y = rng.standard_normal((N, sw.d), dtype=np.float32) * np.float32(sw.y_std)
    return table, idx, Y


# ------------------------------------------------ planted structure (convergence study)

@dataclass(frozen=True)
class PlantedTask:
    """Synthetic windows with a learnable rule: ids ~ Zipf(zipf_s) over V, and
    with probability 1 - noise the centre word is a fixed random permutation
    of its left neighbour.  Corrupt centres are uniform.  A held-out set with
    no noise measures the ranking error (fraction of windows that do not
    score above their corrupted copy), the stand-in for the paper's
    unspecified error level."""
    V: int = 1000
    d: int = 64
    win: int = 5
    H: int = 32
    zipf_s: float = 1.0
    noise: float = 0.1
    seed: int = 11
    init_std: float = 0.01

    def workload(self, B: int, lr: float) -> Workload:
        return Workload("planted", V=self.V, d=self.d, win=self.win, H=self.H, B=B, lr=lr,
                        steps=0, zipf_s=self.zipf_s, seed=self.seed, init_std=self.init_std)

    def rule(self) -> np.ndarray:
        return np.random.default_rng([self.seed, 2]).permutation(self.V).astype(np.int32)

    def batch(self, rng: np.random.Generator, n: int, noise: float | None = None):
        """n windows [n][win] int32 and n corrupt centre ids [n] int32."""
        noise = self.noise if noise is None else noise
        c = self.win // 2
        w = zipf_ids(rng, self.V, self.zipf_s, (n, self.win))
        keep = rng.random(n) >= noise
        w[:, c] = np.where(keep, self.rule()[w[:, c - 1]], w[:, c])
        cor = rng.integers(0, self.V, n).astype(np.int32)
        return w, cor

    def held_out(self, n: int = 8192):
        """Noise-free windows and the same windows with the corrupt centre."""
        w, cor = self.batch(np.random.default_rng([self.seed, 3]), n, noise=0.0)
        wc = w.copy()
        wc[:, self.win // 2] = cor
        return w, wc


PLANTED = PlantedTask()
