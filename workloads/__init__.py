"""Seeded synthetic workloads shaped like the paper's experiments.

This module only draws random inputs: the initial output weights V0 and, per
minibatch step, the hidden representations H and the K-sparse targets given as
(index, value) pairs.  It contains none of the method's arithmetic, so both the
HIP path and the fp64 oracle can consume exactly the same bytes.

Layout (row-major, one example per row):
  H    : m x d   float32   (the paper stores the same numbers as a d x m matrix
                            with one example per column, section 3.6 / 4.1.4)
  idx  : m x K   int32     0-based row indices into V, -1 marks an empty slot
  val  : m x K   float32   target values (the paper's T matrix, section 4.1.4)
  V0   : D x d   float32

Distributions (the paper gives only shapes; these are the stated synthetic
stand-ins for its language-model workloads, whose corpus is not available):
  V0, H   ~ N(0, 1/d) entries, so Q0 = V0^T V0 ~ (D/d) I
  values  ~ N(0, 1), or all ones for one-hot (classification) targets
  indices ~ uniform over [0, D) without replacement inside one example, or a
            truncated Zipf law p(i) ~ (i+1)^-s over [0, D) (index 0 most
            frequent), redrawn inside an example until its K indices differ.
"""
from __future__ import annotations

import dataclasses
from typing import Iterator

import numpy as np

LOSS_SQUARED = "squared"
LOSS_SPHERICAL_SOFTMAX = "spherical_softmax"
LOSS_TAYLOR_SOFTMAX = "taylor_softmax"


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    loss: str
    D: int
    d: int
    m: int
    K: int
    index_dist: str = "uniform"      # "uniform" | "zipf"
    value_dist: str = "normal"       # "normal" | "ones"
    zipf_s: float = 1.1
    lr: float = 0.01
    eps: float = 1e-3                # spherical softmax epsilon
    steps: int = 100
    seed: int = 0

    def describe(self) -> dict:
        return dataclasses.asdict(self)


# The workloads the measurements are quoted on (with the sweep below), and the Taylor
# softmax on the spherical softmax's shapes and target recipe.
WORKLOADS = {
    "sq_D2k_d32_m16_K3": Workload("sq_D2k_d32_m16_K3", LOSS_SQUARED, 2000, 32, 16, 3,
                                  steps=100),
    "sq_D200k_d500_m128_K5": Workload("sq_D200k_d500_m128_K5", LOSS_SQUARED, 200_000, 500,
                                      128, 5, steps=1000),
    "sphsm_D200k_d500_m128_zipf": Workload("sphsm_D200k_d500_m128_zipf",
                                           LOSS_SPHERICAL_SOFTMAX, 200_000, 500, 128, 1,
                                           index_dist="zipf", value_dist="ones",
                                           steps=1000),
    "sq_D800k_d512_m256_K10_zipf": Workload("sq_D800k_d512_m256_K10_zipf", LOSS_SQUARED,
                                            800_000, 512, 256, 10, index_dist="zipf",
                                            steps=500),
    "taylor_D200k_d500_m128_zipf": Workload("taylor_D200k_d500_m128_zipf",
                                            LOSS_TAYLOR_SOFTMAX, 200_000, 500, 128, 1,
                                            index_dist="zipf", value_dist="ones",
                                            steps=1000),
}


def sweep_workloads(m: int = 512, K: int = 5) -> list[Workload]:
    """The D x d sweep comparing the factored and naive paths (squared error).

    D runs from 2k (below the flop crossover D ~ (10 d^2 + 3 m d + m^2) / (3 d),
    about 1.7k at d = 256) up to 1M, so that the measured crossover is bracketed.
    """
    out = []
    for D in (2_000, 5_000, 10_000, 20_000, 50_000, 200_000, 1_000_000):
        for d in (256, 512, 1024):
            out.append(Workload(f"sq_sweep_D{D}_d{d}_m{m}", LOSS_SQUARED, D, d, m, K,
                                steps=50))
    return out


def make_v0(rng: np.random.Generator, D: int, d: int) -> np.ndarray:
    """V0 (D x d, float32) with N(0, 1/d) entries."""
    v = rng.standard_normal((D, d), dtype=np.float32)
    v *= np.float32(1.0 / np.sqrt(d))
    return v


class ZipfSampler:
    """Inverse-CDF sampler of the truncated Zipf law p(i) ~ (i+1)^-s on [0, D)."""

    def __init__(self, D: int, s: float):
        w = np.arange(1, D + 1, dtype=np.float64) ** (-s)
        c = np.cumsum(w)
        self.cdf = c / c[-1]
        self.D = D

    def draw(self, rng: np.random.Generator, size) -> np.ndarray:
        u = rng.random(size)
        return np.minimum(np.searchsorted(self.cdf, u, side="right"), self.D - 1)

    def p(self, i: int) -> float:
        return float(self.cdf[i] - (self.cdf[i - 1] if i > 0 else 0.0))


def _distinct_rows(idx: np.ndarray, redraw) -> np.ndarray:
    """Redraw entries until every row of idx holds K distinct values."""
    m, K = idx.shape
    if K <= 1:
        return idx
    for j in range(m):
        row = idx[j]
        while len(np.unique(row)) < K:
            seen = set()
            for k in range(K):
                while int(row[k]) in seen:
                    row[k] = redraw()
                seen.add(int(row[k]))
        idx[j] = row
    return idx


def make_targets(rng: np.random.Generator, w: Workload, m: int | None = None,
                 zipf: ZipfSampler | None = None) -> tuple[np.ndarray, np.ndarray]:
    """(idx int32 m x K, val float32 m x K) for one minibatch."""
    m = w.m if m is None else m
    K = w.K
    if w.index_dist == "uniform":
        if K > w.D:
            raise ValueError("K distinct indices need K <= D")
        idx = rng.integers(0, w.D, size=(m, K), dtype=np.int64)
        idx = _distinct_rows(idx, lambda: int(rng.integers(0, w.D)))
    elif w.index_dist == "zipf":
        zipf = zipf or ZipfSampler(w.D, w.zipf_s)
        idx = zipf.draw(rng, (m, K)).astype(np.int64)
        idx = _distinct_rows(idx, lambda: int(zipf.draw(rng, 1)[0]))
    else:
        raise ValueError(w.index_dist)
    if w.value_dist == "normal":
        val = rng.standard_normal((m, K), dtype=np.float32)
    elif w.value_dist == "ones":
        val = np.ones((m, K), dtype=np.float32)
    else:
        raise ValueError(w.value_dist)
    return idx.astype(np.int32), val


def make_h(rng: np.random.Generator, m: int, d: int) -> np.ndarray:
    h = rng.standard_normal((m, d), dtype=np.float32)
    h *= np.float32(1.0 / np.sqrt(d))
    return h


class Stream:
    """Deterministic stream: V0 first, then per step H, idx, val from one PCG64."""

    def __init__(self, w: Workload, seed: int | None = None, with_v0: bool = True):
        self.w = w
        self.rng = np.random.default_rng(w.seed if seed is None else seed)
        self.zipf = ZipfSampler(w.D, w.zipf_s) if w.index_dist == "zipf" else None
        self.V0 = make_v0(self.rng, w.D, w.d) if with_v0 else None

    def batch(self, m: int | None = None):
        m = self.w.m if m is None else m
        H = make_h(self.rng, m, self.w.d)
        idx, val = make_targets(self.rng, self.w, m, self.zipf)
        return H, idx, val

    def batches(self, n: int) -> Iterator[tuple[np.ndarray, np.ndarray, np.ndarray]]:
        for _ in range(n):
            yield self.batch()
