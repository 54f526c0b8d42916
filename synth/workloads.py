"""Seeded synthetic workloads shaped like the paper's training setting.

The paper trains output layers with a vocabulary-sized sparse target
(D between 1e4 and 8e5 words, hidden size d around 300-500, minibatches of
m = 128; section 4 and Table 1).  Its corpus is not available here, so every
input is synthetic: each named configuration fixes D, d, m, K, the target index
distribution (uniform or bounded Zipf over a frequency-sorted vocabulary), the
target values, the scale of H and the initialisation of V and U.

Nothing in this module computes any part of the output-layer step; it draws
numbers only.  Every array is float32 / int32, C-contiguous, and is a pure
function of (configuration, seed, stream, step), so the CPU oracle and the GPU
library receive bit-identical inputs.
"""
from __future__ import annotations

import dataclasses
import math
from functools import lru_cache
from typing import Optional, Tuple

import numpy as np

# Base entropy for the named configurations: seed of configuration c is BASE + c.
BASE_ENTROPY = 14127091

# Independent random streams per workload.
_STREAM_INIT = 0
_STREAM_H = 1
_STREAM_Y = 2


@dataclasses.dataclass(frozen=True)
class WorkloadConfig:
    """Shape and distributions of one synthetic workload.

    idx_dist   'uniform' (each index equally likely) or 'zipf' (rank r = index+1
               has probability proportional to r**-zipf_s, r = 1..D).
    distinct   draw the K indices of an example without replacement.
    val_dist   'normal' (N(0,1)), 'one' (all 1.0) or 'poisson2p1' (Poisson(2)+1).
    h_scale    standard deviation of the N(0, h_scale^2) entries of H.
    v_bound    V0 entries are U(-v_bound, v_bound).
    u_init     'identity', 'random' (I + N(0, (0.3/sqrt(d))^2) entries; tests only) or
               'spectrum' (Q1 diag(s) Q2^T with Haar-random orthogonal Q1, Q2 and
               s = 1 except s[:len(u_sigma)] = u_sigma; tests only).
    pad_frac   fraction of target slots replaced by the padding index -1 (tests only).
    dup_frac   fraction of target slots that copy another slot's index of the same
               example, so that an index repeats inside one example (tests only).
    """

    name: str
    D: int
    d: int
    m: int
    K: int
    loss: str = "squared"  # 'squared' or 'spherical'
    lr: float = 1e-3
    steps: int = 1000
    idx_dist: str = "uniform"
    zipf_s: float = 1.0
    distinct: bool = True
    val_dist: str = "normal"
    h_scale: Optional[float] = None  # None means 1/sqrt(d)
    v_bound: Optional[float] = None  # None means 1/sqrt(d)
    u_init: str = "identity"
    u_sigma: Tuple[float, ...] = ()
    sph_eps: float = 1e-3
    pad_frac: float = 0.0
    dup_frac: float = 0.0
    entropy: int = BASE_ENTROPY

    @property
    def h_std(self) -> float:
        return self.h_scale if self.h_scale is not None else 1.0 / math.sqrt(self.d)

    @property
    def v_half_width(self) -> float:
        return self.v_bound if self.v_bound is not None else 1.0 / math.sqrt(self.d)

    def replace(self, **kw) -> "WorkloadConfig":
        return dataclasses.replace(self, **kw)


def _named_configs() -> dict:
    c1 = WorkloadConfig(
        name="c1_tiny_squared", D=2000, d=32, m=16, K=5, loss="squared", lr=0.01,
        steps=100, idx_dist="uniform", distinct=True, val_dist="normal",
        h_scale=1.0, v_bound=0.01, entropy=BASE_ENTROPY + 1,
    )
    # Same as c1 with H scaled by 1/sqrt(d): a well-conditioned diagnostic of c1.
    c1s = c1.replace(name="c1s_tiny_scaled", h_scale=None, entropy=BASE_ENTROPY + 11)
    c2 = WorkloadConfig(
        name="c2_paper_squared", D=200_000, d=500, m=128, K=10, loss="squared",
        lr=1e-3, steps=1000, idx_dist="uniform", distinct=True, val_dist="normal",
        entropy=BASE_ENTROPY + 2,
    )
    c3 = WorkloadConfig(
        name="c3_spherical_onehot", D=200_000, d=500, m=128, K=1, loss="spherical",
        lr=1e-3, steps=1000, idx_dist="zipf", zipf_s=1.0, distinct=True,
        val_dist="one", sph_eps=1e-3, entropy=BASE_ENTROPY + 3,
    )
    c4 = WorkloadConfig(
        name="c4_large_vocab_skew", D=1_000_000, d=512, m=256, K=64, loss="squared",
        lr=1e-3, steps=1000, idx_dist="zipf", zipf_s=1.1, distinct=True,
        val_dist="poisson2p1", entropy=BASE_ENTROPY + 4,
    )
    c5 = WorkloadConfig(
        name="c5_wide_large_batch", D=500_000, d=1024, m=512, K=32, loss="squared",
        lr=1e-3, steps=2000, idx_dist="uniform", distinct=True, val_dist="normal",
        entropy=BASE_ENTROPY + 5,
    )
    return {"c1": c1, "c1s": c1s, "c2": c2, "c3": c3, "c4": c4, "c5": c5}


CONFIGS = _named_configs()


def get_config(name: str, **overrides) -> WorkloadConfig:
    cfg = CONFIGS[name]
    return cfg.replace(**overrides) if overrides else cfg


@lru_cache(maxsize=8)
def _zipf_cdf(D: int, s: float) -> np.ndarray:
    ranks = np.arange(1, D + 1, dtype=np.float64)
    w = ranks ** (-s)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    return cdf


def bounded_zipf_sampler(D: int, s: float):
    """Inverse-CDF sampler of index = rank - 1 with P(rank r) proportional to r**-s, r = 1..D."""
    cdf = _zipf_cdf(int(D), float(s))

    def draw(rng: np.random.Generator, n: int) -> np.ndarray:
        u = rng.random(n)
        out = np.searchsorted(cdf, u, side="right")
        np.minimum(out, D - 1, out=out)
        return out.astype(np.int64)

    return draw


def _rng(cfg: WorkloadConfig, stream: int, step: int) -> np.random.Generator:
    ss = np.random.SeedSequence(entropy=cfg.entropy, spawn_key=(stream, step))
    return np.random.default_rng(ss)


class Workload:
    """Random access to the initial state and to the minibatch of every step."""

    def __init__(self, cfg: WorkloadConfig):
        self.cfg = cfg
        if cfg.idx_dist == "zipf":
            self._zipf = bounded_zipf_sampler(cfg.D, cfg.zipf_s)
        else:
            self._zipf = None

    # ---------------------------------------------------------------- init
    def init_V(self) -> np.ndarray:
        c = self.cfg
        rng = _rng(c, _STREAM_INIT, 0)
        V = rng.random((c.D, c.d), dtype=np.float32)
        a = np.float32(c.v_half_width)
        V *= np.float32(2.0) * a
        V -= a
        return V

    def init_U(self) -> np.ndarray:
        c = self.cfg
        if c.u_init == "identity":
            return np.eye(c.d, dtype=np.float32)
        if c.u_init == "random":
            rng = _rng(c, _STREAM_INIT, 1)
            U = np.eye(c.d) + rng.standard_normal((c.d, c.d)) * (0.3 / math.sqrt(c.d))
            return np.ascontiguousarray(U, dtype=np.float32)
        if c.u_init == "spectrum":
            rng = _rng(c, _STREAM_INIT, 2)
            s = np.ones(c.d)
            s[: len(c.u_sigma)] = c.u_sigma
            q = []
            for _ in range(2):
                a, r = np.linalg.qr(rng.standard_normal((c.d, c.d)))
                q.append(a * np.sign(np.diag(r)))
            return np.ascontiguousarray((q[0] * s) @ q[1].T, dtype=np.float32)
        raise ValueError(f"unknown u_init {c.u_init!r}")

    # ------------------------------------------------------------- batches
    def _draw_indices(self, rng: np.random.Generator) -> np.ndarray:
        c = self.cfg
        if c.idx_dist == "uniform":
            draw = lambda n: rng.integers(0, c.D, size=n, dtype=np.int64)  # noqa: E731
        elif c.idx_dist == "zipf":
            draw = lambda n: self._zipf(rng, n)  # noqa: E731
        else:
            raise ValueError(f"unknown idx_dist {c.idx_dist!r}")
        if not c.distinct:
            return draw(c.m * c.K).reshape(c.m, c.K)
        if c.K > c.D:
            raise ValueError("cannot draw K distinct indices from fewer than K rows")
        out = np.empty((c.m, c.K), dtype=np.int64)
        for i in range(c.m):
            chosen: list = []
            seen: set = set()
            while len(chosen) < c.K:
                for v in draw(2 * c.K + 8).tolist():
                    if v not in seen:
                        seen.add(v)
                        chosen.append(v)
                        if len(chosen) == c.K:
                            break
            out[i] = chosen
        return out

    def _draw_values(self, rng: np.random.Generator) -> np.ndarray:
        c = self.cfg
        shape = (c.m, c.K)
        if c.val_dist == "normal":
            return rng.standard_normal(shape, dtype=np.float32)
        if c.val_dist == "one":
            return np.ones(shape, dtype=np.float32)
        if c.val_dist == "poisson2p1":
            return (rng.poisson(2.0, size=shape) + 1).astype(np.float32)
        raise ValueError(f"unknown val_dist {c.val_dist!r}")

    def batch(self, step: int) -> Tuple[np.ndarray, np.ndarray, np.ndarray]:
        """(H[m x d] float32, Y_idx[m x K] int32, Y_val[m x K] float32) of one step.

        Row i of H is the last hidden representation h of example i; row i of
        (Y_idx, Y_val) holds its K (index, value) target pairs, -1 = padding.
        """
        c = self.cfg
        rh = _rng(c, _STREAM_H, step)
        H = rh.standard_normal((c.m, c.d), dtype=np.float32)
        H *= np.float32(c.h_std)
        ry = _rng(c, _STREAM_Y, step)
        idx = self._draw_indices(ry)
        val = self._draw_values(ry)
        if c.dup_frac > 0.0 and c.K > 1:
            mask = ry.random((c.m, c.K)) < c.dup_frac
            mask[:, 0] = False
            src = ry.integers(0, c.K, size=(c.m, c.K))
            for i, k in zip(*np.nonzero(mask)):
                idx[i, k] = idx[i, src[i, k] % k]
        if c.pad_frac > 0.0:
            mask = ry.random((c.m, c.K)) < c.pad_frac
            idx[mask] = -1
        return (
            np.ascontiguousarray(H),
            np.ascontiguousarray(idx.astype(np.int32)),
            np.ascontiguousarray(val.astype(np.float32)),
        )
