"""Seeded synthetic inputs for the rotated W2A4 linear.

This module draws random numbers and nothing else: it holds no step of the
quantized-linear method (no rotation, no scale rule, no rounding to a level
set, no packing).  Both the CPU oracle's tests and the GPU benchmark take
their inputs from here, so that the two sides see identical bytes.

The paper's own workloads are LLaMA-2-7B and LLaMA-3.1-8B linears (Sec. 4.1)
whose rotated weights are near-Gaussian (Sec. 4.2) and whose activations carry
per-channel outliers (Sec. 3.1, activation-max figure).  The checkpoints and
calibration text are not available, so these generators stand in for them:

* weights  ``W = fp32(0.02 * Student-t(5))`` of shape ``[N, K]``;
* activations ``x = fp16(z * g)`` with ``z ~ N(0, 1)`` and a per-channel gain
  ``g`` that is 20 or 30 on a few seeded outlier channels and 1 elsewhere;
* for the throughput benchmark only, decoded integer levels drawn i.i.d. with
  the per-level shares that the paper's bucket table reports for the level
  set, and per-row fp16 scales near the value the row rule gives on these
  weights.

Every stream is ``PCG64(SeedSequence([0, cfg, layer, slot, kind]))``; the root
seed 0 mirrors the paper's calibration sampling seed.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

# kinds of random stream
KIND_W = 0        # fp32 weights
KIND_X = 1        # fp16 activations
KIND_OUTLIER = 2  # choice of outlier channels
KIND_LEVELS = 3   # benchmark-only level draws
KIND_SCALES = 4   # benchmark-only scale draws

# linear slots inside one transformer layer
LINEARS = ("q", "k", "v", "o", "gate", "up", "down")
LINEAR_ID = {name: i for i, name in enumerate(LINEARS)}
# the four activation sites that feed those linears
SITE_OF = {"q": 0, "k": 0, "v": 0, "o": 1, "gate": 2, "up": 2, "down": 3}

# level-set format ids (same numbering as the C ABI)
FMT_W2_MNZ = 0
FMT_W2_POT = 1
FMT_W4_SYM = 2


def rng(cfg: int, layer: int, slot: int, kind: int) -> np.random.Generator:
    """The seeded stream for one (config, layer, slot, kind)."""
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([0, cfg, layer, slot, kind])))


@dataclass(frozen=True)
class LinearShape:
    name: str
    N: int      # output features
    K: int      # input features
    block: int  # Hadamard block size for this linear's input


@dataclass(frozen=True)
class Config:
    idx: int
    label: str
    linears: tuple
    Ms: tuple
    layers: int
    fmt_of_layer: tuple            # level-set format per layer
    outlier_count: tuple = field(default=())   # per K: number of outlier channels
    outlier_gain: float = 20.0

    def n_outliers(self, K: int) -> int:
        if self.outlier_count == ("two",):
            return 2
        return int(round(0.01 * K))


def _llama2_layer():
    return (
        LinearShape("q", 4096, 4096, 4096), LinearShape("k", 4096, 4096, 4096),
        LinearShape("v", 4096, 4096, 4096), LinearShape("o", 4096, 4096, 4096),
        LinearShape("gate", 11008, 4096, 4096), LinearShape("up", 11008, 4096, 4096),
        LinearShape("down", 4096, 11008, 64),
    )


def _llama31_layer():
    return (
        LinearShape("q", 4096, 4096, 4096), LinearShape("k", 1024, 4096, 4096),
        LinearShape("v", 1024, 4096, 4096), LinearShape("o", 4096, 4096, 4096),
        LinearShape("gate", 14336, 4096, 4096), LinearShape("up", 14336, 4096, 4096),
        LinearShape("down", 4096, 14336, 2048),
    )


CONFIGS = {
    0: Config(0, "tiny single linear 512x256, M=4, MNZ",
              (LinearShape("lin", 512, 256, 256),), (4,), 1, (FMT_W2_MNZ,), ("two",), 20.0),
    1: Config(1, "LLaMA-2-7B layer decode, M=1, MNZ", _llama2_layer(), (1,), 1,
              (FMT_W2_MNZ,), ("two",), 20.0),
    2: Config(2, "LLaMA-3.1-8B 32-layer decode, M in {1,4,16}, MNZ", _llama31_layer(), (1, 4, 16), 32,
              (FMT_W2_MNZ,) * 32, ("pct",), 30.0),
    3: Config(3, "LLaMA-3.1-8B MLP, PoT-MNZ, M in {1,8,64}",
              tuple(s for s in _llama31_layer() if s.name in ("gate", "up", "down")), (1, 8, 64), 32,
              (FMT_W2_POT,) * 32, ("pct",), 30.0),
    4: Config(4, "LLaMA-3.1-8B prefill M=2048, layers 0-15 W4, 16-31 W2 MNZ", _llama31_layer(), (2048,), 32,
              (FMT_W4_SYM,) * 16 + (FMT_W2_MNZ,) * 16, ("pct",), 30.0),
}


def weights_fp32(cfg: int, layer: int, linear: str, N: int, K: int) -> np.ndarray:
    """Unrotated fp32 weights ``0.02 * t(5)``, shape [N, K] (out x in)."""
    g = rng(cfg, layer, LINEAR_ID.get(linear, 0), KIND_W)
    return (0.02 * g.standard_t(5, size=(N, K))).astype(np.float32)


def outlier_channels(cfg: int, layer: int, site: int, K: int, count: int) -> np.ndarray:
    """Sorted indices of ``count`` distinct outlier input channels."""
    g = rng(cfg, layer, site, KIND_OUTLIER)
    return np.sort(g.choice(K, size=count, replace=False))


def activations_fp16(cfg: int, layer: int, site: int, M: int, K: int,
                     n_outliers: int, gain: float) -> np.ndarray:
    """fp16 activations [M, K]: N(0,1) with ``n_outliers`` channels scaled by ``gain``."""
    g = rng(cfg, layer, site, KIND_X)
    z = g.standard_normal(size=(M, K))
    gains = np.ones(K)
    if n_outliers > 0:
        gains[outlier_channels(cfg, layer, site, K, n_outliers)] = gain
    return (z * gains[None, :]).astype(np.float16)


def config_activations(c: Config, layer: int, site: int, M: int, K: int) -> np.ndarray:
    return activations_fp16(c.idx, layer, site, M, K, c.n_outliers(K), c.outlier_gain)


# ---------------------------------------------------------------------------
# benchmark-only level and scale draws
# ---------------------------------------------------------------------------
# Per-level shares (ascending level order) from the paper's RTN bucket table
# (Table "bucket-summary", Sec. 4.5.1), used as categorical probabilities.
SHARES_MNZ = (15.95, 34.04, 34.05, 15.96)
SHARES_POT = (17.27, 32.72, 32.73, 17.27)
LEVELS_MNZ_HALF = (-3, -1, 1, 3)
LEVELS_POT = (-4, -1, 1, 4)
# W4: a discretized normal of standard deviation 1.93 level steps on -7..7.
W4_SD = 1.93

# nominal per-row scale of each format on 0.02*t(5) weights (RMS = 0.0258)
NOMINAL_SCALE = {FMT_W2_MNZ: 0.0129, FMT_W2_POT: 0.0099, FMT_W4_SYM: 0.0135}


def _level_table(fmt: int):
    if fmt == FMT_W2_MNZ:
        vals, p = LEVELS_MNZ_HALF, np.array(SHARES_MNZ)
    elif fmt == FMT_W2_POT:
        vals, p = LEVELS_POT, np.array(SHARES_POT)
    elif fmt == FMT_W4_SYM:
        vals = tuple(range(-7, 8))
        cdf = [0.5 * (1 + math.erf((v + 0.5) / (W4_SD * math.sqrt(2)))) for v in range(-8, 8)]
        p = np.diff(np.array(cdf))
        p[0] += cdf[0]
        p[-1] += 1 - cdf[-1]
    else:
        raise ValueError(f"unknown format {fmt}")
    p = np.asarray(p, dtype=np.float64)
    return np.asarray(vals, dtype=np.int8), p / p.sum()


def draw_levels(fmt: int, N: int, K: int, cfg: int = 0, layer: int = 0, slot: int = 0) -> np.ndarray:
    """int8 decoded levels [N, K] drawn i.i.d. from the format's level shares."""
    vals, p = _level_table(fmt)
    g = rng(cfg, layer, slot, KIND_LEVELS)
    u = g.random(size=(N, K))
    # bucket index = number of cumulative-share edges <= u (what a right-sided search returns)
    idx = np.zeros((N, K), dtype=np.int8)
    for e in np.cumsum(p)[:-1]:
        idx += u >= e
    return vals[idx]


def draw_scales(fmt: int, N: int, cfg: int = 0, layer: int = 0, slot: int = 0) -> np.ndarray:
    """fp16 per-row scales [N] spread log-normally (5%) around the nominal value."""
    g = rng(cfg, layer, slot, KIND_SCALES)
    return (NOMINAL_SCALE[fmt] * np.exp(0.05 * g.standard_normal(N))).astype(np.float16)


def draw_levels_torch(fmt: int, N: int, K: int, seed: int, device):
    """Device-side twin of :func:`draw_levels` for the large benchmark stacks.

    Same categorical distribution; a torch generator supplies the uniforms, so
    the bytes differ from the numpy draw.  Used only where no oracle compares.
    """
    import torch
    vals, p = _level_table(fmt)
    g = torch.Generator(device=device)
    g.manual_seed(int(seed))
    u = torch.rand((N, K), generator=g, device=device, dtype=torch.float32)
    edges = torch.tensor(np.cumsum(p)[:-1], dtype=torch.float32, device=device)
    idx = torch.bucketize(u, edges, right=True)
    del u
    return torch.tensor(vals, dtype=torch.int8, device=device)[idx]
