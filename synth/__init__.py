"""Seeded synthetic inputs for the fused W4A4 + sparse-residual linear layer.

This module only draws random numbers: it produces the full-precision weight
``W`` (fp32, ``[N, K]``) and activation ``X`` (fp16, ``[M, K]``) of one linear
layer, plus the residual block budget of a workload.  It holds none of the
method's arithmetic (no quantisation, no residual, no block scoring): both the
CPU oracle and the GPU library receive these arrays as their inputs.

Recipe (synthetic stand-ins for the LLaMA3 / Qwen3 layers the paper measures;
the paper's real weights and calibration text are not available):

* ``W``: i.i.d. normal, standard deviation 0.02, fp32.  Each entry is
  independently an outlier with probability 0.005 and is then multiplied by 20
  (sign kept).
* ``X``: i.i.d. standard normal; 4 distinct seeded input channels are
  multiplied by 30; the result is rounded to fp16 (round to nearest even).
* Skewed variant (Qwen3-32B-shaped layers): 8 seeded 128-row output bands are
  "hot".  A designated set of ``nnzb`` 128x128 blocks is drawn, ``n_hot`` of
  them inside the bands and the rest outside; every outlier is placed inside a
  designated block (overall outlier count unchanged in expectation), so that
  residual-norm block selection returns exactly the designated set.
* Seeds: ``0x4D51 + 1000 * config + 10 * shape_index``; independent streams per
  tensor (``W`` = 0, outlier mask = 1, ``X`` = 2, channel picks = 3, skew
  bands = 4) via numpy's ``SeedSequence``.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Tuple

import numpy as np

BLOCK = 128          # residual block edge and weight group length along K
SIGMA_W = 0.02
P_OUTLIER = 0.005
OUTLIER_MULT = 20.0
N_OUTLIER_CH = 4
CH_MULT = 30.0

STREAM_W, STREAM_MASK, STREAM_X, STREAM_CH, STREAM_BANDS = 0, 1, 2, 3, 4


def seed_for(config: int, shape_index: int) -> int:
    return 0x4D51 + 1000 * config + 10 * shape_index


def _rng(seed: int, stream: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, stream]))


def budget(N: int, K: int, density_pct: float) -> int:
    """Residual block budget: floor(rho * NB * KB + 0.5), in exact arithmetic."""
    nblocks = (N // BLOCK) * (K // BLOCK)
    # density given in percent; use integer arithmetic where it is integral
    if float(density_pct).is_integer():
        return (int(density_pct) * nblocks + 50) // 100
    return int(np.floor(density_pct / 100.0 * nblocks + 0.5))


def gen_weight(N: int, K: int, seed: int,
               designated: Optional[np.ndarray] = None) -> np.ndarray:
    """fp32 weight [N, K].  ``designated``: optional bool [N/128, K/128] block
    mask; when given, all outliers fall inside the designated blocks."""
    w = _rng(seed, STREAM_W).standard_normal((N, K), dtype=np.float32)
    w *= np.float32(SIGMA_W)
    u = _rng(seed, STREAM_MASK).random((N, K), dtype=np.float32)
    if designated is None:
        mask = u < np.float32(P_OUTLIER)
    else:
        nb, kb = designated.shape
        n_des = int(designated.sum())
        if n_des == 0:
            return w
        p_in = min(1.0, P_OUTLIER * N * K / (n_des * BLOCK * BLOCK))
        inside = np.repeat(np.repeat(designated, BLOCK, axis=0), BLOCK, axis=1)
        mask = (u < np.float32(p_in)) & inside
    w[mask] *= np.float32(OUTLIER_MULT)
    return w


def gen_act(M: int, K: int, seed: int) -> np.ndarray:
    """fp16 activation [M, K] with N_OUTLIER_CH channels scaled by CH_MULT."""
    x = _rng(seed, STREAM_X).standard_normal((M, K), dtype=np.float32)
    ch = _rng(seed, STREAM_CH).choice(K, size=min(N_OUTLIER_CH, K), replace=False)
    x[:, ch] *= np.float32(CH_MULT)
    return x.astype(np.float16)


def skew_blocks(N: int, K: int, nnzb: int, seed: int,
                n_bands: int = 8, hot_frac: float = 0.8) -> Tuple[np.ndarray, int]:
    """Designated residual blocks for the skewed workload.

    Returns (bool mask [N/128, K/128], n_hot) where n_hot blocks lie in
    ``n_bands`` seeded block-rows and the remaining ``nnzb - n_hot`` elsewhere.
    """
    NB, KB = N // BLOCK, K // BLOCK
    rng = _rng(seed, STREAM_BANDS)
    n_bands = min(n_bands, NB)
    bands = np.sort(rng.choice(NB, size=n_bands, replace=False))
    in_band = np.zeros((NB, KB), dtype=bool)
    in_band[bands, :] = True
    band_idx = np.flatnonzero(in_band.ravel())
    out_idx = np.flatnonzero(~in_band.ravel())
    n_hot = min(int(round(hot_frac * nnzb)), band_idx.size)
    n_cold = nnzb - n_hot
    if n_cold > out_idx.size:          # tiny grids: top up the bands
        n_cold = out_idx.size
        n_hot = nnzb - n_cold
    pick = np.concatenate([
        rng.choice(band_idx, size=n_hot, replace=False),
        rng.choice(out_idx, size=n_cold, replace=False) if n_cold else np.zeros(0, np.int64),
    ])
    mask = np.zeros(NB * KB, dtype=bool)
    mask[pick] = True
    return mask.reshape(NB, KB), n_hot


@dataclass
class Layer:
    """One synthetic linear layer: weight shape, residual density and seed,
    with the token counts ``ms`` it is exercised at (same weights for every M)."""
    name: str
    K: int
    N: int
    density_pct: float
    seed: int
    ms: Tuple[int, ...]
    skewed: bool = False

    @property
    def nnzb(self) -> int:
        return budget(self.N, self.K, self.density_pct)

    def designated(self) -> Optional[np.ndarray]:
        if not self.skewed or self.nnzb == 0:
            return None
        return skew_blocks(self.N, self.K, self.nnzb, self.seed)[0]

    def weight(self) -> np.ndarray:
        return gen_weight(self.N, self.K, self.seed, designated=self.designated())

    def act(self, M: int) -> np.ndarray:
        return gen_act(M, self.K, self.seed)


def workloads() -> List[Layer]:
    """Every layer of the five workload families.

    1: single 1024->1024 layer, M=64.
    2: LLaMA3-8B attention projection 4096->4096, M in {1, 16, 256, 4096}.
    3: LLaMA3-8B MLP 4096->14336 and 14336->4096, M=4096, density {0,5,10,20}%
       (one weight per shape; the density only changes the budget).
    4: Qwen3-32B 5120->5120, 5120->1024 and MLP 5120<->25600, M in {1,32,2048},
       skewed residual placement.
    5: LLaMA3-70B MLP 8192->28672 and 28672->8192, M=8192.
    """
    out: List[Layer] = [Layer("c1_1024", 1024, 1024, 10, seed_for(1, 0), (64,))]
    out.append(Layer("c2_4096", 4096, 4096, 10, seed_for(2, 0), (1, 16, 256, 4096)))
    for i, (k, n, tag) in enumerate(((4096, 14336, "up"), (14336, 4096, "down"))):
        for d in (0, 5, 10, 20):
            out.append(Layer(f"c3_{tag}_d{d}", k, n, d, seed_for(3, i), (4096,)))
    for i, (k, n, tag) in enumerate(((5120, 5120, "qo"), (5120, 1024, "kv"),
                                     (5120, 25600, "up"), (25600, 5120, "down"))):
        out.append(Layer(f"c4_{tag}", k, n, 10, seed_for(4, i), (1, 32, 2048), skewed=True))
    for i, (k, n, tag) in enumerate(((8192, 28672, "up"), (28672, 8192, "down"))):
        out.append(Layer(f"c5_{tag}", k, n, 10, seed_for(5, i), (8192,)))
    return out


def table5_workloads() -> List[Layer]:
    """Qwen3-8B GEMM operators with concatenated outputs (the shapes of the
    paper's kernel-fusion latency table, out x in): qkv 6144 x 4096, o
    4096 x 4096, gate_up 24576 x 4096, down 4096 x 12288; 10 % residual
    density; prefill M = batch x 2048 tokens (the input length of the paper's
    serving runs) and decode M = batch, for batch 4, 8, 16, 32."""
    ms = (4, 8, 16, 32, 4 * 2048, 8 * 2048, 16 * 2048, 32 * 2048)
    out: List[Layer] = []
    for i, (k, n, tag) in enumerate(((4096, 6144, "qkv"), (4096, 4096, "o"),
                                     (4096, 24576, "gate_up"), (12288, 4096, "down"))):
        out.append(Layer(f"t5_{tag}", k, n, 10, seed_for(6, i), ms))
    return out


def workload(name: str) -> Layer:
    for w in workloads() + table5_workloads():
        if w.name == name:
            return w
    raise KeyError(name)
