"""Seeded synthetic inputs shared by the tests, the smoke check and the bench.

This module draws random numbers and shapes them like the activations of the
diffusion transformers the paper evaluates (PixArt-Sigma, SANA and
FLUX.1-schnell, Sec. 4.1): token-major bf16 matrices with heavy-tailed values
and a few outlier channels (the outlier problem the paper starts from, Sec. 1).
The real activations need model weights and prompt sets that are not
available, so these generators stand in for them; no item of any dataset is
used.  It holds none of the quantizer's arithmetic: it only produces inputs
(activations, Kronecker factors, SmoothQuant multipliers) for both the HIP
path and the oracle.

Recipe per workload (seed = SeedSequence(index).spawn(4) -> values, outlier
channels, outlier rows, factors):
  values      N(0,1) | Laplace(0,1) | Student-t(nu=3), drawn in fp64, scaled
              in fp32 by the outlier multipliers, rounded to bf16
              (round-to-nearest-even, torch CPU cast);
  outliers    round(frac * d) distinct channels times a factor; optionally
              round(frac_rows * M) distinct token rows times a factor;
  factors     A = I + 0.1 N(0,1) (a x a), B likewise (b x b), each redrawn
              until its 2-norm condition number is below 10; one shared pair
              or one pair per 32-column block.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

# name -> (index, M, d, dist, outlier channel frac, channel factor,
#          outlier row frac, row factor, (a, b), per_block_factors)
WORKLOADS = {
    "tiny_256x1152": (0, 256, 1152, "normal", 0.01, 30.0, 0.0, 1.0, (4, 8), False),
    "pixart_8192x1152": (1, 8192, 1152, "normal", 0.01, 30.0, 0.001, 10.0, (4, 8), False),
    "pixart_8192x4608": (1, 8192, 4608, "normal", 0.01, 30.0, 0.001, 10.0, (4, 8), False),
    "sana_4096x2240": (2, 4096, 2240, "laplace", 0.02, 20.0, 0.0, 1.0, (4, 8), False),
    "sana_4096x5600": (2, 4096, 5600, "laplace", 0.02, 20.0, 0.0, 1.0, (4, 8), False),
    "flux_4608x3072": (3, 4608, 3072, "student_t3", 0.005, 50.0, 0.0, 1.0, (4, 8), False),
    "flux_4608x12288": (3, 4608, 12288, "student_t3", 0.005, 50.0, 0.0, 1.0, (4, 8), False),
    "large_18432x12288": (4, 18432, 12288, "student_t3", 0.005, 50.0, 0.0, 1.0, (4, 8), True),
    "large_18432x12288_2x16": (4, 18432, 12288, "student_t3", 0.005, 50.0, 0.0, 1.0, (2, 16),
                               True),
}


@dataclass
class Workload:
    name: str
    X: np.ndarray            # [M, d] uint16 bf16 bit patterns
    A: np.ndarray            # [nfac, a, a] fp32
    B: np.ndarray            # [nfac, b, b] fp32
    mult: np.ndarray         # [d] fp32 SmoothQuant multipliers 1/s_c
    meta: dict = field(default_factory=dict)


def to_bf16_bits(x32: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round-to-nearest-even (torch CPU cast)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x32, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy()


def _draw(rng, dist, shape):
    if dist == "normal":
        return rng.standard_normal(shape)
    if dist == "laplace":
        return rng.laplace(0.0, 1.0, shape)
    if dist == "student_t3":
        return rng.standard_t(3.0, shape)
    raise ValueError(dist)


def activations(M, d, dist="normal", seed=0, chan_frac=0.01, chan_factor=30.0, row_frac=0.0,
                row_factor=1.0, seeds=None):
    """bf16 activation matrix [M, d] with outlier channels (and rows)."""
    if seeds is None:
        seeds = np.random.SeedSequence(seed).spawn(4)
    rv, rc, rr = (np.random.default_rng(s) for s in seeds[:3])
    x = _draw(rv, dist, (M, d)).astype(np.float32)
    n_ch = int(round(chan_frac * d))
    if n_ch > 0:
        ch = rc.choice(d, size=n_ch, replace=False)
        x[:, ch] *= np.float32(chan_factor)
    n_rows = int(round(row_frac * M))
    if n_rows > 0:
        rows = rr.choice(M, size=n_rows, replace=False)
        x[rows, :] *= np.float32(row_factor)
    return to_bf16_bits(x)


def near_identity(rng, n, count=1, max_cond=10.0):
    """`count` matrices I + 0.1 N(0,1) of size n x n, each with cond2 < max_cond."""
    out = np.empty((count, n, n), dtype=np.float32)
    for f in range(count):
        while True:
            m = np.eye(n) + 0.1 * rng.standard_normal((n, n))
            if np.linalg.cond(m) < max_cond:
                out[f] = m.astype(np.float32)
                break
    return out


def factors(a, b, nfac=1, seed=0, rng=None):
    """Kronecker factor pairs A [nfac, a, a], B [nfac, b, b]."""
    if rng is None:
        rng = np.random.default_rng(seed)
    A = near_identity(rng, a, nfac)
    B = near_identity(rng, b, nfac)
    return A, B


def lu_params(nfac=1, seed=0):
    """Random LU parameters (a_k, b_k, c_k) of five 2x2 factors per factor pair,
    [nfac, 5, 3] fp32: a_k = 1 + 0.15 N, b_k = 0.3 + 0.15 N, c_k = 0.15 N (a
    perturbed start in the spirit of a calibrated transform; every a_k stays
    well away from 0)."""
    rng = np.random.default_rng(seed)
    lu = (rng.normal(size=(nfac, 5, 3)) * 0.15).astype(np.float32)
    lu[..., 0] += np.float32(1.0)
    lu[..., 1] += np.float32(0.3)
    return lu


def weights(o, d, seed=0, chan_frac=0.01, chan_factor=4.0):
    """bf16 weight matrix [o, d] of a linear layer: N(0, 1/d) entries (the
    usual initialisation scale), with round(chan_frac * d) input channels
    scaled by chan_factor so that the weight side has outlier columns too."""
    rv, rc = (np.random.default_rng(s) for s in np.random.SeedSequence(seed).spawn(2))
    w = (rv.standard_normal((o, d)) / np.sqrt(d)).astype(np.float32)
    n_ch = int(round(chan_frac * d))
    if n_ch > 0:
        ch = rc.choice(d, size=n_ch, replace=False)
        w[:, ch] *= np.float32(chan_factor)
    return to_bf16_bits(w)


def calib_layer(R, o, d, seed=0, dist="student_t3", chan_frac=0.005, chan_factor=50.0):
    """A synthetic layer for the calibration of Sec. 3.3: calibration
    activations X [R, d] (R = samples x tokens, the FLUX recipe of
    ``activations``: Student-t(3) values and 0.5% outlier channels x50) and a
    weight W [o, d] (``weights``).  Returns (X, W) as bf16 bit patterns."""
    ss = np.random.SeedSequence([seed, 7]).spawn(2)
    X = activations(R, d, dist, chan_frac=chan_frac, chan_factor=chan_factor,
                    seeds=np.random.SeedSequence(ss[0].entropy).spawn(4))
    W = weights(o, d, seed=int(ss[1].generate_state(1)[0]))
    return X, W


def activations_device(R, d, seed=0, chan_frac=0.005, chan_factor=50.0, device="cuda", chunk=8192):
    """The FLUX activation recipe of ``activations`` drawn on the device with
    torch's generator, for sizes too large to draw on the host (calibration
    sets of 128 samples x 4608 tokens): Student-t(3) values as z / sqrt(chi2_3 / 3)
    (z and the three chi-square terms standard normal), round(chan_frac * d)
    channels times chan_factor, rounded to bf16.  Not bit-identical to
    ``activations`` (another generator); used for timing only."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    X = torch.empty((R, d), dtype=torch.bfloat16, device=device)
    ch = torch.randperm(d, generator=g, device=device)[: max(1, int(round(chan_frac * d)))]
    for r0 in range(0, R, chunk):
        r1 = min(R, r0 + chunk)
        z = torch.randn((r1 - r0, d), generator=g, device=device)
        c = (torch.randn((r1 - r0, d, 3), generator=g, device=device) ** 2).sum(-1) / 3.0
        t = z / c.sqrt()
        t[:, ch] *= chan_factor
        X[r0:r1] = t.to(torch.bfloat16)
    return X


def smoothquant_multipliers(X_bits: np.ndarray) -> np.ndarray:
    """Per-channel multipliers m_c = 1 / s_c with s_c = max_r |X[r, c]|^0.5
    (migration strength alpha = 0.5, beta = 0), computed in fp64 and rounded
    to fp32; an all-zero channel gets 1."""
    x = (X_bits.astype(np.uint32) << 16).view(np.float32)
    amax = np.abs(x).max(axis=0).astype(np.float64)
    m = np.where(amax > 0, 1.0 / np.sqrt(np.where(amax > 0, amax, 1.0)), 1.0)
    return m.astype(np.float32)


def workload(name: str, rows: int | None = None) -> Workload:
    """Build a named workload; `rows` optionally truncates M (same seeds)."""
    idx, M, d, dist, cf, cfac, rf, rfac, (a, b), per_block = WORKLOADS[name]
    seeds = np.random.SeedSequence(idx).spawn(4)
    Mr = M if rows is None else min(rows, M)
    X = activations(M, d, dist, chan_frac=cf, chan_factor=cfac, row_frac=rf, row_factor=rfac,
                    seeds=seeds)
    if Mr != M:
        X = np.ascontiguousarray(X[:Mr])
    nfac = d // 32 if per_block else 1
    A, B = factors(a, b, nfac, rng=np.random.default_rng(seeds[3]))
    mult = smoothquant_multipliers(X)
    meta = {"index": idx, "M": Mr, "d": d, "dist": dist, "chan_frac": cf, "chan_factor": cfac,
            "row_frac": rf, "row_factor": rfac, "a": a, "b": b, "nfac": nfac,
            "seed": f"SeedSequence({idx}).spawn(4)"}
    return Workload(name, X, A, B, mult, meta)
