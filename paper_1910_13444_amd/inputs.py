"""Seeded synthetic inputs for the PI-GAN training step.

This module is shared by the HIP path's tests and benchmark and by the CPU
oracle's tests.  It draws random numbers only; it holds none of the method's
arithmetic (no network evaluation, no derivatives, no losses).

Recipe (stands in for the paper's Hanford datasets, which are not available):
  * sensor locations x ~ U[0,1]^d, fixed per seed and shared by every sample;
  * collocation points x ~ U[0,1]^d drawn independently per sample (the paper
    redraws its free f-sensors for every realisation, Sec. III.A.1);
  * noise z ~ N(0, I_{n_z}) per sample; the teacher has its own noise z';
  * generator, discriminator and teacher weights are Glorot-normal,
    std = sqrt(2 / (fan_in + fan_out)), untruncated, with zero biases.
All arrays are float32 (what the device path consumes).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .configs import Workload, n_params, n_params_trunk

_ROLES = ("genY", "genU", "disc", "teachY", "teachU", "z", "z_teach", "xc", "xsY", "xsU", "f")


def _rngs(seed: int) -> dict[str, np.random.Generator]:
    kids = np.random.SeedSequence(seed).spawn(len(_ROLES))
    return {r: np.random.default_rng(k) for r, k in zip(_ROLES, kids)}


def glorot_mlp(rng: np.random.Generator, in_dim: int, L: int, W: int) -> np.ndarray:
    """One packed parameter vector [W1, b1, ..., W_L, b_L, w_out, b_out] (float32)."""
    out = np.zeros(n_params(in_dim, L, W), dtype=np.float32)
    off = 0
    fan_in = in_dim
    for _ in range(L):
        std = np.sqrt(2.0 / (fan_in + W))
        out[off:off + W * fan_in] = rng.standard_normal(W * fan_in) * std
        off += W * fan_in + W          # bias stays zero
        fan_in = W
    std = np.sqrt(2.0 / (W + 1))
    out[off:off + W] = rng.standard_normal(W) * std
    return out


def glorot_trunk(rng: np.random.Generator, in_dim: int, L: int, W: int) -> np.ndarray:
    """One packed trunk vector [W1, b1, ..., W_L, b_L, w_Y, b_Y, w_u, b_u] (float32):
    Glorot-normal layers as glorot_mlp, the two heads as one 2 x W matrix."""
    out = np.zeros(n_params_trunk(in_dim, L, W), dtype=np.float32)
    off = 0
    fan_in = in_dim
    for _ in range(L):
        std = np.sqrt(2.0 / (fan_in + W))
        out[off:off + W * fan_in] = rng.standard_normal(W * fan_in) * std
        off += W * fan_in + W
        fan_in = W
    std = np.sqrt(2.0 / (W + 2))
    for _ in range(2):
        out[off:off + W] = rng.standard_normal(W) * std
        off += W + 1
    return out


@dataclass
class StepInputs:
    """Everything one training step consumes except the real snapshots."""
    pY: np.ndarray        # [G, nY]   fp32 master weights of the Y generator
    pU: np.ndarray        # [G, nU]
    pD: np.ndarray        # [G, nD]
    tY: np.ndarray        # [G, nY]   teacher weights (produce the "real" snapshots)
    tU: np.ndarray        # [G, nU]
    z: np.ndarray         # [G, S, n_z]
    z_teach: np.ndarray   # [G, B_r, n_z]
    xc: np.ndarray        # [G, S, P, d]
    xsY: np.ndarray       # [G, n_sY, d]
    xsU: np.ndarray       # [G, n_sU, d]
    f: np.ndarray | None  # [G, S, P] or None (then f_const is used)
    f_const: float
    w_group: np.ndarray   # [G]
    pT: np.ndarray | None = None   # [G, nT] shared-trunk weights (trunk workloads; then pY..tU are None)
    tT: np.ndarray | None = None   # [G, nT] teacher trunk


def make_inputs(wl: Workload, seed: int | None = None, f_array: bool = False,
                S: int | None = None, B_r: int | None = None) -> StepInputs:
    """Draw the inputs of one step.  ``S``/``B_r`` override the sample counts
    (a reduced-sample draw uses the same weights and sensor locations)."""
    seed = wl.seed if seed is None else seed
    S = wl.S if S is None else S
    B_r = wl.B_r if B_r is None else B_r
    r = _rngs(seed)
    G = wl.G

    def nets(rng, in_dim, L, W):
        return np.stack([glorot_mlp(rng, in_dim, L, W) for _ in range(G)])

    pT = tT = None
    if wl.arch == "trunk":
        pT = np.stack([glorot_trunk(r["genY"], wl.in_dim, wl.L, wl.W) for _ in range(G)])
        tT = np.stack([glorot_trunk(r["teachY"], wl.in_dim, wl.L, wl.W) for _ in range(G)])
        pY = pU = tY = tU = None
    else:
        pY = nets(r["genY"], wl.in_dim, wl.L, wl.W)
        pU = nets(r["genU"], wl.in_dim, wl.L, wl.W)
        tY = nets(r["teachY"], wl.in_dim, wl.L, wl.W)
        tU = nets(r["teachU"], wl.in_dim, wl.L, wl.W)
    pD = nets(r["disc"], wl.n_in, wl.L_D, wl.W_D)
    z = r["z"].standard_normal((G, S, wl.n_z)).astype(np.float32)
    zt = r["z_teach"].standard_normal((G, B_r, wl.n_z)).astype(np.float32)
    xc = r["xc"].random((G, S, wl.P, wl.d)).astype(np.float32)
    xsY = r["xsY"].random((G, wl.n_sY, wl.d)).astype(np.float32)
    xsU = r["xsU"].random((G, wl.n_sU, wl.d)).astype(np.float32)
    f = r["f"].standard_normal((G, S, wl.P)).astype(np.float32) if f_array else None
    wg = np.full((G,), wl.w_group, dtype=np.float32)
    return StepInputs(pY, pU, pD, tY, tU, z, zt, xc, xsY, xsU, f, wl.f_const, wg, pT, tT)
