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


# ---------------------------------------------------------------------------
# Hierarchical subdomains (Sec. III.B.1, domain decomposition): one generator,
# one discriminator per subdomain of every level, all levels partitioning the
# whole domain.  Stand-in for the paper's METIS partitions of the Hanford site:
# nested regular grids of the unit square with sides `sides` (e.g. 1, 2, 4 ->
# 1 + 4 + 16 subdomains).  Sensors and collocation points are stratified over
# the finest grid's cells (the same count in every cell), so every
# discriminator can take the same number of sensors from its subdomain
# (coarser levels take sparser subsets, as the paper balances them).
# ---------------------------------------------------------------------------

@dataclass
class Hierarchy:
    sides: tuple            # grid side per level, coarsest first; each divides the finest
    idxY: np.ndarray        # [D, mY] int32 indices into the Y sensors
    idxU: np.ndarray        # [D, mU] int32 indices into the u sensors
    idxF: np.ndarray        # [D, nF] int32 indices into each sample's collocation points (free sensors)
    w: np.ndarray           # [D] float32 weight 1 / (levels * subdomains of the level)
    level: np.ndarray       # [D] level of each discriminator

    @property
    def D(self) -> int:
        return int(self.idxY.shape[0])


def _cells_of(side: int, fine: int, ci: int, cj: int) -> list[int]:
    """Finest cells (row-major index) inside subdomain (ci, cj) of a side x side grid."""
    r = fine // side
    return [(ci * r + a) * fine + (cj * r + b) for a in range(r) for b in range(r)]


def _pick(side: int, fine: int, ci: int, cj: int, m: int, per_cell: int) -> list[int]:
    """m indices (sensors or points, per_cell per finest cell) spread evenly
    over subdomain (ci, cj): m / k from each of its k cells when m >= k, else
    the first one of every cell of an evenly spaced q x q sub-grid (m = q^2)."""
    cells = _cells_of(side, fine, ci, cj)
    k = len(cells)
    if m >= k:
        if m % k or m // k > per_cell:
            raise ValueError("sensor or point counts do not divide over the subdomain's cells")
        return [c * per_cell + j for c in cells for j in range(m // k)]
    r = fine // side
    q = int(round(m ** 0.5))
    if q * q != m or r % q:
        raise ValueError("a subdomain with more cells than picks needs a square pick count dividing its side")
    st = r // q
    return [((ci * r + a * st + st // 2) * fine + (cj * r + b * st + st // 2)) * per_cell
            for a in range(q) for b in range(q)]


def make_hierarchy(sides, m_sensors: int, n_free: int, per_cell_sensors: int, per_cell_points: int) -> Hierarchy:
    """Index lists of every subdomain's discriminator.  Sensors of finest cell
    c are c * per_cell_sensors + [0, per_cell_sensors); points of cell c are
    c * per_cell_points + [0, per_cell_points).  A subdomain covering k cells
    takes m_sensors / k sensors and n_free / k points from each (the first
    ones), or, when it has more cells than picks, one from each cell of an
    evenly spaced sub-grid (so hundreds of finest subdomains still leave the
    coarse critics a modest input)."""
    fine = sides[-1]
    idxY, idxF, w, level = [], [], [], []
    for lv, side in enumerate(sides):
        for ci in range(side):
            for cj in range(side):
                idxY.append(_pick(side, fine, ci, cj, m_sensors, per_cell_sensors))
                idxF.append(_pick(side, fine, ci, cj, n_free, per_cell_points))
                w.append(1.0 / (len(sides) * side * side))
                level.append(lv)
    idxY = np.array(idxY, np.int32)
    return Hierarchy(tuple(sides), idxY, idxY.copy(), np.array(idxF, np.int32), np.array(w, np.float32),
                     np.array(level, np.int32))


def stratified_points(rng: np.random.Generator, lead: tuple, fine: int, per_cell: int) -> np.ndarray:
    """[*lead, fine*fine*per_cell, 2] points, per_cell uniform points in each
    cell of a fine x fine grid of the unit square (cell-major order)."""
    u = rng.random(lead + (fine * fine, per_cell, 2))
    ci = np.arange(fine * fine) // fine
    cj = np.arange(fine * fine) % fine
    off = np.stack([ci, cj], axis=-1).astype(np.float64)[:, None, :]
    return ((off + u) / fine).reshape(lead + (fine * fine * per_cell, 2)).astype(np.float32)


@dataclass
class HierInputs:
    base: StepInputs        # weights (G = 1 generator pair), z, stratified xc / xsY / xsU, f
    hier: Hierarchy
    pD: np.ndarray          # [D, nD] one critic per subdomain
    xf_real: np.ndarray     # [B_r, P, 2] free-sensor locations of the real snapshots


def make_hier_inputs(wl: Workload, sides=(1, 2, 4), m_sensors: int = 16, n_free: int = 16,
                     seed: int | None = None, S: int | None = None, B_r: int | None = None) -> HierInputs:
    """Inputs of a hierarchical step (2-D): the workload's generator pair (or,
    for arch "hier_trunk", a shared trunk in base.pT / base.tT) and sample
    counts; sensors and collocation points stratified over the finest
    cells (n_sY, n_sU and P must be multiples of the cell count); one
    Glorot-normal critic per subdomain on n_in = 2 m_sensors + n_free (1 + d)."""
    if wl.d != 2:
        raise ValueError("the hierarchy is built on the unit square (d = 2)")
    fine = sides[-1]
    cells = fine * fine
    if wl.n_sY % cells or wl.n_sU % cells or wl.P % cells:
        raise ValueError("n_sY, n_sU and P must be multiples of the finest cell count")
    seed = wl.seed if seed is None else seed
    base = make_inputs(wl.with_(arch="trunk" if wl.trunk_gen else "pair"), seed=seed, S=S, B_r=B_r)
    r = np.random.default_rng(np.random.SeedSequence(seed).spawn(len(_ROLES) + 2)[-1])
    Sn, G = base.z.shape[1], base.z.shape[0]
    base.xsY = stratified_points(r, (G,), fine, wl.n_sY // cells)
    base.xsU = stratified_points(r, (G,), fine, wl.n_sU // cells)
    base.xc = stratified_points(r, (G, Sn), fine, wl.P // cells)
    hier = make_hierarchy(sides, m_sensors, n_free, min(wl.n_sY, wl.n_sU) // cells, wl.P // cells)
    n_in = 2 * m_sensors + n_free * (1 + wl.d)
    rd = np.random.default_rng(np.random.SeedSequence(seed).spawn(len(_ROLES) + 3)[-1])
    pD = np.stack([glorot_mlp(rd, n_in, wl.L_D, wl.W_D) for _ in range(hier.D)])
    xf_real = stratified_points(rd, (base.z_teach.shape[1],), fine, wl.P // cells)
    return HierInputs(base, hier, pD, xf_real)
