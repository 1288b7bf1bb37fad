"""Algorithmic work of one PI-GAN training step (what the method must compute).

Only matrix products count, at 2*M*N*K.  Not counted: tanh and the derivative
carry, the residual, reductions, weight casts, any recompute or chunking.

Generator (per network, per group), with value rows n_v = S*n_s + S*P and
stream rows R = S*n_s + c*S*P (c = 1+d for Y, 1+2d for u; sensor rows carry
the value stream only):
  forward   first layer x-part 2*d*W*n_v, z-part 2*n_z*W*S (once per sample),
            hidden 2*W^2*R per layer (L-1 layers), output 2*W*R
  backward  weight gradient and input cotangent of every hidden layer and the
            output layer (2x their forward), first-layer weight gradient
            (same count as its forward)
Domain decomposition: one generator pair and n_critics critics on
n_in = 2 m_sensors + n_free (1 + d) inputs each.
Shared trunk (trunk_flops): one network on R = S*(n_sY + n_sU) + (1+2d)*S*P
rows with a two-output head.
Discriminator on R_D = S + B_r rows:
  forward   2*R_D*(n_in*W_D + (L_D-1)*W_D^2 + W_D)
  backward  weight gradients (same as forward) + input cotangents of layers
            2..L_D and the output 2*R_D*((L_D-1)*W_D^2 + W_D) + first-layer
            input cotangent for the fake rows 2*S*n_in*W_D
"""
from __future__ import annotations

from .configs import Workload


def gen_flops(wl: Workload, c: int, n_s: int, S: int | None = None) -> float:
    S = wl.S if S is None else S
    W, L, d = wl.W, wl.L, wl.d
    n_v = S * n_s + S * wl.P
    R = S * n_s + c * S * wl.P
    first = 2.0 * d * W * n_v + 2.0 * wl.n_z * W * S
    rest = (L - 1) * 2.0 * W * W * R + 2.0 * W * R
    return 2.0 * first + 3.0 * rest


def disc_flops(wl: Workload, S: int | None = None, B_r: int | None = None) -> float:
    S = wl.S if S is None else S
    B_r = wl.B_r if B_r is None else B_r
    RD = S + B_r
    W, L = wl.W_D, wl.L_D
    n_in = wl.n_in_hier if wl.is_hier else wl.n_in
    fwd = 2.0 * RD * (n_in * W + (L - 1) * W * W + W)
    bwd = fwd + 2.0 * RD * ((L - 1) * W * W + W) + 2.0 * S * n_in * W
    return fwd + bwd


def trunk_flops(wl: Workload, S: int | None = None) -> float:
    """Shared trunk (one network, both sensor sets, 1 + 2d streams at the
    collocation points, a two-output head); the residual adds are not matrix
    work and are not counted."""
    S = wl.S if S is None else S
    W, L, d = wl.W, wl.L, wl.d
    n_s = wl.n_sY + wl.n_sU
    n_v = S * n_s + S * wl.P
    R = S * n_s + (1 + 2 * d) * S * wl.P
    first = 2.0 * d * W * n_v + 2.0 * wl.n_z * W * S
    rest = (L - 1) * 2.0 * W * W * R + 2.0 * 2 * W * R
    return 2.0 * first + 3.0 * rest


def step_flops(wl: Workload, S: int | None = None, B_r: int | None = None) -> float:
    """Algorithmic FLOPs of one training step over all groups."""
    if wl.trunk_gen:
        gen = trunk_flops(wl, S)
    else:
        gen = gen_flops(wl, wl.c_Y, wl.n_sY, S) + gen_flops(wl, wl.c_U, wl.n_sU, S)
    if wl.is_hier:   # one generator, one critic per subdomain
        return gen + wl.n_critics * disc_flops(wl, S, B_r)
    return wl.G * (gen + disc_flops(wl, S, B_r))


def collocation_points(wl: Workload, S: int | None = None) -> int:
    return wl.G * (wl.S if S is None else S) * wl.P
