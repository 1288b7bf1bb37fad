"""Workload shapes for the PI-GAN training step.

Each workload fixes the two generator MLPs (log-conductivity Y and head u), the
discriminator MLP, the number of noise samples S, collocation points per sample
P, the Y/u sensor counts and the number of independent subdomain groups G.

The shapes follow the paper's problem statement: the generator takes one
spatial location plus the noise vector as a narrow input and the sensors of a
realisation become rows of a larger batch (Sec. III.C, "Single Node
optimizations"); the discriminator sees a whole sensor snapshot as one input
(same section); subdomains each own a discriminator and their loss terms are
weighted by 1/(levels * subdomains in the level) (Sec. III.B.1).
"""
from __future__ import annotations

from dataclasses import dataclass, replace


@dataclass(frozen=True)
class Workload:
    name: str
    dtype: str          # storage / MFMA operand type: "fp32", "bf16" or "fp16"
    G: int              # independent subdomain groups
    d: int              # spatial dimensions
    n_z: int            # noise dimension
    L: int              # generator hidden tanh layers
    W: int              # generator width
    S: int              # noise samples per step
    P: int              # collocation points per sample
    n_sY: int           # log-conductivity sensors
    n_sU: int           # head sensors
    L_D: int            # discriminator hidden tanh layers
    W_D: int            # discriminator width
    B_r: int            # real snapshots per step
    f_const: float      # source term used when no f array is given
    lambda_pde: float = 1.0
    seed: int = 1910
    arch: str = "pair"  # "pair": two tanh MLPs (Y, u); "trunk": one shared trunk, two heads;
                        # "hier": one pair and one critic per subdomain of a hierarchy;
                        # "hier_trunk": the shared trunk and one critic per subdomain
    sides: tuple = ()   # hier: grid side of each level (coarsest first)
    m_sensors: int = 0  # hier: Y (and u) sensors of every critic
    n_free: int = 0     # hier: free sensors of every critic

    @property
    def n_critics(self) -> int:
        return sum(k * k for k in self.sides) if self.is_hier else self.G

    @property
    def is_hier(self) -> bool:
        return self.arch in ("hier", "hier_trunk")

    @property
    def trunk_gen(self) -> bool:
        return self.arch in ("trunk", "hier_trunk")

    @property
    def n_in_hier(self) -> int:
        return 2 * self.m_sensors + self.n_free * (1 + self.d)

    @property
    def n_in(self) -> int:
        return self.n_sY + self.n_sU

    @property
    def in_dim(self) -> int:
        return self.d + self.n_z

    @property
    def c_Y(self) -> int:
        return 1 + self.d

    @property
    def c_U(self) -> int:
        return 1 + 2 * self.d

    @property
    def w_group(self) -> float:
        # one level of G subdomains: weight 1/(levels * subdomains)
        return 1.0 / self.G

    def gen_shape(self) -> tuple[int, int, int]:
        return (self.in_dim, self.L, self.W)

    def disc_shape(self) -> tuple[int, int, int]:
        return (self.n_in, self.L_D, self.W_D)

    def with_(self, **kw) -> "Workload":
        return replace(self, **kw)


def n_params(in_dim: int, L: int, W: int) -> int:
    """Parameter count of a tanh MLP packed as
    [W1 (W x in_dim, row-major), b1, W2 (W x W), b2, ..., W_L, b_L, w_out (W), b_out]."""
    return W * in_dim + W + (L - 1) * (W * W + W) + W + 1


def n_params_trunk(in_dim: int, L: int, W: int) -> int:
    """Parameter count of a shared trunk packed as
    [W1, b1, ..., W_L, b_L, w_Y (W), b_Y, w_u (W), b_u]."""
    return n_params(in_dim, L, W) + W + 1


C1 = Workload("darcy1d_toy_fp32", "fp32", G=1, d=1, n_z=4, L=3, W=32, S=64, P=32,
              n_sY=8, n_sU=8, L_D=2, W_D=32, B_r=64, f_const=1.0, seed=1911)
C2 = Workload("darcy2d_w128_bf16", "bf16", G=1, d=2, n_z=20, L=4, W=128, S=256, P=1024,
              n_sY=200, n_sU=200, L_D=3, W_D=256, B_r=256, f_const=0.0, seed=1912)
C3 = Workload("darcy2d_sd1000_w512_bf16", "bf16", G=1, d=2, n_z=64, L=6, W=512, S=512, P=4096,
              n_sY=1000, n_sU=1000, L_D=4, W_D=1024, B_r=512, f_const=0.0, seed=1913)
C4 = Workload("subdomains16_w256_bf16", "bf16", G=16, d=2, n_z=32, L=4, W=256, S=128, P=1024,
              n_sY=125, n_sU=125, L_D=3, W_D=512, B_r=128, f_const=0.0, seed=1914)
C5 = Workload("bigstep_w1024_disc2048_bf16", "bf16", G=1, d=2, n_z=128, L=6, W=1024, S=1024,
              P=2048, n_sY=4096, n_sU=4096, L_D=5, W_D=2048, B_r=1024, f_const=0.0, seed=1915)
C5H = C5.with_(name="bigstep_w1024_disc2048_fp16", dtype="fp16")

# The paper's own generator: one shared trunk of 5 x 128, 11 x 512 or 21 x 1024
# tanh layers (Sec. III.C) with residual blocks and two heads, on the sample,
# point and sensor counts of the 2-D, thousand-sensor and large-step workloads.
T5 = C2.with_(name="trunk5x128_darcy2d_bf16", L=5, arch="trunk", seed=1921)
T11 = C3.with_(name="trunk11x512_sd1000_bf16", L=11, arch="trunk", seed=1922)
T21 = C5.with_(name="trunk21x1024_bigstep_bf16", L=21, arch="trunk", seed=1923)

# Domain decomposition (Sec. III.B.1): the 2-D workload's generator pair and
# samples, 1 + 4 + 16 subdomain critics (3 x 256 each) on the paper's snapshot
# (16 Y + 16 u sensors, 16 free sensors with their coordinates), no residual
# penalty (the source enters through the critics).
H2 = C2.with_(name="hier21_darcy2d_bf16", n_sY=256, n_sU=256, lambda_pde=0.0, arch="hier", sides=(1, 2, 4),
              m_sensors=16, n_free=16, seed=1931)

# The paper's full method on the 2-D workload: the shared 5 x 128 trunk and
# the same 1 + 4 + 16 subdomain critics.
HT5 = H2.with_(name="hier21_trunk5x128_darcy2d_bf16", L=5, arch="hier_trunk", seed=1932)

# A hierarchy at the scale of the paper's finest level (hundreds of
# subdomains): 1 + 16 + 256 critics of 3 x 256, each on 4 Y + 4 u sensors and
# 4 free sensors of its subdomain (coarse levels take evenly spaced cells).
H273 = H2.with_(name="hier273_darcy2d_bf16", n_sY=1024, n_sU=1024, sides=(1, 4, 16), m_sensors=4, n_free=4,
                seed=1933)

WORKLOADS = {w.name: w for w in (C1, C2, C3, C4, C5, C5H, T5, T11, T21, H2, HT5, H273)}
ALIASES = {"c1": C1, "c2": C2, "c3": C3, "c4": C4, "c5": C5, "c5h": C5H, "t5": T5, "t11": T11, "t21": T21,
           "h2": H2, "ht5": HT5, "h273": H273}


def get(name: str) -> Workload:
    key = name.lower()
    if key in ALIASES:
        return ALIASES[key]
    return WORKLOADS[name]
