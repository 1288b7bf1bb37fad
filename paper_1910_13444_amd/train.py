"""Training loop on one GPU around the C-ABI training step.

Host logic only: every gradient and every parameter update runs in
libpigan.so kernels (pigan_train_step_grads, pigan_trunk_step_grads,
pigan_hier_step_grads or pigan_hier_trunk_step_grads, and pigan_adam_update)
on the current stream.

* fp32 master weights updated by Adam (the paper keeps single-precision
  master weights, Sec. III.C, and names no optimizer).
* Adaptive loss scaling (Sec. III.C): with dynamic scaling the step's
  non-finite flag is read after each call; a flagged step is skipped (the
  update kernel also reads the flag on the device), halves the scale, and
  `growth_interval` clean steps in a row double it.  Without dynamic scaling
  nothing is synchronised.
* Model-exchange schedules of the paper's generator and critic workers
  (Sec. III.D.2) on one device: "sequential" -- n_critic critic updates, then
  one generator update against the updated critic; "parallel" -- each network
  takes steps_per_exchange updates against the copy of the other it received
  at the last exchange, then the copies are exchanged (device copies).
* Optional critic gradient penalty (lambda_gp > 0, the WGAN-GP member of the
  critic family the paper cites, Sec. I.C, Sec. II.C): every step call takes
  fresh mixing weights, one per (critic, pair), uniform on [0, 1) from a
  seeded device generator (or from a caller's function of the call index).
"""
from __future__ import annotations

import ctypes as C
from dataclasses import dataclass

import torch

from . import pigan
from .configs import Workload


class Adam:
    """fp32 Adam state for one device parameter tensor."""

    def __init__(self, params: torch.Tensor, lr: float, beta1: float = 0.5, beta2: float = 0.9, eps: float = 1e-8):
        if params.dtype != torch.float32 or not params.is_cuda or not params.is_contiguous():
            raise ValueError("params must be a contiguous fp32 device tensor")
        self.p = params
        self.m = torch.zeros_like(params)
        self.v = torch.zeros_like(params)
        self.lr, self.beta1, self.beta2, self.eps = float(lr), float(beta1), float(beta2), float(eps)
        self.t = 0

    def step(self, grads: torch.Tensor, skip: torch.Tensor | None = None, count: bool = True):
        """Apply one update (skipped on the device when *skip != 0).  `count`
        advances the update counter (False when the host knows the step was
        skipped, so the bias correction follows the applied updates only)."""
        if count:
            self.t += 1
        t = max(self.t, 1)
        pigan._check(pigan.lib().pigan_adam_update(
            self.p.numel(), pigan._ptr(self.p, "params"), pigan._ptr(grads, "grads", self.p.numel()),
            pigan._ptr(self.m, "m"), pigan._ptr(self.v, "v"), self.lr, self.beta1, self.beta2, self.eps, t,
            None if skip is None else pigan._ptr(skip, "skip", 1, dtype=torch.int32), pigan._stream()))


class LossScaler:
    """Dynamic loss scale (halve on a non-finite step, double after
    growth_interval clean steps)."""

    def __init__(self, init_scale: float = 2.0 ** 15, growth_interval: int = 2000, min_scale: float = 1.0):
        self.scale = float(init_scale)
        self.growth_interval = int(growth_interval)
        self.min_scale = float(min_scale)
        self.good = 0

    def update(self, nonfinite: bool) -> bool:
        if nonfinite:
            self.scale = max(self.min_scale, self.scale * 0.5)
            self.good = 0
            return True
        self.good += 1
        if self.good >= self.growth_interval:
            self.scale *= 2.0
            self.good = 0
        return False


@dataclass
class TrainConfig:
    schedule: str = "sequential"       # or "parallel"
    n_critic: int = 1                  # sequential: critic updates per generator update
    steps_per_exchange: int = 1        # parallel: updates of each network between exchanges
    lr_g: float = 1e-4
    lr_d: float = 1e-4
    beta1: float = 0.5
    beta2: float = 0.9
    eps: float = 1e-8
    dynamic_loss_scale: bool = False   # fp16: adaptive loss scaling
    init_scale: float = 2.0 ** 15
    growth_interval: int = 2000
    chunk_S: int = 0
    lambda_gp: float = 0.0             # critic gradient penalty weight (0: none)
    gp_seed: int = 0                   # seed of the penalty's mixing weights


class Trainer:
    """Owns the master weights (generator: pY and pU, or the trunk pT; critic
    pD: [G, nD], or [D, nD] for the subdomain critics of a hierarchy), their
    Adam states, the loss scale and the schedule.  `inputs` are the batch's
    device tensors: z, xc, xsY, xsU, real, w_group (and optionally f); for a
    hierarchy (arch "hier" or "hier_trunk", one generator, no group axis) z,
    xc, xsY, xsU, real, idxY, idxU, idxF, w_disc (and optionally f).
    With cfg.lambda_gp > 0, gp_eps_fn(call_index) -> [critics, min(S, B_r)]
    fp32 device tensor supplies the penalty's mixing weights of each step
    call (default: uniform draws from a device generator seeded gp_seed)."""

    def __init__(self, wl: Workload, gen: list[torch.Tensor], pD: torch.Tensor, inputs: dict, cfg: TrainConfig,
                 gp_eps_fn=None):
        self.wl, self.cfg, self.inp = wl, cfg, inputs
        lgp = float(cfg.lambda_gp)
        self.trunk = wl.trunk_gen
        self.hier = wl.is_hier
        if cfg.schedule not in ("sequential", "parallel"):
            raise ValueError(f"unknown schedule {cfg.schedule!r}")
        if self.hier:
            S, B_r, D = inputs["z"].shape[0], inputs["real"].shape[1], inputs["w_disc"].shape[0]
            m = (inputs["idxY"].shape[1], inputs["idxU"].shape[1], inputs["idxF"].shape[1])
            if self.trunk:
                self.desc = pigan.hier_trunk_desc(wl, D, *m, S=S, B_r=B_r, chunk_S=cfg.chunk_S,
                                                  lambda_pde=wl.lambda_pde, lambda_gp=lgp)
                self.step_fn = pigan.HierTrunkStep(self.desc)
            else:
                self.desc = pigan.hier_desc(wl, D, *m, S=S, B_r=B_r, chunk_S=cfg.chunk_S, lambda_pde=wl.lambda_pde,
                                            lambda_gp=lgp)
                self.step_fn = pigan.HierStep(self.desc)
            n_crit = D
        elif self.trunk:
            S, B_r = inputs["z"].shape[1], inputs["real"].shape[1]
            self.desc = pigan.trunk_desc(wl, S=S, B_r=B_r, chunk_S=cfg.chunk_S, lambda_gp=lgp)
            self.step_fn = pigan.TrunkStep(self.desc)
            n_crit = inputs["z"].shape[0]
        else:
            S, B_r = inputs["z"].shape[1], inputs["real"].shape[1]
            self.desc = pigan.step_desc(wl, S=S, B_r=B_r, chunk_S=cfg.chunk_S, lambda_gp=lgp)
            self.step_fn = pigan.TrainStep(self.desc)
            n_crit = inputs["z"].shape[0]
        self.gp_shape = (n_crit, min(S, B_r))
        self.gp_eps_fn = gp_eps_fn
        self.gp_gen = None
        if lgp > 0 and gp_eps_fn is None:
            self.gp_gen = torch.Generator(device=inputs["z"].device)
            self.gp_gen.manual_seed(int(cfg.gp_seed))
        self.calls = 0
        self.gen = [g.contiguous() for g in gen]
        self.pD = pD.contiguous()
        self.opt_g = [Adam(g, cfg.lr_g, cfg.beta1, cfg.beta2, cfg.eps) for g in self.gen]
        self.opt_d = Adam(self.pD, cfg.lr_d, cfg.beta1, cfg.beta2, cfg.eps)
        self.scaler = LossScaler(cfg.init_scale, cfg.growth_interval) if cfg.dynamic_loss_scale else None
        self.losses: list[torch.Tensor] = []
        self.skipped = 0
        # parallel schedule: each worker's copy of the other network
        self.gen_copy = [g.clone() for g in self.gen]
        self.pD_copy = self.pD.clone()

    def _gp_eps(self):
        if self.cfg.lambda_gp <= 0:
            return None
        if self.gp_eps_fn is not None:
            return self.gp_eps_fn(self.calls)
        return torch.rand(self.gp_shape, generator=self.gp_gen, device=self.pD.device, dtype=torch.float32)

    def _call(self, gen, pD, critic_only=False):
        """One step call.  critic_only skips the generators' reverse pass (their
        gradients are then not computed: grads_g holds stale buffers) and, for
        the paired and trunk steps, their collocation rows and the residual
        (the call's L_pde is recorded as 0)."""
        if self.scaler is not None:
            self.desc.loss_scale = self.scaler.scale
        self.desc.critic_only = int(critic_only)
        i = self.inp
        eps = self._gp_eps()
        self.calls += 1
        if self.hier:
            idx = (i["idxY"], i["idxU"], i["idxF"], i["real"], i["w_disc"])
            if self.trunk:
                o = self.step_fn(gen[0], pD, i["z"], i["xc"], i["xsY"], i["xsU"], *idx, f=i.get("f"),
                                 f_const=self.wl.f_const, gp_eps=eps)
                grads_g = [o.gT]
            else:
                o = self.step_fn(gen[0], gen[1], pD, i["z"], i["xc"], i["xsY"], i["xsU"], *idx, f=i.get("f"),
                                 f_const=self.wl.f_const, gp_eps=eps)
                grads_g = [o.gY, o.gU]
        elif self.trunk:
            o = self.step_fn(gen[0], pD, i["z"], i["xc"], i["xsY"], i["xsU"], i["real"], f=i.get("f"),
                             f_const=self.wl.f_const, w_group=i["w_group"], gp_eps=eps)
            grads_g = [o.gT]
        else:
            o = self.step_fn(gen[0], gen[1], pD, i["z"], i["xc"], i["xsY"], i["xsU"], i["real"], f=i.get("f"),
                             f_const=self.wl.f_const, w_group=i["w_group"], gp_eps=eps)
            grads_g = [o.gY, o.gU]
        self.losses.append(o.loss.clone())
        skipped = False
        if self.scaler is not None:
            skipped = self.scaler.update(bool(o.nonfinite.item()))
            self.skipped += int(skipped)
        return o, grads_g, skipped

    def _update_g(self, grads_g, flag, skipped):
        for opt, g in zip(self.opt_g, grads_g):
            opt.step(g, skip=flag, count=not skipped)

    def _update_d(self, gD, flag, skipped):
        self.opt_d.step(gD, skip=flag, count=not skipped)

    def round(self):
        """One round of the schedule."""
        cfg = self.cfg
        if cfg.schedule == "sequential":
            for _ in range(cfg.n_critic):
                o, _, sk = self._call(self.gen, self.pD, critic_only=True)
                self._update_d(o.gD, o.nonfinite, sk)
            o, grads_g, sk = self._call(self.gen, self.pD)
            self._update_g(grads_g, o.nonfinite, sk)
        else:
            for _ in range(cfg.steps_per_exchange):
                o, grads_g, sk = self._call(self.gen, self.pD_copy)
                self._update_g(grads_g, o.nonfinite, sk)
                o, _, sk = self._call(self.gen_copy, self.pD, critic_only=True)
                self._update_d(o.gD, o.nonfinite, sk)
            for c, g in zip(self.gen_copy, self.gen):
                c.copy_(g)
            self.pD_copy.copy_(self.pD)

    def run(self, n_rounds: int) -> torch.Tensor:
        for _ in range(n_rounds):
            self.round()
        return torch.stack(self.losses) if self.losses else torch.empty(0)
