"""fp64 oracle of the training loop around the step (TEST INFRASTRUCTURE: only
the tests may import it; it shares no code with the HIP path).

* Parameter update on fp32 master weights (Sec. III.C keeps a single-precision
  copy of the weights and accumulates gradients in it).  The paper names no
  optimizer; the update is Adam (Kingma and Ba, 2015) in its textbook form:
  m = b1 m + (1 - b1) g, v = b2 v + (1 - b2) g^2, and
  p = p - lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps).
  A step whose gradient is not finite leaves p, m and v unchanged.
* Adaptive loss scaling (Sec. III.C): the loss is multiplied by a scale before
  the reverse pass and the gradients divided by it; a step with a non-finite
  gradient is skipped and halves the scale, and `growth_interval` finite steps
  in a row double it.
* Model-exchange schedules (Sec. III.D.2, "Model Exchange") on one device:
  sequential -- the critic is trained for n_critic steps, then the generator
  against the updated critic; parallel -- both train for `steps_per_exchange`
  steps against the copy of the other network they received at the last
  exchange, then the copies are exchanged.
"""
from __future__ import annotations

import numpy as np


def adam_update(p, g, m, v, t: int, lr: float, beta1: float, beta2: float, eps: float, skip: bool = False):
    """One Adam update (t >= 1 counts the updates including this one).
    Returns new (p, m, v); unchanged when skip."""
    p = np.asarray(p, np.float64)
    if skip:
        return p.copy(), np.asarray(m, np.float64).copy(), np.asarray(v, np.float64).copy()
    g = np.asarray(g, np.float64)
    m = beta1 * np.asarray(m, np.float64) + (1.0 - beta1) * g
    v = beta2 * np.asarray(v, np.float64) + (1.0 - beta2) * g * g
    mhat = m / (1.0 - beta1 ** t)
    vhat = v / (1.0 - beta2 ** t)
    return p - lr * mhat / (np.sqrt(vhat) + eps), m, v


class LossScaler:
    """Dynamic loss scale: halve on a non-finite step (which is skipped),
    double after `growth_interval` finite steps in a row."""

    def __init__(self, init_scale: float = 2.0 ** 15, growth_interval: int = 2000, min_scale: float = 1.0):
        self.scale = float(init_scale)
        self.growth_interval = int(growth_interval)
        self.min_scale = float(min_scale)
        self.good = 0

    def update(self, nonfinite: bool) -> bool:
        """Record one step; returns True when the step must be skipped."""
        if nonfinite:
            self.scale = max(self.min_scale, self.scale * 0.5)
            self.good = 0
            return True
        self.good += 1
        if self.good >= self.growth_interval:
            self.scale *= 2.0
            self.good = 0
        return False


def train(step_fn, pG, pD, n_steps: int, schedule: str = "sequential", n_critic: int = 1,
          steps_per_exchange: int = 1, lr_g: float = 1e-4, lr_d: float = 1e-4, beta1: float = 0.5,
          beta2: float = 0.9, eps: float = 1e-8):
    """Run `n_steps` rounds of the schedule.

    step_fn(pG, pD) -> (loss[3], gG, gD): gradients of L_G w.r.t. the generator
    weights pG and of L_D w.r.t. the critic weights pD at the same batch.
    Sequential: a round is n_critic critic updates, then one generator update
    (each with the latest weights).  Parallel: a round is steps_per_exchange
    updates of each network against its frozen copy of the other, then the
    exchange.  Returns (pG, pD, losses) with the losses of every step call.
    """
    pG = np.asarray(pG, np.float64).copy()
    pD = np.asarray(pD, np.float64).copy()
    mG, vG = np.zeros_like(pG), np.zeros_like(pG)
    mD, vD = np.zeros_like(pD), np.zeros_like(pD)
    tG = tD = 0
    losses = []
    for _ in range(n_steps):
        if schedule == "sequential":
            for _ in range(n_critic):
                loss, _, gD = step_fn(pG, pD)
                losses.append(loss)
                tD += 1
                pD, mD, vD = adam_update(pD, gD, mD, vD, tD, lr_d, beta1, beta2, eps)
            loss, gG, _ = step_fn(pG, pD)
            losses.append(loss)
            tG += 1
            pG, mG, vG = adam_update(pG, gG, mG, vG, tG, lr_g, beta1, beta2, eps)
        elif schedule == "parallel":
            D_seen_by_G = pD.copy()      # the generator worker's copy of the critic
            G_seen_by_D = pG.copy()      # the critic worker's copy of the generator
            for _ in range(steps_per_exchange):
                loss, gG, _ = step_fn(pG, D_seen_by_G)
                losses.append(loss)
                tG += 1
                pG, mG, vG = adam_update(pG, gG, mG, vG, tG, lr_g, beta1, beta2, eps)
                loss, _, gD = step_fn(G_seen_by_D, pD)
                losses.append(loss)
                tD += 1
                pD, mD, vD = adam_update(pD, gD, mD, vD, tD, lr_d, beta1, beta2, eps)
        else:
            raise ValueError(f"unknown schedule {schedule!r}")
    return pG, pD, np.array(losses)
