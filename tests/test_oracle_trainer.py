"""Pins of the training-loop oracle (oracle/trainer.py): the Adam update
against torch.optim.Adam (an independent implementation), its first-step and
scale-invariance properties, descent on a convex quadratic, the loss scaler's
state machine, and which weights each schedule's gradient calls see."""
import numpy as np
import torch

from oracle.trainer import LossScaler, adam_update, train


def test_adam_matches_torch():
    rng = np.random.default_rng(0)
    p0 = rng.standard_normal(50)
    grads = [rng.standard_normal(50) * (1 + k) for k in range(7)]
    lr, b1, b2, eps = 3e-3, 0.5, 0.9, 1e-8
    p, m, v = p0.copy(), np.zeros(50), np.zeros(50)
    for t, g in enumerate(grads, 1):
        p, m, v = adam_update(p, g, m, v, t, lr, b1, b2, eps)
    pt = torch.tensor(p0, dtype=torch.float64, requires_grad=True)
    opt = torch.optim.Adam([pt], lr=lr, betas=(b1, b2), eps=eps)
    for g in grads:
        opt.zero_grad()
        pt.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
    assert np.allclose(p, pt.detach().numpy(), rtol=0, atol=1e-14)


def test_adam_first_step_moves_every_coordinate_by_lr():
    rng = np.random.default_rng(1)
    p0 = rng.standard_normal(20)
    g = rng.standard_normal(20)
    p1, _, _ = adam_update(p0, g, np.zeros(20), np.zeros(20), 1, 0.01, 0.9, 0.999, 0.0)
    assert np.allclose(p1, p0 - 0.01 * np.sign(g), rtol=0, atol=1e-15)


def test_adam_is_invariant_to_gradient_scale():
    rng = np.random.default_rng(2)
    p = q = rng.standard_normal(10)
    m1 = v1 = m2 = v2 = np.zeros(10)
    for t in range(1, 6):
        g = rng.standard_normal(10)
        p, m1, v1 = adam_update(p, g, m1, v1, t, 0.01, 0.5, 0.9, 0.0)
        q, m2, v2 = adam_update(q, 1024.0 * g, m2, v2, t, 0.01, 0.5, 0.9, 0.0)
    assert np.allclose(p, q, rtol=0, atol=1e-13)


def test_adam_descends_a_convex_quadratic():
    a = np.linspace(0.5, 5.0, 16)
    p = np.ones(16) * 2.0
    m = v = np.zeros(16)
    f0 = 0.5 * (a * p * p).sum()
    for t in range(1, 801):
        p, m, v = adam_update(p, a * p, m, v, t, 0.05, 0.9, 0.999, 1e-8)
    assert 0.5 * (a * p * p).sum() < f0 * 1e-3


def test_adam_skip_leaves_state():
    p, m, v = np.ones(3), np.full(3, 0.1), np.full(3, 0.2)
    q, mm, vv = adam_update(p, np.array([np.inf, 1.0, 2.0]), m, v, 4, 0.1, 0.5, 0.9, 1e-8, skip=True)
    assert np.array_equal(q, p) and np.array_equal(mm, m) and np.array_equal(vv, v)


def test_loss_scaler_state_machine():
    s = LossScaler(init_scale=1024.0, growth_interval=3, min_scale=1.0)
    assert s.update(True) and s.scale == 512.0
    assert not s.update(False) and not s.update(False) and s.scale == 512.0
    assert not s.update(False) and s.scale == 1024.0          # third finite step in a row doubles
    assert s.update(True) and s.scale == 512.0 and s.good == 0
    for _ in range(20):
        s.update(True)
    assert s.scale == 1.0                                       # clamped at min_scale


def _recording_game():
    """Bilinear game L = pG . A pD: records the (pG, pD) each call sees."""
    A = np.array([[1.0, 2.0], [-1.0, 0.5]])
    seen = []

    def step(pG, pD):
        seen.append((pG.copy(), pD.copy()))
        return np.zeros(3), A @ pD, A.T @ pG
    return step, seen


def test_sequential_schedule_uses_latest_weights():
    step, seen = _recording_game()
    pG, pD, losses = train(step, np.array([1.0, -1.0]), np.array([0.5, 2.0]), n_steps=2, schedule="sequential",
                           n_critic=2, lr_g=0.1, lr_d=0.1)
    assert len(seen) == 6 and len(losses) == 6
    # the critic changes between its two calls; the generator call sees the critic after both updates
    assert not np.array_equal(seen[0][1], seen[1][1])
    assert not np.array_equal(seen[1][1], seen[2][1])
    assert np.array_equal(seen[0][0], seen[2][0])              # generator unchanged until its own update
    assert not np.array_equal(seen[2][0], seen[3][0])


def test_parallel_schedule_trains_against_frozen_copies():
    step, seen = _recording_game()
    pG0, pD0 = np.array([1.0, -1.0]), np.array([0.5, 2.0])
    train(step, pG0, pD0, n_steps=2, schedule="parallel", steps_per_exchange=3, lr_g=0.1, lr_d=0.1)
    assert len(seen) == 12
    first = seen[:6]
    # generator calls (even) see the critic copy of the last exchange; critic calls (odd) the generator copy
    assert all(np.array_equal(c[1], pD0) for c in first[0::2])
    assert all(np.array_equal(c[0], pG0) for c in first[1::2])
    assert not np.array_equal(first[0][0], first[2][0])        # each network does move between exchanges
    assert not np.array_equal(first[1][1], first[3][1])
    second = seen[6:]
    # after the exchange both copies are the other network's latest weights
    assert np.array_equal(second[0][1], second[1][1]) and np.array_equal(second[0][0], second[1][0])
