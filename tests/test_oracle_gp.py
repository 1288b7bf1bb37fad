"""Pins of the oracle's critic gradient penalty
P = w lambda mean_b (||grad_v D(x_b)|| - 1)^2, x_b = eps_b R_b + (1 - eps_b) F_b:

* the input gradient against central differences of D in input space;
* P and dP/dphi against a single-layer closed form written out directly;
* dP/dphi against central differences of P over every critic weight;
* dP/dphi against torch.autograd double reverse mode (create_graph=True);
* invariants: eps = 1 makes P independent of the fake rows, P is linear in
  lambda and w, and the penalty term of the step is additive over chunks."""
import numpy as np
import pytest
import torch

import oracle
from paper_1910_13444_amd.inputs import glorot_mlp

SHAPE = (5, 2, 4)          # n_in, hidden layers, width


def _net(seed, shape=SHAPE, scale=1.0):
    rng = np.random.default_rng(seed)
    p = glorot_mlp(rng, *shape).astype(np.float64) * scale
    n_in, L, W = shape
    # non-zero biases so no layer is odd-symmetric
    layers, wo, bo = oracle.unpack(p, n_in, L, W)
    p = oracle.pack([(Wl, rng.standard_normal(W) * 0.3) for Wl, _ in layers], wo, 0.2)
    return p


def _pair(seed, n, n_in):
    rng = np.random.default_rng(seed)
    return rng.standard_normal((n, n_in)), rng.standard_normal((n, n_in)), rng.random(n)


def test_input_grad_matches_finite_differences():
    p = _net(1)
    X = np.random.default_rng(2).standard_normal((3, SHAPE[0]))
    g = oracle.critic_input_grad(p, SHAPE, X)
    h = 1e-6
    fd = np.zeros_like(X)
    for i in range(SHAPE[0]):
        e = np.zeros(SHAPE[0])
        e[i] = h
        fd[:, i] = (oracle.mlp_forward(p, SHAPE, X + e) - oracle.mlp_forward(p, SHAPE, X - e)) / (2 * h)
    assert np.abs(g - fd).max() < 1e-8 * max(1.0, np.abs(fd).max())


def test_single_layer_closed_form():
    # D(v) = w . tanh(A v + b) + c  =>  grad_v D = A^T (w * (1 - tanh^2(A v + b)))
    shape = (3, 1, 4)
    rng = np.random.default_rng(3)
    A = rng.standard_normal((4, 3))
    b = rng.standard_normal(4) * 0.5
    w = rng.standard_normal(4)
    p = oracle.pack([(A, b)], w, 0.7)
    F, R, eps = _pair(4, 6, 3)
    X = eps[:, None] * R + (1 - eps[:, None]) * F
    t = np.tanh(X @ A.T + b)
    g = (w * (1 - t * t)) @ A
    nrm = np.linalg.norm(g, axis=1)
    lam, wg = 10.0, 0.25
    P_ref = wg * lam * np.mean((nrm - 1) ** 2)
    P, grad = oracle.gradient_penalty(p, shape, F, R, eps, lam, w=wg)
    assert abs(P - P_ref) < 1e-12 * max(1.0, P_ref)
    # dP/dw_j = wg lam (2/n) sum_b (|g_b|-1)/|g_b| g_b . A_j (1 - t_bj^2): closed form of one block
    c = (2 * wg * lam / len(X)) * ((nrm - 1) / nrm)[:, None] * g
    gw_ref = ((c @ A.T) * (1 - t * t)).sum(axis=0)
    _, gw_out, _ = oracle.unpack(grad, *shape)
    assert np.abs(gw_out - gw_ref).max() < 1e-12 * max(1.0, np.abs(gw_ref).max())


def test_weight_gradient_matches_finite_differences():
    p = _net(5)
    F, R, eps = _pair(6, 3, SHAPE[0])
    lam = 3.0
    _, grad = oracle.gradient_penalty(p, SHAPE, F, R, eps, lam, w=0.5)
    h = 1e-6
    fd = np.zeros_like(p)
    for k in range(p.size):
        e = np.zeros_like(p)
        e[k] = h
        fd[k] = (oracle.gradient_penalty(p + e, SHAPE, F, R, eps, lam, w=0.5)[0] -
                 oracle.gradient_penalty(p - e, SHAPE, F, R, eps, lam, w=0.5)[0]) / (2 * h)
    assert np.abs(grad - fd).max() < 1e-7 * max(1.0, np.abs(fd).max())


def test_weight_gradient_matches_autograd():
    torch.set_default_dtype(torch.float64)
    p = _net(7, shape=(6, 3, 5))
    shape = (6, 3, 5)
    F, R, eps = _pair(8, 4, 6)
    lam, wg = 10.0, 1.0 / 16
    pt = torch.tensor(p, requires_grad=True)
    n_in, L, W = shape
    off, layers = 0, []
    fan = n_in
    for _ in range(L):
        Wm = pt[off:off + W * fan].reshape(W, fan)
        off += W * fan
        layers.append((Wm, pt[off:off + W]))
        off += W
        fan = W
    wo, bo = pt[off:off + W], pt[off + W]
    e = torch.tensor(eps)[:, None]
    x = (e * torch.tensor(R) + (1 - e) * torch.tensor(F)).requires_grad_(True)
    h = x
    for Wm, b in layers:
        h = torch.tanh(h @ Wm.T + b)
    D = h @ wo + bo
    g = torch.autograd.grad(D.sum(), x, create_graph=True)[0]
    P = wg * lam * ((g.norm(dim=1) - 1) ** 2).mean()
    P.backward()
    Po, grad = oracle.gradient_penalty(p, shape, F, R, eps, lam, w=wg)
    assert abs(Po - P.item()) < 1e-12 * max(1.0, abs(P.item()))
    ref = pt.grad.numpy()
    assert np.abs(grad - ref).max() < 1e-11 * max(1.0, np.abs(ref).max())


def test_invariants():
    p = _net(9)
    F, R, eps = _pair(10, 5, SHAPE[0])
    one = np.ones_like(eps)
    P1, g1 = oracle.gradient_penalty(p, SHAPE, F, R, one, 2.0)
    P2, g2 = oracle.gradient_penalty(p, SHAPE, F + 5.0, R, one, 2.0)
    assert P1 == P2 and np.array_equal(g1, g2)
    Pa, ga = oracle.gradient_penalty(p, SHAPE, F, R, eps, 1.0, w=1.0)
    Pb, gb = oracle.gradient_penalty(p, SHAPE, F, R, eps, 3.0, w=0.5)
    assert abs(Pb - 1.5 * Pa) < 1e-12 * Pa
    assert np.abs(gb - 1.5 * ga).max() < 1e-12 * np.abs(ga).max()
    # additivity: two halves with the global count equal the whole
    Pw, gw = oracle.gradient_penalty(p, SHAPE, F, R, eps, 2.0)
    Ph0, gh0 = oracle.gradient_penalty(p, SHAPE, F[:2], R[:2], eps[:2], 2.0, n_total=5)
    Ph1, gh1 = oracle.gradient_penalty(p, SHAPE, F[2:], R[2:], eps[2:], 2.0, n_total=5)
    assert abs(Ph0 + Ph1 - Pw) < 1e-12 * Pw
    assert np.abs(gh0 + gh1 - gw).max() < 1e-12 * np.abs(gw).max()


def test_step_penalty_chunking_and_zero():
    from _tiny import TINY2
    from paper_1910_13444_amd.inputs import make_inputs
    wl = TINY2
    inp = make_inputs(wl)
    real = oracle.real_snapshots(wl, inp)
    n_gp = min(wl.S, wl.B_r)
    eps = np.random.default_rng(11).random((wl.G, n_gp))
    base = oracle.train_step(wl, inp, real)
    a = oracle.train_step(wl, inp, real, lambda_gp=10.0, gp_eps=eps)
    b = oracle.train_step(wl, inp, real, lambda_gp=10.0, gp_eps=eps, chunk_S=2)
    assert np.all(a["P_gp"] > 0)
    for k in ("gY", "gU"):
        assert np.array_equal(a[k], base[k])          # the penalty touches the critic only
    assert np.abs(a["loss"][:, 0] - base["loss"][:, 0] - a["P_gp"]).max() < 1e-12
    for k in ("gD", "loss", "P_gp"):
        assert np.abs(np.asarray(a[k]) - np.asarray(b[k])).max() < 1e-12 * max(1.0, np.abs(a[k]).max())
    z = oracle.train_step(wl, inp, real, lambda_gp=0.0, gp_eps=eps)
    assert np.array_equal(z["gD"], base["gD"])
