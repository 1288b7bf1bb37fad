"""Pin the oracle to closed forms (no dependence on its own recursion).

* One hidden tanh layer: G(x) = sum_j c_j tanh(w_j x + beta_j) + b has
  G' = sum_j c_j w_j sech^2(.) and G'' = -2 sum_j c_j w_j^2 tanh(.) sech^2(.);
  sech is evaluated through cosh, a path the oracle never takes.
* Two-dimensional separable units give the Laplacian as a sum of 1-D forms.
* Darcy residual (Eq. 1 with k = exp(Y), Eq. 2) on analytic (Y, u) pairs.
"""
import numpy as np

import oracle


def _one_layer_params(W1, b1, w_out, b_out):
    return np.concatenate([W1.reshape(-1), b1, w_out, [b_out]])


def test_single_layer_1d_jets():
    rng = np.random.default_rng(0)
    W, n_z = 5, 3
    W1 = rng.standard_normal((W, 1 + n_z))
    b1 = rng.standard_normal(W)
    c = rng.standard_normal(W)
    b = 0.3
    p = _one_layer_params(W1, b1, c, b)
    x = rng.random((7, 1))
    z = rng.standard_normal((1, n_z))
    out = oracle.gen_forward(p, (1 + n_z, 1, W), 1, x, np.repeat(z, 7, axis=0), 2)
    beta = W1[:, 1:] @ z[0] + b1
    w = W1[:, 0]
    arg = x * w + beta                       # [7, W]
    sech2 = 1.0 / np.cosh(arg) ** 2
    G = np.tanh(arg) @ c + b
    G1 = sech2 @ (c * w)
    G2 = (-2.0 * np.tanh(arg) * sech2) @ (c * w * w)
    np.testing.assert_allclose(out["y"], G, rtol=1e-13, atol=1e-14)
    np.testing.assert_allclose(out["dy"][0], G1, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(out["ddy"][0], G2, rtol=1e-12, atol=1e-14)


def test_separable_2d_laplacian():
    # units 0..2 see only x1, units 3..5 see only x2
    rng = np.random.default_rng(1)
    W, n_z = 6, 2
    W1 = rng.standard_normal((W, 2 + n_z))
    W1[:3, 1] = 0.0
    W1[3:, 0] = 0.0
    b1 = rng.standard_normal(W)
    c = rng.standard_normal(W)
    p = _one_layer_params(W1, b1, c, -0.1)
    x = rng.random((5, 2))
    z = rng.standard_normal((5, n_z))
    out = oracle.gen_forward(p, (2 + n_z, 1, W), 2, x, z, 2)
    arg = x @ W1[:, :2].T + z @ W1[:, 2:].T + b1
    sech2 = 1.0 / np.cosh(arg) ** 2
    th = np.tanh(arg)
    lap = (-2.0 * th * sech2 * (W1[:, 0] ** 2 + W1[:, 1] ** 2)) @ c
    np.testing.assert_allclose(out["ddy"].sum(axis=0), lap, rtol=1e-12, atol=1e-14)
    # d/dx1 only sees units 0..2
    d1 = (sech2[:, :3] * W1[:3, 0]) @ c[:3]
    np.testing.assert_allclose(out["dy"][0], d1, rtol=1e-12, atol=1e-14)


def _const_net(in_dim, L, W, c):
    n = W * in_dim + W + (L - 1) * (W * W + W) + W + 1
    p = np.zeros(n)
    p[-1] = c
    return p


def _single_unit_net(in_dim, W, d, wvec, beta, alpha):
    """L=1 net whose output is alpha * tanh(wvec . x + beta) + 0 (unit 0 only)."""
    W1 = np.zeros((W, in_dim))
    W1[0, :d] = wvec
    b1 = np.zeros(W)
    b1[0] = beta
    w_out = np.zeros(W)
    w_out[0] = alpha
    return _one_layer_params(W1, b1, w_out, 0.0)


def test_residual_constant_Y():
    # Y = c, u = alpha tanh(w x + beta):  r = -e^c u'' - f = 2 e^c alpha w^2 t sech^2 - f
    c, alpha, w, beta = 0.4, 1.3, 2.1, -0.2
    in_dim, W = 3, 4
    pY = _const_net(in_dim, 1, W, c)
    pU = _single_unit_net(in_dim, W, 1, [w], beta, alpha)
    x = np.linspace(0.05, 0.95, 9)[:, None]
    z = np.zeros((9, 2))
    f = np.linspace(-1, 1, 9)
    jY = oracle.gen_forward(pY, (in_dim, 1, W), 1, x, z, 1)
    jU = oracle.gen_forward(pU, (in_dim, 1, W), 1, x, z, 2)
    r = oracle.darcy_residual(jY["y"], jY["dy"], jU["dy"], jU["ddy"], f)
    arg = w * x[:, 0] + beta
    expect = 2.0 * np.exp(c) * alpha * w * w * np.tanh(arg) / np.cosh(arg) ** 2 - f
    np.testing.assert_allclose(r, expect, rtol=1e-12, atol=1e-14)


def test_residual_coupled_pair_2d():
    # Y = g tanh(v.x + e), u = a tanh(w.x + b)
    # r = -e^Y (grad Y . grad u + lap u) - f
    in_dim, W, d = 4, 3, 2
    g, v, e = 0.7, np.array([1.1, -0.6]), 0.15
    a, w, b = -0.9, np.array([0.8, 1.7]), -0.3
    pY = _single_unit_net(in_dim, W, d, v, e, g)
    pU = _single_unit_net(in_dim, W, d, w, b, a)
    rng = np.random.default_rng(3)
    x = rng.random((11, 2))
    z = rng.standard_normal((11, 2))
    f = 0.25
    jY = oracle.gen_forward(pY, (in_dim, 1, W), d, x, z, 1)
    jU = oracle.gen_forward(pU, (in_dim, 1, W), d, x, z, 2)
    r = oracle.darcy_residual(jY["y"], jY["dy"], jU["dy"], jU["ddy"], np.full(11, f))
    aY = x @ v + e
    aU = x @ w + b
    Y = g * np.tanh(aY)
    sY = 1.0 / np.cosh(aY) ** 2
    sU = 1.0 / np.cosh(aU) ** 2
    gradY = g * sY[:, None] * v[None, :]
    gradU = a * sU[:, None] * w[None, :]
    lapU = -2.0 * a * np.tanh(aU) * sU * (w @ w)
    expect = -np.exp(Y) * ((gradY * gradU).sum(axis=1) + lapU) - f
    np.testing.assert_allclose(r, expect, rtol=1e-12, atol=1e-14)


def test_plain_mlp_matches_manual():
    # the discriminator's value path against an independent loop
    rng = np.random.default_rng(4)
    in_dim, L, W = 5, 2, 4
    from paper_1910_13444_amd.inputs import glorot_mlp
    p = glorot_mlp(rng, in_dim, L, W).astype(np.float64)
    V = rng.standard_normal((6, in_dim))
    y = oracle.mlp_forward(p, (in_dim, L, W), V)
    off = 0
    for n in range(6):
        h = V[n]
        off = 0
        fan = in_dim
        for _ in range(L):
            Wm = p[off:off + W * fan].reshape(W, fan)
            off += W * fan
            bb = p[off:off + W]
            off += W
            h = np.array([np.tanh(sum(Wm[i, k] * h[k] for k in range(fan)) + bb[i]) for i in range(W)])
            fan = W
        val = sum(p[off + i] * h[i] for i in range(W)) + p[off + W]
        assert abs(val - y[n]) < 1e-13
