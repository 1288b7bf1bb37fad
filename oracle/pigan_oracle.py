"""Plain fp64 CPU oracle of the PI-GAN training step (arXiv 1910.13444).

TEST INFRASTRUCTURE.  Only the tests, the package smoke check and the
benchmark's CPU-baseline leg may import this module.  It shares no code with
the HIP path and imports nothing from it.

What is computed (all in float64, NumPy only, no blocking or fusion beyond what
the definitions state):

* Generator networks G(x, z) for Y = log k and for the head u: a tanh MLP on the
  narrow input [x_1..x_d, z_1..z_nz] (one location plus the noise vector,
  Sec. III.C "Single Node optimizations"), L tanh layers of width W, then a
  linear scalar output.  Or the paper's own generator (same section): one
  shared tanh trunk with residual skips over pairs of layers and a linear
  two-output head (Y, u); see trunk_forward.
* Exact spatial jets (value, d/dx_i, d^2/dx_i^2) of the generator, carried
  forward layer by layer by the chain rule.  The paper obtains the source term
  f by applying the differential operator to the generator with automatic
  differentiation (Sec. III.B.1, "Baseline Architecture"); the jets are the
  exact derivatives that operation produces.
* The Darcy residual r = -div(exp(Y) grad u) - f, from the Darcy equation
  (Eq. 1) with the lognormal conductivity k = exp(Y) (Eq. 2), expanded as
  -exp(Y) (grad Y . grad u + lap u) - f.
* Sensor snapshots [Y at the Y sensors | u at the u sensors] per noise sample
  and the discriminator, a tanh MLP on the whole snapshot (Sec. III.C).
* WGAN critic losses per subdomain group, weighted by the subdomain weight
  (Sec. III.B.1): L_D = w (mean D(fake) - mean D(real)),
  L_adv = -w mean D(fake), L_pde = w lambda mean r^2, L_G = L_adv + L_pde.
* Optionally the critic's gradient penalty (the WGAN-GP member of the WGAN
  family the paper cites): P = w lambda_gp mean_b (||grad_v D(x_b)|| - 1)^2 at
  x_b = eps_b R_b + (1 - eps_b) F_b, added to L_D.
* Exact weight gradients of L_D (discriminator) and L_G (both generators) by
  an explicit reverse pass.  Losses are means, so the step is additive over
  sample chunks, the same identity the paper uses to fold subdomain losses into
  its data-parallel gradient sum (Sec. III.D.1).

Parameter packing (float32 master copy in, float64 internally):
[W1 (W x in_dim, row-major), b1, W2 (W x W), b2, ..., W_L, b_L, w_out (W), b_out].

Pins: see tests/test_oracle_*.py (closed forms, finite differences of the jets
and of every weight gradient, torch.autograd in float64, invariants).
"""
from __future__ import annotations

import numpy as np

F64 = np.float64


# ----------------------------------------------------------------------------
# parameter packing
# ----------------------------------------------------------------------------

def unpack(params, in_dim: int, L: int, W: int):
    """Split a packed parameter vector into ([(W_l, b_l)], w_out, b_out)."""
    p = np.asarray(params, dtype=F64).reshape(-1)
    layers = []
    off = 0
    fan = in_dim
    for _ in range(L):
        Wl = p[off:off + W * fan].reshape(W, fan)
        off += W * fan
        bl = p[off:off + W]
        off += W
        layers.append((Wl, bl))
        fan = W
    w_out = p[off:off + W]
    off += W
    b_out = float(p[off])
    off += 1
    if off != p.size:
        raise ValueError(f"parameter vector has {p.size} entries, shape needs {off}")
    return layers, w_out, b_out


def pack(layer_grads, gw_out, gb_out) -> np.ndarray:
    parts = []
    for gW, gb in layer_grads:
        parts.append(np.asarray(gW, F64).reshape(-1))
        parts.append(np.asarray(gb, F64).reshape(-1))
    parts.append(np.asarray(gw_out, F64).reshape(-1))
    parts.append(np.array([gb_out], F64))
    return np.concatenate(parts)


# ----------------------------------------------------------------------------
# tanh and its derivatives with respect to the pre-activation a
# ----------------------------------------------------------------------------

def _tanh_derivs(a):
    t = np.tanh(a)
    s = 1.0 - t * t                  # dt/da
    sp = -2.0 * t * s                # d2t/da2
    spp = 2.0 * s * (3.0 * t * t - 1.0)   # d3t/da3
    return t, s, sp, spp


# ----------------------------------------------------------------------------
# generator: forward jets and reverse pass
# ----------------------------------------------------------------------------

def gen_forward(params, shape, d: int, X, Z, order: int, keep: bool = False):
    """Evaluate a generator and its spatial jets at rows (X[n], Z[n]).

    X: [N, d] locations, Z: [N, n_z] noise (one row per evaluation point).
    order 0: value only; 1: value and d/dx_i; 2: also d^2/dx_i^2 (pure second
    derivatives only: the Laplacian needs no mixed terms).
    Returns dict(y=[N], dy=[d, N] or None, ddy=[d, N] or None, cache).
    """
    in_dim, L, W = shape
    layers, w_out, b_out = unpack(params, in_dim, L, W)
    X = np.asarray(X, F64)
    Z = np.asarray(Z, F64)
    N = X.shape[0]
    W1, b1 = layers[0]
    # layer 1 on the concatenated input [x ; z]
    a = X @ W1[:, :d].T + Z @ W1[:, d:].T + b1
    # d a / d x_i is column i of W1; the second derivative of a is zero
    da = [np.broadcast_to(W1[:, i], (N, W)).copy() for i in range(d)] if order >= 1 else []
    dda = [np.zeros((N, W), F64) for _ in range(d)] if order >= 2 else []
    cache = []
    h = dh = ddh = None
    for l in range(L):
        if l > 0:
            Wl, bl = layers[l]
            Wq = Wl.T
            a = h @ Wq + bl                  # bias enters the value only
            da = [g @ Wq for g in dh]
            dda = [g @ Wq for g in ddh]
        t, s, sp, _ = _tanh_derivs(a)
        if keep:
            cache.append((a, list(da), list(dda), (h, dh, ddh)))
        h = t
        dh = [s * g for g in da]
        ddh = [s * g2 + sp * g1 * g1 for g1, g2 in zip(da, dda)]
    y = h @ w_out + b_out
    out = dict(y=y,
               dy=np.stack([g @ w_out for g in dh]) if order >= 1 else None,
               ddy=np.stack([g @ w_out for g in ddh]) if order >= 2 else None)
    if keep:
        out["cache"] = cache
        out["top"] = (h, dh, ddh)
    return out


def gen_backward(params, shape, d: int, X, Z, fwd, g_y, g_dy=None, g_ddy=None) -> np.ndarray:
    """Reverse pass of gen_forward (keep=True) for output cotangents.

    g_y: [N]; g_dy, g_ddy: [d, N] or None.  Returns the packed gradient (fp64).
    """
    in_dim, L, W = shape
    layers, w_out, b_out = unpack(params, in_dim, L, W)
    X = np.asarray(X, F64)
    Z = np.asarray(Z, F64)
    N = X.shape[0]
    hL, dhL, ddhL = fwd["top"]
    order = 0 if not dhL else (1 if not ddhL else 2)
    g_y = np.asarray(g_y, F64)
    g_dy = [np.asarray(g_dy[i], F64) for i in range(d)] if order >= 1 else []
    g_ddy = [np.asarray(g_ddy[i], F64) for i in range(d)] if order >= 2 else []
    # output layer y = w_out . h (+ b_out on the value only)
    gw_out = hL.T @ g_y
    for i in range(len(g_dy)):
        gw_out = gw_out + dhL[i].T @ g_dy[i]
    for i in range(len(g_ddy)):
        gw_out = gw_out + ddhL[i].T @ g_ddy[i]
    gb_out = g_y.sum()
    gh = np.outer(g_y, w_out)
    gdh = [np.outer(g, w_out) for g in g_dy]
    gddh = [np.outer(g, w_out) for g in g_ddy]
    grads = [None] * L
    for l in reversed(range(L)):
        a, da, dda, prev = fwd["cache"][l]
        t, s, sp, spp = _tanh_derivs(a)
        # h = t(a); h'_i = s a'_i; h''_i = s a''_i + s' a'_i^2
        ga = s * gh
        for i in range(len(gdh)):
            ga = ga + sp * da[i] * gdh[i]
        for i in range(len(gddh)):
            ga = ga + (sp * dda[i] + spp * da[i] * da[i]) * gddh[i]
        gda = []
        for i in range(len(gdh)):
            g = s * gdh[i]
            if gddh:
                g = g + 2.0 * sp * da[i] * gddh[i]
            gda.append(g)
        gdda = [s * g for g in gddh]
        ga = ga
        if l > 0:
            Wl, _ = layers[l]
            h, dh, ddh = prev
            gW = ga.T @ h
            for i in range(len(gda)):
                gW = gW + gda[i].T @ dh[i]
            for i in range(len(gdda)):
                gW = gW + gdda[i].T @ ddh[i]
            grads[l] = (gW, ga.sum(axis=0))
            Wq = Wl
            gh = ga @ Wq
            gdh = [g @ Wq for g in gda]
            gddh = [g @ Wq for g in gdda]
        else:
            gW1 = np.zeros((W, in_dim), F64)
            gW1[:, :d] = ga.T @ X
            gW1[:, d:] = ga.T @ Z
            for i in range(len(gda)):
                gW1[:, i] += gda[i].sum(axis=0)   # a'_i = W1[:, i] for every row
            grads[0] = (gW1, ga.sum(axis=0))
    return pack(grads, gw_out, gb_out)


# ----------------------------------------------------------------------------
# shared-trunk generator: one network with a log-conductivity head and a head
# for u (the paper's own generator, Sec. III.C "Single Node optimizations")
# ----------------------------------------------------------------------------

def trunk_unpack(params, in_dim: int, L: int, W: int):
    """Split a packed trunk vector [W1, b1, ..., W_L, b_L, w_Y, b_Y, w_u, b_u]
    into ([(W_l, b_l)], [(w_Y, b_Y), (w_u, b_u)])."""
    p = np.asarray(params, dtype=F64).reshape(-1)
    layers = []
    off = 0
    fan = in_dim
    for _ in range(L):
        Wl = p[off:off + W * fan].reshape(W, fan)
        off += W * fan
        bl = p[off:off + W]
        off += W
        layers.append((Wl, bl))
        fan = W
    heads = []
    for _ in range(2):
        w = p[off:off + W]
        off += W
        b = float(p[off])
        off += 1
        heads.append((w, b))
    if off != p.size:
        raise ValueError(f"parameter vector has {p.size} entries, trunk shape needs {off}")
    return layers, heads


def trunk_pack(layer_grads, head_grads) -> np.ndarray:
    parts = []
    for gW, gb in layer_grads:
        parts.append(np.asarray(gW, F64).reshape(-1))
        parts.append(np.asarray(gb, F64).reshape(-1))
    for gw, gb in head_grads:
        parts.append(np.asarray(gw, F64).reshape(-1))
        parts.append(np.array([gb], F64))
    return np.concatenate(parts)


def trunk_skip(l: int) -> bool:
    """Whether layer l (1-based) adds the activation of layer l - 2: after the
    first layer, every pair of layers is one residual block whose output is
    its second tanh plus the block's input (the paper's depths 5, 11 and 21
    are one layer plus 2, 5 and 10 such blocks)."""
    return l >= 3 and l % 2 == 1


def trunk_forward(params, shape, d: int, X, Z, order: int, keep: bool = False):
    """Evaluate the trunk and the jets of both heads at rows (X[n], Z[n]).

    h_1 = tanh(W_1 [x ; z] + b_1); h_l = tanh(W_l h_{l-1} + b_l), plus h_{l-2}
    when trunk_skip(l).  Heads Y = w_Y . h_L + b_Y and u = w_u . h_L + b_u
    (biases on the value only).  The skip is linear, so every jet stream of
    h_{l-2} is added to the same stream of h_l.  Returns dict(Y, dY, ddY, u,
    du, ddu) with dY/du [d, N] (order >= 1) and ddY/ddu [d, N] (order 2).
    """
    in_dim, L, W = shape
    layers, heads = trunk_unpack(params, in_dim, L, W)
    X = np.asarray(X, F64)
    Z = np.asarray(Z, F64)
    N = X.shape[0]
    W1, b1 = layers[0]
    a = X @ W1[:, :d].T + Z @ W1[:, d:].T + b1
    da = [np.broadcast_to(W1[:, i], (N, W)).copy() for i in range(d)] if order >= 1 else []
    dda = [np.zeros((N, W), F64) for _ in range(d)] if order >= 2 else []
    acts = [None]          # acts[l] = (h, dh, ddh) of layer l, 1-based
    cache = []
    h = dh = ddh = None
    for l in range(1, L + 1):
        if l > 1:
            Wl, bl = layers[l - 1]
            Wq = Wl.T
            a = h @ Wq + bl
            da = [g @ Wq for g in dh]
            dda = [g @ Wq for g in ddh]
        t, s, sp, _ = _tanh_derivs(a)
        if keep:
            cache.append((a, list(da), list(dda), (h, dh, ddh)))
        nh = t
        ndh = [s * g for g in da]
        nddh = [s * g2 + sp * g1 * g1 for g1, g2 in zip(da, dda)]
        if trunk_skip(l):
            sh, sdh, sddh = acts[l - 2]
            nh = nh + sh
            ndh = [g + gs for g, gs in zip(ndh, sdh)]
            nddh = [g + gs for g, gs in zip(nddh, sddh)]
        h = nh
        dh = [g for g in ndh]
        ddh = [g for g in nddh]
        acts.append((h, dh, ddh))
    out = {}
    for name, (w, b) in zip(("Y", "u"), heads):
        out[name] = h @ w + b
        out["d" + name] = np.stack([g @ w for g in dh]) if order >= 1 else None
        out["dd" + name] = np.stack([g @ w for g in ddh]) if order >= 2 else None
    if keep:
        out["cache"] = cache
        out["top"] = (h, dh, ddh)
    return out


def trunk_backward(params, shape, d: int, X, Z, fwd, gY=None, gdY=None, gddY=None, gu=None, gdu=None, gddu=None) -> np.ndarray:
    """Reverse pass of trunk_forward (keep=True) for cotangents of the head
    jets (each [N] or [d, N]; None means zero).  Returns the packed gradient."""
    in_dim, L, W = shape
    layers, heads = trunk_unpack(params, in_dim, L, W)
    X = np.asarray(X, F64)
    Z = np.asarray(Z, F64)
    N = X.shape[0]
    hL, dhL, ddhL = fwd["top"]
    nd1, nd2 = len(dhL), len(ddhL)

    def cot(v, nd):
        if nd == 0:
            return []
        return [np.zeros(N, F64) if v is None else np.asarray(v[i], F64) for i in range(nd)]

    g_heads = [(np.zeros(N, F64) if gY is None else np.asarray(gY, F64), cot(gdY, nd1), cot(gddY, nd2)),
               (np.zeros(N, F64) if gu is None else np.asarray(gu, F64), cot(gdu, nd1), cot(gddu, nd2))]
    head_grads = []
    gh = np.zeros((N, W), F64)
    gdh = [np.zeros((N, W), F64) for _ in range(nd1)]
    gddh = [np.zeros((N, W), F64) for _ in range(nd2)]
    for (w, _), (g0, g1, g2) in zip(heads, g_heads):
        gw = hL.T @ g0
        for i in range(nd1):
            gw = gw + dhL[i].T @ g1[i]
        for i in range(nd2):
            gw = gw + ddhL[i].T @ g2[i]
        head_grads.append((gw, g0.sum()))
        gh = gh + np.outer(g0, w)
        gdh = [a + np.outer(g, w) for a, g in zip(gdh, g1)]
        gddh = [a + np.outer(g, w) for a, g in zip(gddh, g2)]
    pending = {}           # layer l - 2 -> total cotangent of h_l carried by the skip
    grads = [None] * L
    for l in range(L, 0, -1):
        if l in pending:   # h_l is the input of a residual block: add the skip's cotangent
            sg, sdg, sddg = pending.pop(l)
            gh = gh + sg
            gdh = [a + b for a, b in zip(gdh, sdg)]
            gddh = [a + b for a, b in zip(gddh, sddg)]
        if trunk_skip(l):
            pending[l - 2] = (gh, list(gdh), list(gddh))
        a, da, dda, prev = fwd["cache"][l - 1]
        t, s, sp, spp = _tanh_derivs(a)
        ga = s * gh
        for i in range(nd1):
            ga = ga + sp * da[i] * gdh[i]
        for i in range(nd2):
            ga = ga + (sp * dda[i] + spp * da[i] * da[i]) * gddh[i]
        gda = []
        for i in range(nd1):
            g = s * gdh[i]
            if nd2:
                g = g + 2.0 * sp * da[i] * gddh[i]
            gda.append(g)
        gdda = [s * g for g in gddh]
        ga = ga
        if l > 1:
            Wl, _ = layers[l - 1]
            h, dh, ddh = prev
            gW = ga.T @ h
            for i in range(nd1):
                gW = gW + gda[i].T @ dh[i]
            for i in range(nd2):
                gW = gW + gdda[i].T @ ddh[i]
            grads[l - 1] = (gW, ga.sum(axis=0))
            Wq = Wl
            gh = ga @ Wq
            gdh = [g @ Wq for g in gda]
            gddh = [g @ Wq for g in gdda]
        else:
            gW1 = np.zeros((W, in_dim), F64)
            gW1[:, :d] = ga.T @ X
            gW1[:, d:] = ga.T @ Z
            for i in range(nd1):
                gW1[:, i] += gda[i].sum(axis=0)
            grads[0] = (gW1, ga.sum(axis=0))
    return trunk_pack(grads, head_grads)


# ----------------------------------------------------------------------------
# plain tanh MLP (discriminator)
# ----------------------------------------------------------------------------

def mlp_forward(params, shape, V, keep: bool = False):
    """D(v) = w_out . h_L + b_out with h_l = tanh(W_l h_{l-1} + b_l), h_0 = v.

    keep=True also returns the cache (activations h_0..h_L, pre-activations)."""
    in_dim, L, W = shape
    layers, w_out, b_out = unpack(params, in_dim, L, W)
    h = np.asarray(V, F64)
    hs = [h]
    pre = []
    for Wl, bl in layers:
        a = h @ Wl.T + bl
        pre.append(a)
        h = np.tanh(a)
        hs.append(h)
    y = h @ w_out + b_out
    return (y, dict(h=hs, a=pre)) if keep else y


def mlp_backward(params, shape, cache, g_y, want_input_grad: bool = False):
    in_dim, L, W = shape
    layers, w_out, b_out = unpack(params, in_dim, L, W)
    hs = cache["h"]
    g_y = np.asarray(g_y, F64)
    tops = hs[1:]
    gw_out = tops[-1].T @ g_y
    gb_out = g_y.sum()
    gh = np.outer(g_y, w_out)
    grads = [None] * L
    for l in reversed(range(L)):
        t = tops[l]
        ga = (1.0 - t * t) * gh
        grads[l] = (ga.T @ hs[l], ga.sum(axis=0))
        gh = ga @ layers[l][0]
    g = pack(grads, gw_out, gb_out)
    return (g, gh) if want_input_grad else g


# ----------------------------------------------------------------------------
# gradient penalty of the critic (optional term of the critic loss)
# ----------------------------------------------------------------------------
# The paper trains WGAN critics and cites the gradient-penalty member of that
# family (Sec. I.C, Sec. II.C) without writing it out.  Its definition:
#   x_b = eps_b R_b + (1 - eps_b) F_b                (one pair per row b)
#   P   = w lambda_gp mean_b (||grad_v D(x_b)||_2 - 1)^2
# is added to the critic loss L_D, and its gradient to the critic weights.

def critic_input_grad(params, shape, V):
    """g_b = dD/dv at every row v_b of V: the reverse pass of D to its input."""
    _, cache = mlp_forward(params, shape, V, keep=True)
    _, g = mlp_backward(params, shape, cache, np.ones(np.asarray(V).shape[0], F64), want_input_grad=True)
    return g


def tangent_output_grad(params, shape, V, Cdir):
    """Weight gradient of J = sum_b dD(v_b + t c_b)/dt |_{t=0}.

    The directional derivative is carried forward with the activations
    (h, h_dot), h_dot_0 = c:  a = W h + b,  a_dot = W h_dot,  h = tanh(a),
    h_dot = s a_dot  (s = 1 - tanh^2);  J = sum_b w_out . h_dot_L.  Its
    reverse pass, with s' = ds/da = -2 t s:
      g_a     = s g_h + s' a_dot g_hdot,     g_adot = s g_hdot,
      dJ/dW_l = g_a^T h_{l-1} + g_adot^T h_dot_{l-1},  dJ/db_l = sum_b g_a,
      g_h(l-1) = g_a W_l,  g_hdot(l-1) = g_adot W_l;
    at the top g_h = 0, g_hdot = w_out, dJ/dw_out = sum_b h_dot_L, dJ/db_out = 0."""
    in_dim, L, W = shape
    layers, w_out, b_out = unpack(params, in_dim, L, W)
    h = np.asarray(V, F64)
    hd = np.asarray(Cdir, F64)
    hs, hds, ts, ads = [h], [hd], [], []
    for Wl, bl in layers:
        Wq = Wl
        a = h @ Wq.T + bl
        ad = hd @ Wq.T
        t = np.tanh(a)
        h = t
        hd = (1.0 - t * t) * ad
        ts.append(t)
        ads.append(ad)
        hs.append(h)
        hds.append(hd)
    gw_out = hds[-1].sum(axis=0)
    g_h = np.zeros_like(hs[-1])
    g_hd = np.tile(w_out, (hs[-1].shape[0], 1))
    grads = [None] * L
    for l in reversed(range(L)):
        t, ad = ts[l], ads[l]
        sl = 1.0 - t * t
        g_a = sl * g_h - 2.0 * t * sl * ad * g_hd
        g_ad = sl * g_hd
        grads[l] = (g_a.T @ hs[l] + g_ad.T @ hds[l], g_a.sum(axis=0))
        Wq = layers[l][0]
        g_h = g_a @ Wq
        g_hd = g_ad @ Wq
    return pack(grads, gw_out, 0.0)


def gradient_penalty(params, shape, F, R, eps, lambda_gp, w=1.0, n_total=None):
    """P (summed over these pairs with the 1/n_total of the mean) and dP/dphi.

    dP/dphi = sum_b c_b . dg_b/dphi with c_b = dP/dg_b held fixed, and
    c_b . g_b is the directional derivative of D at x_b along c_b, so dP/dphi
    is tangent_output_grad along c.  A row with g_b = 0 has no gradient
    direction; it contributes P but no weight gradient."""
    w = float(w)                                  # a float32 weight would round P to single precision
    eps = np.asarray(eps, F64)[:, None]
    X = eps * np.asarray(R, F64) + (1.0 - eps) * np.asarray(F, F64)
    n = X.shape[0] if n_total is None else n_total
    g = critic_input_grad(params, shape, X)
    nrm = np.sqrt((g * g).sum(axis=1))
    P = w * lambda_gp * float(((nrm - 1.0) ** 2).sum()) / n
    with np.errstate(divide="ignore", invalid="ignore"):
        coef = np.where(nrm > 0, (nrm - 1.0) / nrm, 0.0)
    Cdir = (2.0 * w * lambda_gp / n) * coef[:, None] * g
    return P, tangent_output_grad(params, shape, X, Cdir)


# ----------------------------------------------------------------------------
# Darcy residual (Eq. 1 with k = exp(Y), Eq. 2)
# ----------------------------------------------------------------------------

def darcy_residual(Y, dY, dU, ddU, f):
    """r = -div(exp(Y) grad u) - f = -exp(Y) (sum_i dY_i dU_i + sum_i ddU_i) - f."""
    Y = np.asarray(Y, F64)
    flux_div = (np.asarray(dY, F64) * np.asarray(dU, F64)).sum(axis=0) + np.asarray(ddU, F64).sum(axis=0)
    return -np.exp(Y) * flux_div - np.asarray(f, F64)


# ----------------------------------------------------------------------------
# row builders: sensors are shared by all samples, collocation points are per
# sample; every row carries its sample's noise vector
# ----------------------------------------------------------------------------

def sensor_rows(xs, z):
    """Rows (s, j) for s in samples, j in sensors: X [S*n, d], Z [S*n, n_z]."""
    xs = np.asarray(xs, F64)
    z = np.asarray(z, F64)
    S, n = z.shape[0], xs.shape[0]
    return np.tile(xs, (S, 1)), np.repeat(z, n, axis=0)


def colloc_rows(xc, z):
    """Rows (s, p): xc [S, P, d] per sample, or [P, d] shared by every sample."""
    xc = np.asarray(xc, F64)
    z = np.asarray(z, F64)
    S = z.shape[0]
    if xc.ndim == 2:
        xc = np.broadcast_to(xc, (S,) + xc.shape)
    P = xc.shape[1]
    return xc.reshape(S * P, -1), np.repeat(z, P, axis=0)


def gen_jets(params, shape, d, z, x, order):
    """Jets [1 + order*d, S, P] (value, d/dx_i, d^2/dx_i^2) at points x of each sample."""
    X, Z = colloc_rows(x, z)
    S = np.asarray(z).shape[0]
    out = gen_forward(params, shape, d, X, Z, order)
    P = X.shape[0] // S
    comps = [out["y"][None]]
    if order >= 1:
        comps.append(out["dy"])
    if order >= 2:
        comps.append(out["ddy"])
    return np.concatenate(comps, axis=0).reshape(-1, S, P)


def snapshots(pY, pU, shape, d, xsY, xsU, z):
    """Sensor snapshots [S, n_sY + n_sU] = [Y at Y sensors | u at u sensors]."""
    S = np.asarray(z).shape[0]
    XY, ZY = sensor_rows(xsY, z)
    XU, ZU = sensor_rows(xsU, z)
    yY = gen_forward(pY, shape, d, XY, ZY, 0)["y"].reshape(S, -1)
    yU = gen_forward(pU, shape, d, XU, ZU, 0)["y"].reshape(S, -1)
    return np.concatenate([yY, yU], axis=1)


# ----------------------------------------------------------------------------
# the training step
# ----------------------------------------------------------------------------

def train_step_group(gshape, dshape, d, pY, pU, pD, z, xc, xsY, xsU, f, real,
                     w=1.0, lambda_pde=1.0, chunk_S=None, lambda_gp=0.0, gp_eps=None):
    """One subdomain group's losses and gradients.

    Returns dict(L_D, L_adv, L_pde, gY, gU, gD, P_gp) with gradients of
    L_D (discriminator weights) and of L_G = L_adv + L_pde (generator weights).
    ``f`` is an [S, P] array.  Samples are processed in chunks of ``chunk_S``
    (all at once by default); the result does not depend on the chunking.
    With lambda_gp > 0 the gradient penalty on the pairs (F_b, R_b),
    b < min(S, B), with mixing weights gp_eps[b] is added to L_D (and reported
    as P_gp) and its gradient to the critic weights.
    """
    z = np.asarray(z, F64)
    xc = np.asarray(xc, F64)
    f = np.asarray(f, F64)
    real = np.asarray(real, F64)
    S, P = xc.shape[0], xc.shape[1]
    B = real.shape[0]
    nY = np.asarray(xsY).shape[0]
    chunk_S = S if not chunk_S else chunk_S
    gY = np.zeros(np.asarray(pY).size, F64)
    gU = np.zeros(np.asarray(pU).size, F64)
    gD = np.zeros(np.asarray(pD).size, F64)
    sum_DF = 0.0
    sum_r2 = 0.0
    P_gp = 0.0
    n_gp = min(S, B)

    # real snapshots: dL_D/dD(real_b) = -w/B
    DR, hsR = mlp_forward(pD, dshape, real, keep=True)
    gD += mlp_backward(pD, dshape, hsR, np.full(B, -w / B, F64))
    sum_DR = DR.sum()

    for s0 in range(0, S, chunk_S):
        sl = slice(s0, min(S, s0 + chunk_S))
        zc = z[sl]
        Sc = zc.shape[0]
        # --- generators at the sensors (value only) -> fake snapshots
        XY, ZY = sensor_rows(xsY, zc)
        XU, ZU = sensor_rows(xsU, zc)
        fY_s = gen_forward(pY, gshape, d, XY, ZY, 0, keep=True)
        fU_s = gen_forward(pU, gshape, d, XU, ZU, 0, keep=True)
        F = np.concatenate([fY_s["y"].reshape(Sc, -1), fU_s["y"].reshape(Sc, -1)], axis=1)
        # --- generators at the collocation points with jets
        XC, ZC = colloc_rows(xc[sl], zc)
        jY = gen_forward(pY, gshape, d, XC, ZC, 1, keep=True)
        jU = gen_forward(pU, gshape, d, XC, ZC, 2, keep=True)
        fc = f[sl].reshape(-1)
        r = darcy_residual(jY["y"], jY["dy"], jU["dy"], jU["ddy"], fc)
        sum_r2 += float((r * r).sum())
        # --- discriminator on the fake snapshots: dL_D/dD(F_s) = w/S
        DF, hsF = mlp_forward(pD, dshape, F, keep=True)
        sum_DF += float(DF.sum())
        gDc, gF = mlp_backward(pD, dshape, hsF, np.full(Sc, w / S, F64), want_input_grad=True)
        gD += gDc
        # --- gradient penalty on this chunk's pairs (F_b, R_b), b < n_gp
        if lambda_gp != 0.0:
            b1 = min(n_gp, s0 + Sc)
            if b1 > s0:
                Pc, gPc = gradient_penalty(pD, dshape, F[:b1 - s0], real[s0:b1], np.asarray(gp_eps, F64)[s0:b1],
                                           lambda_gp, w=w, n_total=n_gp)
                P_gp += Pc
                gD += gPc
        # L_adv = -w mean D(F): its snapshot cotangent is the negated L_D one
        gF = -gF
        # --- residual cotangents: dL_pde/dr = 2 w lambda r / (S P)
        q = 2.0 * w * lambda_pde * r / (S * P)
        eY = np.exp(jY["y"])
        g_Yval = q * (r + fc)                       # dr/dY = -exp(Y)(...) = r + f
        g_Ydy = np.stack([-q * eY * jU["dy"][i] for i in range(d)])
        g_Udy = np.stack([-q * eY * jY["dy"][i] for i in range(d)])
        g_Uddy = np.stack([-q * eY for _ in range(d)])
        g_Uval = np.zeros_like(r)                   # u itself does not enter r
        # --- reverse passes through both generators
        gY += gen_backward(pY, gshape, d, XY, ZY, fY_s, gF[:, :nY].reshape(-1))
        gU += gen_backward(pU, gshape, d, XU, ZU, fU_s, gF[:, nY:].reshape(-1))
        gY += gen_backward(pY, gshape, d, XC, ZC, jY, g_Yval, g_Ydy)
        gU += gen_backward(pU, gshape, d, XC, ZC, jU, g_Uval, g_Udy, g_Uddy)

    L_D = w * (sum_DF / S - sum_DR / B) + P_gp
    L_adv = -w * sum_DF / S
    L_pde = w * lambda_pde * sum_r2 / (S * P)
    return dict(L_D=L_D, L_adv=L_adv, L_pde=L_pde, gY=gY, gU=gU, gD=gD, P_gp=P_gp)


def train_step(wl, inp, real, lambda_pde=None, chunk_S=None, lambda_gp=0.0, gp_eps=None):
    """All groups of a workload.  ``inp`` is an inputs.StepInputs-like object,
    ``real`` the real snapshots [G, B_r, n_in].  Returns dict of stacked arrays:
    loss [G, 3] (L_D, L_adv, L_pde), gY [G, nY], gU [G, nU], gD [G, nD], and
    P_gp [G] (the gradient penalty, included in L_D; gp_eps is [G, min(S, B_r)])."""
    lam = wl.lambda_pde if lambda_pde is None else lambda_pde
    gshape = (wl.d + wl.n_z, wl.L, wl.W)
    dshape = (wl.n_sY + wl.n_sU, wl.L_D, wl.W_D)
    G = inp.z.shape[0]
    S, P = inp.xc.shape[1], inp.xc.shape[2]
    outs = []
    for g in range(G):
        f = inp.f[g] if inp.f is not None else np.full((S, P), inp.f_const)
        outs.append(train_step_group(gshape, dshape, wl.d, inp.pY[g], inp.pU[g], inp.pD[g],
                                     inp.z[g], inp.xc[g], inp.xsY[g], inp.xsU[g], f, real[g],
                                     w=float(inp.w_group[g]), lambda_pde=lam, chunk_S=chunk_S, lambda_gp=lambda_gp,
                                     gp_eps=None if gp_eps is None else gp_eps[g]))
    return dict(loss=np.array([[o["L_D"], o["L_adv"], o["L_pde"]] for o in outs]),
                gY=np.stack([o["gY"] for o in outs]),
                gU=np.stack([o["gU"] for o in outs]),
                gD=np.stack([o["gD"] for o in outs]),
                P_gp=np.array([o["P_gp"] for o in outs]))


def trunk_snapshots(pT, shape, d, xsY, xsU, z):
    """Sensor snapshots of a trunk generator: [Y head at Y sensors | u head at u sensors]."""
    S = np.asarray(z).shape[0]
    XY, ZY = sensor_rows(xsY, z)
    XU, ZU = sensor_rows(xsU, z)
    yY = trunk_forward(pT, shape, d, XY, ZY, 0)["Y"].reshape(S, -1)
    yU = trunk_forward(pT, shape, d, XU, ZU, 0)["u"].reshape(S, -1)
    return np.concatenate([yY, yU], axis=1)


def train_step_group_trunk(gshape, dshape, d, pT, pD, z, xc, xsY, xsU, f, real,
                           w=1.0, lambda_pde=1.0, chunk_S=None, lambda_gp=0.0, gp_eps=None):
    """One group's losses and gradients with the shared-trunk generator.

    Same losses as train_step_group (including its optional critic gradient
    penalty on the pairs (F_b, R_b), b < min(S, B)); both heads come from one
    network, so one gradient gT of L_G = L_adv + L_pde is returned.  Returns
    dict(L_D, L_adv, L_pde, gT, gD, P_gp)."""
    z = np.asarray(z, F64)
    xc = np.asarray(xc, F64)
    f = np.asarray(f, F64)
    real = np.asarray(real, F64)
    S, P = xc.shape[0], xc.shape[1]
    B = real.shape[0]
    nY = np.asarray(xsY).shape[0]
    chunk_S = S if not chunk_S else chunk_S
    gT = np.zeros(np.asarray(pT).size, F64)
    gD = np.zeros(np.asarray(pD).size, F64)
    sum_DF = 0.0
    sum_r2 = 0.0
    P_gp = 0.0
    n_gp = min(S, B)
    DR, hsR = mlp_forward(pD, dshape, real, keep=True)
    gD += mlp_backward(pD, dshape, hsR, np.full(B, -w / B, F64))
    sum_DR = DR.sum()
    for s0 in range(0, S, chunk_S):
        sl = slice(s0, min(S, s0 + chunk_S))
        zc = z[sl]
        Sc = zc.shape[0]
        # trunk at the Y sensors (Y head) and at the u sensors (u head)
        XY, ZY = sensor_rows(xsY, zc)
        XU, ZU = sensor_rows(xsU, zc)
        fY_s = trunk_forward(pT, gshape, d, XY, ZY, 0, keep=True)
        fU_s = trunk_forward(pT, gshape, d, XU, ZU, 0, keep=True)
        F = np.concatenate([fY_s["Y"].reshape(Sc, -1), fU_s["u"].reshape(Sc, -1)], axis=1)
        # trunk at the collocation points: jets of both heads
        XC, ZC = colloc_rows(xc[sl], zc)
        jc = trunk_forward(pT, gshape, d, XC, ZC, 2, keep=True)
        fc = f[sl].reshape(-1)
        r = darcy_residual(jc["Y"], jc["dY"], jc["du"], jc["ddu"], fc)
        sum_r2 += float((r * r).sum())
        DF, hsF = mlp_forward(pD, dshape, F, keep=True)
        sum_DF += float(DF.sum())
        gDc, gF = mlp_backward(pD, dshape, hsF, np.full(Sc, w / S, F64), want_input_grad=True)
        gD += gDc
        if lambda_gp != 0.0:
            b1 = min(n_gp, s0 + Sc)
            if b1 > s0:
                Pc, gPc = gradient_penalty(pD, dshape, F[:b1 - s0], real[s0:b1], np.asarray(gp_eps, F64)[s0:b1],
                                           lambda_gp, w=w, n_total=n_gp)
                P_gp += Pc
                gD += gPc
        gF = -gF
        q = 2.0 * w * lambda_pde * r / (S * P)
        eY = np.exp(jc["Y"])
        g_Yval = q * (r + fc)
        g_Ydy = np.stack([-q * eY * jc["du"][i] for i in range(d)])
        g_Udy = np.stack([-q * eY * jc["dY"][i] for i in range(d)])
        g_Uddy = np.stack([-q * eY for _ in range(d)])
        gT += trunk_backward(pT, gshape, d, XY, ZY, fY_s, gY=gF[:, :nY].reshape(-1))
        gT += trunk_backward(pT, gshape, d, XU, ZU, fU_s, gu=gF[:, nY:].reshape(-1))
        gT += trunk_backward(pT, gshape, d, XC, ZC, jc, gY=g_Yval, gdY=g_Ydy, gdu=g_Udy, gddu=g_Uddy)
    L_D = w * (sum_DF / S - sum_DR / B) + P_gp
    L_adv = -w * sum_DF / S
    L_pde = w * lambda_pde * sum_r2 / (S * P)
    return dict(L_D=L_D, L_adv=L_adv, L_pde=L_pde, gT=gT, gD=gD, P_gp=P_gp)


def train_step_trunk(wl, inp, real, lambda_pde=None, chunk_S=None, lambda_gp=0.0, gp_eps=None):
    """All groups of a trunk workload (inp.pT holds the trunk weights).
    Returns loss [G, 3], gT [G, nT], gD [G, nD], P_gp [G] (gp_eps is
    [G, min(S, B_r)] when lambda_gp > 0)."""
    lam = wl.lambda_pde if lambda_pde is None else lambda_pde
    gshape = (wl.d + wl.n_z, wl.L, wl.W)
    dshape = (wl.n_sY + wl.n_sU, wl.L_D, wl.W_D)
    G = inp.z.shape[0]
    S, P = inp.xc.shape[1], inp.xc.shape[2]
    outs = []
    for g in range(G):
        f = inp.f[g] if inp.f is not None else np.full((S, P), inp.f_const)
        outs.append(train_step_group_trunk(gshape, dshape, wl.d, inp.pT[g], inp.pD[g], inp.z[g], inp.xc[g],
                                           inp.xsY[g], inp.xsU[g], f, real[g], w=float(inp.w_group[g]),
                                           lambda_pde=lam, chunk_S=chunk_S, lambda_gp=lambda_gp,
                                           gp_eps=None if gp_eps is None else gp_eps[g]))
    return dict(loss=np.array([[o["L_D"], o["L_adv"], o["L_pde"]] for o in outs]),
                gT=np.stack([o["gT"] for o in outs]),
                gD=np.stack([o["gD"] for o in outs]),
                P_gp=np.array([o["P_gp"] for o in outs]))


def real_snapshots_trunk(wl, inp):
    """Teacher snapshots [G, B_r, n_in] of a trunk workload (teacher trunk inp.tT)."""
    gshape = (wl.d + wl.n_z, wl.L, wl.W)
    return np.stack([trunk_snapshots(inp.tT[g], gshape, wl.d, inp.xsY[g], inp.xsU[g], inp.z_teach[g])
                     for g in range(inp.z.shape[0])])


def train_step_hier(gshape, dshape, d, pY, pU, pDs, z, xc, xsY, xsU, f, idxY, idxU, idxF, real, w,
                    lambda_pde=0.0, chunk_S=None, trunk=False, lambda_gp=0.0, gp_eps=None):
    """Domain decomposition (Sec. III.B.1): one generator pair, one critic per
    subdomain of every level.  Critic k sees the paper's snapshot of its
    subdomain: [Y at Y sensors idxY[k] | u at u sensors idxU[k] | the
    generated source f = -div(exp(Y) grad u) at the free sensors idxF[k] (a
    subset of each sample's collocation points) | those free sensors'
    coordinates], real[k] its real snapshots ([B, n_in], f = 0 there).
    Weights w[k] = 1 / (levels * subdomains of the level).  Losses per critic:
    L_D[k] = w_k (mean D_k(fake) - mean D_k(real)), L_adv[k] = -w_k mean D_k(fake);
    the generator loss is sum_k L_adv[k] + L_pde with L_pde = lambda mean r^2.
    With trunk=True the generator is the shared trunk pY (pU unused): its Y
    head at the Y sensors, its u head at the u sensors, both heads' jets at the
    collocation points; gY is then the trunk's gradient and gU is empty.
    With lambda_gp > 0 every critic k also takes the gradient penalty of
    gradient_penalty on its pairs (F_b, R_b), b < min(S, B), with mixing
    weights gp_eps[k, b], weight w_k; it is added to L_D[k] and reported as
    P_gp[k].
    Returns dict(L_D [D], L_adv [D], L_pde, gY, gU, gD [D, nD], P_gp [D])."""
    z = np.asarray(z, F64)
    xc = np.asarray(xc, F64)
    f = np.asarray(f, F64)
    S, P = xc.shape[0], xc.shape[1]
    D = len(pDs)
    chunk_S = S if not chunk_S else chunk_S
    gY = np.zeros(np.asarray(pY).size, F64)
    gU = np.zeros(0 if trunk else np.asarray(pU).size, F64)
    gD = np.zeros((D, np.asarray(pDs[0]).size), F64)
    sum_DF = np.zeros(D)
    sum_DR = np.zeros(D)
    sum_r2 = 0.0
    P_gp = np.zeros(D)
    n_gp = min(S, np.asarray(real[0]).shape[0])
    for k in range(D):
        Rk = np.asarray(real[k], F64)
        DR, hsR = mlp_forward(pDs[k], dshape, Rk, keep=True)
        gD[k] += mlp_backward(pDs[k], dshape, hsR, np.full(Rk.shape[0], -w[k] / Rk.shape[0], F64))
        sum_DR[k] = DR.sum()
    B = np.asarray(real[0]).shape[0]
    nYs, nUs = np.asarray(xsY).shape[0], np.asarray(xsU).shape[0]
    for s0 in range(0, S, chunk_S):
        sl = slice(s0, min(S, s0 + chunk_S))
        zc = z[sl]
        Sc = zc.shape[0]
        XY, ZY = sensor_rows(xsY, zc)
        XU, ZU = sensor_rows(xsU, zc)
        XC, ZC = colloc_rows(xc[sl], zc)
        if trunk:
            fY_s = trunk_forward(pY, gshape, d, XY, ZY, 0, keep=True)
            fU_s = trunk_forward(pY, gshape, d, XU, ZU, 0, keep=True)
            Ys = fY_s["Y"].reshape(Sc, nYs)
            Us = fU_s["u"].reshape(Sc, nUs)
            jc = trunk_forward(pY, gshape, d, XC, ZC, 2, keep=True)
            jY = dict(y=jc["Y"], dy=jc["dY"])
            jU = dict(y=jc["u"], dy=jc["du"], ddy=jc["ddu"])
        else:
            fY_s = gen_forward(pY, gshape, d, XY, ZY, 0, keep=True)
            fU_s = gen_forward(pU, gshape, d, XU, ZU, 0, keep=True)
            Ys = fY_s["y"].reshape(Sc, nYs)
            Us = fU_s["y"].reshape(Sc, nUs)
            jY = gen_forward(pY, gshape, d, XC, ZC, 1, keep=True)
            jU = gen_forward(pU, gshape, d, XC, ZC, 2, keep=True)
        fc = f[sl].reshape(-1)
        r = darcy_residual(jY["y"], jY["dy"], jU["dy"], jU["ddy"], fc)
        sum_r2 += float((r * r).sum())
        Nf = (r + fc).reshape(Sc, P)                    # the generated source at every point
        gYs = np.zeros((Sc, nYs))
        gUs = np.zeros((Sc, nUs))
        gN = np.zeros((Sc, P))
        for k in range(D):
            iY, iU, iF = np.asarray(idxY[k]), np.asarray(idxU[k]), np.asarray(idxF[k])
            F = np.concatenate([Ys[:, iY], Us[:, iU], Nf[:, iF], xc[sl][:, iF, :].reshape(Sc, -1)], axis=1)
            DF, hsF = mlp_forward(pDs[k], dshape, F, keep=True)
            sum_DF[k] += float(DF.sum())
            gDc, gF = mlp_backward(pDs[k], dshape, hsF, np.full(Sc, w[k] / S, F64), want_input_grad=True)
            gD[k] += gDc
            if lambda_gp != 0.0:
                b1 = min(n_gp, s0 + Sc)
                if b1 > s0:
                    Pc, gPc = gradient_penalty(pDs[k], dshape, F[:b1 - s0], np.asarray(real[k], F64)[s0:b1],
                                               np.asarray(gp_eps, F64)[k, s0:b1], lambda_gp, w=w[k],
                                               n_total=n_gp)
                    P_gp[k] += Pc
                    gD[k] += gPc
            gF = -gF                                      # L_adv = -w mean D(F)
            nY_, nU_, nF_ = len(iY), len(iU), len(iF)
            np.add.at(gYs, (slice(None), iY), gF[:, :nY_])
            np.add.at(gUs, (slice(None), iU), gF[:, nY_:nY_ + nU_])
            np.add.at(gN, (slice(None), iF), gF[:, nY_ + nU_:nY_ + nU_ + nF_])
            # the coordinates are inputs, not generated: their cotangent is dropped
        # cotangent of r (= of the generated source) from the penalty and the critics
        q = 2.0 * lambda_pde * r / (S * P) + gN.reshape(-1)
        eY = np.exp(jY["y"])
        g_Yval = q * (r + fc)
        g_Ydy = np.stack([-q * eY * jU["dy"][i] for i in range(d)])
        g_Udy = np.stack([-q * eY * jY["dy"][i] for i in range(d)])
        g_Uddy = np.stack([-q * eY for _ in range(d)])
        if trunk:
            gY += trunk_backward(pY, gshape, d, XY, ZY, fY_s, gY=gYs.reshape(-1))
            gY += trunk_backward(pY, gshape, d, XU, ZU, fU_s, gu=gUs.reshape(-1))
            gY += trunk_backward(pY, gshape, d, XC, ZC, jc, gY=g_Yval, gdY=g_Ydy, gdu=g_Udy, gddu=g_Uddy)
        else:
            gY += gen_backward(pY, gshape, d, XY, ZY, fY_s, gYs.reshape(-1))
            gU += gen_backward(pU, gshape, d, XU, ZU, fU_s, gUs.reshape(-1))
            gY += gen_backward(pY, gshape, d, XC, ZC, jY, g_Yval, g_Ydy)
            gU += gen_backward(pU, gshape, d, XC, ZC, jU, np.zeros_like(r), g_Udy, g_Uddy)
    w = np.asarray(w, F64)
    return dict(L_D=w * (sum_DF / S - sum_DR / B) + P_gp, L_adv=-w * sum_DF / S,
                L_pde=lambda_pde * sum_r2 / (S * P), gY=gY, gU=gU, gD=gD, P_gp=P_gp)


def real_snapshots_hier(wl, hin, trunk_teacher=None):
    """Real snapshots [D, B_r, n_in] of a hierarchical step: the teacher pair
    at each critic's Y and u sensors, f = 0 at its free sensors (the true field
    satisfies the equation with the paper's zero source), and the coordinates
    of the real realisations' free sensors (hin.xf_real)."""
    b = hin.base
    gshape = (wl.d + wl.n_z, wl.L, wl.W)
    if trunk_teacher is not None:
        Y = trunk_snapshots(trunk_teacher, gshape, wl.d, b.xsY[0], b.xsU[0], b.z_teach[0])
    else:
        Y = snapshots(b.tY[0], b.tU[0], gshape, wl.d, b.xsY[0], b.xsU[0], b.z_teach[0])
    nY = b.xsY.shape[1]
    Yv, Uv = Y[:, :nY], Y[:, nY:]
    B = Y.shape[0]
    h = hin.hier
    out = []
    for k in range(h.D):
        out.append(np.concatenate([Yv[:, h.idxY[k]], Uv[:, h.idxU[k]], np.zeros((B, h.idxF.shape[1])),
                                   hin.xf_real[:, h.idxF[k], :].reshape(B, -1)], axis=1))
    return np.stack(out)


def real_snapshots(wl, inp):
    """Teacher snapshots [G, B_r, n_in] from the teacher weights and noise z'."""
    gshape = (wl.d + wl.n_z, wl.L, wl.W)
    return np.stack([snapshots(inp.tY[g], inp.tU[g], gshape, wl.d, inp.xsY[g], inp.xsU[g],
                               inp.z_teach[g]) for g in range(inp.z.shape[0])])
