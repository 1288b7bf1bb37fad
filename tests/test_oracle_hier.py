"""Pins of the oracle's domain-decomposition step (train_step_hier): reduction
to the plain step, central differences of every generator and critic weight
gradient (with free sensors and the residual penalty both active), invariance
under permuting the critics, the zero-critic limit, and chunking."""
import numpy as np
import pytest

import oracle
from paper_1910_13444_amd import configs
from paper_1910_13444_amd.inputs import glorot_mlp, make_hier_inputs

WL = configs.C2.with_(n_sY=16, n_sU=16, S=3, P=16, B_r=2, W=5, W_D=4, L=2, L_D=1, n_z=2, dtype="fp32", seed=77)


def _setup(wl=WL, sides=(1, 2), m=4, nf=4):
    hi = make_hier_inputs(wl, sides=sides, m_sensors=m, n_free=nf)
    real = oracle.real_snapshots_hier(wl, hi)
    return hi, real


def _run(wl, hi, real, pY=None, pU=None, pDs=None, lam=0.5, chunk=None, idx=None, w=None):
    b, h = hi.base, hi.hier
    iY, iU, iF = idx if idx is not None else (h.idxY, h.idxU, h.idxF)
    dshape = (real.shape[2], wl.L_D, wl.W_D)
    return oracle.train_step_hier(wl.gen_shape(), dshape, wl.d, b.pY[0] if pY is None else pY,
                                  b.pU[0] if pU is None else pU, hi.pD if pDs is None else pDs, b.z[0], b.xc[0],
                                  b.xsY[0], b.xsU[0], np.full((wl.S, wl.P), 0.3), iY, iU, iF, real,
                                  h.w if w is None else w, lambda_pde=lam, chunk_S=chunk)


def test_one_critic_on_every_sensor_is_the_plain_step():
    wl = WL
    hi, _ = _setup()
    b = hi.base
    inp_real = oracle.real_snapshots(wl, b)[0]                 # [B, n_sY + n_sU]
    pD = glorot_mlp(np.random.default_rng(1), wl.n_sY + wl.n_sU, wl.L_D, wl.W_D).astype(np.float64)
    idx = (np.arange(wl.n_sY)[None], np.arange(wl.n_sU)[None], np.zeros((1, 0), np.int64))
    o = _run(wl, hi, inp_real[None], pDs=pD[None], idx=idx, w=np.array([0.7]), lam=0.9)
    ref = oracle.train_step_group(wl.gen_shape(), wl.disc_shape(), wl.d, b.pY[0], b.pU[0], pD, b.z[0], b.xc[0],
                                  b.xsY[0], b.xsU[0], np.full((wl.S, wl.P), 0.3), inp_real, w=0.7, lambda_pde=0.9 / 0.7)
    # the plain step weights its residual by w too: lambda_pde / w there equals lambda_pde here
    assert np.isclose(o["L_D"][0], ref["L_D"], rtol=1e-13)
    assert np.isclose(o["L_adv"][0] + o["L_pde"], ref["L_adv"] + ref["L_pde"], rtol=1e-13)
    assert np.allclose(o["gY"], ref["gY"], rtol=1e-12, atol=1e-15)
    assert np.allclose(o["gU"], ref["gU"], rtol=1e-12, atol=1e-15)
    assert np.allclose(o["gD"][0], ref["gD"], rtol=1e-12, atol=1e-15)


def test_hier_grads_fd():
    wl = WL
    hi, real = _setup()
    o = _run(wl, hi, real)
    b = hi.base
    h = 1e-6

    def LG(pY, pU):
        r = _run(wl, hi, real, pY=pY, pU=pU)
        return r["L_adv"].sum() + r["L_pde"]

    for name, p0 in (("Y", b.pY[0].astype(np.float64)), ("U", b.pU[0].astype(np.float64))):
        fd = np.zeros_like(p0)
        for k in range(p0.size):
            e = np.zeros_like(p0)
            e[k] = h
            if name == "Y":
                fd[k] = (LG(p0 + e, b.pU[0]) - LG(p0 - e, b.pU[0])) / (2 * h)
            else:
                fd[k] = (LG(b.pY[0], p0 + e) - LG(b.pY[0], p0 - e)) / (2 * h)
        g = o["g" + name]
        assert np.abs(g - fd).max() <= 1e-6 * max(1.0, np.abs(fd).max()), name
        assert np.abs(g).max() > 1e-4
    pDs = hi.pD.astype(np.float64)
    for k in (0, 3):
        fd = np.zeros(pDs.shape[1])
        for j in range(pDs.shape[1]):
            pp, pm = pDs.copy(), pDs.copy()
            pp[k, j] += h
            pm[k, j] -= h
            fd[j] = (_run(wl, hi, real, pDs=pp)["L_D"].sum() - _run(wl, hi, real, pDs=pm)["L_D"].sum()) / (2 * h)
        assert np.abs(o["gD"][k] - fd).max() <= 1e-6 * max(1.0, np.abs(fd).max())


def test_permuting_the_critics():
    wl = WL
    hi, real = _setup()
    h = hi.hier
    perm = np.array([3, 0, 4, 1, 2])
    a = _run(wl, hi, real)
    b = _run(wl, hi, real[perm], pDs=hi.pD[perm], idx=(h.idxY[perm], h.idxU[perm], h.idxF[perm]), w=h.w[perm])
    assert np.allclose(b["L_D"], a["L_D"][perm], rtol=1e-12, atol=1e-16)
    assert np.allclose(b["gD"], a["gD"][perm], rtol=1e-12, atol=1e-16)
    assert np.allclose(b["gY"], a["gY"], rtol=1e-11, atol=1e-16)
    assert np.allclose(b["gU"], a["gU"], rtol=1e-11, atol=1e-16)


def test_zero_critics_leave_the_residual_gradient():
    """Critics with zero output weights see nothing: the generator gradient is
    the residual penalty's alone, as in the plain step with a zero critic."""
    wl = WL
    hi, real = _setup()
    pDs = hi.pD.astype(np.float64).copy()
    nD = pDs.shape[1]
    pDs[:, nD - wl.W_D - 1:] = 0.0
    o = _run(wl, hi, real, pDs=pDs, lam=0.8)
    b = hi.base
    pD1 = np.zeros(configs.n_params(wl.n_sY + wl.n_sU, wl.L_D, wl.W_D))
    ref = oracle.train_step_group(wl.gen_shape(), wl.disc_shape(), wl.d, b.pY[0], b.pU[0], pD1, b.z[0], b.xc[0],
                                  b.xsY[0], b.xsU[0], np.full((wl.S, wl.P), 0.3),
                                  oracle.real_snapshots(wl, b)[0], w=1.0, lambda_pde=0.8)
    assert np.allclose(o["gY"], ref["gY"], rtol=1e-12, atol=1e-16)
    assert np.allclose(o["gU"], ref["gU"], rtol=1e-12, atol=1e-16)
    assert np.allclose(o["L_adv"], 0.0) and np.isclose(o["L_pde"], ref["L_pde"], rtol=1e-13)


def test_hier_chunking():
    wl = WL
    hi, real = _setup()
    a = _run(wl, hi, real)
    b = _run(wl, hi, real, chunk=1)
    for k in ("L_D", "L_adv", "gY", "gU", "gD"):
        assert np.allclose(a[k], b[k], rtol=1e-12, atol=1e-15)


def _trunk_setup():
    wl = WL.with_(arch="hier_trunk", L=3, W=4)
    hi = make_hier_inputs(wl, sides=(1, 2), m_sensors=4, n_free=4)
    real = oracle.real_snapshots_hier(wl, hi, trunk_teacher=hi.base.tT[0])
    return wl, hi, real


def _run_trunk(wl, hi, real, pT=None, pDs=None, lam=0.5, idx=None, w=None):
    b, h = hi.base, hi.hier
    iY, iU, iF = idx if idx is not None else (h.idxY, h.idxU, h.idxF)
    return oracle.train_step_hier(wl.gen_shape(), (real.shape[2], wl.L_D, wl.W_D), wl.d,
                                  b.pT[0] if pT is None else pT, None, hi.pD if pDs is None else pDs, b.z[0],
                                  b.xc[0], b.xsY[0], b.xsU[0], np.full((wl.S, wl.P), 0.3), iY, iU, iF, real,
                                  h.w if w is None else w, lambda_pde=lam, trunk=True)


def test_trunk_hier_one_critic_is_the_trunk_step():
    wl, hi, _ = _trunk_setup()
    b = hi.base
    real = oracle.real_snapshots_trunk(wl, b)[0]
    pD = glorot_mlp(np.random.default_rng(2), wl.n_sY + wl.n_sU, wl.L_D, wl.W_D).astype(np.float64)
    idx = (np.arange(wl.n_sY)[None], np.arange(wl.n_sU)[None], np.zeros((1, 0), np.int64))
    o = _run_trunk(wl, hi, real[None], pDs=pD[None], idx=idx, w=np.array([0.6]), lam=0.9)
    ref = oracle.train_step_group_trunk(wl.gen_shape(), wl.disc_shape(), wl.d, b.pT[0], pD, b.z[0], b.xc[0],
                                        b.xsY[0], b.xsU[0], np.full((wl.S, wl.P), 0.3), real, w=0.6,
                                        lambda_pde=0.9 / 0.6)
    assert np.isclose(o["L_D"][0], ref["L_D"], rtol=1e-13)
    assert np.allclose(o["gY"], ref["gT"], rtol=1e-12, atol=1e-15)
    assert np.allclose(o["gD"][0], ref["gD"], rtol=1e-12, atol=1e-15)


def test_trunk_hier_grads_fd():
    wl, hi, real = _trunk_setup()
    o = _run_trunk(wl, hi, real)
    p0 = hi.base.pT[0].astype(np.float64)
    h = 1e-6
    fd = np.zeros_like(p0)
    for k in range(p0.size):
        e = np.zeros_like(p0)
        e[k] = h
        a = _run_trunk(wl, hi, real, pT=p0 + e)
        b = _run_trunk(wl, hi, real, pT=p0 - e)
        fd[k] = ((a["L_adv"].sum() + a["L_pde"]) - (b["L_adv"].sum() + b["L_pde"])) / (2 * h)
    assert np.abs(o["gY"] - fd).max() <= 1e-6 * max(1.0, np.abs(fd).max())
    assert np.abs(o["gY"]).max() > 1e-4


def test_hier_gradient_penalty_fd():
    """Each subdomain critic's gradient penalty: central differences of the
    summed L_D (with the penalties) in two critics' weights; the generator
    gradients are unchanged; each P_gp[k] > 0 is added to L_D[k]."""
    wl = WL
    hi, real = _setup()
    h = hi.hier
    eps = np.random.default_rng(9).random((h.D, min(wl.S, real.shape[1])))
    lam = 4.0

    def run(pDs):
        b = hi.base
        return oracle.train_step_hier(wl.gen_shape(), (real.shape[2], wl.L_D, wl.W_D), wl.d, b.pY[0], b.pU[0], pDs,
                                      b.z[0], b.xc[0], b.xsY[0], b.xsU[0], np.full((wl.S, wl.P), 0.3), h.idxY,
                                      h.idxU, h.idxF, real, h.w, lambda_pde=0.5, lambda_gp=lam, gp_eps=eps)
    pDs = hi.pD.astype(np.float64)
    o = run(pDs)
    o0 = _run(wl, hi, real)
    assert np.all(o["P_gp"] > 0)
    assert np.allclose(o["L_D"], o0["L_D"] + o["P_gp"], rtol=1e-13)
    assert np.array_equal(o["gY"], o0["gY"]) and np.array_equal(o["gU"], o0["gU"])
    hstep = 1e-6
    for k in (0, 3):
        fd = np.zeros(pDs.shape[1])
        for j in range(pDs.shape[1]):
            pp, pm = pDs.copy(), pDs.copy()
            pp[k, j] += hstep
            pm[k, j] -= hstep
            fd[j] = (run(pp)["L_D"].sum() - run(pm)["L_D"].sum()) / (2 * hstep)
        assert np.abs(o["gD"][k] - fd).max() <= 1e-6 * max(1.0, np.abs(fd).max())
        assert np.abs(o["gD"][k] - o0["gD"][k]).max() > 1e-5
