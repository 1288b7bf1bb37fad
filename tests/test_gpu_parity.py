"""GPU parity: the HIP path through the C-ABI against the fp64 oracle on the
same seeded inputs.

Metric: normwise relative error per tensor (every jet component, the residual
r and r + f separately, every layer's weight and bias gradient, each loss),
with max|d| / max|oracle| printed beside it.  Bar: 1e-5 in fp32 mode, 2e-2 in
bf16/fp16 mode, for every tensor."""
import sys

import numpy as np
import pytest

import oracle
from paper_1910_13444_amd import configs, pigan
from paper_1910_13444_amd.inputs import glorot_mlp, make_inputs
from _parity import TOL, amax_rel, check, rel, run_step_gpu, step_errors, to_dev
from _tiny import TINY1, TINY2, TINY3

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


# ---------------------------------------------------------------------------
# generator jets
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("dtype", ["fp32", "bf16", "fp16"])
@pytest.mark.parametrize("d,order,x_shared,L,W,S,P", [
    (1, 2, False, 3, 32, 5, 37),
    (2, 2, False, 3, 128, 3, 211),
    (2, 2, False, 3, 128, 20, 500),
    (1, 2, False, 3, 128, 4, 300),
    (2, 1, False, 2, 128, 3, 97),
    (2, 1, True, 2, 64, 4, 100),
    (2, 0, False, 4, 256, 2, 150),
    (3, 2, False, 2, 128, 2, 70),
    (3, 1, False, 2, 512, 2, 45),
])
def test_gen_forward(dtype, d, order, x_shared, L, W, S, P):
    _say(f"gen_forward dtype={dtype} d={d} order={order} shared={x_shared} L={L} W={W} S={S} P={P}")
    import torch
    rng = np.random.default_rng(100 + d * 10 + order)
    n_z = 5
    shape = (d + n_z, L, W)
    p = np.stack([glorot_mlp(rng, *shape), glorot_mlp(rng, *shape)])  # G = 2
    p[:, -1] = 0.3
    z = rng.standard_normal((2, S, n_z)).astype(np.float32)
    x = rng.random((2, P, d) if x_shared else (2, S, P, d)).astype(np.float32)
    jet = pigan.gen_forward(to_dev(p), shape, d, to_dev(z), to_dev(x), order, dtype=dtype, x_shared=x_shared)
    torch.cuda.synchronize()
    jet = jet.cpu().numpy()
    for g in range(2):
        ref = oracle.gen_jets(p[g], shape, d, z[g], x[g], order)
        errs = {f"g{g}.c{k}": rel(jet[g, k], ref[k]) for k in range(ref.shape[0])}
        check(errs, TOL[dtype], "gen_forward")


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
def test_gen_forward_saturated(dtype):
    """Every hidden unit saturated: biases of magnitude 5 to 10 put |a| in
    about [4, 11], where 1 - tanh^2 computed from tanh in fp32 loses most of
    its digits (s = 4.5e-7 at |a| = 8 next to an fp32 spacing of 6e-8 near 1)
    while the jets are built from s alone.  The oracle's fp64 1 - tanh^2
    keeps about 1e-6 relative accuracy up to |a| = 12."""
    _say(f"gen_forward saturated units dtype={dtype}")
    import torch
    from oracle.pigan_oracle import unpack
    rng = np.random.default_rng(77)
    d, n_z, L, W, S, P = 2, 5, 3, 128, 3, 200
    shape = (d + n_z, L, W)
    p = glorot_mlp(rng, *shape)
    off = 0
    fan = d + n_z
    for _ in range(L):                       # biases +-[5, 10]
        off += W * fan
        p[off:off + W] = rng.choice([-1.0, 1.0], W) * rng.uniform(5.0, 10.0, W)
        off += W
        fan = W
    p = p[None]
    z = rng.standard_normal((1, S, n_z)).astype(np.float32)
    x = rng.random((1, S, P, d)).astype(np.float32)
    layers, _, _ = unpack(p[0], *shape)
    a1 = x[0].reshape(-1, d) @ layers[0][0][:, :d].T.astype(np.float64) + \
        np.repeat(z[0], P, 0) @ layers[0][0][:, d:].T.astype(np.float64) + layers[0][1]
    assert np.abs(a1).min() > 3.5 and np.abs(a1).max() < 12.0
    jet = pigan.gen_forward(to_dev(p), shape, d, to_dev(z), to_dev(x), 2, dtype=dtype)
    torch.cuda.synchronize()
    jet = jet.cpu().numpy()[0]
    ref = oracle.gen_jets(p[0], shape, d, z[0], x[0], 2)
    assert np.abs(ref[1:]).max() < 1e-2 * np.abs(ref[0]).max()   # the derivative jets are small: s is tiny
    check({f"c{k}": rel(jet[k], ref[k]) for k in range(ref.shape[0])}, TOL[dtype], "gen_forward saturated",
          maxe={f"c{k}": amax_rel(jet[k], ref[k]) for k in range(ref.shape[0])})


def test_pde_residual():
    import torch
    rng = np.random.default_rng(5)
    for d in (1, 2, 3):
        G, M = 3, 1234
        jY = rng.standard_normal((G, 1 + d, M)).astype(np.float32) * 0.5
        jU = rng.standard_normal((G, 1 + 2 * d, M)).astype(np.float32)
        f = rng.standard_normal((G, M)).astype(np.float32)
        for ff, fc in ((f, 0.0), (None, 0.75)):
            r = pigan.pde_residual(to_dev(jY), to_dev(jU), d, None if ff is None else to_dev(ff), fc)
            torch.cuda.synchronize()
            r = r.cpu().numpy()
            fv = ff if ff is not None else np.full((G, M), fc)
            for g in range(G):
                ref = oracle.darcy_residual(jY[g, 0], jY[g, 1:], jU[g, 1:1 + d], jU[g, 1 + d:], fv[g])
                assert rel(r[g], ref) < 1e-6
                assert rel(r[g] + fv[g], ref + fv[g]) < 1e-6


@pytest.mark.parametrize("dtype", ["fp32", "bf16"])
@pytest.mark.parametrize("n_in,L,W,B", [(16, 2, 32, 64), (250, 3, 64, 37), (400, 2, 256, 70)])
def test_disc_forward(dtype, n_in, L, W, B):
    _say(f"disc_forward dtype={dtype} n_in={n_in} L={L} W={W} B={B}")
    import torch
    rng = np.random.default_rng(n_in)
    shape = (n_in, L, W)
    p = np.stack([glorot_mlp(rng, *shape) for _ in range(2)])
    p[:, -1] = -0.2
    snap = rng.standard_normal((2, B, n_in)).astype(np.float32)
    sc = pigan.disc_forward(to_dev(p), shape, to_dev(snap), dtype=dtype)
    torch.cuda.synchronize()
    sc = sc.cpu().numpy()
    for g in range(2):
        ref = oracle.mlp_forward(p[g], shape, snap[g])
        check({f"g{g}": rel(sc[g], ref)}, TOL[dtype], "disc_forward")


# ---------------------------------------------------------------------------
# training step
# ---------------------------------------------------------------------------
STEP_CASES = {
    "tiny2d_fp32": (TINY2.with_(W=32, W_D=32), dict(f_array=True)),
    "tiny1d_fp32": (TINY1.with_(W=32, W_D=64), {}),
    "tiny3d_groups_fp32": (TINY3.with_(W=64, W_D=32, S=3, P=40), {}),
    "c1_full_fp32": (configs.C1, {}),
    "c2_S3_ragged_bf16": (configs.C2.with_(S=3, P=1000, B_r=3), {}),
    "c2_S3_fp32": (configs.C2.with_(S=3, P=333, B_r=4, dtype="fp32"), dict(f_array=True)),
    "c4_groups_S2_bf16": (configs.C4.with_(S=2, P=96, B_r=2), {}),
    "c3_S2_bf16": (configs.C3.with_(S=2, P=256, B_r=2), {}),
    "c5_S2_bf16": (configs.C5.with_(S=2, P=128, B_r=2), {}),
    # ragged collocation rows (R not a multiple of the 32-row weight-gradient
    # stage, points not a multiple of the 32-point reverse tile) at widths
    # 512 and 256, whose weight gradients take the 256 x 256 and 128 x 256 tiles
    "c3_S2_ragged_bf16": (configs.C3.with_(S=2, P=250, B_r=2), {}),
    "c4_groups_S2_ragged_bf16": (configs.C4.with_(S=2, P=100, B_r=2), {}),
    "c2_S3_ragged_bf16_f": (configs.C2.with_(S=3, P=1000, B_r=3), dict(f_array=True)),
    "c3_S2_fp32": (configs.C3.with_(S=2, P=256, B_r=2, dtype="fp32"), {}),
    "c4_groups_S2_fp32": (configs.C4.with_(S=2, P=96, B_r=2, dtype="fp32"), {}),
    "c5_S2_fp32": (configs.C5.with_(S=2, P=128, B_r=2, dtype="fp32"), {}),
}


_EXACT = {}


def _oracle_step(wl, inp, key):
    """Exact oracle result (cached per input key) and the real snapshots."""
    if key not in _EXACT:
        real = oracle.real_snapshots(wl, inp)
        _EXACT[key] = (real, oracle.train_step(wl, inp, real))
    return _EXACT[key]


def _step_case(wl, inp, key, label, **kw):
    real, ref = _oracle_step(wl, inp, key)
    out = run_step_gpu(wl, inp, real, **kw)
    assert out["nonfinite"] == 0
    check(step_errors(wl, out, ref), TOL[wl.dtype], label, maxe=step_errors(wl, out, ref, amax_rel))


@pytest.mark.parametrize("case", list(STEP_CASES))
def test_train_step(case):
    wl, kw = STEP_CASES[case]
    _say(f"train_step case={case} dtype={wl.dtype} G={wl.G} S={wl.S} P={wl.P} W={wl.W} W_D={wl.W_D}")
    inp = make_inputs(wl, **kw)
    _step_case(wl, inp, (wl.seed, wl.S, wl.P, wl.G, str(kw)), case)


def test_train_step_fp16_loss_scale():
    wl = configs.C5H.with_(S=2, P=128, B_r=2)
    _say("train_step fp16 C5-shaped with loss scale 1024")
    inp = make_inputs(wl)
    _step_case(wl, inp, (wl.seed, wl.S, wl.P, wl.G, "{}"), "c5_fp16", loss_scale=1024.0)


def test_chunking_matches_unchunked():
    wl = configs.C2.with_(S=5, P=300, B_r=4)
    _say("chunking S=5 chunk 2 vs whole")
    inp = make_inputs(wl, f_array=True)
    real = oracle.real_snapshots(wl, inp)
    a = run_step_gpu(wl, inp, real)
    b = run_step_gpu(wl, inp, real, chunk_S=2)
    errs = {k: rel(b[k], a[k]) for k in ("gY", "gU", "gD", "loss")}
    check(errs, 1e-5, "chunking")


def test_deterministic():
    wl = configs.C2.with_(S=4, P=512, B_r=4)
    _say("determinism")
    inp = make_inputs(wl)
    real = oracle.real_snapshots(wl, inp)
    a = run_step_gpu(wl, inp, real)
    b = run_step_gpu(wl, inp, real)
    for k in ("gY", "gU", "gD", "loss"):
        np.testing.assert_array_equal(a[k], b[k])


def test_nonfinite_flag():
    wl = configs.C1.with_(S=4, P=16, B_r=4)
    _say("nonfinite flag")
    inp = make_inputs(wl)
    real = oracle.real_snapshots(wl, inp)
    assert run_step_gpu(wl, inp, real)["nonfinite"] == 0
    inp.z[0, 1, 0] = np.nan
    assert run_step_gpu(wl, inp, real)["nonfinite"] == 1
