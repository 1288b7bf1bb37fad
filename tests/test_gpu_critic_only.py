"""The critic-only step (descriptor field critic_only = 1, used for the
critic updates of the training schedules): the critic's gradient and its
losses must be those of the full step, bit for bit (the skipped work feeds
neither), for the paired, shared-trunk and domain-decomposition steps, with
and without the gradient penalty and with several sample chunks.  The paired
and trunk steps skip the collocation rows too and report L_pde = 0; the
domain-decomposition steps evaluate the residual (their critics read the
generated source) and report it."""
import numpy as np
import pytest

import oracle
from paper_1910_13444_amd import configs
from paper_1910_13444_amd.inputs import make_hier_inputs, make_inputs
from _parity import run_hier_gpu, run_hier_trunk_gpu, run_step_gpu, run_trunk_gpu

pytestmark = pytest.mark.gpu


def _same(a, b, residual=False):
    assert a["nonfinite"] == 0 and b["nonfinite"] == 0
    for k in ("gD",) + (("P_gp",) if "P_gp" in a else ()):
        np.testing.assert_array_equal(b[k], a[k])
    if residual:
        np.testing.assert_array_equal(b["loss"], a["loss"])
    else:
        np.testing.assert_array_equal(b["loss"][:, :2], a["loss"][:, :2])
        assert (b["loss"][:, 2] == 0).all() and (a["loss"][:, 2] != 0).any()


@pytest.mark.parametrize("dtype,chunk,lgp", [("bf16", 0, 0.0), ("bf16", 2, 0.0), ("fp32", 2, 0.7)])
def test_critic_only_pair(dtype, chunk, lgp):
    wl = configs.C2.with_(S=5, P=256, B_r=3, dtype=dtype)
    print(f"critic-only pair step dtype={dtype} chunk_S={chunk} lambda_gp={lgp}", flush=True)
    inp = make_inputs(wl)
    real = oracle.real_snapshots(wl, inp)
    eps = np.random.default_rng(3).random((wl.G, 3)).astype(np.float32) if lgp > 0 else None
    kw = dict(chunk_S=chunk, lambda_gp=lgp, gp_eps=eps)
    _same(run_step_gpu(wl, inp, real, **kw), run_step_gpu(wl, inp, real, critic_only=True, **kw))


def test_critic_only_trunk():
    wl = configs.T5.with_(S=3, P=256, B_r=3)
    print("critic-only trunk step bf16", flush=True)
    inp = make_inputs(wl)
    real = oracle.real_snapshots_trunk(wl, inp)
    _same(run_trunk_gpu(wl, inp, real), run_trunk_gpu(wl, inp, real, critic_only=True))


@pytest.mark.parametrize("trunk", [False, True], ids=["pair", "trunk"])
def test_critic_only_hier(trunk):
    base = configs.HT5 if trunk else configs.C2.with_(n_sY=256, n_sU=256)
    wl = base.with_(S=4, P=256, B_r=4, seed=98)
    print(f"critic-only hierarchical step trunk={trunk} bf16", flush=True)
    hi = make_hier_inputs(wl, sides=(1, 2, 4), m_sensors=16, n_free=16)
    if trunk:
        real = oracle.real_snapshots_hier(wl, hi, trunk_teacher=hi.base.tT[0])
        a = run_hier_trunk_gpu(wl, hi, real, lam=0.5)
        b = run_hier_trunk_gpu(wl, hi, real, lam=0.5, critic_only=True)
    else:
        real = oracle.real_snapshots_hier(wl, hi)
        a = run_hier_gpu(wl, hi, real, lam=0.5)
        b = run_hier_gpu(wl, hi, real, lam=0.5, critic_only=True)
    _same(a, b, residual=True)
