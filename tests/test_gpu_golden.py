"""Parity with every collocation point and sensor of the two largest
single-network workloads (6x512 generators at 4096 points with the 4x1024
critic on 2000 sensors; 6x1024 generators at 2048 points with the 5x2048
critic on 8192 sensors), at 8 noise samples, bf16, against stored fp64
oracle values (tests/golden/make_golden.py writes them from oracle/ alone).

Every loss and bias / output-layer gradient is compared in full; each
weight-gradient matrix G through its norm and the sketches G r and s^T G
(normwise relative errors, which estimate the matrix's own), with the
element-wise error over 256 stored elements printed beside them."""
import os

import numpy as np
import pytest

from paper_1910_13444_amd import configs
from paper_1910_13444_amd.inputs import make_inputs
from _parity import TOL, check, rel, run_step_gpu

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))
S_RED = 8


def _tensors(in_dim, L, W):
    out, off, fan = [], 0, in_dim
    for l in range(1, L + 1):
        out.append((f"W{l}", slice(off, off + W * fan), (W, fan)))
        off += W * fan
        out.append((f"b{l}", slice(off, off + W), None))
        off += W
        fan = W
    out.append(("w_out", slice(off, off + W), None))
    out.append(("b_out", slice(off + W, off + W + 1), None))
    return out


def _compare(g_gpu, shape, prefix, gold, errs, maxe):
    g = np.asarray(g_gpu[0], np.float64)
    for name, sl, mshape in _tensors(*shape):
        key = f"{prefix}.{name}"
        if mshape is None:
            errs[key] = rel(g[sl], gold[key])
            continue
        M = g[sl].reshape(mshape)
        errs[key + ".Gr"] = rel(M @ gold[key + ".r"], gold[key + ".Gr"])
        errs[key + ".sG"] = rel(gold[key + ".s"] @ M, gold[key + ".sG"])
        errs[key + ".norm"] = abs(np.linalg.norm(M) - gold[key + ".norm"][0]) / gold[key + ".norm"][0]
        ref = gold[key + ".val"]
        maxe[key] = float(np.abs(M.ravel()[gold[key + ".idx"]] - ref).max() / np.abs(ref).max())


@pytest.mark.parametrize("wl0", [configs.C3, configs.C5], ids=["w512_p4096", "w1024_p2048"])
def test_step_all_points_reduced_samples(wl0):
    wl = wl0.with_(S=S_RED, B_r=S_RED)
    print(f"stored-oracle step {wl.name} S={wl.S} P={wl.P} sensors={wl.n_sY}+{wl.n_sU}", flush=True)
    gold = np.load(os.path.join(HERE, "golden", f"step_{wl0.name}_S{S_RED}.npz"))
    inp = make_inputs(wl)
    cs = np.array([np.float64(a).sum() for a in (inp.pY, inp.pU, inp.pD, inp.z, inp.xc, inp.xsY, inp.xsU)])
    np.testing.assert_array_equal(cs, gold["inputs_checksum"])      # same seeded draw as the stored step
    out = run_step_gpu(wl, inp, gold["real"])
    assert out["nonfinite"] == 0
    errs, maxe = {}, {}
    for i, k in enumerate(("L_D", "L_adv", "L_pde")):
        errs[k] = rel(out["loss"][:, i], gold["loss"][:, i])
    _compare(out["gY"], wl.gen_shape(), "gY", gold, errs, maxe)
    _compare(out["gU"], wl.gen_shape(), "gU", gold, errs, maxe)
    _compare(out["gD"], wl.disc_shape(), "gD", gold, errs, maxe)
    check(errs, TOL[wl.dtype], f"stored oracle {wl.name}", maxe=maxe)
