"""GPU parity of the training step with the critic gradient penalty
(pigan_train_step_grads_gp) against the fp64 oracle: every critic weight
gradient, L_D (which includes the penalty) and the penalty itself; the
generator gradients are the plain step's, bit for bit; chunking and a real
batch smaller than the fake batch (fewer pairs than samples)."""
import numpy as np
import pytest

import oracle
from paper_1910_13444_amd import configs
from paper_1910_13444_amd.inputs import make_inputs
from _parity import TOL, amax_rel, check, rel, run_step_gpu, step_errors
from _tiny import TINY2

pytestmark = pytest.mark.gpu

LAM = 10.0

CASES = {
    "tiny2d_fp32": TINY2.with_(W=32, W_D=32),
    "c1_full_fp32": configs.C1,
    "c2_S3_bf16": configs.C2.with_(S=3, P=256, B_r=3),
    "c4_groups_S2_bf16": configs.C4.with_(S=2, P=96, B_r=2),
    "c2_S4_fp32": configs.C2.with_(S=4, P=128, B_r=4, dtype="fp32"),
}


def _eps(wl, S, B):
    return np.random.default_rng(wl.seed + 5).random((wl.G, min(S, B))).astype(np.float32)


def _case(wl, label, chunk_S=0, B_r=None):
    print(f"gradient penalty case={label} dtype={wl.dtype} G={wl.G} S={wl.S} W_D={wl.W_D}", flush=True)
    inp = make_inputs(wl)
    real = oracle.real_snapshots(wl, inp)
    if B_r is not None:
        real = real[:, :B_r].copy()
    eps = _eps(wl, wl.S, real.shape[1])
    ref = oracle.train_step(wl, inp, real, lambda_gp=LAM, gp_eps=eps)
    out = run_step_gpu(wl, inp, real, chunk_S=chunk_S, lambda_gp=LAM, gp_eps=eps)
    assert out["nonfinite"] == 0
    assert np.all(ref["P_gp"] > 0)
    plain = run_step_gpu(wl, inp, real, chunk_S=chunk_S)
    np.testing.assert_array_equal(out["gY"], plain["gY"])
    np.testing.assert_array_equal(out["gU"], plain["gU"])
    errs = step_errors(wl, out, ref)
    if wl.dtype == "fp32":
        # the penalty's own weight gradient, isolated from the critic term
        ref_plain = oracle.train_step(wl, inp, real)
        errs["gD_penalty_part"] = max(rel(out["gD"][g] - plain["gD"][g], ref["gD"][g] - ref_plain["gD"][g])
                                      for g in range(wl.G))
    check(errs, TOL[wl.dtype], label, maxe=step_errors(wl, out, ref, amax_rel))


@pytest.mark.parametrize("case", list(CASES))
def test_step_with_gradient_penalty(case):
    _case(CASES[case], case)


def test_gradient_penalty_chunked_and_fewer_pairs():
    wl = configs.C2.with_(S=5, P=128, B_r=5, dtype="fp32")
    _case(wl, "c2_S5_chunk2_fp32", chunk_S=2)
    _case(wl, "c2_S5_Br3_fp32", chunk_S=2, B_r=3)
