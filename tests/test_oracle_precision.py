"""Pins of the oracle's precision models (used only to size the parity bar of
ill-conditioned tensors): the bf16 rounding matches torch's round-to-nearest-
even conversion, fp16 matches numpy's, and each model stays close to, but not
equal to, the exact result."""
import numpy as np
import torch

import oracle
from oracle.pigan_oracle import _round_bf16
from paper_1910_13444_amd.inputs import make_inputs
from _parity import rel
from _tiny import TINY2


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = rng.standard_normal(200000) * 10.0 ** rng.integers(-30, 30, 200000)
    # exact ties: bf16 has 8 significant bits, so values with 9 bits end in a tie
    ties = (rng.integers(256, 512, 2000) * 2.0 + 1.0) * 2.0 ** rng.integers(-20, 20, 2000)
    x = np.concatenate([x, ties, -ties])
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(_round_bf16(x), ref)


def test_precision_models_are_close_but_not_exact():
    wl = TINY2.with_(W=16, W_D=16, S=3, P=8)
    inp = make_inputs(wl, f_array=True)
    real = np.random.default_rng(1).standard_normal((1, wl.B_r, wl.n_in))
    ex = oracle.train_step(wl, inp, real)
    for prec, lo, hi in (("fp32", 1e-9, 1e-5), ("bf16", 1e-5, 5e-2), ("fp16", 1e-6, 1e-2)):
        m = oracle.train_step(wl, inp, real, prec=prec)
        for k in ("gY", "gU", "gD"):
            e = rel(m[k], ex[k])
            assert lo < e < hi, (prec, k, e)
    # the fp32 model leaves the module's working type untouched
    assert oracle.pigan_oracle.F64 is np.float64
