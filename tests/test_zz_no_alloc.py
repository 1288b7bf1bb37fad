"""pigan_train_step_grads_noalloc (the step with its workspace in the
library's fixed device array) against pigan_train_step_grads on the same
inputs: two calls in a row, the second smaller, in fp32 and bf16; the
outputs must be identical (same plan, same kernels).  A step needing more
than the array is refused before anything is launched."""
import numpy as np
import pytest

import oracle
from paper_1910_13444_amd import configs, pigan
from paper_1910_13444_amd.inputs import make_inputs
from _parity import to_dev

pytestmark = pytest.mark.gpu


def _outputs(wl, inp, real, noalloc):
    import torch
    desc = pigan.step_desc(wl, S=inp.z.shape[1], B_r=real.shape[1])
    step = pigan.TrainStep(desc, noalloc=noalloc)
    o = step(to_dev(inp.pY), to_dev(inp.pU), to_dev(inp.pD), to_dev(inp.z), to_dev(inp.xc), to_dev(inp.xsY),
             to_dev(inp.xsU), to_dev(real), f=None if inp.f is None else to_dev(inp.f), f_const=inp.f_const,
             w_group=to_dev(inp.w_group))
    torch.cuda.synchronize()
    return {k: getattr(o, k).cpu().numpy().copy() for k in ("gY", "gU", "gD", "loss", "nonfinite")}


@pytest.mark.parametrize("wls", [
    (configs.C1, configs.C1.with_(S=16, P=16, B_r=16)),
    (configs.C2.with_(S=4, P=256, B_r=4), configs.C2.with_(S=2, P=128, B_r=2)),
], ids=["fp32_toy", "bf16_2d"])
def test_noalloc_step_matches_workspace_step(wls):
    for wl in wls:                      # the second call is smaller than the first
        print(f"no-allocation step {wl.name} S={wl.S} P={wl.P}", flush=True)
        inp = make_inputs(wl, f_array=True)
        real = oracle.real_snapshots(wl, inp)
        a = _outputs(wl, inp, real, noalloc=False)
        b = _outputs(wl, inp, real, noalloc=True)
        assert int(b["nonfinite"][0]) == 0
        for k in ("gY", "gU", "gD", "loss"):
            np.testing.assert_array_equal(b[k], a[k])


def test_noalloc_step_refuses_a_step_beyond_its_array():
    import torch
    wl = configs.C2                      # about 5.6 GiB of workspace
    desc = pigan.step_desc(wl)
    assert pigan.workspace_bytes(desc) > (128 << 20)
    dummy = torch.zeros(1, device="cuda")
    st = pigan.lib().pigan_train_step_grads_noalloc(pigan.C.byref(desc), *[pigan.C.c_void_p(dummy.data_ptr())] * 8,
                                                   0.0, *[pigan.C.c_void_p(dummy.data_ptr())] * 8, None)
    assert st == 3                       # PIGAN_EWORKSPACE, nothing launched
    assert b"holds" in pigan.lib().pigan_last_error()
