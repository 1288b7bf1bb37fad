"""A training step captured in a HIP graph: every replay, with eager work and
synchronisations between replays, reproduces the eager call's outputs bit for
bit (the library launches only kernels, so the graph holds no memset or copy
nodes), and a replay after the inputs change follows the new inputs."""
import sys

import numpy as np
import pytest
import torch

import oracle
from paper_1910_13444_amd import configs, pigan
from paper_1910_13444_amd.inputs import make_inputs
from _parity import to_dev

pytestmark = pytest.mark.gpu


def _outs(o):
    return [t.detach().cpu().clone() for t in (o.gY, o.gU, o.gD, o.loss, o.nonfinite)]


@pytest.mark.parametrize("dtype,chunk", [("bf16", 0), ("fp32", 2)])
def test_graph_replays_match_eager(dtype, chunk):
    wl = configs.C2.with_(S=5, P=256, B_r=4, dtype=dtype, seed=61)
    print(f"graph replay: C2-shaped {dtype} S=5 chunk_S={chunk}", flush=True)
    sys.stdout.flush()
    inp = make_inputs(wl)
    real = oracle.real_snapshots(wl, inp)
    d = dict(pY=to_dev(inp.pY), pU=to_dev(inp.pU), pD=to_dev(inp.pD), z=to_dev(inp.z), xc=to_dev(inp.xc),
             xsY=to_dev(inp.xsY), xsU=to_dev(inp.xsU), real=to_dev(real), w=to_dev(inp.w_group))
    step = pigan.TrainStep(pigan.step_desc(wl, chunk_S=chunk))

    def call():
        return step(d["pY"], d["pU"], d["pD"], d["z"], d["xc"], d["xsY"], d["xsU"], d["real"], f=None,
                    f_const=wl.f_const, w_group=d["w"])
    eager = _outs(call())
    torch.cuda.synchronize()
    g = pigan.StepGraph(call)
    for rep in range(3):
        for t in (step.out.gY, step.out.gU, step.out.gD, step.out.loss):
            t.fill_(float("nan"))                     # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = _outs(step.out)
        for a, b in zip(got, eager):
            assert torch.equal(a, b), f"replay {rep} differs from the eager call"
    # new inputs, same buffers: the replay follows them
    d["pD"].mul_(1.5)
    ref = _outs(call())
    for t in (step.out.gY, step.out.gU, step.out.gD, step.out.loss):
        t.zero_()
    g.replay()
    torch.cuda.synchronize()
    for a, b in zip(_outs(step.out), ref):
        assert torch.equal(a, b)
    assert not torch.equal(ref[2], eager[2])


def test_graph_replays_trunk_and_hierarchy():
    """The same for the shared-trunk step and the domain-decomposition step
    (grouped critic launches, the snapshot gather and the cotangent scatter)."""
    from paper_1910_13444_amd.inputs import make_hier_inputs
    print("graph replay: trunk 5x128 and 1 + 4 + 16 critic hierarchy, bf16", flush=True)
    wl = configs.T5.with_(S=3, P=256, B_r=3, seed=62)
    inp = make_inputs(wl)
    real = oracle.real_snapshots_trunk(wl, inp)
    dt = dict(pT=to_dev(inp.pT), pD=to_dev(inp.pD), z=to_dev(inp.z), xc=to_dev(inp.xc), xsY=to_dev(inp.xsY),
              xsU=to_dev(inp.xsU), real=to_dev(real), w=to_dev(inp.w_group))
    tstep = pigan.TrunkStep(pigan.trunk_desc(wl))

    def tcall():
        return tstep(dt["pT"], dt["pD"], dt["z"], dt["xc"], dt["xsY"], dt["xsU"], dt["real"], f_const=wl.f_const,
                     w_group=dt["w"])

    wh = configs.H2.with_(S=3, P=1024, B_r=3, seed=63)
    hi = make_hier_inputs(wh, sides=wh.sides, m_sensors=wh.m_sensors, n_free=wh.n_free)
    b, h = hi.base, hi.hier
    realh = oracle.real_snapshots_hier(wh, hi)

    def ti(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()
    dh = dict(pY=to_dev(b.pY[0]), pU=to_dev(b.pU[0]), pD=to_dev(hi.pD), z=to_dev(b.z[0]), xc=to_dev(b.xc[0]),
              xsY=to_dev(b.xsY[0]), xsU=to_dev(b.xsU[0]), iY=ti(h.idxY), iU=ti(h.idxU), iF=ti(h.idxF),
              real=to_dev(realh), w=to_dev(h.w))
    hstep = pigan.HierStep(pigan.hier_desc(wh, h.D, wh.m_sensors, wh.m_sensors, wh.n_free, lambda_pde=0.5))

    def hcall():
        return hstep(dh["pY"], dh["pU"], dh["pD"], dh["z"], dh["xc"], dh["xsY"], dh["xsU"], dh["iY"], dh["iU"],
                     dh["iF"], dh["real"], dh["w"])

    for call, names in ((tcall, ("gT", "gD", "loss", "nonfinite")), (hcall, ("gY", "gU", "gD", "loss", "nonfinite"))):
        o = call()
        eager = [getattr(o, k).detach().cpu().clone() for k in names]
        g = pigan.StepGraph(call)
        for rep in range(3):
            for k in names[:-1]:
                getattr(o, k).fill_(float("nan"))
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            for k, e in zip(names, eager):
                assert torch.equal(getattr(o, k).cpu(), e), f"{k}: replay {rep} differs from the eager call"
