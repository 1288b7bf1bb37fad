"""Helpers of the GPU parity tests: run the HIP path through the C-ABI and
compare it tensor by tensor with the fp64 oracle."""
from __future__ import annotations

import numpy as np

TOL = {"fp32": 1e-5, "bf16": 2e-2, "fp16": 2e-2}


def rel(a, b) -> float:
    a = np.asarray(a, np.float64).ravel()
    b = np.asarray(b, np.float64).ravel()
    den = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / den) if den > 0 else float(np.linalg.norm(a))


def param_slices(in_dim, L, W):
    """(name, slice) of every weight tensor in the packed parameter vector."""
    out = []
    off = 0
    fan = in_dim
    for l in range(1, L + 1):
        out.append((f"W{l}", slice(off, off + W * fan)))
        off += W * fan
        out.append((f"b{l}", slice(off, off + W)))
        off += W
        fan = W
    out.append(("w_out", slice(off, off + W)))
    out.append(("b_out", slice(off + W, off + W + 1)))
    return out


def grad_errors(g_gpu, g_ref, shape, prefix):
    errs = {}
    G = g_ref.shape[0]
    for name, sl in param_slices(*shape):
        if name == "b_out" and shape is not None:
            # a single scalar per group: compare all groups together
            errs[f"{prefix}.{name}"] = rel(g_gpu[:, sl], g_ref[:, sl])
            continue
        errs[f"{prefix}.{name}"] = max(rel(g_gpu[g, sl], g_ref[g, sl]) for g in range(G))
    return errs


def check(errs: dict, tol: float, label: str = ""):
    bad = {k: v for k, v in errs.items() if not (v <= tol)}
    worst = sorted(errs.items(), key=lambda kv: -kv[1])[:6]
    msg = f"{label} tol={tol:g} worst: " + ", ".join(f"{k}={v:.3g}" for k, v in worst)
    print(msg)
    assert not bad, msg


COND_FACTOR = 3.0


def check_conditioned(errs: dict, errs_model: dict, tol: float, label: str = ""):
    """Per-tensor bar: err <= max(tol, COND_FACTOR * err_model), where err_model
    is the distance of the oracle's own precision model (same storage format,
    fp32 accumulation) from the exact result.  A tensor whose value is a sum of
    nearly cancelling terms amplifies storage rounding; the precision model
    measures that amplification on the same inputs."""
    lim = {k: max(tol, COND_FACTOR * errs_model.get(k, 0.0)) for k in errs}
    bad = {k: (v, lim[k]) for k, v in errs.items() if not (v <= lim[k])}
    ratio = sorted(((v / lim[k], k) for k, v in errs.items()), reverse=True)[:6]
    msg = (f"{label} tol={tol:g} worst err/limit: "
           + ", ".join(f"{k}={errs[k]:.3g}/{lim[k]:.3g}" for _, k in ratio))
    print(msg)
    assert not bad, msg


def to_dev(a, dev="cuda"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)


def run_step_gpu(wl, inp, real, chunk_S=0, dtype=None, loss_scale=1.0, lambda_pde=None, lambda_gp=0.0,
                 gp_eps=None):
    """One training step through pigan_train_step_grads (or, with lambda_gp,
    pigan_train_step_grads_gp); returns numpy outputs."""
    import torch
    from paper_1910_13444_amd import pigan
    S = inp.z.shape[1]
    desc = pigan.step_desc(wl, S=S, B_r=real.shape[1], chunk_S=chunk_S, dtype=dtype, loss_scale=loss_scale,
                           lambda_pde=lambda_pde, lambda_gp=lambda_gp)
    step = pigan.TrainStep(desc)
    o = step(to_dev(inp.pY), to_dev(inp.pU), to_dev(inp.pD), to_dev(inp.z), to_dev(inp.xc), to_dev(inp.xsY),
             to_dev(inp.xsU), to_dev(real), f=None if inp.f is None else to_dev(inp.f), f_const=inp.f_const,
             w_group=to_dev(inp.w_group), gp_eps=None if gp_eps is None else to_dev(gp_eps))
    torch.cuda.synchronize()
    out = dict(gY=o.gY.cpu().numpy(), gU=o.gU.cpu().numpy(), gD=o.gD.cpu().numpy(), loss=o.loss.cpu().numpy(),
               nonfinite=int(o.nonfinite.cpu().item()))
    if o.gp is not None:
        out["P_gp"] = o.gp.cpu().numpy()
    return out


def step_errors(wl, out, ref):
    errs = {}
    errs.update(grad_errors(out["gY"], ref["gY"], wl.gen_shape(), "gY"))
    errs.update(grad_errors(out["gU"], ref["gU"], wl.gen_shape(), "gU"))
    errs.update(grad_errors(out["gD"], ref["gD"], wl.disc_shape(), "gD"))
    for i, k in enumerate(("L_D", "L_adv", "L_pde")):
        errs[k] = rel(out["loss"][:, i], ref["loss"][:, i])
    if "P_gp" in out:
        errs["P_gp"] = rel(out["P_gp"], ref["P_gp"])
    return errs


def trunk_slices(in_dim, L, W):
    """(name, slice) of every weight tensor of a packed shared trunk."""
    out = [kv for kv in param_slices(in_dim, L, W) if kv[0] not in ("w_out", "b_out")]
    off = out[-1][1].stop
    out += [("w_Y", slice(off, off + W)), ("b_Y", slice(off + W, off + W + 1)),
            ("w_u", slice(off + W + 1, off + 2 * W + 1)), ("b_u", slice(off + 2 * W + 1, off + 2 * W + 2))]
    return out


def run_trunk_gpu(wl, inp, real, chunk_S=0, dtype=None, loss_scale=1.0, lambda_gp=0.0, gp_eps=None):
    """One training step through pigan_trunk_step_grads (or, with lambda_gp >
    0, pigan_trunk_step_grads_gp); returns numpy outputs."""
    import torch
    from paper_1910_13444_amd import pigan
    desc = pigan.trunk_desc(wl, S=inp.z.shape[1], B_r=real.shape[1], chunk_S=chunk_S, dtype=dtype,
                            loss_scale=loss_scale, lambda_gp=lambda_gp)
    step = pigan.TrunkStep(desc)
    o = step(to_dev(inp.pT), to_dev(inp.pD), to_dev(inp.z), to_dev(inp.xc), to_dev(inp.xsY), to_dev(inp.xsU),
             to_dev(real), f=None if inp.f is None else to_dev(inp.f), f_const=inp.f_const,
             w_group=to_dev(inp.w_group), gp_eps=None if gp_eps is None else to_dev(gp_eps))
    torch.cuda.synchronize()
    out = dict(gT=o.gT.cpu().numpy(), gD=o.gD.cpu().numpy(), loss=o.loss.cpu().numpy(),
               nonfinite=int(o.nonfinite.cpu().item()))
    if o.gp is not None:
        out["P_gp"] = o.gp.cpu().numpy()
    return out


def trunk_errors(wl, out, ref):
    errs = {}
    G = ref["gT"].shape[0]
    for name, sl in trunk_slices(*wl.gen_shape()):
        errs[f"gT.{name}"] = max(rel(out["gT"][g, sl], ref["gT"][g, sl]) for g in range(G))
    errs.update(grad_errors(out["gD"], ref["gD"], wl.disc_shape(), "gD"))
    for i, k in enumerate(("L_D", "L_adv", "L_pde")):
        errs[k] = rel(out["loss"][:, i], ref["loss"][:, i])
    return errs


def run_hier_gpu(wl, hi, real, lam=0.0, chunk_S=0, dtype=None, idx=None, f=None, f_const=0.0, lambda_gp=0.0,
                 gp_eps=None):
    """One domain-decomposition step through pigan_hier_step_grads (or, with
    lambda_gp > 0, pigan_hier_step_grads_gp: then the result has P_gp)."""
    import torch
    from paper_1910_13444_amd import pigan
    b, h = hi.base, hi.hier
    iY, iU, iF = idx if idx is not None else (h.idxY, h.idxU, h.idxF)
    desc = pigan.hier_desc(wl, h.D, iY.shape[1], iU.shape[1], iF.shape[1], S=b.z.shape[1], B_r=real.shape[1],
                           chunk_S=chunk_S, dtype=dtype, lambda_pde=lam, lambda_gp=lambda_gp)
    step = pigan.HierStep(desc)

    def ti(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()
    o = step(to_dev(b.pY[0]), to_dev(b.pU[0]), to_dev(hi.pD), to_dev(b.z[0]), to_dev(b.xc[0]), to_dev(b.xsY[0]),
             to_dev(b.xsU[0]), ti(iY), ti(iU), ti(iF), to_dev(real), to_dev(h.w),
             f=None if f is None else to_dev(f), f_const=f_const, gp_eps=None if gp_eps is None else to_dev(gp_eps))
    torch.cuda.synchronize()
    out = dict(gY=o.gY.cpu().numpy(), gU=o.gU.cpu().numpy(), gD=o.gD.cpu().numpy(), loss=o.loss.cpu().numpy(),
               nonfinite=int(o.nonfinite.cpu().item()))
    if o.gp is not None:
        out["P_gp"] = o.gp.cpu().numpy()
    return out


def run_hier_trunk_gpu(wl, hi, real, lam=0.0, chunk_S=0, dtype=None, f_const=0.0, lambda_gp=0.0, gp_eps=None):
    """One domain-decomposition step with the shared trunk
    (pigan_hier_trunk_step_grads, or its _gp form when lambda_gp > 0)."""
    import torch
    from paper_1910_13444_amd import pigan
    b, h = hi.base, hi.hier
    desc = pigan.hier_trunk_desc(wl, h.D, h.idxY.shape[1], h.idxU.shape[1], h.idxF.shape[1], S=b.z.shape[1],
                                 B_r=real.shape[1], chunk_S=chunk_S, dtype=dtype, lambda_pde=lam,
                                 lambda_gp=lambda_gp)
    step = pigan.HierTrunkStep(desc)

    def ti(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()
    o = step(to_dev(b.pT[0]), to_dev(hi.pD), to_dev(b.z[0]), to_dev(b.xc[0]), to_dev(b.xsY[0]), to_dev(b.xsU[0]),
             ti(h.idxY), ti(h.idxU), ti(h.idxF), to_dev(real), to_dev(h.w), f_const=f_const,
             gp_eps=None if gp_eps is None else to_dev(gp_eps))
    torch.cuda.synchronize()
    out = dict(gY=o.gT.cpu().numpy(), gD=o.gD.cpu().numpy(), loss=o.loss.cpu().numpy(),
               nonfinite=int(o.nonfinite.cpu().item()))
    if o.gp is not None:
        out["P_gp"] = o.gp.cpu().numpy()
    return out


def hier_errors(wl, out, ref, n_in, trunk=False):
    errs = {}
    if trunk:
        for name, sl in trunk_slices(*wl.gen_shape()):
            errs[f"gT.{name}"] = rel(out["gY"][sl], ref["gY"][sl])
    else:
        errs.update(grad_errors(out["gY"][None], ref["gY"][None], wl.gen_shape(), "gY"))
        errs.update(grad_errors(out["gU"][None], ref["gU"][None], wl.gen_shape(), "gU"))
    errs.update(grad_errors(out["gD"], ref["gD"], (n_in, wl.L_D, wl.W_D), "gD"))
    errs["L_D"] = rel(out["loss"][:, 0], ref["L_D"])
    errs["L_adv"] = rel(out["loss"][:, 1], ref["L_adv"])
    errs["L_pde"] = rel(out["loss"][:, 2], np.full(len(ref["L_D"]), ref["L_pde"]))
    if "P_gp" in out:
        errs["P_gp"] = rel(out["P_gp"], ref["P_gp"])
    return errs
