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


def grad_errors(g_gpu, g_ref, shape, prefix, metric=rel):
    errs = {}
    G = g_ref.shape[0]
    for name, sl in param_slices(*shape):
        if name == "b_out" and shape is not None:
            # a single scalar per group: compare all groups together
            errs[f"{prefix}.{name}"] = metric(g_gpu[:, sl], g_ref[:, sl])
            continue
        errs[f"{prefix}.{name}"] = max(metric(g_gpu[g, sl], g_ref[g, sl]) for g in range(G))
    return errs


def amax_rel(a, b) -> float:
    """max |a - b| / max |b| (the element-wise companion of the normwise error)."""
    a = np.asarray(a, np.float64).ravel()
    b = np.asarray(b, np.float64).ravel()
    den = np.abs(b).max() if b.size else 0.0
    return float(np.abs(a - b).max() / den) if den > 0 else float(np.abs(a).max() if a.size else 0.0)


def check(errs: dict, tol: float, label: str = "", maxe: dict | None = None):
    """Assert every normwise error is within tol; print the worst tensors and,
    when given, their element-wise errors max|d| / max|oracle|."""
    bad = {k: v for k, v in errs.items() if not (v <= tol)}
    worst = sorted(errs.items(), key=lambda kv: -kv[1])[:6]
    msg = f"{label} tol={tol:g} worst: " + ", ".join(f"{k}={v:.3g}" for k, v in worst)
    if maxe:
        wm = sorted(maxe.items(), key=lambda kv: -kv[1])[:4]
        msg += " | max-abs: " + ", ".join(f"{k}={v:.3g}" for k, v in wm)
    print(msg, flush=True)
    assert not bad, msg


def to_dev(a, dev="cuda"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)


def run_step_gpu(wl, inp, real, chunk_S=0, dtype=None, loss_scale=1.0, lambda_pde=None, lambda_gp=0.0,
                 gp_eps=None, critic_only=False):
    """One training step through pigan_train_step_grads (or, with lambda_gp,
    pigan_train_step_grads_gp); returns numpy outputs."""
    import torch
    from paper_1910_13444_amd import pigan
    S = inp.z.shape[1]
    desc = pigan.step_desc(wl, S=S, B_r=real.shape[1], chunk_S=chunk_S, dtype=dtype, loss_scale=loss_scale,
                           lambda_pde=lambda_pde, lambda_gp=lambda_gp)
    desc.critic_only = int(critic_only)
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


def step_errors(wl, out, ref, metric=rel):
    errs = {}
    errs.update(grad_errors(out["gY"], ref["gY"], wl.gen_shape(), "gY", metric))
    errs.update(grad_errors(out["gU"], ref["gU"], wl.gen_shape(), "gU", metric))
    errs.update(grad_errors(out["gD"], ref["gD"], wl.disc_shape(), "gD", metric))
    for i, k in enumerate(("L_D", "L_adv", "L_pde")):
        errs[k] = metric(out["loss"][:, i], ref["loss"][:, i])
    if "P_gp" in out:
        errs["P_gp"] = metric(out["P_gp"], ref["P_gp"])
    return errs


def trunk_slices(in_dim, L, W):
    """(name, slice) of every weight tensor of a packed shared trunk."""
    out = [kv for kv in param_slices(in_dim, L, W) if kv[0] not in ("w_out", "b_out")]
    off = out[-1][1].stop
    out += [("w_Y", slice(off, off + W)), ("b_Y", slice(off + W, off + W + 1)),
            ("w_u", slice(off + W + 1, off + 2 * W + 1)), ("b_u", slice(off + 2 * W + 1, off + 2 * W + 2))]
    return out


def run_trunk_gpu(wl, inp, real, chunk_S=0, dtype=None, loss_scale=1.0, lambda_gp=0.0, gp_eps=None,
                  critic_only=False):
    """One training step through pigan_trunk_step_grads (or, with lambda_gp >
    0, pigan_trunk_step_grads_gp); returns numpy outputs."""
    import torch
    from paper_1910_13444_amd import pigan
    desc = pigan.trunk_desc(wl, S=inp.z.shape[1], B_r=real.shape[1], chunk_S=chunk_S, dtype=dtype,
                            loss_scale=loss_scale, lambda_gp=lambda_gp)
    desc.critic_only = int(critic_only)
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


def trunk_errors(wl, out, ref, metric=rel):
    errs = {}
    G = ref["gT"].shape[0]
    for name, sl in trunk_slices(*wl.gen_shape()):
        errs[f"gT.{name}"] = max(metric(out["gT"][g, sl], ref["gT"][g, sl]) for g in range(G))
    errs.update(grad_errors(out["gD"], ref["gD"], wl.disc_shape(), "gD", metric))
    for i, k in enumerate(("L_D", "L_adv", "L_pde")):
        errs[k] = metric(out["loss"][:, i], ref["loss"][:, i])
    if "P_gp" in out and "P_gp" in ref:
        errs["P_gp"] = metric(out["P_gp"], ref["P_gp"])
    return errs


def run_hier_gpu(wl, hi, real, lam=0.0, chunk_S=0, dtype=None, idx=None, f=None, f_const=0.0, lambda_gp=0.0,
                 gp_eps=None, critic_only=False):
    """One domain-decomposition step through pigan_hier_step_grads (or, with
    lambda_gp > 0, pigan_hier_step_grads_gp: then the result has P_gp)."""
    import torch
    from paper_1910_13444_amd import pigan
    b, h = hi.base, hi.hier
    iY, iU, iF = idx if idx is not None else (h.idxY, h.idxU, h.idxF)
    desc = pigan.hier_desc(wl, h.D, iY.shape[1], iU.shape[1], iF.shape[1], S=b.z.shape[1], B_r=real.shape[1],
                           chunk_S=chunk_S, dtype=dtype, lambda_pde=lam, lambda_gp=lambda_gp)
    desc.critic_only = int(critic_only)
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


def run_hier_trunk_gpu(wl, hi, real, lam=0.0, chunk_S=0, dtype=None, f_const=0.0, lambda_gp=0.0, gp_eps=None,
                       critic_only=False):
    """One domain-decomposition step with the shared trunk
    (pigan_hier_trunk_step_grads, or its _gp form when lambda_gp > 0)."""
    import torch
    from paper_1910_13444_amd import pigan
    b, h = hi.base, hi.hier
    desc = pigan.hier_trunk_desc(wl, h.D, h.idxY.shape[1], h.idxU.shape[1], h.idxF.shape[1], S=b.z.shape[1],
                                 B_r=real.shape[1], chunk_S=chunk_S, dtype=dtype, lambda_pde=lam,
                                 lambda_gp=lambda_gp)
    desc.critic_only = int(critic_only)
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


def hier_errors(wl, out, ref, n_in, trunk=False, metric=rel):
    errs = {}
    if trunk:
        for name, sl in trunk_slices(*wl.gen_shape()):
            errs[f"gT.{name}"] = metric(out["gY"][sl], ref["gY"][sl])
    else:
        errs.update(grad_errors(out["gY"][None], ref["gY"][None], wl.gen_shape(), "gY", metric))
        errs.update(grad_errors(out["gU"][None], ref["gU"][None], wl.gen_shape(), "gU", metric))
    errs.update(grad_errors(out["gD"], ref["gD"], (n_in, wl.L_D, wl.W_D), "gD", metric))
    errs["L_D"] = metric(out["loss"][:, 0], ref["L_D"])
    errs["L_adv"] = metric(out["loss"][:, 1], ref["L_adv"])
    errs["L_pde"] = metric(out["loss"][:, 2], np.full(len(ref["L_D"]), ref["L_pde"]))
    if "P_gp" in out:
        errs["P_gp"] = metric(out["P_gp"], ref["P_gp"])
    return errs
