"""Benchmark of the PI-GAN training step on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c5]

The default workload is the largest single-network configuration: generators
6 x 1024 tanh (z in R^128), 1024 noise samples x 2048 collocation points,
4096 + 4096 sensors, critic 5 x 2048 tanh on the 8192-value snapshot, bf16.

A step is one call of pigan_train_step_grads: both generators' jets at every
(collocation point x noise sample) pair and at the sensors, the Darcy
residual, the discriminator on fake and real snapshots, and every weight
gradient.  Inputs are seeded synthetic data resident in HBM before the timed
region starts.  Prints ONE JSON line on stdout; diagnostics go to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_TFLOPS = {"bf16": 2516.6, "fp16": 2516.6, "fp32": 157.3}
PEAK_GBS = 8000.0
METRIC = "PI-GAN train-step TFLOP/s (bf16 MFMA) + collocation points/s, 1 MI355X"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def device_inputs(wl, dev):
    import numpy as np
    import torch

    from paper_1910_13444_amd import pigan
    from paper_1910_13444_amd.inputs import make_inputs

    if wl.is_hier:
        return hier_inputs(wl, dev)
    inp = make_inputs(wl)

    def t(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)

    d = dict(pD=t(inp.pD), z=t(inp.z), xc=t(inp.xc), xsY=t(inp.xsY), xsU=t(inp.xsU), w_group=t(inp.w_group))
    if wl.arch == "trunk":
        d["pT"] = t(inp.pT)
        # real snapshots for timing: a seeded teacher pair of plain generators
        # of the trunk's depth and width (same sensors and teacher noise)
        teach = make_inputs(wl.with_(arch="pair"))
        tY, tU = teach.tY, teach.tU
    else:
        d["pY"], d["pU"] = t(inp.pY), t(inp.pU)
        tY, tU = inp.tY, inp.tU
    # real snapshots: the seeded teacher generators at the sensors, on the device
    shape = wl.gen_shape()
    zt = t(inp.z_teach)
    yY = pigan.gen_forward(t(tY), shape, wl.d, zt, d["xsY"], 0, dtype="fp32", x_shared=True)
    yU = pigan.gen_forward(t(tU), shape, wl.d, zt, d["xsU"], 0, dtype="fp32", x_shared=True)
    d["real"] = torch.cat([yY[:, 0], yU[:, 0]], dim=-1).contiguous()
    torch.cuda.synchronize()
    return d, inp


def hier_inputs(wl, dev):
    """Device inputs of a domain-decomposition step: the generator (pair or
    shared trunk), the stratified sensors and points, the critics' index lists
    and weights, and real snapshots per critic (a teacher pair at its sensors
    on the device, f = 0 at its free sensors, their coordinates)."""
    import numpy as np
    import torch

    from paper_1910_13444_amd import pigan
    from paper_1910_13444_amd.inputs import make_hier_inputs, make_inputs

    hi = make_hier_inputs(wl, sides=wl.sides, m_sensors=wl.m_sensors, n_free=wl.n_free)
    b, h = hi.base, hi.hier

    def t(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev)

    def ti(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(dev)
    d = dict(pD=t(hi.pD), z=t(b.z[0]), xc=t(b.xc[0]), xsY=t(b.xsY[0]),
             xsU=t(b.xsU[0]), idxY=ti(h.idxY), idxU=ti(h.idxU), idxF=ti(h.idxF), w_disc=t(h.w))
    if wl.trunk_gen:
        d["pT"] = t(b.pT[0])
        teach = make_inputs(wl.with_(arch="pair"))   # same teacher noise, plain teacher pair
        tY, tU = teach.tY, teach.tU
    else:
        d["pY"], d["pU"] = t(b.pY[0]), t(b.pU[0])
        tY, tU = b.tY, b.tU
    shape = wl.gen_shape()
    zt = t(b.z_teach)
    yY = pigan.gen_forward(t(tY), shape, wl.d, zt, t(b.xsY), 0, dtype="fp32", x_shared=True)[0, 0]
    yU = pigan.gen_forward(t(tU), shape, wl.d, zt, t(b.xsU), 0, dtype="fp32", x_shared=True)[0, 0]
    xf = t(hi.xf_real)                                            # [B, P, 2]
    Bn = yY.shape[0]
    real = []
    for k in range(h.D):
        real.append(torch.cat([yY[:, d["idxY"][k].long()], yU[:, d["idxU"][k].long()],
                               torch.zeros(Bn, h.idxF.shape[1], device=dev),
                               xf[:, d["idxF"][k].long(), :].reshape(Bn, -1)], dim=1))
    d["real"] = torch.stack(real).contiguous()
    torch.cuda.synchronize()
    return d, hi


KERNEL_SOURCES = ("common.h", "gemm.hip", "pointwise.hip")


def kernel_source_hash():
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_1910_13444_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def recorded_traffic(key, wl):
    """HBM bytes per launch of the launch shape `key` on this workload, from a
    committed counter summary (profiles/*.traffic.json: FETCH_SIZE and
    WRITE_SIZE per dispatch, scaled by a known-size copy).  None when no
    summary covers it or the kernel sources changed since it was taken."""
    import glob
    src = kernel_source_hash()
    for f in sorted(glob.glob(os.path.join(ROOT, "profiles", "*.traffic.json"))):
        with open(f) as fh:
            rec = json.load(fh)
        if rec.get("workload") != wl.name or rec.get("kernel_sources_sha256") != src:
            continue
        v = rec.get("hbm_bytes_per_launch", {}).get(key)
        if v is not None:
            return float(v)
    return None


def measured_peaks(dev):
    """Achievable rates on this GPU from two micro-benchmarks (context for
    the roofline): a 2 GiB device-to-device copy (bytes read + written per
    second) and an 8192^3 bf16 matrix product through the vendor BLAS."""
    import torch
    out = {}
    n = 1 << 31
    a = torch.empty(n, dtype=torch.uint8, device=dev)
    b = torch.empty_like(a)
    b.copy_(a)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(5):
        b.copy_(a)
    e1.record()
    torch.cuda.synchronize()
    out["copy_GBps"] = 2.0 * n * 5 / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del a, b
    m = 8192
    x = torch.randn(m, m, dtype=torch.bfloat16, device=dev)
    y = torch.randn(m, m, dtype=torch.bfloat16, device=dev)
    torch.matmul(x, y)
    e0.record()
    for _ in range(10):
        torch.matmul(x, y)
    e1.record()
    torch.cuda.synchronize()
    out["bf16_gemm_TFLOPs"] = 2.0 * m ** 3 * 10 / (e0.elapsed_time(e1) * 1e-3) / 1e12
    del x, y
    torch.cuda.empty_cache()
    return out


def run_steps(step, d, wl, k):
    for _ in range(k):
        if wl.arch == "hier_trunk":
            step(d["pT"], d["pD"], d["z"], d["xc"], d["xsY"], d["xsU"], d["idxY"], d["idxU"], d["idxF"],
                 d["real"], d["w_disc"], f=None, f_const=wl.f_const, gp_eps=d.get("gp_eps"))
        elif wl.arch == "hier":
            step(d["pY"], d["pU"], d["pD"], d["z"], d["xc"], d["xsY"], d["xsU"], d["idxY"], d["idxU"], d["idxF"],
                 d["real"], d["w_disc"], f=None, f_const=wl.f_const, gp_eps=d.get("gp_eps"))
        elif wl.arch == "trunk":
            step(d["pT"], d["pD"], d["z"], d["xc"], d["xsY"], d["xsU"], d["real"], f=None, f_const=wl.f_const,
                 w_group=d["w_group"], gp_eps=d.get("gp_eps"))
        else:
            step(d["pY"], d["pU"], d["pD"], d["z"], d["xc"], d["xsY"], d["xsU"], d["real"], f=None,
                 f_const=wl.f_const, w_group=d["w_group"], gp_eps=d.get("gp_eps"))


def cpu_baseline(wl, budget_s: float = 15.0):
    """The fp64 oracle on a bounded sample of the same workload (S' noise
    samples, all collocation points and sensors), scaled to TFLOP/s."""
    import numpy as np

    import oracle
    from paper_1910_13444_amd import flops
    from paper_1910_13444_amd.inputs import make_inputs

    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        cores = os.cpu_count() or 1

    def timed(S):
        w2 = wl.with_(S=S, B_r=min(wl.B_r, S))
        inp = make_inputs(w2)
        real = np.random.default_rng(0).standard_normal((w2.G, w2.B_r, w2.n_in)).astype(np.float32)
        t0 = time.perf_counter()
        if w2.arch == "trunk":
            oracle.train_step_trunk(w2, inp, real)
        else:
            oracle.train_step(w2, inp, real)
        return w2, time.perf_counter() - t0

    # one sample first; a larger sample only when one takes well under the budget
    w2, t2 = timed(1)
    S = int(max(1, min(wl.S, round(budget_s / max(t2, 1e-3)))))
    if S >= 2:
        w2, t2 = timed(S)
    f = flops.step_flops(w2, S=w2.S, B_r=w2.B_r)
    return {"value": f / t2 / 1e12, "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
            "sample": f"{w2.S} of {wl.S} noise samples (B_r={w2.B_r}), all {wl.P} collocation points "
                      f"and all sensors per sample, fp64 NumPy, {t2:.2f} s",
            "collocation_points_per_s": w2.G * w2.S * wl.P / t2}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="c5")
    ap.add_argument("--chunk-S", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true")
    ap.add_argument("--graph", action="store_true",
                    help="time replays of one step captured in a HIP graph instead of eager calls")
    ap.add_argument("--no-peaks", action="store_true", help="skip the copy / GEMM micro-benchmarks")
    ap.add_argument("--lambda-gp", type=float, default=0.0,
                    help="add the critic gradient penalty with this weight (seeded mixing weights)")
    ap.add_argument("--copy-calib", type=int, default=0, metavar="BYTES",
                    help="first run one plain device-to-device copy of BYTES bytes (a known-size reference "
                         "dispatch for scaling HBM byte counters)")
    a = ap.parse_args()

    if a.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print(f"bench.py measures one GPU only: the PI-GAN step is built and timed on a single MI355X "
              f"(requested --gpus {a.gpus}); multi-GPU execution is not implemented.", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_1910_13444_amd import configs, flops, pigan

    wl = configs.get(a.workload)
    dev = torch.device("cuda:0")
    pigan.lib()
    log(f"bench: workload {wl.name} dtype {wl.dtype} S={wl.S} P={wl.P} W={wl.W} L={wl.L}")
    if a.copy_calib > 0:
        src = torch.ones(a.copy_calib, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"bench: calibration copy of {a.copy_calib} bytes done")
        del src, dst
    d, inp = device_inputs(wl, dev)
    if a.lambda_gp > 0:
        import numpy as np
        n_crit = wl.n_critics if wl.is_hier else wl.G       # one row of mixing weights per critic
        eps = np.random.default_rng(wl.seed + 5).random((n_crit, min(wl.S, wl.B_r)), dtype=np.float32)
        d["gp_eps"] = torch.from_numpy(eps).to(dev)
    if wl.is_hier:
        if wl.trunk_gen:
            step = pigan.HierTrunkStep(pigan.hier_trunk_desc(wl, wl.n_critics, wl.m_sensors, wl.m_sensors, wl.n_free,
                                                             chunk_S=a.chunk_S, lambda_pde=wl.lambda_pde,
                                                             lambda_gp=a.lambda_gp), device=dev)
        else:
            step = pigan.HierStep(pigan.hier_desc(wl, wl.n_critics, wl.m_sensors, wl.m_sensors, wl.n_free,
                                                  chunk_S=a.chunk_S, lambda_pde=wl.lambda_pde,
                                                  lambda_gp=a.lambda_gp), device=dev)
    elif wl.arch == "trunk":
        step = pigan.TrunkStep(pigan.trunk_desc(wl, chunk_S=a.chunk_S, lambda_gp=a.lambda_gp), device=dev)
    else:
        step = pigan.TrainStep(pigan.step_desc(wl, chunk_S=a.chunk_S, lambda_gp=a.lambda_gp), device=dev)
    log(f"bench: workspace {step.ws_bytes / 2**30:.2f} GiB; warmup {a.warmup}")
    run_steps(step, d, wl, a.warmup)
    torch.cuda.synchronize()
    nf = int(step.out.nonfinite.item())

    graph = pigan.StepGraph(lambda: run_steps(step, d, wl, 1)) if a.graph else None

    # timed region
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    ev0.record()
    if graph is not None:
        for _ in range(a.steps):
            graph.replay()
    else:
        run_steps(step, d, wl, a.steps)
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    ms = ev0.elapsed_time(ev1) / a.steps
    log(f"bench: {a.steps} steps, {ms:.3f} ms/step (wall {wall * 1e3 / a.steps:.3f} ms/step)")

    F = flops.step_flops(wl)
    pts = flops.collocation_points(wl)
    tflops = F / (ms * 1e-3) / 1e12

    # per-kernel timing: the same steps again with HIP events around every launch
    roof = None
    kernels = None
    step_roof = None
    if not a.no_profile:
        pigan.profile_enable(True)
        run_steps(step, d, wl, a.steps)
        torch.cuda.synchronize()
        stats = pigan.profile_read()
        pigan.profile_enable(False)
        tot = sum(s["total_ms"] for s in stats)
        kernels = {s["name"]: {"launches_per_step": s["launches"] / a.steps,
                               "ms_per_step": s["total_ms"] / a.steps,
                               "share": s["total_ms"] / tot if tot else 0.0,
                               "alg_flops_per_step": s["flops"] / a.steps,
                               "alg_bytes_per_step": s["bytes"] / a.steps} for s in stats}
        # the step's own roofline: every launch at the faster of its two
        # bounds (algorithmic FLOPs at the dense peak, algorithmic bytes at
        # 8 TB/s); launches that record neither count zero, so this is a
        # lower bound on the step time
        bound_s = sum(max(s["flops"] / (PEAK_TFLOPS[wl.dtype] * 1e12), s["bytes"] / (PEAK_GBS * 1e9))
                      for s in stats) / a.steps
        step_roof = {"bound_ms": bound_s * 1e3, "frac": bound_s * 1e3 / ms,
                     "mfma_bound_share": sum(s["total_ms"] for s in stats
                                             if s["flops"] / (PEAK_TFLOPS[wl.dtype] * 1e12) >
                                             s["bytes"] / (PEAK_GBS * 1e9)) / tot if tot else 0.0}
        dom = max(stats, key=lambda s: s["total_ms"])
        avg_ms = dom["total_ms"] / dom["launches"]
        fl = dom["flops"] / dom["launches"]
        by = dom["bytes"] / dom["launches"]
        ridge = PEAK_TFLOPS[wl.dtype] * 1e12 / (PEAK_GBS * 1e9)
        traffic = recorded_traffic(dom["name"], wl)
        if by > 0 and fl / by < ridge:
            ach = by / (avg_ms * 1e-3) / 1e9
            roof = {"kernel": dom["name"], "bound": "hbm", "achieved": ach, "peak": PEAK_GBS, "unit": "GB/s",
                    "frac": ach / PEAK_GBS, "traffic": traffic, "traffic_unit": "HBM bytes per launch", "avg_launch_ms": avg_ms,
                    "launches_per_step": dom["launches"] / a.steps, "alg_bytes_per_launch": by,
                    "alg_flops_per_launch": fl}
        else:
            ach = fl / (avg_ms * 1e-3) / 1e12
            pk = PEAK_TFLOPS[wl.dtype]
            roof = {"kernel": dom["name"], "bound": "mfma", "achieved": ach, "peak": pk, "unit": "TFLOP/s",
                    "frac": ach / pk, "traffic": traffic, "traffic_unit": "HBM bytes per launch", "avg_launch_ms": avg_ms,
                    "launches_per_step": dom["launches"] / a.steps, "alg_bytes_per_launch": by,
                    "alg_flops_per_launch": fl}
        for k, v in sorted(kernels.items(), key=lambda kv: -kv[1]["ms_per_step"]):
            log(f"  {k:12s} {v['ms_per_step']:.4f} ms/step  {100 * v['share']:.1f}%  "
                f"launches/step {v['launches_per_step']:.0f}")

    peaks = None if a.no_peaks else measured_peaks(dev)
    # the oracle baseline covers the paired and shared-trunk steps
    cpu = None if (a.no_cpu_baseline or wl.is_hier) else cpu_baseline(wl)

    out = {
        "metric": METRIC, "value": tflops, "unit": "TFLOP/s", "n_gpus": 1, "steps": a.steps,
        "warmup": a.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": wl.dtype, "data": "synthetic",
        "config": {"workload": wl.name, "G": wl.G, "d": wl.d, "n_z": wl.n_z,
                   "gen": (f"shared trunk {wl.L}x{wl.W} tanh, residual blocks, 2 heads" if wl.trunk_gen
                           else f"{wl.L}x{wl.W} tanh"),
                   "critics": (f"{wl.n_critics} subdomain critics, levels {list(wl.sides)}, "
                               f"{wl.n_in_hier} inputs each" if wl.is_hier else wl.G),
                   "disc": f"{wl.L_D}x{wl.W_D} tanh on {wl.n_in}", "S": wl.S, "P": wl.P,
                   "sensors": [wl.n_sY, wl.n_sU], "B_r": wl.B_r, "chunk_S": a.chunk_S, "lambda_gp": a.lambda_gp,
                   "launch": "hip_graph" if a.graph else "eager",
                   "collocation_points_per_step": pts, "alg_flops_per_step": F},
        "collocation_points_per_s": pts / (ms * 1e-3),
        "mfma_frac_step": tflops / PEAK_TFLOPS[wl.dtype],
        "nonfinite": nf,
        "roofline": roof,
        "step_roofline": step_roof,
        "measured_peaks": peaks,
        "cpu_baseline": cpu,
        "kernels": kernels,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
