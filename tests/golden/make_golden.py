"""Writes the stored expected values of the reduced-sample parity tests:
the fp64 oracle's training step on the 6x512 workload (4096 collocation
points, 1000 + 1000 sensors, 4x1024 critic) and the 6x1024 workload (2048
collocation points, 4096 + 4096 sensors, 5x2048 critic) with 8 noise samples
and 8 real snapshots and every collocation point and sensor of the full
workload.

Calls only oracle/ and the seeded input generator.  Per workload one
step_<name>_S8.npz holds the three losses, every bias and output-layer
gradient in full, and for every weight-gradient matrix its Frobenius norm,
the two sketches G r and s^T G with seeded Gaussian r and s (stored too), and
256 sampled elements; plus the real snapshots and checksums of the inputs.

    python tests/golden/make_golden.py        # about 4 minutes on 8 cores
"""
import os
import sys

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))
sys.path.insert(0, os.path.dirname(HERE))

import oracle                                              # noqa: E402
from paper_1910_13444_amd import configs                   # noqa: E402
from paper_1910_13444_amd.inputs import make_inputs        # noqa: E402

S_RED = 8
WORKLOADS = (configs.C3, configs.C5)


def reduced(wl):
    return wl.with_(S=S_RED, B_r=S_RED)


def tensors(in_dim, L, W):
    """(name, slice, matrix shape or None) of every tensor of a packed MLP."""
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


def input_checksums(inp):
    return np.array([np.float64(a).sum() for a in (inp.pY, inp.pU, inp.pD, inp.z, inp.xc, inp.xsY, inp.xsU)])


def summarise(grad, shape, prefix, rng, out):
    """grad: [G, n_params] of one network (G = 1 here)."""
    g = np.asarray(grad[0], np.float64)
    for name, sl, mshape in tensors(*shape):
        key = f"{prefix}.{name}"
        if mshape is None:
            out[key] = g[sl]
            continue
        M = g[sl].reshape(mshape)
        r = rng.standard_normal(mshape[1])
        s = rng.standard_normal(mshape[0])
        idx = rng.choice(M.size, 256, replace=False)
        out[key + ".norm"] = np.array([np.linalg.norm(M)])
        out[key + ".r"] = r
        out[key + ".s"] = s
        out[key + ".Gr"] = M @ r
        out[key + ".sG"] = s @ M
        out[key + ".idx"] = idx.astype(np.int64)
        out[key + ".val"] = M.ravel()[idx]


def main():
    for wl0 in WORKLOADS:
        wl = reduced(wl0)
        print(f"oracle step {wl.name} S={wl.S} P={wl.P}", flush=True)
        inp = make_inputs(wl)
        real = oracle.real_snapshots(wl, inp)
        ref = oracle.train_step(wl, inp, real)
        rng = np.random.default_rng(20191030)
        out = {"loss": np.asarray(ref["loss"], np.float64), "real": real.astype(np.float32),
               "inputs_checksum": input_checksums(inp)}
        summarise(ref["gY"], wl.gen_shape(), "gY", rng, out)
        summarise(ref["gU"], wl.gen_shape(), "gU", rng, out)
        summarise(ref["gD"], wl.disc_shape(), "gD", rng, out)
        path = os.path.join(HERE, f"step_{wl0.name}_S{S_RED}.npz")
        np.savez_compressed(path, **out)
        print(f"wrote {path} ({os.path.getsize(path) / 1e6:.2f} MB)", flush=True)


if __name__ == "__main__":
    main()
