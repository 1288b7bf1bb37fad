"""ctypes binding of libpigan.so (argument marshalling only).

Every step of the PI-GAN hot path runs in the library's HIP kernels; this
module only checks torch tensors (device, dtype, contiguity, sizes), passes
their device pointers and the current HIP stream, and turns non-OK statuses
into exceptions.  There is no CPU fallback: without the built library every
call raises.
"""
from __future__ import annotations

import ctypes as C
import os
import re
from dataclasses import dataclass

import torch

from .configs import Workload, n_params

_HERE = os.path.dirname(os.path.abspath(__file__))
# PIGAN_LIBRARY selects another build of the same sources (the host-sanitized
# one of the CPU argument-check tests)
LIB_PATH = os.environ.get("PIGAN_LIBRARY") or os.path.join(_HERE, "libpigan.so")
HEADER = os.path.join(os.path.dirname(_HERE), "include", "pigan.h")

OK, EINVAL, ENOTSUP, EWORKSPACE, EDEVICE = 0, 1, 2, 3, 4
STATUS_NAMES = {0: "OK", 1: "EINVAL", 2: "ENOTSUP", 3: "EWORKSPACE", 4: "EDEVICE"}
DTYPES = {"fp32": 0, "bf16": 1, "fp16": 2}


class PiganError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


class Mlp(C.Structure):
    _fields_ = [("n_groups", C.c_int32), ("in_dim", C.c_int32), ("n_hidden", C.c_int32), ("width", C.c_int32)]


class StepDesc(C.Structure):
    _fields_ = [("genY", Mlp), ("genU", Mlp), ("disc", Mlp),
                ("d", C.c_int32), ("n_z", C.c_int32), ("S", C.c_int32), ("P", C.c_int32),
                ("n_sY", C.c_int32), ("n_sU", C.c_int32), ("B_r", C.c_int32), ("chunk_S", C.c_int32),
                ("dt", C.c_int32), ("lambda_pde", C.c_float), ("lambda_gp", C.c_float),
                ("loss_scale", C.c_float), ("critic_only", C.c_int32)]


class TrunkDesc(C.Structure):
    _fields_ = [("trunk", Mlp), ("disc", Mlp),
                ("d", C.c_int32), ("n_z", C.c_int32), ("S", C.c_int32), ("P", C.c_int32),
                ("n_sY", C.c_int32), ("n_sU", C.c_int32), ("B_r", C.c_int32), ("chunk_S", C.c_int32),
                ("dt", C.c_int32), ("lambda_pde", C.c_float), ("loss_scale", C.c_float),
                ("lambda_gp", C.c_float), ("critic_only", C.c_int32)]


class HierDesc(C.Structure):
    _fields_ = [("genY", Mlp), ("genU", Mlp), ("disc", Mlp),
                ("d", C.c_int32), ("n_z", C.c_int32), ("S", C.c_int32), ("P", C.c_int32),
                ("n_sY", C.c_int32), ("n_sU", C.c_int32), ("B_r", C.c_int32), ("chunk_S", C.c_int32),
                ("mY", C.c_int32), ("mU", C.c_int32), ("nF", C.c_int32),
                ("dt", C.c_int32), ("lambda_pde", C.c_float), ("loss_scale", C.c_float),
                ("lambda_gp", C.c_float), ("critic_only", C.c_int32)]


class HierTrunkDesc(C.Structure):
    _fields_ = [("trunk", Mlp), ("disc", Mlp),
                ("d", C.c_int32), ("n_z", C.c_int32), ("S", C.c_int32), ("P", C.c_int32),
                ("n_sY", C.c_int32), ("n_sU", C.c_int32), ("B_r", C.c_int32), ("chunk_S", C.c_int32),
                ("mY", C.c_int32), ("mU", C.c_int32), ("nF", C.c_int32),
                ("dt", C.c_int32), ("lambda_pde", C.c_float), ("loss_scale", C.c_float),
                ("lambda_gp", C.c_float), ("critic_only", C.c_int32)]


class KernelStat(C.Structure):
    _fields_ = [("name", C.c_char * 48), ("launches", C.c_int64), ("total_ms", C.c_double),
                ("flops", C.c_double), ("bytes", C.c_double)]


_lib = None
P = C.c_void_p


def lib():
    """Open libpigan.so (raises if it has not been built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_1910_13444_amd.build`")
    L = C.CDLL(LIB_PATH)
    i32, i64, f32, sz = C.c_int32, C.c_int64, C.c_float, C.c_size_t
    sigs = {
        "pigan_mlp_n_params": (i64, [P]),
        "pigan_gen_forward_workspace": (sz, [P, i32, i32, i32, i32, i32]),
        "pigan_gen_forward": (i32, [P, P, i32, P, P, i32, i32, i32, i32, i32, P, P, sz, P]),
        "pigan_pde_residual": (i32, [i32, i32, i64, P, P, P, f32, P, P]),
        "pigan_disc_forward_workspace": (sz, [P, i32, i32]),
        "pigan_disc_forward": (i32, [P, P, P, i32, i32, P, P, sz, P]),
        "pigan_workspace_bytes": (sz, [P]),
        "pigan_train_step_grads": (i32, [P, P, P, P, P, P, P, P, P, f32, P, P, P, P, P, P, P, P, sz, P]),
        "pigan_train_step_grads_gp": (i32, [P, P, P, P, P, P, P, P, P, f32, P, P, P, P, P, P, P, P, P, P, sz, P]),
        "pigan_train_step_grads_noalloc": (i32, [P, P, P, P, P, P, P, P, P, f32, P, P, P, P, P, P, P, P]),
        "pigan_adam_update": (i32, [i64, P, P, P, P, f32, f32, f32, f32, i32, P, P]),
        "pigan_hier_workspace_bytes": (sz, [P]),
        "pigan_hier_step_grads": (i32, [P, P, P, P, P, P, P, P, P, f32, P, P, P, P, P, P, P, P, P, P, P, sz, P]),
        "pigan_hier_step_grads_gp": (i32, [P, P, P, P, P, P, P, P, P, f32, P, P, P, P, P, P, P, P, P, P, P, P, P, sz,
                                           P]),
        "pigan_hier_trunk_workspace_bytes": (sz, [P]),
        "pigan_hier_trunk_step_grads": (i32, [P, P, P, P, P, P, P, P, f32, P, P, P, P, P, P, P, P, P, P, sz, P]),
        "pigan_hier_trunk_step_grads_gp": (i32, [P, P, P, P, P, P, P, P, f32, P, P, P, P, P, P, P, P, P, P, P, P, sz,
                                                 P]),
        "pigan_trunk_param_count": (i64, [P]),
        "pigan_trunk_workspace_bytes": (sz, [P]),
        "pigan_trunk_step_grads": (i32, [P, P, P, P, P, P, P, P, f32, P, P, P, P, P, P, P, sz, P]),
        "pigan_trunk_step_grads_gp": (i32, [P, P, P, P, P, P, P, P, f32, P, P, P, P, P, P, P, P, P, sz, P]),
        "pigan_last_error": (C.c_char_p, []),
        "pigan_profile_enable": (i32, [i32]),
        "pigan_profile_read": (i32, [P, i32, P]),
    }
    for name, (res, args) in sigs.items():
        fn = getattr(L, name)
        fn.restype = res
        fn.argtypes = args
    _lib = L
    return L


def declared_symbols() -> list[str]:
    """Function names declared in include/pigan.h."""
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(pigan_[a-z0-9_]+)\s*\(", txt)))


def _check(status: int):
    if status != OK:
        raise PiganError(status, lib().pigan_last_error().decode())


def _ptr(t: torch.Tensor | None, name: str, numel: int | None = None, dtype=torch.float32):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} has {t.numel()} elements, expected {numel}")
    return C.c_void_p(t.data_ptr())


def _stream():
    return C.c_void_p(torch.cuda.current_stream().cuda_stream)


def mlp(G: int, in_dim: int, L: int, W: int) -> Mlp:
    return Mlp(G, in_dim, L, W)


def _workspace(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


# ---------------------------------------------------------------------------
# entry points
# ---------------------------------------------------------------------------

def gen_forward(params: torch.Tensor, shape: tuple[int, int, int], d: int, z: torch.Tensor, x: torch.Tensor,
                order: int, dtype: str = "bf16", x_shared: bool = False, out: torch.Tensor | None = None,
                ws: torch.Tensor | None = None) -> torch.Tensor:
    """Generator jets [G, 1 + order*d, S, P] at points x ([G,S,P,d] or [G,P,d] shared)."""
    in_dim, L, W = shape
    G, S, n_z = z.shape
    Pn = x.shape[-2]
    net = Mlp(G, in_dim, L, W)
    dt = DTYPES[dtype]
    need = lib().pigan_gen_forward_workspace(C.byref(net), d, S, Pn, order, dt)
    if need == 0:  # invalid shape: let the library report why
        _check(lib().pigan_gen_forward(C.byref(net), None, d, None, None, 0, S, Pn, order, dt, None, None, 0, None))
    if out is None:
        out = torch.empty((G, 1 + order * d, S, Pn), dtype=torch.float32, device=z.device)
    if ws is None or ws.numel() < need:
        ws = _workspace(need, z.device)
    xn = G * (Pn if x_shared else S * Pn) * d
    st = lib().pigan_gen_forward(C.byref(net), _ptr(params, "params", G * n_params(in_dim, L, W)), d,
                                 _ptr(z, "z"), _ptr(x, "x", xn), int(bool(x_shared)), S, Pn, order, dt,
                                 _ptr(out, "jet", G * (1 + order * d) * S * Pn), _ptr(ws, "ws", dtype=torch.uint8),
                                 ws.numel(), _stream())
    _check(st)
    return out


def pde_residual(jetY: torch.Tensor, jetU: torch.Tensor, d: int, f: torch.Tensor | None = None,
                 f_const: float = 0.0, out: torch.Tensor | None = None) -> torch.Tensor:
    """r = -div(exp(Y) grad u) - f from jets [G,1+d,M] and [G,1+2d,M]."""
    G = jetY.shape[0]
    M = jetY[0, 0].numel()
    if out is None:
        out = torch.empty((G, M), dtype=torch.float32, device=jetY.device)
    st = lib().pigan_pde_residual(d, G, M, _ptr(jetY, "jetY", G * (1 + d) * M), _ptr(jetU, "jetU", G * (1 + 2 * d) * M),
                                  _ptr(f, "f", G * M), float(f_const), _ptr(out, "r", G * M), _stream())
    _check(st)
    return out


def disc_forward(params: torch.Tensor, shape: tuple[int, int, int], snap: torch.Tensor, dtype: str = "bf16",
                 out: torch.Tensor | None = None, ws: torch.Tensor | None = None) -> torch.Tensor:
    in_dim, L, W = shape
    G, B, n_in = snap.shape
    net = Mlp(G, in_dim, L, W)
    dt = DTYPES[dtype]
    need = lib().pigan_disc_forward_workspace(C.byref(net), B, dt)
    if need == 0:
        _check(lib().pigan_disc_forward(C.byref(net), None, None, B, dt, None, None, 0, None))
    if out is None:
        out = torch.empty((G, B), dtype=torch.float32, device=snap.device)
    if ws is None or ws.numel() < need:
        ws = _workspace(need, snap.device)
    st = lib().pigan_disc_forward(C.byref(net), _ptr(params, "params", G * n_params(in_dim, L, W)),
                                  _ptr(snap, "snap", G * B * in_dim), B, dt, _ptr(out, "score", G * B),
                                  _ptr(ws, "ws", dtype=torch.uint8), ws.numel(), _stream())
    _check(st)
    return out


def step_desc(wl: Workload, S: int | None = None, B_r: int | None = None, chunk_S: int = 0,
              dtype: str | None = None, lambda_pde: float | None = None, loss_scale: float = 1.0,
              lambda_gp: float = 0.0) -> StepDesc:
    S = wl.S if S is None else S
    B_r = wl.B_r if B_r is None else B_r
    return StepDesc(Mlp(wl.G, wl.in_dim, wl.L, wl.W), Mlp(wl.G, wl.in_dim, wl.L, wl.W),
                    Mlp(wl.G, wl.n_in, wl.L_D, wl.W_D), wl.d, wl.n_z, S, wl.P, wl.n_sY, wl.n_sU, B_r, chunk_S,
                    DTYPES[dtype or wl.dtype], wl.lambda_pde if lambda_pde is None else lambda_pde, lambda_gp,
                    loss_scale)


def workspace_bytes(desc: StepDesc) -> int:
    return int(lib().pigan_workspace_bytes(C.byref(desc)))


@dataclass
class StepOut:
    gY: torch.Tensor
    gU: torch.Tensor
    gD: torch.Tensor
    loss: torch.Tensor
    nonfinite: torch.Tensor
    gp: torch.Tensor | None = None      # [G] critic gradient penalty (included in loss[:, 0])


class TrainStep:
    """Holds the workspace and output buffers of repeated training steps.
    noalloc=True calls pigan_train_step_grads_noalloc instead: no workspace
    is allocated, the library's fixed device array serves as workspace."""

    def __init__(self, desc: StepDesc, device="cuda", noalloc: bool = False):
        self.desc = desc
        self.noalloc = noalloc
        self.device = torch.device(device)
        G = desc.genY.n_groups
        self.nY = n_params(desc.genY.in_dim, desc.genY.n_hidden, desc.genY.width)
        self.nU = n_params(desc.genU.in_dim, desc.genU.n_hidden, desc.genU.width)
        self.nD = n_params(desc.disc.in_dim, desc.disc.n_hidden, desc.disc.width)
        need = workspace_bytes(desc)
        if need == 0:
            _check(lib().pigan_train_step_grads(C.byref(desc), *([None] * 8), 0.0, *([None] * 8), 0, None))
        self.ws_bytes = need
        self.ws = None if noalloc else _workspace(need, self.device)
        f32 = dict(dtype=torch.float32, device=self.device)
        self.out = StepOut(torch.empty((G, self.nY), **f32), torch.empty((G, self.nU), **f32),
                           torch.empty((G, self.nD), **f32), torch.empty((G, 3), **f32),
                           torch.zeros((1,), dtype=torch.int32, device=self.device),
                           torch.zeros((G,), **f32) if desc.lambda_gp != 0.0 else None)

    def __call__(self, pY, pU, pD, z, xc, xsY, xsU, real, f=None, f_const=0.0, w_group=None,
                 gp_eps=None) -> StepOut:
        """gp_eps: [G, min(S, B_r)] mixing weights of the critic gradient
        penalty (required when the descriptor's lambda_gp is non-zero)."""
        d = self.desc
        G, S, Pn = d.genY.n_groups, d.S, d.P
        o = self.out
        args = [C.byref(d), _ptr(pY, "pY", G * self.nY), _ptr(pU, "pU", G * self.nU), _ptr(pD, "pD", G * self.nD),
                _ptr(z, "z", G * S * d.n_z), _ptr(xc, "xc", G * S * Pn * d.d), _ptr(xsY, "xsY", G * d.n_sY * d.d),
                _ptr(xsU, "xsU", G * d.n_sU * d.d), _ptr(f, "f", G * S * Pn), float(f_const),
                _ptr(real, "real", G * d.B_r * (d.n_sY + d.n_sU)), _ptr(w_group, "w_group", G)]
        outs = [_ptr(o.gY, "gY"), _ptr(o.gU, "gU"), _ptr(o.gD, "gD"), _ptr(o.loss, "loss")]
        tail = [_ptr(o.nonfinite, "nonfinite", 1, dtype=torch.int32), _ptr(self.ws, "ws", dtype=torch.uint8),
                self.ws_bytes, _stream()]
        if self.noalloc:
            st = lib().pigan_train_step_grads_noalloc(*args, *outs, _ptr(o.nonfinite, "nonfinite", 1,
                                                                         dtype=torch.int32), _stream())
        elif d.lambda_gp != 0.0:
            eps = _ptr(gp_eps, "gp_eps", G * min(S, d.B_r))
            st = lib().pigan_train_step_grads_gp(*args, eps, *outs, _ptr(o.gp, "gp", G), *tail)
        else:
            st = lib().pigan_train_step_grads(*args, *outs, *tail)
        _check(st)
        return o


def trunk_desc(wl: Workload, S: int | None = None, B_r: int | None = None, chunk_S: int = 0,
               dtype: str | None = None, lambda_pde: float | None = None, loss_scale: float = 1.0,
               lambda_gp: float = 0.0) -> TrunkDesc:
    S = wl.S if S is None else S
    B_r = wl.B_r if B_r is None else B_r
    return TrunkDesc(Mlp(wl.G, wl.in_dim, wl.L, wl.W), Mlp(wl.G, wl.n_in, wl.L_D, wl.W_D), wl.d, wl.n_z, S, wl.P,
                     wl.n_sY, wl.n_sU, B_r, chunk_S, DTYPES[dtype or wl.dtype],
                     wl.lambda_pde if lambda_pde is None else lambda_pde, loss_scale, lambda_gp)


def trunk_workspace_bytes(desc: TrunkDesc) -> int:
    return int(lib().pigan_trunk_workspace_bytes(C.byref(desc)))


@dataclass
class TrunkOut:
    gT: torch.Tensor
    gD: torch.Tensor
    loss: torch.Tensor
    nonfinite: torch.Tensor
    gp: torch.Tensor | None = None    # [G] gradient penalty (when lambda_gp > 0)


class TrunkStep:
    """Repeated training steps with the shared-trunk generator."""

    def __init__(self, desc: TrunkDesc, device="cuda"):
        self.desc = desc
        self.device = torch.device(device)
        G = desc.trunk.n_groups
        self.nT = int(lib().pigan_trunk_param_count(C.byref(desc.trunk)))
        self.nD = n_params(desc.disc.in_dim, desc.disc.n_hidden, desc.disc.width)
        need = trunk_workspace_bytes(desc)
        if need == 0:
            _check(lib().pigan_trunk_step_grads(C.byref(desc), *([None] * 7), 0.0, *([None] * 7), 0, None))
        self.ws_bytes = need
        self.ws = _workspace(need, self.device)
        f32 = dict(dtype=torch.float32, device=self.device)
        self.out = TrunkOut(torch.empty((G, self.nT), **f32), torch.empty((G, self.nD), **f32),
                            torch.empty((G, 3), **f32), torch.zeros((1,), dtype=torch.int32, device=self.device),
                            torch.empty((G,), **f32) if desc.lambda_gp > 0 else None)

    def __call__(self, pT, pD, z, xc, xsY, xsU, real, f=None, f_const=0.0, w_group=None, gp_eps=None) -> TrunkOut:
        d = self.desc
        G, S, Pn = d.trunk.n_groups, d.S, d.P
        o = self.out
        args = [C.byref(d), _ptr(pT, "pT", G * self.nT), _ptr(pD, "pD", G * self.nD), _ptr(z, "z", G * S * d.n_z),
                _ptr(xc, "xc", G * S * Pn * d.d), _ptr(xsY, "xsY", G * d.n_sY * d.d),
                _ptr(xsU, "xsU", G * d.n_sU * d.d), _ptr(f, "f", G * S * Pn), float(f_const),
                _ptr(real, "real", G * d.B_r * (d.n_sY + d.n_sU)), _ptr(w_group, "w_group", G)]
        tail = [_ptr(o.nonfinite, "nonfinite", 1, dtype=torch.int32), _ptr(self.ws, "ws", dtype=torch.uint8),
                self.ws_bytes, _stream()]
        if d.lambda_gp > 0:
            eps = _ptr(gp_eps, "gp_eps", G * min(S, d.B_r))
            st = lib().pigan_trunk_step_grads_gp(*args, eps, _ptr(o.gT, "gT"), _ptr(o.gD, "gD"),
                                                 _ptr(o.loss, "loss"), _ptr(o.gp, "gp", G), *tail)
        else:
            st = lib().pigan_trunk_step_grads(*args, _ptr(o.gT, "gT"), _ptr(o.gD, "gD"), _ptr(o.loss, "loss"),
                                              *tail)
        _check(st)
        return o


def hier_desc(wl: Workload, D: int, mY: int, mU: int, nF: int, S: int | None = None, B_r: int | None = None,
              chunk_S: int = 0, dtype: str | None = None, lambda_pde: float = 0.0,
              loss_scale: float = 1.0, lambda_gp: float = 0.0) -> HierDesc:
    S = wl.S if S is None else S
    B_r = wl.B_r if B_r is None else B_r
    n_in = mY + mU + nF * (1 + wl.d)
    return HierDesc(Mlp(1, wl.in_dim, wl.L, wl.W), Mlp(1, wl.in_dim, wl.L, wl.W), Mlp(D, n_in, wl.L_D, wl.W_D),
                    wl.d, wl.n_z, S, wl.P, wl.n_sY, wl.n_sU, B_r, chunk_S, mY, mU, nF, DTYPES[dtype or wl.dtype],
                    lambda_pde, loss_scale, lambda_gp)


@dataclass
class HierOut:
    gY: torch.Tensor
    gU: torch.Tensor
    gD: torch.Tensor      # [D, nD]
    loss: torch.Tensor    # [D, 3]: L_D[k], L_adv[k], L_pde
    nonfinite: torch.Tensor
    gp: torch.Tensor | None = None    # [D] every critic's gradient penalty (when lambda_gp > 0)


class HierStep:
    """Repeated domain-decomposition steps: one generator pair, D critics."""

    def __init__(self, desc: HierDesc, device="cuda"):
        self.desc = desc
        self.device = torch.device(device)
        D = desc.disc.n_groups
        self.nY = n_params(desc.genY.in_dim, desc.genY.n_hidden, desc.genY.width)
        self.nU = n_params(desc.genU.in_dim, desc.genU.n_hidden, desc.genU.width)
        self.nD = n_params(desc.disc.in_dim, desc.disc.n_hidden, desc.disc.width)
        need = int(lib().pigan_hier_workspace_bytes(C.byref(desc)))
        if need == 0:
            _check(lib().pigan_hier_step_grads(C.byref(desc), *([None] * 8), 0.0, *([None] * 10), None, 0, None))
        self.ws_bytes = need
        self.ws = _workspace(need, self.device)
        f32 = dict(dtype=torch.float32, device=self.device)
        self.out = HierOut(torch.empty((self.nY,), **f32), torch.empty((self.nU,), **f32),
                           torch.empty((D, self.nD), **f32), torch.empty((D, 3), **f32),
                           torch.zeros((1,), dtype=torch.int32, device=self.device),
                           torch.empty((D,), **f32) if desc.lambda_gp > 0 else None)

    def __call__(self, pY, pU, pD, z, xc, xsY, xsU, idxY, idxU, idxF, real, w_disc, f=None, f_const=0.0,
                 gp_eps=None) -> HierOut:
        """gp_eps: [D, min(S, B_r)] mixing weights of the critics' gradient
        penalty (required when the descriptor's lambda_gp is non-zero)."""
        d = self.desc
        D, S, Pn = d.disc.n_groups, d.S, d.P
        o = self.out
        i32 = torch.int32
        args = [C.byref(d), _ptr(pY, "pY", self.nY), _ptr(pU, "pU", self.nU), _ptr(pD, "pD", D * self.nD),
                _ptr(z, "z", S * d.n_z), _ptr(xc, "xc", S * Pn * d.d), _ptr(xsY, "xsY", d.n_sY * d.d),
                _ptr(xsU, "xsU", d.n_sU * d.d), _ptr(f, "f", S * Pn), float(f_const),
                _ptr(idxY, "idxY", D * d.mY, dtype=i32), _ptr(idxU, "idxU", D * d.mU, dtype=i32),
                _ptr(idxF, "idxF", D * d.nF, dtype=i32), _ptr(real, "real", D * d.B_r * d.disc.in_dim),
                _ptr(w_disc, "w_disc", D)]
        outs = [_ptr(o.gY, "gY"), _ptr(o.gU, "gU"), _ptr(o.gD, "gD"), _ptr(o.loss, "loss")]
        tail = [_ptr(o.nonfinite, "nonfinite", 1, dtype=i32), _ptr(self.ws, "ws", dtype=torch.uint8), self.ws_bytes,
                _stream()]
        if d.lambda_gp > 0:
            eps = _ptr(gp_eps, "gp_eps", D * min(S, d.B_r))
            st = lib().pigan_hier_step_grads_gp(*args, eps, *outs, _ptr(o.gp, "gp", D), *tail)
        else:
            st = lib().pigan_hier_step_grads(*args, *outs, *tail)
        _check(st)
        return o


def hier_trunk_desc(wl: Workload, D: int, mY: int, mU: int, nF: int, S: int | None = None,
                    B_r: int | None = None, chunk_S: int = 0, dtype: str | None = None, lambda_pde: float = 0.0,
                    loss_scale: float = 1.0, lambda_gp: float = 0.0) -> HierTrunkDesc:
    S = wl.S if S is None else S
    B_r = wl.B_r if B_r is None else B_r
    n_in = mY + mU + nF * (1 + wl.d)
    return HierTrunkDesc(Mlp(1, wl.in_dim, wl.L, wl.W), Mlp(D, n_in, wl.L_D, wl.W_D), wl.d, wl.n_z, S, wl.P,
                         wl.n_sY, wl.n_sU, B_r, chunk_S, mY, mU, nF, DTYPES[dtype or wl.dtype], lambda_pde,
                         loss_scale, lambda_gp)


@dataclass
class HierTrunkOut:
    gT: torch.Tensor
    gD: torch.Tensor      # [D, nD]
    loss: torch.Tensor    # [D, 3]: L_D[k], L_adv[k], L_pde
    nonfinite: torch.Tensor
    gp: torch.Tensor | None = None    # [D] every critic's gradient penalty (when lambda_gp > 0)


class HierTrunkStep:
    """Repeated domain-decomposition steps with the shared-trunk generator."""

    def __init__(self, desc: HierTrunkDesc, device="cuda"):
        self.desc = desc
        self.device = torch.device(device)
        D = desc.disc.n_groups
        self.nT = int(lib().pigan_trunk_param_count(C.byref(desc.trunk)))
        self.nD = n_params(desc.disc.in_dim, desc.disc.n_hidden, desc.disc.width)
        need = int(lib().pigan_hier_trunk_workspace_bytes(C.byref(desc)))
        if need == 0:
            _check(lib().pigan_hier_trunk_step_grads(C.byref(desc), *([None] * 7), 0.0, *([None] * 10), 0, None))
        self.ws_bytes = need
        self.ws = _workspace(need, self.device)
        f32 = dict(dtype=torch.float32, device=self.device)
        self.out = HierTrunkOut(torch.empty((self.nT,), **f32), torch.empty((D, self.nD), **f32),
                                torch.empty((D, 3), **f32), torch.zeros((1,), dtype=torch.int32, device=self.device),
                                torch.empty((D,), **f32) if desc.lambda_gp > 0 else None)

    def __call__(self, pT, pD, z, xc, xsY, xsU, idxY, idxU, idxF, real, w_disc, f=None, f_const=0.0,
                 gp_eps=None) -> HierTrunkOut:
        d = self.desc
        D, S, Pn = d.disc.n_groups, d.S, d.P
        o = self.out
        i32 = torch.int32
        args = [C.byref(d), _ptr(pT, "pT", self.nT), _ptr(pD, "pD", D * self.nD), _ptr(z, "z", S * d.n_z),
                _ptr(xc, "xc", S * Pn * d.d), _ptr(xsY, "xsY", d.n_sY * d.d), _ptr(xsU, "xsU", d.n_sU * d.d),
                _ptr(f, "f", S * Pn), float(f_const),
                _ptr(idxY, "idxY", D * d.mY, dtype=i32), _ptr(idxU, "idxU", D * d.mU, dtype=i32),
                _ptr(idxF, "idxF", D * d.nF, dtype=i32), _ptr(real, "real", D * d.B_r * d.disc.in_dim),
                _ptr(w_disc, "w_disc", D)]
        outs = [_ptr(o.gT, "gT"), _ptr(o.gD, "gD"), _ptr(o.loss, "loss")]
        tail = [_ptr(o.nonfinite, "nonfinite", 1, dtype=i32), _ptr(self.ws, "ws", dtype=torch.uint8), self.ws_bytes,
                _stream()]
        if d.lambda_gp > 0:
            eps = _ptr(gp_eps, "gp_eps", D * min(S, d.B_r))
            st = lib().pigan_hier_trunk_step_grads_gp(*args, eps, *outs, _ptr(o.gp, "gp", D), *tail)
        else:
            st = lib().pigan_hier_trunk_step_grads(*args, *outs, *tail)
        _check(st)
        return o


class StepGraph:
    """A step call captured once in a HIP graph (torch.cuda.CUDAGraph) and
    replayed: the same kernels on the same device buffers, launched as one
    graph (no per-kernel launch gaps).  `fn` issues the work on the current
    stream and takes no arguments (e.g. a lambda around a TrainStep call with
    fixed device tensors); it runs once eagerly on a side stream first.  The
    library's launches are all kernels (no memset or host synchronisation), so
    every replay recomputes the outputs from the current contents of the
    inputs."""

    def __init__(self, fn):
        self.fn = fn
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            fn()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        self.graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(self.graph):
            fn()
        torch.cuda.synchronize()

    def replay(self):
        self.graph.replay()


def profile_enable(on: bool = True):
    _check(lib().pigan_profile_enable(1 if on else 0))


def profile_read() -> list[dict]:
    arr = (KernelStat * 64)()
    n = C.c_int32(0)
    _check(lib().pigan_profile_read(arr, 64, C.byref(n)))
    return [dict(name=arr[i].name.decode(), launches=arr[i].launches, total_ms=arr[i].total_ms,
                 flops=arr[i].flops, bytes=arr[i].bytes) for i in range(min(n.value, 64))]
