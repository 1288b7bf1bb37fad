"""GPU checks of the training loop: the Adam update kernel against the oracle
update, the GPU trainer against the oracle trainer for both exchange schedules,
dynamic loss scaling in fp16, and the residual loss falling while training."""
import sys

import numpy as np
import pytest
import torch

import oracle
from oracle.trainer import adam_update, train as oracle_train
from paper_1910_13444_amd import configs, pigan
from paper_1910_13444_amd.configs import Workload
from paper_1910_13444_amd.inputs import make_inputs
from paper_1910_13444_amd.train import Adam, TrainConfig, Trainer
from _parity import rel, to_dev

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def test_adam_kernel_matches_oracle():
    _say("adam kernel: n=100003, 3 updates, then a flagged (skipped) update")
    rng = np.random.default_rng(3)
    n = 100003
    p0 = rng.standard_normal(n).astype(np.float32)
    p = to_dev(p0)
    opt = Adam(p, lr=1e-3, beta1=0.5, beta2=0.9, eps=1e-8)
    pr, m, v = p0.astype(np.float64), np.zeros(n), np.zeros(n)
    for t in range(1, 4):
        g = (rng.standard_normal(n) * 10.0 ** rng.integers(-3, 2, n)).astype(np.float32)
        opt.step(to_dev(g))
        pr, m, v = adam_update(pr, g, m, v, t, 1e-3, 0.5, 0.9, 1e-8)
    torch.cuda.synchronize()
    pg = p.cpu().numpy().astype(np.float64)
    # the master weights are fp32: each update rounds p (|p| ~ 1, ulp ~ 1.2e-7),
    # so the weights agree to ~1e-7 relative while their change (~3 lr) carries
    # a few 1e-5 relative rounding; both bars follow from that
    err_p = rel(pg, pr)
    err_d = rel(pg - p0, pr - p0)
    print(f"adam update rel err: weights {err_p:.3g}, weight change {err_d:.3g}")
    assert err_p <= 1e-6 and err_d <= 1e-4
    assert rel(opt.m.cpu().numpy(), m) <= 1e-6 and rel(opt.v.cpu().numpy(), v) <= 1e-6
    before = p.clone()
    flag = torch.ones(1, dtype=torch.int32, device="cuda")
    opt.step(to_dev(np.full(n, np.inf, np.float32)), skip=flag)
    torch.cuda.synchronize()
    assert torch.equal(before, p)


TW = Workload("train_tiny", "fp32", G=1, d=2, n_z=3, L=3, W=32, S=3, P=16, n_sY=4, n_sU=3,
              L_D=2, W_D=32, B_r=3, f_const=0.5, seed=41)


def _oracle_step_fn(wl, inp, real):
    gshape, dshape = wl.gen_shape(), wl.disc_shape()
    f = np.full((wl.S, wl.P), wl.f_const)
    if wl.arch == "trunk":
        def fn(pG, pD):
            o = oracle.train_step_group_trunk(gshape, dshape, wl.d, pG, pD, inp.z[0], inp.xc[0], inp.xsY[0],
                                              inp.xsU[0], f, real[0], w=float(inp.w_group[0]))
            return np.array([o["L_D"], o["L_adv"], o["L_pde"]]), o["gT"], o["gD"]
    else:
        nY = inp.pY.shape[1]

        def fn(pG, pD):
            o = oracle.train_step_group(gshape, dshape, wl.d, pG[:nY], pG[nY:], pD, inp.z[0], inp.xc[0],
                                        inp.xsY[0], inp.xsU[0], f, real[0], w=float(inp.w_group[0]))
            return (np.array([o["L_D"], o["L_adv"], o["L_pde"]]), np.concatenate([o["gY"], o["gU"]]), o["gD"])
    return fn


def _critic_calls(schedule, rounds, n_critic=2, steps_per_exchange=2):
    """Which step calls of the schedule are critic updates (in call order)."""
    one = [True] * n_critic + [False] if schedule == "sequential" else [False, True] * steps_per_exchange
    return np.array(one * rounds)


def _without_critic_residual(ref_losses, schedule, rounds=3):
    """The oracle loop's losses as the GPU loop records them: the critic-only
    calls of the paired and trunk steps do not evaluate the residual and
    report L_pde = 0."""
    out = np.array(ref_losses, dtype=np.float64).copy()
    out[_critic_calls(schedule, rounds), ..., 2] = 0.0
    return out


def _gpu_trainer(wl, inp, real, cfg):
    gen = [to_dev(inp.pT)] if wl.arch == "trunk" else [to_dev(inp.pY), to_dev(inp.pU)]
    dev = dict(z=to_dev(inp.z), xc=to_dev(inp.xc), xsY=to_dev(inp.xsY), xsU=to_dev(inp.xsU), real=to_dev(real),
               w_group=to_dev(inp.w_group))
    return Trainer(wl, gen, to_dev(inp.pD), dev, cfg)


@pytest.mark.parametrize("schedule,arch", [("sequential", "pair"), ("parallel", "pair"), ("sequential", "trunk")])
def test_trainer_matches_oracle(schedule, arch):
    wl = TW.with_(arch=arch, L=3 if arch == "pair" else 5)
    _say(f"trainer {schedule} {arch}: 3 rounds fp32 vs the oracle loop")
    inp = make_inputs(wl)
    real = oracle.real_snapshots_trunk(wl, inp) if arch == "trunk" else oracle.real_snapshots(wl, inp)
    cfg = TrainConfig(schedule=schedule, n_critic=2, steps_per_exchange=2, lr_g=1e-3, lr_d=2e-3)
    tr = _gpu_trainer(wl, inp, real, cfg)
    losses = tr.run(3).cpu().numpy()
    pG0 = inp.pT[0] if arch == "trunk" else np.concatenate([inp.pY[0], inp.pU[0]])
    pG, pD, ref_losses = oracle_train(_oracle_step_fn(wl, inp, real), pG0, inp.pD[0], 3, schedule=schedule,
                                      n_critic=2, steps_per_exchange=2, lr_g=1e-3, lr_d=2e-3)
    ref_losses = _without_critic_residual(ref_losses, schedule)
    gpu_G = np.concatenate([g.cpu().numpy().ravel() for g in tr.gen])
    gpu_D = tr.pD.cpu().numpy().ravel()
    eG = rel(gpu_G - pG0, pG - pG0)
    eD = rel(gpu_D - inp.pD[0], pD - inp.pD[0])
    eL = rel(losses.reshape(ref_losses.shape), ref_losses)
    print(f"weight change rel err: generator {eG:.3g}, critic {eD:.3g}; losses {eL:.3g}")
    assert losses.shape[0] == ref_losses.shape[0]
    # losses at the fp32 bar; weight changes within 2e-5 (Adam's normalised update
    # divides by sqrt(v) + eps, so coordinates with tiny gradients amplify their
    # error; measured at most 4.1e-6 over these schedules)
    assert eG <= 2e-5 and eD <= 2e-5 and eL <= 1e-5


def test_dynamic_loss_scale_fp16_skips_overflow():
    wl = configs.C2.with_(S=2, P=64, B_r=2, dtype="fp16", seed=43)
    _say("trainer fp16 with an overflowing initial loss scale 2^40")
    inp = make_inputs(wl)
    real = oracle.real_snapshots(wl, inp)
    cfg = TrainConfig(dynamic_loss_scale=True, init_scale=2.0 ** 40, growth_interval=1000, lr_g=1e-4, lr_d=1e-4)
    tr = _gpu_trainer(wl, inp, real, cfg)
    pD0 = tr.pD.clone()
    gen0 = [g.clone() for g in tr.gen]
    # critic step (critic only: the adversarial path is fp32 and does not
    # overflow), then the generator step, whose fp16 reverse pass overflows
    tr.round()
    torch.cuda.synchronize()
    assert tr.skipped == 1 and tr.scaler.scale == 2.0 ** 39
    assert all(torch.equal(a, b) for a, b in zip(gen0, tr.gen))   # skipped on the device: weights untouched
    assert not torch.equal(pD0, tr.pD)
    # the scale comes down to one at which steps stop overflowing: some block
    # of 4 rounds (8 step calls) runs without a skip within 60 rounds
    clean = False
    for _ in range(15):
        before = tr.skipped
        tr.run(4)
        torch.cuda.synchronize()
        if tr.skipped == before:
            clean = True
            break
    print(f"scale 2^{np.log2(tr.scaler.scale):.0f}, skipped {tr.skipped}")
    assert clean and tr.scaler.scale < 2.0 ** 39
    assert not any(torch.equal(a, b) for a, b in zip(gen0, tr.gen))
    assert torch.isfinite(tr.pD).all() and all(torch.isfinite(g).all() for g in tr.gen)


def test_training_reduces_the_residual():
    """The 1-D Darcy toy (fp32): the residual penalty is a direct term of the
    generator loss, so training lowers it."""
    wl = configs.C1
    _say("trainer C1 toy: 150 rounds, residual loss must drop")
    inp = make_inputs(wl)
    real = oracle.real_snapshots(wl, inp)
    cfg = TrainConfig(n_critic=1, lr_g=2e-3, lr_d=2e-3)
    tr = _gpu_trainer(wl, inp, real, cfg)
    losses = tr.run(150).cpu().numpy()[:, 0, :]    # [calls, 3]; critic then generator call per round
    gen_calls = losses[1::2]                       # (critic-only calls report no residual)
    first, last = gen_calls[:4, 2].mean(), gen_calls[-4:, 2].mean()
    print(f"L_pde first {first:.4g} last {last:.4g}; L_D last {losses[-1, 0]:.4g}")
    assert np.isfinite(losses).all()
    assert last < 0.5 * first


HW = configs.C2.with_(n_sY=16, n_sU=16, S=3, P=16, B_r=2, W=32, W_D=32, L=3, L_D=2, n_z=3, dtype="fp32",
                      lambda_pde=0.5, f_const=0.3, seed=45)


@pytest.mark.parametrize("schedule,arch", [("sequential", "hier"), ("parallel", "hier_trunk")])
def test_hier_trainer_matches_oracle(schedule, arch):
    """The training loop of the domain-decomposition step: one generator
    (pair or shared trunk) and 1 + 4 subdomain critics updated together."""
    from paper_1910_13444_amd.inputs import make_hier_inputs
    wl = HW.with_(arch=arch, L=3 if arch == "hier" else 5)
    _say(f"hier trainer {schedule} {arch}: 3 rounds fp32 vs the oracle loop")
    hi = make_hier_inputs(wl, sides=(1, 2), m_sensors=4, n_free=4)
    b, h = hi.base, hi.hier
    trunk = arch == "hier_trunk"
    real = oracle.real_snapshots_hier(wl, hi, trunk_teacher=b.tT[0] if trunk else None)
    f = np.full((wl.S, wl.P), wl.f_const)
    dshape = (real.shape[2], wl.L_D, wl.W_D)
    nY = 0 if trunk else b.pY.shape[1]

    def fn(pG, pD):
        pY, pU = (pG, None) if trunk else (pG[:nY], pG[nY:])
        o = oracle.train_step_hier(wl.gen_shape(), dshape, wl.d, pY, pU, pD, b.z[0], b.xc[0], b.xsY[0], b.xsU[0], f,
                                   h.idxY, h.idxU, h.idxF, real, h.w, lambda_pde=wl.lambda_pde, trunk=trunk)
        loss = np.stack([o["L_D"], o["L_adv"], np.full(len(o["L_D"]), o["L_pde"])], 1)
        return loss, (o["gY"] if trunk else np.concatenate([o["gY"], o["gU"]])), o["gD"]

    def ti(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()
    dev = dict(z=to_dev(b.z[0]), xc=to_dev(b.xc[0]), xsY=to_dev(b.xsY[0]), xsU=to_dev(b.xsU[0]), real=to_dev(real),
               idxY=ti(h.idxY), idxU=ti(h.idxU), idxF=ti(h.idxF), w_disc=to_dev(h.w))
    gen = [to_dev(b.pT[0])] if trunk else [to_dev(b.pY[0]), to_dev(b.pU[0])]
    cfg = TrainConfig(schedule=schedule, n_critic=2, steps_per_exchange=2, lr_g=1e-3, lr_d=2e-3)
    tr = Trainer(wl, gen, to_dev(hi.pD), dev, cfg)
    losses = tr.run(3).cpu().numpy()
    pG0 = b.pT[0] if trunk else np.concatenate([b.pY[0], b.pU[0]])
    pG, pD, ref_losses = oracle_train(fn, pG0, hi.pD, 3, schedule=schedule, n_critic=2, steps_per_exchange=2,
                                      lr_g=1e-3, lr_d=2e-3)
    gpu_G = np.concatenate([g.cpu().numpy().ravel() for g in tr.gen])
    gpu_D = tr.pD.cpu().numpy()
    eG = rel(gpu_G - pG0, pG - pG0)
    eD = rel(gpu_D - hi.pD, pD - hi.pD)
    eL = rel(losses, ref_losses)
    print(f"weight change rel err: generator {eG:.3g}, critics {eD:.3g}; losses {eL:.3g}")
    assert losses.shape == ref_losses.shape
    # losses at the fp32 bar; weight changes within 2e-5 (Adam's normalised update
    # divides by sqrt(v) + eps, so coordinates with tiny gradients amplify their
    # error; measured at most 4.1e-6 over these schedules)
    assert eG <= 2e-5 and eD <= 2e-5 and eL <= 1e-5


@pytest.mark.parametrize("schedule,arch", [("sequential", "pair"), ("parallel", "trunk"), ("sequential", "hier")])
def test_trainer_with_gradient_penalty_matches_oracle(schedule, arch):
    """The training loop with the critics' gradient penalty: each step call
    takes its own mixing weights (a seeded host sequence fed to both sides in
    call order); 3 rounds fp32 against the oracle loop."""
    lgp = 5.0
    rng = np.random.default_rng(47)
    if arch == "hier":
        from paper_1910_13444_amd.inputs import make_hier_inputs
        wl = HW.with_(arch="hier", seed=48)
        hi = make_hier_inputs(wl, sides=(1, 2), m_sensors=4, n_free=4)
        b, h = hi.base, hi.hier
        real = oracle.real_snapshots_hier(wl, hi)
        n_crit, pD0 = h.D, hi.pD
    else:
        wl = TW.with_(arch=arch, L=3 if arch == "pair" else 5, seed=49)
        inp = make_inputs(wl)
        real = oracle.real_snapshots_trunk(wl, inp) if arch == "trunk" else oracle.real_snapshots(wl, inp)
        n_crit, pD0 = wl.G, inp.pD[0]
    n_gp = min(wl.S, real.shape[1])
    eps = [rng.random((n_crit, n_gp)).astype(np.float32) for _ in range(40)]
    _say(f"trainer {schedule} {arch} with gradient penalty {lgp}: 3 rounds fp32 vs the oracle loop")
    calls = [0]

    def next_eps():
        e = eps[calls[0]]
        calls[0] += 1
        return e

    cfg = TrainConfig(schedule=schedule, n_critic=2, steps_per_exchange=2, lr_g=1e-3, lr_d=2e-3, lambda_gp=lgp)
    if arch == "hier":
        f = np.full((wl.S, wl.P), wl.f_const)
        dshape = (real.shape[2], wl.L_D, wl.W_D)
        nY = b.pY.shape[1]

        def fn(pG, pD):
            o = oracle.train_step_hier(wl.gen_shape(), dshape, wl.d, pG[:nY], pG[nY:], pD, b.z[0], b.xc[0], b.xsY[0],
                                       b.xsU[0], f, h.idxY, h.idxU, h.idxF, real, h.w, lambda_pde=wl.lambda_pde,
                                       lambda_gp=lgp, gp_eps=next_eps())
            loss = np.stack([o["L_D"], o["L_adv"], np.full(len(o["L_D"]), o["L_pde"])], 1)
            return loss, np.concatenate([o["gY"], o["gU"]]), o["gD"]

        def ti(a):
            return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()
        dev = dict(z=to_dev(b.z[0]), xc=to_dev(b.xc[0]), xsY=to_dev(b.xsY[0]), xsU=to_dev(b.xsU[0]),
                   real=to_dev(real), idxY=ti(h.idxY), idxU=ti(h.idxU), idxF=ti(h.idxF), w_disc=to_dev(h.w))
        gen = [to_dev(b.pY[0]), to_dev(b.pU[0])]
        pG0 = np.concatenate([b.pY[0], b.pU[0]])
        tr = Trainer(wl, gen, to_dev(pD0), dev, cfg, gp_eps_fn=lambda k: to_dev(eps[k]))
    else:
        gshape, dshape = wl.gen_shape(), wl.disc_shape()
        f = np.full((wl.S, wl.P), wl.f_const)
        nY = 0 if arch == "trunk" else inp.pY.shape[1]

        def fn(pG, pD):
            e = next_eps()[0]
            if arch == "trunk":
                o = oracle.train_step_group_trunk(gshape, dshape, wl.d, pG, pD, inp.z[0], inp.xc[0], inp.xsY[0],
                                                  inp.xsU[0], f, real[0], w=float(inp.w_group[0]), lambda_gp=lgp,
                                                  gp_eps=e)
                return np.array([o["L_D"], o["L_adv"], o["L_pde"]]), o["gT"], o["gD"]
            o = oracle.train_step_group(gshape, dshape, wl.d, pG[:nY], pG[nY:], pD, inp.z[0], inp.xc[0], inp.xsY[0],
                                        inp.xsU[0], f, real[0], w=float(inp.w_group[0]), lambda_gp=lgp, gp_eps=e)
            return np.array([o["L_D"], o["L_adv"], o["L_pde"]]), np.concatenate([o["gY"], o["gU"]]), o["gD"]
        pG0 = inp.pT[0] if arch == "trunk" else np.concatenate([inp.pY[0], inp.pU[0]])
        tr = _gpu_trainer(wl, inp, real, cfg)
        tr.gp_eps_fn = lambda k: to_dev(eps[k])
    losses = tr.run(3).cpu().numpy()
    pG, pD, ref_losses = oracle_train(fn, pG0, pD0, 3, schedule=schedule, n_critic=2, steps_per_exchange=2,
                                      lr_g=1e-3, lr_d=2e-3)
    if arch != "hier":
        ref_losses = _without_critic_residual(ref_losses, schedule)
    assert tr.calls == calls[0]
    gpu_G = np.concatenate([g.cpu().numpy().ravel() for g in tr.gen])
    gpu_D = tr.pD.cpu().numpy().reshape(np.shape(pD))
    eG = rel(gpu_G - pG0, pG - pG0)
    eD = rel(gpu_D - pD0, pD - pD0)
    eL = rel(losses.reshape(ref_losses.shape), ref_losses)
    print(f"weight change rel err: generator {eG:.3g}, critic {eD:.3g}; losses {eL:.3g}")
    # losses at the fp32 bar; weight changes within 2e-5 (Adam's normalised update
    # divides by sqrt(v) + eps, so coordinates with tiny gradients amplify their
    # error; measured at most 4.1e-6 over these schedules)
    assert eG <= 2e-5 and eD <= 2e-5 and eL <= 1e-5
