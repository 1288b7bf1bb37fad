"""The C-ABI library loads, exports every symbol include/pigan.h declares, and
rejects invalid arguments on the host before touching the device (these calls
return before any HIP call, so they run without a GPU)."""
import ctypes as C
import os

import pytest

from paper_1910_13444_amd import configs, pigan

pytestmark = pytest.mark.skipif(not os.path.exists(pigan.LIB_PATH), reason="libpigan.so not built")

FAKE = C.c_void_p(4096)   # never dereferenced: every case below fails validation first


def test_exports_every_declared_symbol():
    L = pigan.lib()
    names = pigan.declared_symbols()
    assert "pigan_train_step_grads" in names and len(names) >= 11
    for n in names:
        assert hasattr(L, n), n


def test_n_params_matches_packing():
    L = pigan.lib()
    for wl in (configs.C1, configs.C2, configs.C5):
        m = pigan.Mlp(1, wl.in_dim, wl.L, wl.W)
        assert L.pigan_mlp_n_params(C.byref(m)) == configs.n_params(wl.in_dim, wl.L, wl.W)


def _step(desc, ws_bytes, ptr=FAKE, f=None, wg=None):
    L = pigan.lib()
    args = [ptr] * 8
    args[7] = f        # f may be null
    return L.pigan_train_step_grads(C.byref(desc), *args[:7], f, 0.0, ptr, wg, ptr, ptr, ptr, ptr, ptr, ptr,
                                    ws_bytes, None)


@pytest.mark.parametrize("field,value,status", [
    ("d", 0, pigan.EINVAL), ("d", 4, pigan.EINVAL), ("n_z", 0, pigan.EINVAL), ("S", 0, pigan.EINVAL),
    ("P", -1, pigan.EINVAL), ("n_sY", 0, pigan.EINVAL), ("B_r", 0, pigan.EINVAL), ("chunk_S", -2, pigan.EINVAL),
    ("lambda_gp", -0.5, pigan.EINVAL), ("loss_scale", 0.0, pigan.EINVAL), ("lambda_pde", -1.0, pigan.EINVAL),
    ("dt", 7, pigan.EINVAL), ("critic_only", 2, pigan.EINVAL), ("critic_only", -1, pigan.EINVAL),
])
def test_step_rejects_bad_descriptor(field, value, status):
    d = pigan.step_desc(configs.C1)
    setattr(d, field, value)
    assert _step(d, 1 << 40) == status
    assert pigan.lib().pigan_last_error()
    assert pigan.workspace_bytes(d) == 0


def _step_gp(desc, ws_bytes, eps, ptr=FAKE):
    L = pigan.lib()
    return L.pigan_train_step_grads_gp(C.byref(desc), *([ptr] * 7), None, 0.0, ptr, None, eps, ptr, ptr, ptr, ptr,
                                       None, ptr, ptr, ws_bytes, None)


def test_gradient_penalty_entry_validation():
    d = pigan.step_desc(configs.C1, lambda_gp=10.0)
    need = pigan.workspace_bytes(d)
    assert need > pigan.workspace_bytes(pigan.step_desc(configs.C1)) > 0   # the penalty's buffers
    assert _step(d, need) == pigan.ENOTSUP             # the plain entry has no mixing weights
    assert b"pigan_train_step_grads_gp" in pigan.lib().pigan_last_error()
    assert _step_gp(d, need, None) == pigan.EINVAL     # lambda_gp > 0 needs gp_eps
    d.lambda_gp = float("nan")
    assert _step_gp(d, need, FAKE) == pigan.EINVAL
    assert pigan.workspace_bytes(d) == 0
    d = pigan.step_desc(configs.C1, lambda_gp=10.0)
    assert _step_gp(d, need - 1, FAKE) == pigan.EWORKSPACE


def test_step_rejects_inconsistent_shapes():
    d = pigan.step_desc(configs.C1)
    d.genY.in_dim += 1
    assert _step(d, 1 << 40) == pigan.EINVAL
    d = pigan.step_desc(configs.C1)
    d.disc.in_dim += 1
    assert _step(d, 1 << 40) == pigan.EINVAL
    d = pigan.step_desc(configs.C1)
    d.genU.n_groups = 2
    assert _step(d, 1 << 40) == pigan.EINVAL
    d = pigan.step_desc(configs.C1)
    d.genY.width = 48           # not a supported width
    assert _step(d, 1 << 40) == pigan.ENOTSUP


def test_step_rejects_null_and_small_workspace():
    d = pigan.step_desc(configs.C1)
    need = pigan.workspace_bytes(d)
    assert need > 0
    assert _step(d, need, ptr=None) == pigan.EINVAL           # null inputs
    L = pigan.lib()
    args = [FAKE] * 7
    st = L.pigan_train_step_grads(C.byref(d), *args, None, 0.0, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE, None,
                                  need, None)
    assert st == pigan.EWORKSPACE                               # null workspace
    assert _step(d, need - 1) == pigan.EWORKSPACE
    # misaligned workspace
    st = L.pigan_train_step_grads(C.byref(d), *args, None, 0.0, FAKE, None, FAKE, FAKE, FAKE, FAKE, FAKE,
                                  C.c_void_p(4096 + 16), need, None)
    assert st == pigan.EINVAL


def test_workspace_grows_with_chunk():
    d = pigan.step_desc(configs.C2)
    full = pigan.workspace_bytes(d)
    d.chunk_S = 32
    part = pigan.workspace_bytes(d)
    assert 0 < part < full


def test_auto_chunk_keeps_large_steps_bounded():
    for wl in (configs.C3, configs.C5):
        assert 0 < pigan.workspace_bytes(pigan.step_desc(wl)) <= (128 << 30)
    import ctypes as C
    assert 0 < pigan.lib().pigan_trunk_workspace_bytes(C.byref(pigan.trunk_desc(configs.T21))) <= (128 << 30)


def test_gen_forward_and_disc_forward_validation():
    L = pigan.lib()
    net = pigan.Mlp(1, 6, 2, 32)
    assert L.pigan_gen_forward_workspace(C.byref(net), 2, 4, 8, 2, 1) > 0
    assert L.pigan_gen_forward_workspace(C.byref(net), 2, 4, 8, 3, 1) == 0   # order 3
    st = L.pigan_gen_forward(C.byref(net), FAKE, 7, FAKE, FAKE, 0, 4, 8, 1, 1, FAKE, FAKE, 1 << 30, None)
    assert st == pigan.EINVAL                                                 # in_dim <= d
    st = L.pigan_gen_forward(C.byref(net), FAKE, 2, FAKE, FAKE, 0, 4, 8, 1, 1, FAKE, FAKE, 16, None)
    assert st == pigan.EWORKSPACE
    dnet = pigan.Mlp(1, 250, 3, 64)
    assert L.pigan_disc_forward_workspace(C.byref(dnet), 16, 0) > 0
    st = L.pigan_disc_forward(C.byref(dnet), FAKE, FAKE, 0, 0, FAKE, FAKE, 1 << 30, None)
    assert st == pigan.EINVAL
    st = L.pigan_pde_residual(0, 1, 10, FAKE, FAKE, None, 0.0, FAKE, None)
    assert st == pigan.EINVAL
    st = L.pigan_pde_residual(2, 1, 10, None, FAKE, None, 0.0, FAKE, None)
    assert st == pigan.EINVAL


# ---------------------------------------------------------------------------
# shared trunk and parameter update
# ---------------------------------------------------------------------------

def test_trunk_param_count_matches_packing():
    L = pigan.lib()
    for wl in (configs.T5, configs.T11, configs.T21):
        m = pigan.Mlp(1, wl.in_dim, wl.L, wl.W)
        assert L.pigan_trunk_param_count(C.byref(m)) == configs.n_params_trunk(wl.in_dim, wl.L, wl.W)
    assert L.pigan_trunk_param_count(None) == 0


def _trunk_step(desc, ws_bytes, ptr=FAKE, ws=FAKE):
    return pigan.lib().pigan_trunk_step_grads(C.byref(desc), *([ptr] * 6), None, 0.0, ptr, None, ptr, ptr, ptr, ptr,
                                              ws, ws_bytes, None)


@pytest.mark.parametrize("field,value", [("d", 0), ("n_z", 0), ("S", 0), ("P", 0), ("n_sU", 0), ("B_r", 0),
                                         ("chunk_S", -1), ("loss_scale", -1.0), ("lambda_pde", -2.0), ("dt", 9),
                                         ("critic_only", 3)])
def test_trunk_step_rejects_bad_descriptor(field, value):
    d = pigan.trunk_desc(configs.T5)
    setattr(d, field, value)
    assert _trunk_step(d, 1 << 40) == pigan.EINVAL
    assert pigan.trunk_workspace_bytes(d) == 0


def test_trunk_step_validation():
    d = pigan.trunk_desc(configs.T5)
    need = pigan.trunk_workspace_bytes(d)
    assert need > 0
    assert _trunk_step(d, need, ptr=None) == pigan.EINVAL
    assert _trunk_step(d, need - 1) == pigan.EWORKSPACE
    assert _trunk_step(d, need, ws=None) == pigan.EWORKSPACE
    assert _trunk_step(d, need, ws=C.c_void_p(4096 + 64)) == pigan.EINVAL      # misaligned workspace
    d.trunk.width = 96                                                           # neither divides nor fills 256
    assert _trunk_step(d, 1 << 40) == pigan.ENOTSUP
    d = pigan.trunk_desc(configs.T5)
    d.disc.in_dim = 7
    assert _trunk_step(d, 1 << 40) == pigan.EINVAL
    assert pigan.lib().pigan_trunk_step_grads(None, *([FAKE] * 6), None, 0.0, FAKE, None, FAKE, FAKE, FAKE, FAKE,
                                              FAKE, 1 << 40, None) == pigan.EINVAL
    assert 0 < pigan.trunk_workspace_bytes(pigan.trunk_desc(configs.T21)) <= (128 << 30)


def test_adam_update_validation():
    L = pigan.lib()

    def adam(n, ptr=FAKE, lr=1e-3, b1=0.5, b2=0.9, eps=1e-8, t=1):
        return L.pigan_adam_update(n, ptr, ptr, ptr, ptr, lr, b1, b2, eps, t, None, None)
    assert adam(0, ptr=None) == pigan.OK            # nothing to update: no launch
    assert adam(-1) == pigan.EINVAL
    assert adam(10, ptr=None) == pigan.EINVAL
    assert adam(10, t=0) == pigan.EINVAL
    assert adam(10, b1=1.0) == pigan.EINVAL and adam(10, b2=-0.1) == pigan.EINVAL
    assert adam(10, lr=float("inf")) == pigan.EINVAL and adam(10, eps=-1.0) == pigan.EINVAL


def _hier(desc, ws_bytes, ptr=FAKE, idx=FAKE, ws=FAKE):
    return pigan.lib().pigan_hier_step_grads(C.byref(desc), *([ptr] * 7), None, 0.0, idx, idx, idx, ptr, ptr, ptr, ptr,
                                             ptr, ptr, ptr, ws, ws_bytes, None)


def test_hier_step_validation():
    wl = configs.C2.with_(n_sY=256, n_sU=256)
    d = pigan.hier_desc(wl, 21, 16, 16, 16)
    need = int(pigan.lib().pigan_hier_workspace_bytes(C.byref(d)))
    assert need > 0
    assert _hier(d, need, ptr=None) == pigan.EINVAL
    assert _hier(d, need, idx=None) == pigan.EINVAL
    assert _hier(d, need - 1) == pigan.EWORKSPACE
    assert _hier(d, need, ws=C.c_void_p(4096 + 32)) == pigan.EINVAL
    for field, value in (("mY", -1), ("nF", -3), ("B_r", 0), ("lambda_pde", -1.0), ("d", 5), ("critic_only", 2)):
        e = pigan.hier_desc(wl, 21, 16, 16, 16)
        setattr(e, field, value)
        assert _hier(e, 1 << 40) == pigan.EINVAL, field
    e = pigan.hier_desc(wl, 21, 16, 16, 16)
    e.genY.n_groups = 2                                    # one generator pair only
    assert _hier(e, 1 << 40) == pigan.EINVAL
    e = pigan.hier_desc(wl, 21, 16, 16, 16)
    e.disc.in_dim = 81                                     # != mY + mU + nF (1 + d)
    assert _hier(e, 1 << 40) == pigan.EINVAL
    e = pigan.hier_desc(wl, 21, 0, 0, 0)
    assert _hier(e, 1 << 40) == pigan.EINVAL


def _hier_trunk(desc, ws_bytes, ptr=FAKE, idx=FAKE, ws=FAKE):
    return pigan.lib().pigan_hier_trunk_step_grads(C.byref(desc), *([ptr] * 6), None, 0.0, idx, idx, idx, ptr, ptr,
                                                   ptr, ptr, ptr, ptr, ws, ws_bytes, None)


def test_hier_trunk_step_validation():
    wl = configs.HT5
    d = pigan.hier_trunk_desc(wl, 21, 16, 16, 16)
    need = int(pigan.lib().pigan_hier_trunk_workspace_bytes(C.byref(d)))
    # the trunk sees both sensor sets in one network: a different plan from the pair's
    pair = int(pigan.lib().pigan_hier_workspace_bytes(C.byref(pigan.hier_desc(wl, 21, 16, 16, 16))))
    assert need > 0 and pair > 0 and need != pair
    assert _hier_trunk(d, need, ptr=None) == pigan.EINVAL
    assert _hier_trunk(d, need, idx=None) == pigan.EINVAL
    assert _hier_trunk(d, need - 1) == pigan.EWORKSPACE
    assert _hier_trunk(d, need, ws=C.c_void_p(4096 + 32)) == pigan.EINVAL
    for field, value in (("mY", -1), ("B_r", 0), ("lambda_pde", -1.0), ("loss_scale", 0.0)):
        e = pigan.hier_trunk_desc(wl, 21, 16, 16, 16)
        setattr(e, field, value)
        assert _hier_trunk(e, 1 << 40) == pigan.EINVAL, field
        assert pigan.lib().pigan_hier_trunk_workspace_bytes(C.byref(e)) == 0
    e = pigan.hier_trunk_desc(wl, 21, 16, 16, 16)
    e.trunk.n_groups = 2                                   # one generator for the whole domain
    assert _hier_trunk(e, 1 << 40) == pigan.EINVAL
    e = pigan.hier_trunk_desc(wl, 21, 16, 16, 16)
    e.trunk.in_dim = wl.in_dim + 1
    assert _hier_trunk(e, 1 << 40) == pigan.EINVAL
    assert pigan.lib().pigan_hier_trunk_step_grads(None, *([None] * 7), 0.0, *([None] * 10), 0, None) == pigan.EINVAL


def test_trunk_gradient_penalty_validation():
    wl = configs.T5
    d = pigan.trunk_desc(wl, lambda_gp=10.0)
    need = int(pigan.lib().pigan_trunk_workspace_bytes(C.byref(d)))
    plain = int(pigan.lib().pigan_trunk_workspace_bytes(C.byref(pigan.trunk_desc(wl))))
    assert need > plain > 0                                # the penalty's buffers
    args = (C.byref(d), *([FAKE] * 7), 0.0, FAKE, FAKE)
    # the plain entry refuses a penalty, the penalty entry needs the mixing weights
    assert pigan.lib().pigan_trunk_step_grads(*args, FAKE, FAKE, FAKE, FAKE, FAKE, need, None) == pigan.ENOTSUP
    assert pigan.lib().pigan_trunk_step_grads_gp(*args, None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, need,
                                                 None) == pigan.EINVAL
    e = pigan.trunk_desc(wl, lambda_gp=-1.0)
    assert pigan.lib().pigan_trunk_step_grads_gp(C.byref(e), *([FAKE] * 7), 0.0, FAKE, FAKE, FAKE, FAKE, FAKE,
                                                 FAKE, FAKE, FAKE, FAKE, need, None) == pigan.EINVAL
    assert pigan.lib().pigan_trunk_step_grads(*args, FAKE, FAKE, FAKE, FAKE, FAKE, need, None) == pigan.ENOTSUP
    assert b"pigan_trunk_step_grads_gp" in pigan.lib().pigan_last_error()


def test_hier_gradient_penalty_validation():
    """Both hierarchical _gp entry points: the penalty's buffers are in the
    workspace, the plain entries refuse a penalty and name the _gp entry, the
    _gp entries need the mixing weights and a finite lambda_gp >= 0."""
    L = pigan.lib()
    for wl, mk, ws_fn, plain_fn, gp_fn, n_gen in (
            (configs.H2, pigan.hier_desc, L.pigan_hier_workspace_bytes, L.pigan_hier_step_grads,
             L.pigan_hier_step_grads_gp, 2),
            (configs.HT5, pigan.hier_trunk_desc, L.pigan_hier_trunk_workspace_bytes, L.pigan_hier_trunk_step_grads,
             L.pigan_hier_trunk_step_grads_gp, 1)):
        d = mk(wl, 21, 16, 16, 16, lambda_gp=10.0)
        need = int(ws_fn(C.byref(d)))
        plain = int(ws_fn(C.byref(mk(wl, 21, 16, 16, 16))))
        assert need > plain > 0, wl.name
        head = (C.byref(d), *([FAKE] * (n_gen + 5)), None, 0.0, FAKE, FAKE, FAKE, FAKE, FAKE)
        outs = (FAKE,) * (n_gen + 2)
        assert plain_fn(*head, *outs, FAKE, FAKE, need, None) == pigan.ENOTSUP
        assert gp_fn.__name__.encode() in L.pigan_last_error()
        assert gp_fn(*head, None, *outs, FAKE, FAKE, FAKE, need, None) == pigan.EINVAL      # no gp_eps
        assert gp_fn(*head, FAKE, *outs, FAKE, FAKE, FAKE, need - 1, None) == pigan.EWORKSPACE
        for bad in (-1.0, float("inf")):
            e = mk(wl, 21, 16, 16, 16, lambda_gp=bad)
            assert int(ws_fn(C.byref(e))) == 0
            assert gp_fn(C.byref(e), *head[1:], FAKE, *outs, FAKE, FAKE, FAKE, 1 << 40, None) == pigan.EINVAL


def test_critic_only_step_needs_no_generator_gradients():
    """critic_only = 1: the generators' gradient outputs may be NULL; the
    full step still requires them."""
    L = pigan.lib()
    d = pigan.step_desc(configs.C1)
    need = pigan.workspace_bytes(d)

    def call(desc, gY):
        return L.pigan_train_step_grads(C.byref(desc), *([FAKE] * 7), None, 0.0, FAKE, None, gY, gY, FAKE, FAKE,
                                        FAKE, FAKE, need - 1, None)
    assert call(d, None) == pigan.EINVAL
    d.critic_only = 1
    assert call(d, None) == pigan.EWORKSPACE       # past the pointer checks; stops at the workspace size
