"""GPU tests of the torch.optim adapter (``paper_2608_20818_amd.PRMOptimizer``):
a small two-layer model trained for a few steps, its 2-D weights checked
against the oracle's PRM step and its biases against the oracle's AdamW step,
plus save / resume through ``state_dict``.  Gradients come from torch's
autograd on the GPU (not from libprm) and are copied to the host for the
oracle."""
import copy
import os
import sys

import numpy as np
import pytest
import torch

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import paper_2608_20818_amd as prm  # noqa: E402
import prm_case as pc  # noqa: E402
from oracle import prm_oracle as po  # noqa: E402

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

HID, D_IN, BATCH = 320, 96, 64
HP = dict(lr=0.02, K=2, beta=0.95, weight_decay=0.1, gamma=0.15, aux_lr=1e-3, aux_betas=(0.9, 0.95),
          aux_eps=1e-8, aux_weight_decay=0.01)


def make_model(seed=20818):
    rng = np.random.default_rng(seed)
    model = torch.nn.Sequential(torch.nn.Linear(D_IN, HID), torch.nn.GELU(), torch.nn.Linear(HID, D_IN)).cuda()
    with torch.no_grad():
        for p in model.parameters():
            p.copy_(torch.tensor(rng.normal(0.0, 0.05, size=tuple(p.shape)), dtype=torch.float32))
    x = torch.tensor(rng.normal(size=(BATCH, D_IN)), dtype=torch.float32, device="cuda")
    y = torch.tensor(rng.normal(size=(BATCH, D_IN)), dtype=torch.float32, device="cuda")
    return model, x, y


def backward(model, x, y, scale=1.0, seed=0):
    """Loss gradients plus seeded Gaussian noise on the 2-D ones, at half their
    RMS: a batch of 64 gives exactly rank-deficient weight gradients, whose
    NS5 direction the bf16 path only meets within its wider envelope (the
    precision-envelope tests cover that regime); minibatch noise makes real
    gradients full-rank, as in the synthetic DiT workloads."""
    model.zero_grad(set_to_none=False)
    loss = scale * ((model(x) - y) ** 2).mean()
    loss.backward()
    rng = np.random.default_rng([94, seed])
    with torch.no_grad():
        for p in model.parameters():
            if p.ndim == 2:
                r = torch.tensor(rng.normal(size=tuple(p.shape)), dtype=torch.float32, device="cuda")
                p.grad.add_(r * (0.5 * float(p.grad.pow(2).mean().sqrt())))
    torch.cuda.synchronize()


def host(model):
    return [pc.to_host(p) for p in model.parameters()], [pc.to_host(p.grad) for p in model.parameters()]


def oracle_configs():
    cfg = prm.config_default(K=HP["K"], lr=HP["lr"], wd=HP["weight_decay"], gamma=HP["gamma"], beta=HP["beta"],
                             param_dtype=prm.F32, grad_dtype=prm.F32)
    aoc = po.AdamWConfig(lr=pc.f32(HP["aux_lr"]), beta1=pc.f32(0.9), beta2=pc.f32(0.95), eps=pc.f32(1e-8),
                         wd=pc.f32(HP["aux_weight_decay"]))
    return pc.oracle_config(cfg), aoc


def test_two_steps_against_the_oracle():
    """t = 0 (NS5 refresh) and t = 1 (row-wise step) for the weights; AdamW
    updates 1 and 2 for the biases."""
    model, x, y = make_model()
    opt = prm.PRMOptimizer(model.parameters(), **HP)
    oc, aoc = oracle_configs()
    lr = pc.f32(HP["lr"])
    params = list(model.parameters())
    Mo = [np.zeros(p.shape) for p in params]   # momenta (weights) / first moments (biases)
    Vo = [np.zeros(p.shape) for p in params]   # second moments (biases)
    for t in (0, 1):
        backward(model, x, y, scale=1.0 + t, seed=t)
        P0, G0 = host(model)
        opt.step()
        torch.cuda.synchronize()
        tol = pc.TOL_NS5 if t % HP["K"] == 0 else pc.TOL_ROWWISE
        for i, p in enumerate(params):
            got = pc.to_host(p)
            st = opt.state[p]
            if p.ndim == 2:
                Wo, Mn, Do, rho = po.step_matrix(P0[i], Mo[i], G0[i], t, oc)
                assert rho == (1 if t == 0 else 0)
                bound = lr * tol * np.linalg.norm(Do) * 1.01 + 4e-7 * np.linalg.norm(Wo)
                err = np.linalg.norm(got - Wo)
                print(f"  t={t} W{tuple(p.shape)}: |W - W_oracle| {err:.3e} (bound {bound:.3e})", flush=True)
                assert err <= bound, f"t={t} {tuple(p.shape)}"
                assert pc.rel(pc.to_host(st["momentum"]), Mn) <= pc.TOL_M
                Mo[i] = pc.to_host(st["momentum"])
            else:
                pe, me, ve = po.adamw_step(P0[i], G0[i], Mo[i], Vo[i], t + 1, aoc)
                assert pc.rel(pc.to_host(st["exp_avg"]), me) <= 1e-6
                assert pc.rel(pc.to_host(st["exp_avg_sq"]), ve) <= 1e-6
                assert np.max(np.abs(got - pe)) <= 4e-7 * np.max(np.abs(pe)) + 1e-6 * HP["aux_lr"], f"t={t} bias"
                Mo[i] = pc.to_host(st["exp_avg"])
                Vo[i] = pc.to_host(st["exp_avg_sq"])
    assert opt.param_groups[0]["prm_step"] == 2


def test_state_dict_resume_is_bitwise():
    """Two steps, save, then a third step in the original optimizer and in a
    fresh one that loaded the saved state: identical parameters."""
    model, x, y = make_model(seed=7)
    opt = prm.PRMOptimizer(model.parameters(), **HP)
    for t in range(2):
        backward(model, x, y, scale=1.0 + t, seed=t)
        opt.step()
    # a saved copy (load_state_dict keeps references to the tensors it is given)
    sd = copy.deepcopy(opt.state_dict())
    model2, _, _ = make_model(seed=7)
    with torch.no_grad():
        for p2, p in zip(model2.parameters(), model.parameters()):
            p2.copy_(p)
    opt2 = prm.PRMOptimizer(model2.parameters(), **HP)
    opt2.load_state_dict(sd)
    backward(model, x, y, scale=3.0, seed=2)
    with torch.no_grad():
        for p2, p in zip(model2.parameters(), model.parameters()):
            p2.grad = p.grad.clone()
    opt.step()   # t = 2: a refresh (K = 2)
    opt2.step()
    torch.cuda.synchronize()
    for p2, p in zip(model2.parameters(), model.parameters()):
        assert torch.equal(p2, p), tuple(p.shape)
    assert opt2.param_groups[0]["prm_step"] == 3


def test_missing_gradient_is_refused():
    model, x, y = make_model()
    opt = prm.PRMOptimizer(model.parameters(), **HP)
    with pytest.raises(ValueError):
        opt.step()  # no backward yet: no gradients
