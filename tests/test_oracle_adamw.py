"""Pins of the oracle's auxiliary AdamW update (the non-matrix parameter group).

Each check reaches the expected value by another route: PyTorch's own AdamW
(``torch.optim.AdamW`` in float64 on the CPU, a library routine implementing
the published method), closed forms for constant and zero gradients, and the
paper's printed hyperparameters.  The mutation test plants plausible mistakes
in the oracle and checks that a pin catches each one.
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import prm_oracle as po

GOLD = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "paper_constants.json")))


def rel(a, b):
    return np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300)


def torch_adamw(p0, grads, m0, v0, t0, cfg):
    """Run torch.optim.AdamW (float64, CPU, single-tensor path) from state (m0, v0)
    at update count t0 over the gradient list; returns (p, m, v)."""
    p = torch.nn.Parameter(torch.tensor(p0, dtype=torch.float64))
    opt = torch.optim.AdamW([p], lr=cfg.lr, betas=(cfg.beta1, cfg.beta2), eps=cfg.eps,
                            weight_decay=cfg.wd, foreach=False, fused=False)
    if t0 > 0:
        opt.state[p] = {"step": torch.tensor(float(t0), dtype=torch.float64),
                        "exp_avg": torch.tensor(m0, dtype=torch.float64),
                        "exp_avg_sq": torch.tensor(v0, dtype=torch.float64)}
    for g in grads:
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
    st = opt.state[p]
    return p.detach().numpy(), st["exp_avg"].numpy(), st["exp_avg_sq"].numpy()


def run_oracle(p, grads, m, v, t0, cfg):
    for k, g in enumerate(grads):
        p, m, v = oracle.adamw_step(p, g, m, v, t0 + k + 1, cfg)
    return p, m, v


def test_defaults_match_paper_table():
    gold = GOLD["aux_adamw"]["value"]
    cfg = oracle.AdamWConfig()
    assert cfg.lr == gold["lr"]
    assert (cfg.beta1, cfg.beta2) == tuple(gold["betas"])
    assert cfg.eps == gold["eps"] == GOLD["adamw_eps"]["value"]
    assert cfg.wd == gold["weight_decay"] == GOLD["weight_decay"]["value"]


@pytest.mark.parametrize("t0", [0, 3, 40])
def test_matches_torch_adamw(t0):
    rng = np.random.default_rng(7 + t0)
    n = 257
    cfg = oracle.AdamWConfig(lr=3e-3, wd=0.1)  # large enough that decay and step both show
    p = rng.standard_normal(n) * 0.02
    m = rng.standard_normal(n) * 3e-3 if t0 else np.zeros(n)
    v = (rng.standard_normal(n) ** 2) * 1e-5 if t0 else np.zeros(n)
    grads = [rng.standard_normal(n) * 0.01 * (1 + k) for k in range(4)]
    grads[1][:5] = 0.0                     # zero gradients
    grads[2][5:9] *= 1e-9                  # gradients far below eps
    po_, mo, vo = run_oracle(p, grads, m, v, t0, cfg)
    pt, mt, vt = torch_adamw(p, grads, m, v, t0, cfg)
    assert rel(mo, mt) < 1e-14
    assert rel(vo, vt) < 1e-14
    assert rel(po_ - p, pt - p) < 1e-12
    assert np.max(np.abs(po_ - pt)) < 1e-15


def test_constant_gradient_closed_form():
    # From a zero state, a constant gradient g gives m^ = g and v^ = g^2 at every
    # t, so each update is p <- (1 - eta*lambda) p - eta * g / (|g| + eps):
    # p_T = q^T p_0 - eta * u * (1 - q^T) / (1 - q), q = 1 - eta*lambda.
    cfg = oracle.AdamWConfig(lr=1e-3, wd=0.05)
    g = np.array([0.3, -2e-4, 5.0, -1e-9, 0.0])
    p0 = np.array([0.1, -0.2, 0.3, 0.4, -0.5])
    p, m, v = p0.copy(), np.zeros(5), np.zeros(5)
    T = 7
    for t in range(1, T + 1):
        p, m, v = oracle.adamw_step(p, g, m, v, t, cfg)
    q = 1.0 - cfg.lr * cfg.wd
    u = g / (np.abs(g) + cfg.eps)
    expect = q ** T * p0 - cfg.lr * u * (1.0 - q ** T) / (1.0 - q)
    assert np.allclose(p, expect, rtol=1e-12, atol=1e-16)
    assert np.allclose(m, (1 - cfg.beta1 ** T) * g, rtol=1e-13, atol=0)
    assert np.allclose(v, (1 - cfg.beta2 ** T) * g * g, rtol=1e-13, atol=0)


def test_zero_gradient_is_pure_decay():
    cfg = oracle.AdamWConfig(lr=2e-2, wd=0.3)
    p0 = np.linspace(-1, 1, 9)
    p, m, v = p0, np.zeros(9), np.zeros(9)
    for t in range(1, 4):
        p, m, v = oracle.adamw_step(p, np.zeros(9), m, v, t, cfg)
    assert np.array_equal(m, np.zeros(9)) and np.array_equal(v, np.zeros(9))
    assert np.allclose(p, (1 - cfg.lr * cfg.wd) ** 3 * p0, rtol=1e-15, atol=0)


def test_rejects_t_below_one():
    with pytest.raises(ValueError):
        oracle.adamw_step(np.zeros(2), np.zeros(2), np.zeros(2), np.zeros(2), 0, oracle.AdamWConfig())


def test_byte_model():
    # bf16 p and g: p 2+2, g 2, m 4+4, v 4+4
    assert oracle.adamw_bytes_per_element(2, 2) == 22
    assert oracle.adamw_bytes_per_element(4, 4) == 28


def test_mutations_are_caught(monkeypatch):
    """Plant plausible mistakes in the oracle (on the CPU) and check the torch pin fails."""
    rng = np.random.default_rng(3)
    n = 64
    cfg = oracle.AdamWConfig(lr=3e-3, wd=0.1)
    p = rng.standard_normal(n) * 0.02
    m = rng.standard_normal(n) * 3e-3
    v = rng.standard_normal(n) ** 2 * 1e-5
    grads = [rng.standard_normal(n) * 0.01 for _ in range(2)]
    pt, _, _ = torch_adamw(p, grads, m, v, 2, cfg)

    def pin_holds():
        po_, _, _ = run_oracle(p, grads, m, v, 2, cfg)
        return rel(po_ - p, pt - p) < 1e-12

    assert pin_holds()
    good = po.adamw_step

    def make(mistake):
        def bad(p, g, m, v, t, cfg, lr=None):
            eta = cfg.lr
            if mistake == "l2_instead_of_decoupled":
                g = g + cfg.wd * p  # Adam with L2 regularization
            m1 = cfg.beta1 * m + (1 - cfg.beta1) * g
            v1 = cfg.beta2 * v + (1 - cfg.beta2) * g * g
            bc1, bc2 = 1 - cfg.beta1 ** t, 1 - cfg.beta2 ** t
            if mistake == "no_bias_correction":
                bc1 = bc2 = 1.0
            if mistake == "v_from_g":
                v1 = cfg.beta2 * v + (1 - cfg.beta2) * np.abs(g)
            denom = np.sqrt(v1 / bc2) + cfg.eps
            if mistake == "eps_inside_sqrt":
                denom = np.sqrt(v1 / bc2 + cfg.eps)
            step = (m1 / bc1) / denom
            if mistake == "l2_instead_of_decoupled":
                return p - eta * step, m1, v1
            if mistake == "decay_after_step":
                q = p - eta * step
                return q - eta * cfg.wd * q, m1, v1
            return p - eta * (step + cfg.wd * p), m1, v1
        return bad

    for mistake in ("no_bias_correction", "v_from_g", "eps_inside_sqrt", "l2_instead_of_decoupled",
                    "decay_after_step"):
        monkeypatch.setattr(oracle, "adamw_step", make(mistake))
        assert not pin_holds(), mistake
    monkeypatch.setattr(oracle, "adamw_step", make(None))
    assert pin_holds()
    monkeypatch.setattr(oracle, "adamw_step", good)
    assert pin_holds()
