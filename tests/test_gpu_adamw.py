"""GPU parity of the fused aux-AdamW step (prm_adamw_*) against the fp64 oracle.

Inputs come from ``synth.host_aux`` and expected values from
``oracle.adamw_step`` only.  Bars: the fp32 moments within 1e-6 (relative
Frobenius, per tensor); the parameter, element by element, equal to the
oracle's value up to its storage rounding (half an ulp of its type plus fp32
slack); and, where the update is many ulps of p (large lr), the fp32 update
within 1e-5 relative Frobenius.
"""
import ctypes
import os
import sys

import numpy as np
import pytest
import torch

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import synth  # noqa: E402
import oracle  # noqa: E402
import paper_2608_20818_amd as prm  # noqa: E402
from prm_case import dtype_name, f32, rel, to_device, to_host  # noqa: E402

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

TOL_STATE = 1e-6
TOL_UPDATE = 1e-5
# ragged sizes around the 2048-element chunk and the 4-element piece, an empty
# tensor, and single elements
RAGGED = (1, 3, 7, 2047, 2048, 2049, 4093, 5000, 0, 12, 6143)


def oracle_cfg(c):
    return oracle.AdamWConfig(lr=f32(c.lr), beta1=f32(c.beta1), beta2=f32(c.beta2), eps=f32(c.eps),
                              wd=f32(c.wd))


def f32_ulp(x):
    ax = np.abs(np.asarray(x, dtype=np.float64))
    return 2.0 ** (np.floor(np.log2(np.maximum(ax, 2.0 ** -126))) - 23)


def check_tensor(i, pd, P, p0, M, V, pe, me, ve, scale, check_update=False):
    assert rel(M, me) <= TOL_STATE, (i, rel(M, me))
    assert rel(V, ve) <= TOL_STATE, (i, rel(V, ve))
    # the parameter equals the oracle's up to its storage rounding: half an ulp
    # of the stored type, the fp32 rounding of the decayed p, and fp32 errors of
    # the update term relative to its operands (``scale``: the update with |m|
    # and |g| in place of m and g, where their sum may cancel)
    ulp = synth.bf16_ulp(pe) if pd == prm.BF16 else f32_ulp(pe)
    bound = 0.5 * ulp + 2.0 ** -23 * np.abs(pe) + 16 * 2.0 ** -23 * scale + 1e-30
    ratio = np.abs(P - pe) / bound
    assert ratio.size == 0 or ratio.max() <= 1.0, (i, float(ratio.max()))
    if check_update:
        # an update many fp32 ulps large: its relative error is the arithmetic's
        assert rel(P - p0, pe - p0) <= TOL_UPDATE, (i, rel(P - p0, pe - p0))


def update_scale(ocfg, eta, t, g, m0, v_new):
    eta = ocfg.lr if eta is None else eta
    num = (ocfg.beta1 * np.abs(m0) + (1 - ocfg.beta1) * np.abs(g)) / (1 - ocfg.beta1 ** t)
    return eta * num / (np.sqrt(v_new / (1 - ocfg.beta2 ** t)) + ocfg.eps)


def run_case(numels, pd, gd, steps, *, fresh=False, lr=-1.0, wid=95, check_update=False):
    cfg = prm.adamw_config_default(param_dtype=pd, grad_dtype=gd)
    ocfg = oracle_cfg(cfg)
    eta = None if lr < 0 else f32(lr)
    host = [synth.host_aux(wid, i, n, param_dtype=dtype_name(pd), grad_dtype=dtype_name(gd),
                           steps=range(len(steps))) for i, n in enumerate(numels)]
    dev = torch.device("cuda")
    P = [to_device(h["p"], pd) for h in host]
    M = [torch.zeros(n, device=dev) if fresh else torch.tensor(h["m"], device=dev)
         for h, n in zip(host, numels)]
    V = [torch.zeros(n, device=dev) if fresh else torch.tensor(h["v"], device=dev)
         for h, n in zip(host, numels)]
    opt = prm.AuxAdamW(numels, cfg, stream=torch.cuda.current_stream())
    try:
        for k, t in enumerate(steps):
            print(f"[adamw] {len(numels)} tensors pd={pd} gd={gd} t={t}", flush=True)
            G = [to_device(h[f"g{k}"], gd) for h in host]  # new tensors: the pointer table is re-sent
            p0 = [to_host(x) for x in P]
            m0 = [to_host(x) for x in M]
            v0 = [to_host(x) for x in V]
            opt.step([x if x.numel() else None for x in P], [x if x.numel() else None for x in G],
                     [x if x.numel() else None for x in M], [x if x.numel() else None for x in V], t, lr)
            torch.cuda.synchronize()
            for i in range(len(numels)):
                pe, me, ve = oracle.adamw_step(p0[i], host[i][f"g{k}"], m0[i], v0[i], t, ocfg, eta)
                sc = update_scale(ocfg, eta, t, host[i][f"g{k}"], m0[i], ve)
                check_tensor(i, pd, to_host(P[i]), p0[i], to_host(M[i]), to_host(V[i]), pe, me, ve, sc,
                             check_update)
    finally:
        opt.close()


@pytest.mark.parametrize("pd,gd", [(prm.F32, prm.F32), (prm.BF16, prm.BF16), (prm.F32, prm.BF16),
                                   (prm.BF16, prm.F32)])
def test_ragged_tensors_resumed_state(pd, gd):
    run_case(RAGGED, pd, gd, steps=(4, 5, 6))


@pytest.mark.parametrize("pd", [prm.F32, prm.BF16])
def test_fresh_state_first_updates(pd):
    # t = 1 from zero moments: m^ = g and v^ = g^2 exactly (bias correction)
    run_case(RAGGED, pd, pd, steps=(1, 2), fresh=True)


def test_large_t_and_lr_override():
    # lr 0.05: the update is ~1e7 fp32 ulps of p, so the 1e-5 relative bar on
    # the update itself applies
    run_case((2048, 33, 4096, 5), prm.F32, prm.BF16, steps=(1000, 1001), lr=0.05, check_update=True)


def test_tiny_workload_group():
    run_case(synth.aux_numels(0), prm.F32, prm.F32, steps=(4,), wid=0)


def test_empty_group_and_argument_errors():
    L = prm.load()
    cfg = prm.adamw_config_default(param_dtype=prm.F32, grad_dtype=prm.F32)
    with prm.AuxAdamW([], cfg) as opt:
        opt.step([], [], [], [], 1)  # nothing to do
    x = torch.zeros(64, device="cuda")
    with prm.AuxAdamW([64], cfg) as opt:
        nul = (ctypes.c_void_p * 1)(x.data_ptr())
        assert L.prm_adamw_step(opt._ctx, nul, nul, nul, nul, 0, -1.0) == prm.PRM_EINVAL
        bad = (ctypes.c_void_p * 1)(x.data_ptr() + 4)
        assert L.prm_adamw_step(opt._ctx, bad, nul, nul, nul, 1, -1.0) == prm.PRM_EALIGN
        none = (ctypes.c_void_p * 1)(0)
        assert L.prm_adamw_step(opt._ctx, none, nul, nul, nul, 1, -1.0) == prm.PRM_EINVAL
    torch.cuda.synchronize()
    assert torch.count_nonzero(x).item() == 0  # rejected calls launched nothing


def test_dit4b_group_full_size():
    # the aux group of the DiT-4B-shaped set (43.8 M elements, 292 tensors) at
    # the bench's dtypes, one resumed update, every element against the oracle
    numels = synth.aux_numels(2)
    run_case(numels, prm.BF16, prm.BF16, steps=(4,), wid=2)


def test_bound_step_matches_step():
    numels = (4096, 5, 2049)
    outs = []
    for bound in (False, True):
        cfg = prm.adamw_config_default(param_dtype=prm.BF16, grad_dtype=prm.BF16)
        host = [synth.host_aux(96, i, n, param_dtype="bf16", grad_dtype="bf16") for i, n in enumerate(numels)]
        P = [to_device(h["p"], prm.BF16) for h in host]
        G = [to_device(h["g0"], prm.BF16) for h in host]
        M = [torch.tensor(h["m"], device="cuda") for h in host]
        V = [torch.tensor(h["v"], device="cuda") for h in host]
        with prm.AuxAdamW(numels, cfg) as opt:
            if bound:
                opt.bind(P, G, M, V)
            for t in (4, 5, 6):
                if bound:
                    opt.step_bound(t)
                else:
                    opt.step(P, G, M, V, t)
            torch.cuda.synchronize()
        outs.append([to_host(x) for x in P + M + V])
    for a, b in zip(*outs):
        assert np.array_equal(a, b)
