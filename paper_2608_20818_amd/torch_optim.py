"""A ``torch.optim.Optimizer`` over libprm, for training loops.

Two-dimensional parameters take the Periodic Row-wise Muon step (Alg. 1: one
libprm context over all of them), every other parameter the fused AdamW step
of the non-matrix group (App. "Optimizer and Training Hyperparameters").  This
module only marshals tensors: both updates run in libprm's kernels.  The
optimizer state (fp32 momenta, AdamW moments) lives in ``self.state`` and the
step counter in the first parameter group, so ``state_dict`` /
``load_state_dict`` save and resume a run.
"""
from __future__ import annotations

import torch

from . import BF16, F32, AuxAdamW, Optimizer, adamw_config_default, config_default

_CODE = {torch.float32: F32, torch.bfloat16: BF16}


def _dtype_code(params, what):
    dts = {p.dtype for p in params}
    if len(dts) > 1:
        raise ValueError(f"{what}: one storage type for all of them (got {sorted(str(d) for d in dts)})")
    d = next(iter(dts))
    if d not in _CODE:
        raise ValueError(f"{what}: float32 or bfloat16 storage (got {d})")
    return _CODE[d]


class PRMOptimizer(torch.optim.Optimizer):
    """PRM for the 2-D parameters, AdamW for the rest.

    ``lr`` / ``weight_decay`` / ``K`` / ``beta`` / ``gamma`` and any further
    ``prm_config`` field (``nesterov``, ``ns_plain``, ...) configure the PRM
    step; ``aux_lr``, ``aux_betas``, ``aux_eps`` and ``aux_weight_decay`` the
    AdamW step.  Parameters are contiguous device tensors, float32 or
    bfloat16, one type per group of the two; their gradients have the same
    types.  Every parameter needs a gradient at every step (the library
    steps each group as a whole).  All parameter groups share one ``lr`` and one
    ``aux_lr`` (each library call takes one learning rate); changing them in
    ``param_groups[0]`` between steps is honoured, as a scheduler does.
    """

    def __init__(self, params, lr: float = 5e-3, K: int = 3, beta: float = 0.95, weight_decay: float = 0.01,
                 gamma: float = 0.15, aux_lr: float = 1e-4, aux_betas=(0.9, 0.95), aux_eps: float = 1e-8,
                 aux_weight_decay: float = 0.01, **prm_fields):
        super().__init__(params, dict(lr=lr, aux_lr=aux_lr))
        if len({(g["lr"], g["aux_lr"]) for g in self.param_groups}) != 1:
            raise ValueError("all parameter groups need the same lr and aux_lr")
        ps = [p for g in self.param_groups for p in g["params"]]
        self._mats = [p for p in ps if p.ndim == 2]
        self._aux = [p for p in ps if p.ndim != 2]
        for p in ps:
            if not p.is_cuda or not p.is_contiguous():
                raise ValueError("parameters must be contiguous device tensors")
        self._prm_fields = dict(K=K, beta=beta, wd=weight_decay, gamma=gamma, **prm_fields)
        self._aux_fields = dict(beta1=aux_betas[0], beta2=aux_betas[1], eps=aux_eps, wd=aux_weight_decay)
        self._wcode = _dtype_code(self._mats, "2-D parameters") if self._mats else F32
        self._acode = _dtype_code(self._aux, "other parameters") if self._aux else F32
        self._prm = None
        self._adamw = None
        self.param_groups[0].setdefault("prm_step", 0)

    def _state(self, p, names):
        st = self.state[p]
        for n in names:
            if n not in st:
                st[n] = torch.zeros(p.shape, dtype=torch.float32, device=p.device)
        return [st[n] for n in names]

    @torch.no_grad()
    def step(self, closure=None):
        loss = None
        if closure is not None:
            with torch.enable_grad():
                loss = closure()
        g0 = self.param_groups[0]
        t = int(g0["prm_step"])
        if self._mats:
            grads = [p.grad for p in self._mats]
            if any(g is None for g in grads):
                raise ValueError("every 2-D parameter needs a gradient at every step")
            gcode = _dtype_code(grads, "gradients of the 2-D parameters")
            if self._prm is None:
                cfg = config_default(lr=float(g0["lr"]), param_dtype=self._wcode, grad_dtype=gcode,
                                     **self._prm_fields)
                self._prm = Optimizer([tuple(p.shape) for p in self._mats], cfg)
            M = [self._state(p, ("momentum",))[0] for p in self._mats]
            self._prm.step(self._mats, grads, M, t, lr=float(g0["lr"]))
        if self._aux:
            agrads = [p.grad for p in self._aux]
            if any(g is None for g in agrads):
                raise ValueError("every other parameter needs a gradient at every step (one fused update)")
            if self._adamw is None:
                gcode = _dtype_code(agrads, "gradients of the other parameters")
                cfg = adamw_config_default(lr=float(g0["aux_lr"]), param_dtype=self._acode, grad_dtype=gcode,
                                           **self._aux_fields)
                self._adamw = AuxAdamW([p.numel() for p in self._aux], cfg)
            mv = [self._state(p, ("exp_avg", "exp_avg_sq")) for p in self._aux]
            # AdamW's bias corrections count this optimizer's steps from 1
            self._adamw.step(self._aux, agrads, [m for m, _ in mv], [v for _, v in mv], t + 1,
                             lr=float(g0["aux_lr"]))
        g0["prm_step"] = t + 1
        return loss
