"""Helpers of the GPU parity tests: run libprm and the oracle on the same seeded
inputs and measure the differences.  Inputs come from ``synth`` only; expected
values come from ``oracle`` only."""
from __future__ import annotations

import math

import numpy as np

import synth
from oracle import prm_oracle as po

TOL_ROWWISE = 1e-5   # relative Frobenius error of D per matrix, fp32 row-wise path
TOL_NS5 = 2e-2       # relative Frobenius error of D per matrix, bf16 NS5 path
TOL_M = 1e-6         # relative Frobenius error of the fp32 momentum


def f32(x: float) -> float:
    return float(np.float32(x))


def oracle_config(cfg) -> po.PRMConfig:
    """Oracle configuration holding the same (fp32) numbers the library reads."""
    return po.PRMConfig(K=cfg.K, beta=f32(cfg.beta), lr=f32(cfg.lr), wd=f32(cfg.wd),
                        gamma=f32(cfg.gamma), eps_rownorm=f32(cfg.eps_rownorm),
                        eps_ns=f32(cfg.eps_ns), nesterov=bool(cfg.nesterov),
                        ema_dampening=bool(cfg.ema_dampening), scale_mode=cfg.scale_mode,
                        never_refresh=bool(cfg.never_refresh),
                        gamma_on_refresh=bool(cfg.gamma_on_refresh),
                        coeffs=(f32(cfg.ns_a), f32(cfg.ns_b), f32(cfg.ns_c)))


def rel(a, b) -> float:
    nb = np.linalg.norm(b)
    na = np.linalg.norm(a - b)
    if nb == 0:
        return 0.0 if na == 0 else math.inf
    return float(na / nb)


def torch_dtype(code):
    import torch
    return torch.bfloat16 if code == 1 else torch.float32


def dtype_name(code):
    return "bf16" if code == 1 else "f32"


def to_device(arr, code, device="cuda"):
    import torch
    return torch.tensor(arr, dtype=torch.float32, device=device).to(torch_dtype(code)).contiguous()


def to_host(t):
    import torch
    return t.detach().to(torch.float64).cpu().numpy()


def host_inputs(shapes, cfg, workload_id=90, steps=(0,)):
    """Seeded (W0, M0, {t: G_t}) per matrix with the configured storage types."""
    out = []
    for i, (m, n) in enumerate(shapes):
        out.append(synth.host_matrix(workload_id, i, m, n, min(m, n),
                                     param_dtype=dtype_name(cfg.param_dtype),
                                     grad_dtype=dtype_name(cfg.grad_dtype), steps=steps))
    return out


def bf16_ulp_diff(gpu, ref_exact):
    """Elementwise distance, in bf16 ulps of the reference, between GPU bf16
    values and the reference rounded to bf16."""
    r = synth.round_to_bf16(ref_exact)
    return np.abs(gpu - r) / synth.bf16_ulp(r)


def bf16_write_bound(W_gpu, W_or, D_gpu, D_or, lr) -> float:
    """Largest ratio |W_gpu - W_or| / (ulp/2 + eta |D_gpu - D_or| + fp32 slack)
    over the elements; <= 1 means the bf16 parameter write is exact up to its
    final rounding."""
    eta = f32(lr)
    ulp = synth.bf16_ulp(W_gpu)
    bound = 0.5 * ulp + eta * np.abs(D_gpu - D_or) * 1.001 + 2.0 ** -22 * (np.abs(W_or) + eta * np.abs(D_or)) + 1e-38
    return float(np.max(np.abs(W_gpu - W_or) / bound))


def ns_chunks(shapes, budget=48 << 30, tile=256, plain=False):
    """Which NS5 workspace chunk each matrix lands in, as the library's planner
    packs them (include/prm.h, prm_init): matrices sorted by padded oriented
    shape (r desc, then c desc, ties in list order) are packed in order into
    chunks of at most `budget` bytes, each matrix taking 4 rp cp bytes for its
    two iterates and 2 rp^2 + 4 rp bytes for each of its split symmetric
    matrices: four on the factored path (oriented c >= 2r), two otherwise
    (regions aligned to 256 bytes).  Returns (chunk index per matrix, largest
    chunk's bytes); tests check the latter against prm_plan_workspace_bytes."""
    def a256(x):
        return (x + 255) // 256 * 256
    rp = [-(-min(m, n) // tile) * tile for m, n in shapes]
    cp = [-(-max(m, n) // tile) * tile for m, n in shapes]
    order = sorted(range(len(shapes)), key=lambda i: (-rp[i], -cp[i], i))
    chunk = [0] * len(shapes)
    k, cur, biggest = -1, 0, 0
    for i in order:
        m, n = shapes[i]
        splits = 4 if (not plain and max(m, n) >= 2 * min(m, n)) else 2
        need = 2 * a256(rp[i] * cp[i] * 2) + splits * (a256(rp[i] * rp[i] * 2) + a256(rp[i] * 4))
        if k < 0 or cur + need > budget:
            k, cur = k + 1, 0
        chunk[i] = k
        cur += need
        biggest = max(biggest, cur)
    return chunk, biggest


def row_errors(A, B):
    """Relative error of every row of A against the same row of B."""
    num = np.linalg.norm(A - B, axis=1)
    den = np.maximum(np.linalg.norm(B, axis=1), 1e-300)
    return num / den
