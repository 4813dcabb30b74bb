"""Seeded synthetic inputs for the Periodic Row-wise Muon optimizer step.

This module is shared by the tests, the benchmark and the oracle-side checks,
so it holds NONE of the method's arithmetic: no momentum rule, no RowNorm, no
Newton-Schulz, no parameter write.  It only draws weights, gradients and
momenta with the shapes and value distributions of the workloads:

* weights   W ~ N(0, 0.02)
* gradients G = U diag(s) V^T + 0.01 N(0, 1), U (m x k) and V (n x k) Haar
  (QR of a Gaussian with diag(R) > 0), s_i = 1/i; k = min(m, n) for the tiny
  workload and k = min(m, n, 128) for the DiT-shaped weight sets
* momentum  the state after three heavy-ball steps from zero with beta = 0.95
  has the same U, V and the distribution
  U diag((1 + beta + beta^2) s) V^T + 0.01 sqrt(1 + beta^2 + beta^4) N(0, 1);
  it is drawn directly from that distribution (one seeded draw).

The auxiliary (non-matrix) group that AdamW updates -- biases, norm scales and
shifts, embedders -- is a list of flat tensors: one bias of width n per matrix,
four h-vectors per block (two norm layers), and four equal embedder-sized
tensors that bring the group to the share the paper's model-configuration
table gives for the matching scale (100% minus the Muon-routed share).  Its
values: p ~ N(0, 0.02), g ~ 0.01 N(0, 1), first moment ~ 0.003 N(0, 1), second
moment ~ 1.4e-5 chi^2_3 / 3 (the scale of a few averaged squared gradients).

Seeds: numpy.random.SeedSequence([20818, workload, matrix, tag]).  Host draws
use PCG64.  Device draws (large workloads) take the thin Haar factors from the
host draw and the large Gaussian terms from a torch generator on the GPU seeded
from the same sequence; any matrix the oracle needs is copied back from the
device so that both sides read identical bytes.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

SEED_ROOT = 20818
TAGS = {"U": 1, "V": 2, "W": 3, "M": 4, "G": 100,  # gradient of step t uses 100 + t
        "AP": 300, "AM": 301, "AV": 302, "AG": 400}   # aux group; its gradient of step t: 400 + t


@dataclass(frozen=True)
class Workload:
    name: str
    shapes: tuple            # ((m, n), ...)
    param_dtype: str         # "f32" | "bf16"
    grad_dtype: str          # "f32" | "bf16"
    K: int
    lr: float
    wd: float
    gamma: float = 0.15
    beta: float = 0.95
    rank_cap: int | None = None   # None: k = min(m, n)
    blocks: int = 0
    hidden: int = 0


def dit_shapes(blocks: int, h: int):
    """Per block: qkv h x 3h, attention out h x h, MLP up h x 4h, MLP down 4h x h,
    adaLN modulation h x 6h."""
    one = ((h, 3 * h), (h, h), (h, 4 * h), (4 * h, h), (h, 6 * h))
    return tuple(s for _ in range(blocks) for s in one)


KINDS = ("qkv", "out", "mlp_up", "mlp_down", "adaln")

WORKLOADS = (
    Workload("tiny", ((256, 256), (256, 256), (256, 768), (256, 1024), (1024, 256), (128, 512)),
             "f32", "f32", K=4, lr=0.02, wd=0.1),
    Workload("dit-1.3b", dit_shapes(24, 2048), "bf16", "bf16", K=5, lr=5e-3, wd=0.01,
             rank_cap=128, blocks=24, hidden=2048),
    Workload("dit-4b", dit_shapes(32, 3072), "bf16", "bf16", K=5, lr=3e-3, wd=0.01,
             rank_cap=128, blocks=32, hidden=3072),
    Workload("dit-9b", dit_shapes(40, 4096), "bf16", "bf16", K=5, lr=2.4e-3, wd=0.01,
             rank_cap=128, blocks=40, hidden=4096),
    Workload("dit-15b", dit_shapes(48, 5120), "bf16", "bf16", K=5, lr=2e-3, wd=0.01,
             rank_cap=128, blocks=48, hidden=5120),
)


# Muon-routed share of the trainable parameters (model-configuration table).
MUON_ROUTED = {"dit-1.3b": 0.9869, "dit-4b": 0.9920, "dit-9b": 0.9948, "dit-15b": 0.9960}


def aux_numels(workload: int) -> tuple:
    """Element counts of the auxiliary AdamW group of a workload."""
    wl = WORKLOADS[workload]
    biases = [n for (_, n) in wl.shapes]
    if wl.name == "tiny":
        return tuple(biases + [256, 256, 7, 1])
    f = MUON_ROUTED[wl.name]
    norms = [wl.hidden] * (4 * wl.blocks)
    total = int(round(sum(m * n for m, n in wl.shapes) * (1.0 - f) / f))
    rest = total - sum(biases) - sum(norms)
    q = rest // 4
    return tuple([q, q, q, rest - 3 * q] + biases + norms)


def host_aux(workload: int, idx: int, numel: int, *, param_dtype: str, grad_dtype: str,
             steps=(0,)) -> dict:
    """Seeded draws of one aux tensor: float32 arrays holding exactly the values
    of the storage dtypes (p in param_dtype, g in grad_dtype, m and v fp32)."""
    def rng(tag, t=0):
        return host_rng(workload, idx, tag, t)

    out = {"p": to_dtype_values(0.02 * rng("AP").standard_normal(numel, dtype=np.float32),
                                param_dtype).astype(np.float32),
           "m": 0.003 * rng("AM").standard_normal(numel, dtype=np.float32),
           "v": (1.4e-5 / 3.0) * 2.0 * rng("AV").standard_gamma(1.5, numel, dtype=np.float32)}
    for t in steps:
        out[f"g{t}"] = to_dtype_values(0.01 * rng("AG", t).standard_normal(numel, dtype=np.float32),
                                       grad_dtype).astype(np.float32)
    return out


def rank_of(wl: Workload, m: int, n: int) -> int:
    k = min(m, n)
    return k if wl.rank_cap is None else min(k, wl.rank_cap)


def seed_sequence(workload: int, mat: int, tag: str, step: int = 0) -> np.random.SeedSequence:
    code = TAGS[tag] + (step if tag in ("G", "AG") else 0)
    return np.random.SeedSequence([SEED_ROOT, int(workload), int(mat), int(code)])


def host_rng(workload: int, mat: int, tag: str, step: int = 0) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed_sequence(workload, mat, tag, step)))


def torch_seed(workload: int, mat: int, tag: str, step: int = 0) -> int:
    return int(seed_sequence(workload, mat, tag, step).generate_state(2, np.uint64)[0] >> 1)


# ---------------------------------------------------------------- bf16 helpers
def round_to_bf16(x) -> np.ndarray:
    """Round float values to the nearest bfloat16 (ties to even); returned as float64."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    nan = np.isnan(f)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    u = (u << 16).astype(np.uint32)
    out = u.view(np.float32).astype(np.float64)
    out[nan] = np.nan
    return out


def bf16_ulp(x) -> np.ndarray:
    """Spacing of bfloat16 numbers at |x| (normal range)."""
    ax = np.abs(np.asarray(x, dtype=np.float64))
    e = np.floor(np.log2(np.maximum(ax, 2.0 ** -126)))
    return 2.0 ** (e - 7)


def to_dtype_values(x, dtype: str) -> np.ndarray:
    """float64 array holding exactly the values the given storage dtype keeps."""
    if dtype == "f32":
        return np.asarray(x, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        return round_to_bf16(x)
    raise ValueError(dtype)


# ---------------------------------------------------------------- host draws
def haar_columns(rng: np.random.Generator, n: int, k: int) -> np.ndarray:
    """n x k matrix with Haar-distributed orthonormal columns (QR, diag(R) > 0)."""
    Z = rng.standard_normal((n, k))
    Q, R = np.linalg.qr(Z)
    d = np.sign(np.diag(R))
    d[d == 0] = 1.0
    return Q * d


def spectrum(k: int) -> np.ndarray:
    return 1.0 / np.arange(1, k + 1, dtype=np.float64)


def host_factors(workload: int, mat: int, m: int, n: int, k: int):
    U = haar_columns(host_rng(workload, mat, "U"), m, k)
    V = haar_columns(host_rng(workload, mat, "V"), n, k)
    return U, V


def host_matrix(workload: int, mat: int, m: int, n: int, k: int, *, param_dtype: str,
                grad_dtype: str, beta: float = 0.95, steps=(0,), noise: float = 0.01):
    """(W0, M0, {t: G_t}) for one matrix as float64 arrays holding exact storage values.

    W0 in ``param_dtype``; M0 in fp32; gradients in ``grad_dtype``.  ``noise``
    is the standard deviation of the Gaussian term of each gradient (0.01 in
    every workload; smaller values give signal-dominated momenta).
    """
    U, V = host_factors(workload, mat, m, n, k)
    s = spectrum(k)
    W0 = 0.02 * host_rng(workload, mat, "W").standard_normal((m, n))
    sig_m = 1.0 + beta + beta * beta
    noise_m = noise * math.sqrt(1.0 + beta ** 2 + beta ** 4)
    M0 = (U * (sig_m * s)) @ V.T + noise_m * host_rng(workload, mat, "M").standard_normal((m, n))
    grads = {}
    for t in steps:
        grads[t] = to_dtype_values(
            (U * s) @ V.T + noise * host_rng(workload, mat, "G", t).standard_normal((m, n)),
            grad_dtype)
    return to_dtype_values(W0, param_dtype), to_dtype_values(M0, "f32"), grads


def host_workload(workload: int, steps=(0,), mats=None):
    """Host draws for every (or the selected) matrix of a workload."""
    wl = WORKLOADS[workload]
    idx = range(len(wl.shapes)) if mats is None else mats
    out = []
    for i in idx:
        m, n = wl.shapes[i]
        out.append(host_matrix(workload, i, m, n, rank_of(wl, m, n), param_dtype=wl.param_dtype,
                               grad_dtype=wl.grad_dtype, beta=wl.beta, steps=steps))
    return out


# ---------------------------------------------------------------- device draws
def device_matrix(workload: int, mat: int, m: int, n: int, k: int, *, param_dtype: str,
                  grad_dtype: str, device, beta: float = 0.95, step: int = 0,
                  want=("W", "M", "G")):
    """Same recipe as ``host_matrix`` drawn on the GPU with torch (for the large
    weight sets).  Returns a dict of device tensors in their storage dtypes."""
    import torch

    dt = {"f32": torch.float32, "bf16": torch.bfloat16}

    def gen(tag, t=0):
        g = torch.Generator(device=device)
        g.manual_seed(torch_seed(workload, mat, tag, t))
        return g

    out = {}
    if "W" in want:
        out["W"] = (0.02 * torch.randn(m, n, generator=gen("W"), device=device)).to(dt[param_dtype])
    if "M" in want or "G" in want:
        # the thin Haar factors are small (m x k, n x k): drawn on the host with
        # the same seeds as host_matrix, so both paths share U and V exactly
        Uh, Vh = host_factors(workload, mat, m, n, k)
        U = torch.tensor(Uh, dtype=torch.float32, device=device)
        V = torch.tensor(Vh, dtype=torch.float32, device=device)
        s = 1.0 / torch.arange(1, k + 1, device=device, dtype=torch.float32)
        if "M" in want:
            sig_m = 1.0 + beta + beta * beta
            noise_m = 0.01 * math.sqrt(1.0 + beta ** 2 + beta ** 4)
            Mx = torch.randn(m, n, generator=gen("M"), device=device)
            Mx.mul_(noise_m).addmm_(U * (sig_m * s), V.t().contiguous())
            out["M"] = Mx
        if "G" in want:
            Gx = torch.randn(m, n, generator=gen("G", step), device=device)
            Gx.mul_(0.01).addmm_(U * s, V.t().contiguous())
            out["G"] = Gx.to(dt[grad_dtype])
    return out
