"""Full-size parity on the DiT-shaped weight sets (configs DiT-1.3B, 4B, 9B and
15B: 120-240 matrices, 1.8-22.7 G elements, bf16 W and G, fp32 M) in the
launch configuration bench.py times.

The oracle cannot run a whole set, so it checks sampled outputs it can
compute one by one:
* refresh step (t = 0; also in precise mode at DiT-1.3B and 4B): 48 oriented rows of NS5 for every kind of matrix of the
  first and the last block (at DiT-15B: five matrices that cover every kind
  and each of its workspace chunks), from the eigendecomposition closed
  form of the oracle (pinned to the five-iteration map on small inputs):
  relative Frobenius error <= 2e-2 over the sampled rows, and the same bound
  on the worst single sampled row (one wrong row among thousands would hardly
  move the matrix error);
* row-wise step (t = 1): 64 oriented rows (stored columns for the tall MLP
  down projection) of every sampled matrix, error <= 1e-5, per row as well;
* momentum rows <= 1e-6; bf16 W rows within half an ulp plus eta |D - D_oracle|.
Up to DiT-9B the non-debug prm_step (what bench.py times) must also produce
bitwise the same W and M as prm_step_debug on the same inputs, and every
matrix of the set is checked, not only the sampled ones:
* row-wise step: every oriented row of D against RowNorm of the same row of
  the new momentum (fp64 on the GPU: a norm and a division), <= 1e-5 per row;
* refresh step: D against the five-iteration map evaluated in fp64 on the GPU
  (torch matrix products) from the step's new momentum, <= 2e-2 per matrix and
  per row.  That fp64 evaluation is itself held to the oracle's closed form on
  the sampled matrices (rows agree to 1e-12), so a batching or indexing error
  in any matrix of any launch shows up.
At DiT-15B (W, M and G take 180 GB) there is no room for that second copy, and
only the sampled matrices get a direction output (NULL entries for the others).
"""
import os
import sys

import numpy as np
import pytest
import torch

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import paper_2608_20818_amd as prm  # noqa: E402
import prm_case as pc  # noqa: E402
import synth  # noqa: E402
from oracle import prm_oracle as po  # noqa: E402

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

SETS = (1, 2, 3, 4)          # DiT-1.3B, 4B, 9B, 15B
NO_COPY = (4,)               # too large for a second copy of W and M
# matrix index = 5 block + kind, kinds qkv, out, mlp up, mlp down, adaLN.
# Refresh samples: both end blocks x every kind; at DiT-15B (closed form about
# 15 s per matrix) qkv, out, mlp up and adaLN of block 0 and the last block's
# mlp down, which lie in its workspace chunks 1, 2, 0, 0 and 1
# (test_fullsize_sample_covers_every_chunk checks this on the CPU)
REFRESH_SAMPLE = {wi: tuple(range(5)) + tuple(range(5 * (synth.WORKLOADS[wi].blocks - 1),
                                                     5 * synth.WORKLOADS[wi].blocks)) for wi in (1, 2, 3)}
REFRESH_SAMPLE[4] = (0, 1, 2, 4, 5 * (synth.WORKLOADS[4].blocks - 1) + 3)
# the fp64 GPU evaluations that check every matrix, against the oracle on the
# same exact inputs (sampled rows): both are fp64, so they agree to rounding
PIN_NS5 = 1e-12
PIN_ROWWISE = 1e-12


def make_set(wi, step):
    WL = synth.WORKLOADS[wi]
    W, M, G = [], [], []
    for i, (m, n) in enumerate(WL.shapes):
        d = synth.device_matrix(wi, i, m, n, synth.rank_of(WL, m, n), param_dtype=WL.param_dtype,
                                grad_dtype=WL.grad_dtype, device="cuda", beta=WL.beta, step=step)
        W.append(d["W"])
        M.append(d["M"])
        G.append(d["G"])
    torch.cuda.synchronize()
    return W, M, G


def config(WL, precise=0):
    return prm.config_default(K=WL.K, lr=WL.lr, wd=WL.wd, gamma=WL.gamma, beta=WL.beta,
                              param_dtype=prm.BF16, grad_dtype=prm.BF16, ns_precise=precise)


def run(wi, step, sample, precise=0, every=None):
    """One step at the given t over the whole set; returns host copies of the
    sampled matrices' inputs and outputs, and (up to DiT-9B) checks the debug
    step against the timed one bitwise.  ``every(i, M_i, D_i)`` (device
    tensors after the step) is called for every matrix that has a direction
    output (with the host inputs of the sampled ones); its results come back
    as a dict."""
    WL = synth.WORKLOADS[wi]
    cfg = config(WL, precise)
    shapes = list(WL.shapes)
    print(f"[fullsize] {WL.name} t={step}: drawing {len(shapes)} matrices", flush=True)
    W, M, G = make_set(wi, step)
    host_in = {i: (pc.to_host(W[i]), pc.to_host(M[i]), pc.to_host(G[i])) for i in sample}
    copy = wi not in NO_COPY
    if copy:
        W2 = [w.clone() for w in W]
        M2 = [m.clone() for m in M]
    D = [torch.empty(s, dtype=torch.float32, device="cuda") if (copy or i in sample) else None
         for i, s in enumerate(shapes)]
    print(f"[fullsize] {WL.name} t={step}: step", flush=True)
    with prm.Optimizer(shapes, cfg) as opt:
        rho = opt.step(W, G, M, step, directions=D)
        if copy:
            rho2 = opt.step(W2, G, M2, step)
        torch.cuda.synchronize()
    assert rho == po.refresh_indicator(step, WL.K)
    if copy:
        assert rho2 == rho
        for a, b in zip(W + M, W2 + M2):
            assert torch.equal(a, b), "timed step differs from the debug step"
        del W2, M2
    out = {i: (pc.to_host(W[i]), pc.to_host(M[i]), pc.to_host(D[i])) for i in sample}
    checked = {}
    if every is not None:
        print(f"[fullsize] {WL.name} t={step}: checking every matrix", flush=True)
        for i in range(len(shapes)):
            if D[i] is not None:
                checked[i] = every(i, M[i], D[i], host_in)
    del W, M, G, D
    torch.cuda.empty_cache()
    return cfg, host_in, out, checked


def oriented_rows(A, m, n, rows):
    return A[rows] if m <= n else A[:, rows].T


def check_rows(WL, cfg, i, rows, Do_rows, host_in, out, tol):
    m, n = WL.shapes[i]
    W0, M0, G = host_in[i]
    Wg, Mg, Dg = out[i]
    oc = pc.oracle_config(cfg)
    Mo = po.momentum_update(M0, G, oc.beta)
    Dg_rows = oriented_rows(Dg, m, n, rows)
    err = pc.rel(Dg_rows, Do_rows)
    worst = float(np.max(pc.row_errors(Dg_rows, Do_rows)))
    print(f"  {i} {m}x{n}: D rows err {err:.3e}, worst row {worst:.3e}", flush=True)
    assert err <= tol, f"matrix {i} {m}x{n}: D err {err:.3e} > {tol}"
    assert worst <= tol, f"matrix {i} {m}x{n}: worst sampled row err {worst:.3e} > {tol}"
    assert pc.rel(oriented_rows(Mg, m, n, rows), oriented_rows(Mo, m, n, rows)) <= pc.TOL_M
    Wo_rows = (1 - oc.lr * oc.wd) * oriented_rows(W0, m, n, rows) - oc.lr * Do_rows
    slack = pc.bf16_write_bound(oriented_rows(Wg, m, n, rows), Wo_rows, Dg_rows, Do_rows, cfg.lr)
    assert slack <= 1.0, f"matrix {i}: W outside the rounding bound ({slack:.3f})"


def oriented64(A, m, n):
    """Oriented fp64 copy of a device matrix (stored rows if m <= n, else columns)."""
    return (A if m <= n else A.t()).to(torch.float64).contiguous()


def ns5_fp64(U, m, n, oc):
    """s(m, n) X_5 for the oriented U: the five-iteration map of eq.
    (app-ns-recurrence) in fp64 torch matrix products on the GPU, a check of
    every matrix of a set (the CPU oracle takes too long for all of them)."""
    a, b, c = oc.coeffs
    X = oriented64(U, m, n)
    X = X / (torch.linalg.vector_norm(X) + oc.eps_ns)
    for _ in range(po.NS_ITERS):
        A = torch.mm(X, X.t().contiguous())
        B = b * A + c * torch.mm(A, A)
        X = a * X + torch.mm(B, X)
    return po.shape_scale(m, n, oc.scale_mode) * X


def rownorm_fp64(U, m, n, oc):
    """gamma s(m, n) RowNorm of the oriented U (eq. rownorm), fp64 on the GPU."""
    X = oriented64(U, m, n)
    nu = torch.linalg.vector_norm(X, dim=1).clamp_min(oc.eps_rownorm)
    return (po.shape_scale(m, n, oc.scale_mode) * oc.gamma) * X / nu[:, None]


def every_matrix(WL, oc, ref, rows_of):
    """Callback for ``run``: D of matrix i against ``ref`` evaluated from the
    step's own new momentum (matrix and worst-row error); for a sampled matrix
    also ``ref`` evaluated from the exact fp64 momentum of the host inputs at
    the sampled rows, which the test holds to the oracle."""
    def f(i, Mi, Di, host_in):
        m, n = WL.shapes[i]
        R = ref(Mi, m, n, oc)
        Dg = oriented64(Di, m, n)
        diff = torch.linalg.vector_norm(Dg - R, dim=1)
        den = torch.linalg.vector_norm(R, dim=1)
        err = float(torch.linalg.vector_norm(diff) / torch.linalg.vector_norm(den))
        worst = float((diff / den.clamp_min(1e-300)).max())
        del R, Dg, diff, den
        exact = None
        if i in rows_of:
            _, M0, G = host_in[i]
            Ue = torch.tensor(po.momentum_update(M0, G, oc.beta), dtype=torch.float64, device="cuda")
            exact = ref(Ue, m, n, oc)[torch.as_tensor(rows_of[i], device="cuda")].cpu().numpy()
            del Ue
        return err, worst, exact
    return f


def check_every(WL, checked, tol):
    errs = {i: e for i, (e, _, _) in checked.items()}
    worst = {i: w for i, (_, w, _) in checked.items()}
    ie, iw = max(errs, key=errs.get), max(worst, key=worst.get)
    print(f"  every matrix ({len(checked)}): largest D err {errs[ie]:.3e} (matrix {ie} {WL.shapes[ie]}), "
          f"worst row {worst[iw]:.3e} (matrix {iw})", flush=True)
    assert errs[ie] <= tol, f"matrix {ie}: D err {errs[ie]:.3e} > {tol}"
    assert worst[iw] <= tol, f"matrix {iw}: worst row err {worst[iw]:.3e} > {tol}"


@pytest.mark.parametrize("wi,precise", [(wi, 0) for wi in SETS] + [(1, 1), (2, 1)],
                         ids=[synth.WORKLOADS[i].name for i in SETS] + ["dit-1.3b-precise", "dit-4b-precise"])
def test_refresh_step_sampled_rows(wi, precise):
    """The default path on every set; the precise mode (hi + lo iterates, the
    plain iterations for every matrix) on DiT-1.3B and DiT-4B."""
    WL = synth.WORKLOADS[wi]
    sample = list(REFRESH_SAMPLE[wi])             # matrices of the first and last block
    rng = np.random.default_rng(7)
    rows_of = {i: np.sort(rng.choice(min(WL.shapes[i]), 48, replace=False)) for i in sample}
    oc = pc.oracle_config(config(WL, precise))
    every = None if wi in NO_COPY else every_matrix(WL, oc, ns5_fp64, rows_of)
    cfg, host_in, out, checked = run(wi, 0, sample, precise, every)
    for i in sample:
        m, n = WL.shapes[i]
        W0, M0, G = host_in[i]
        U = po.momentum_update(M0, G, oc.beta)
        X = po.orient(U)
        rows = rows_of[i]
        Do = po.shape_scale(m, n, oc.scale_mode) * po.ns5_rows_closed_form(X, rows, oc.eps_ns, oc.coeffs)
        check_rows(WL, cfg, i, rows, Do, host_in, out, pc.TOL_NS5)
        if checked:
            pin = pc.rel(checked[i][2], Do)
            print(f"    fp64 GPU map vs oracle closed form, sampled rows: {pin:.1e}", flush=True)
            assert pin <= PIN_NS5, f"matrix {i}: the fp64 check map disagrees with the oracle ({pin:.1e})"
    if checked:
        check_every(WL, checked, pc.TOL_NS5)


@pytest.mark.parametrize("wi", SETS, ids=[synth.WORKLOADS[i].name for i in SETS])
def test_rowwise_step_sampled_rows(wi):
    WL = synth.WORKLOADS[wi]
    L = WL.blocks
    sample = list(range(5)) + list(range(5 * (L - 1), 5 * L))   # first and last block
    if wi in NO_COPY:
        sample = list(range(5)) + [5 * (L - 1) + 3]               # and the last MLP down only
    rng = np.random.default_rng(8)
    rows_of = {i: np.sort(rng.choice(min(WL.shapes[i]), 64, replace=False)) for i in sample}
    oc = pc.oracle_config(config(WL))
    every = None if wi in NO_COPY else every_matrix(WL, oc, rownorm_fp64, rows_of)
    cfg, host_in, out, checked = run(wi, 1, sample, 0, every)
    for i in sample:
        m, n = WL.shapes[i]
        W0, M0, G = host_in[i]
        U = po.momentum_update(M0, G, oc.beta)
        rows = rows_of[i]
        Xr = oriented_rows(U, m, n, rows)
        Do = po.shape_scale(m, n, oc.scale_mode) * oc.gamma * po.rownorm(Xr, oc.eps_rownorm)
        check_rows(WL, cfg, i, rows, Do, host_in, out, pc.TOL_ROWWISE)
        if checked:
            pin = pc.rel(checked[i][2], Do)
            assert pin <= PIN_ROWWISE, f"matrix {i}: the fp64 check map disagrees with the oracle ({pin:.1e})"
    if checked:
        check_every(WL, checked, pc.TOL_ROWWISE)
