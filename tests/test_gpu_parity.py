"""GPU parity: libprm (through the C ABI) against the fp64 oracle on the same
seeded inputs, at sizes the oracle finishes in seconds.  Shapes are chosen to
reach every launch path: wide rows held in registers with 64 / 256 / 512
threads per row, the generic wide path (unaligned or very long rows), the
tall two-pass path with 4-wide and scalar columns, NS5 with padded tiles,
multiple tiles, several workspace chunks, and degenerate 1 x 1, 1 x n and
m x 1 matrices."""
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

RAGGED = [(256, 768), (130, 130), (200, 4104), (40, 17000), (37, 333), (3, 33000),
          (520, 136), (301, 77), (1, 1), (1, 64), (64, 1), (384, 1280), (1024, 256)]


def run_one_step(shapes, cfg, t, workload_id=90, inputs=None):
    """One prm_step_debug at step t on fresh seeded inputs; returns GPU and
    oracle results as float64 host arrays."""
    inputs = inputs or pc.host_inputs(shapes, cfg, workload_id, steps=(t,))
    dev = "cuda"
    W = [pc.to_device(w, cfg.param_dtype) for w, _, _ in inputs]
    M = [pc.to_device(m, 0) for _, m, _ in inputs]
    G = [pc.to_device(g[t], cfg.grad_dtype) for _, _, g in inputs]
    D = [torch.zeros(s, dtype=torch.float32, device=dev) for s in shapes]
    with prm.Optimizer(shapes, cfg) as opt:
        rho = opt.step(W, G, M, t, directions=D)
        torch.cuda.synchronize()
    oc = pc.oracle_config(cfg)
    res = []
    for i, (w0, m0, g) in enumerate(inputs):
        Wo, Mo, Do, rho_o = po.step_matrix(w0, m0, g[t], t, oc)
        res.append(dict(W=pc.to_host(W[i]), M=pc.to_host(M[i]), D=pc.to_host(D[i]),
                        Wo=Wo, Mo=Mo, Do=Do, W0=w0))
        assert rho == rho_o
    return rho, res


def check(res, rho, cfg, shapes, lr):
    tol = pc.TOL_NS5 if rho else pc.TOL_ROWWISE
    for (m, n), r in zip(shapes, res):
        eD = pc.rel(r["D"], r["Do"])
        eM = pc.rel(r["M"], r["Mo"])
        print(f"  {m}x{n} rho={rho} D_err={eD:.3e} M_err={eM:.3e}", flush=True)
        assert eD <= tol, f"{m}x{n} rho={rho}: D rel err {eD:.3e} > {tol}"
        assert eM <= pc.TOL_M, f"{m}x{n}: M rel err {eM:.3e}"
        if cfg.param_dtype == prm.F32:
            # W_gpu - W_oracle = -eta (D_gpu - D_oracle) up to fp32 rounding
            bound = pc.f32(lr) * np.linalg.norm(r["D"] - r["Do"]) * 1.01 + 4e-7 * np.linalg.norm(r["Wo"]) + 1e-30
            assert np.linalg.norm(r["W"] - r["Wo"]) <= bound, f"{m}x{n}: W"
        else:
            # W_gpu = bf16(decay W0 - eta D_gpu): within half a bf16 ulp of the
            # exact update with the GPU's own direction, which differs from the
            # oracle's update by eta |D_gpu - D_oracle|
            slack = pc.bf16_write_bound(r["W"], r["Wo"], r["D"], r["Do"], lr)
            assert slack <= 1.0, f"{m}x{n}: W outside the rounding bound ({slack:.3f})"


@pytest.mark.parametrize("t", [0, 1])
@pytest.mark.parametrize("wdt,gdt,plain", [(1, 1, 0), (0, 0, 0), (1, 0, 0), (0, 1, 0), (1, 1, 1)])
def test_ragged_shapes_all_paths(t, wdt, gdt, plain):
    cfg = prm.config_default(K=4, lr=0.02, wd=0.1, param_dtype=wdt, grad_dtype=gdt, ns_plain=plain)
    rho, res = run_one_step(RAGGED, cfg, t)
    assert rho == (1 if t == 0 else 0)
    check(res, rho, cfg, RAGGED, cfg.lr)


# several 256 x 256 tiles per symmetric product with padding: tiles above the
# diagonal and their mirrors (Gram, square), the fold stage pairs and the
# transposed parameter write of the last apply
MULTI_TILE = [(700, 2000), (1536, 520), (600, 600), (1300, 1800)]


@pytest.mark.parametrize("t,wdt,gdt,plain", [(0, 1, 1, 0), (0, 0, 0, 0), (1, 1, 1, 0), (0, 1, 1, 1), (0, 0, 0, 1)])
def test_multi_tile_symmetric_products(t, wdt, gdt, plain):
    # 700 x 2000 and 1536 x 520 (c >= 2r) run NS5 in the factored form unless
    # ns_plain; 600 x 600 and 1300 x 1800 always run the five iterations
    cfg = prm.config_default(K=4, lr=0.02, wd=0.1, param_dtype=wdt, grad_dtype=gdt, ns_plain=plain)
    rho, res = run_one_step(MULTI_TILE, cfg, t, workload_id=93)
    assert rho == (1 if t == 0 else 0)
    check(res, rho, cfg, MULTI_TILE, cfg.lr)


@pytest.mark.parametrize("t,wdt,gdt", [(0, 1, 1), (0, 0, 0), (4, 0, 1)])
def test_precise_mode_multi_tile(t, wdt, gdt):
    """ns_precise (hi + lo iterates) over several tiles with padding: the
    Gram's three K segments, the apply's two with a fold stage pair in each,
    the hi + lo write of the next iterate, and the parameter write."""
    cfg = prm.config_default(K=4, lr=0.02, wd=0.1, param_dtype=wdt, grad_dtype=gdt, ns_precise=1)
    rho, res = run_one_step(MULTI_TILE, cfg, t, workload_id=95)
    assert rho == 1
    check(res, rho, cfg, MULTI_TILE, cfg.lr)


# the dispatcher's switch between the two exact forms of NS5: oriented
# c >= 2r runs the factored form (split products between two Grams), c < 2r
# the five iterations as written; both sides of the boundary, wide and tall
THRESHOLD = {"factored": [(300, 600), (600, 300), (256, 512)], "plain": [(300, 599), (599, 300), (257, 512)]}


@pytest.mark.parametrize("form", ["factored", "plain"])
@pytest.mark.parametrize("wdt,gdt", [(1, 1), (0, 0)])
def test_factored_form_threshold(form, wdt, gdt):
    shapes = THRESHOLD[form]
    cfg = prm.config_default(K=4, lr=0.02, wd=0.1, param_dtype=wdt, grad_dtype=gdt)
    inputs = pc.host_inputs(shapes, cfg, 94, steps=(0,))
    W = [pc.to_device(w, cfg.param_dtype) for w, _, _ in inputs]
    M = [pc.to_device(m, 0) for _, m, _ in inputs]
    G = [pc.to_device(g[0], cfg.grad_dtype) for _, _, g in inputs]
    D = [torch.zeros(sh, dtype=torch.float32, device="cuda") for sh in shapes]
    with prm.Optimizer(shapes, cfg) as opt:
        opt.profile_enable(True)
        assert opt.step(W, G, M, 0, directions=D) == 1
        torch.cuda.synchronize()
        stats = opt.profile_read()
    # the split product runs only in the factored form; the plain form runs
    # one Gram, one square and one apply launch per iteration
    if form == "factored":
        assert stats["ns_sprod"]["launches"] == 9 and stats["ns_gram"]["launches"] == 2, stats
    else:
        assert stats["ns_sprod"]["launches"] == 0 and stats["ns_gram"]["launches"] == 5, stats
    oc = pc.oracle_config(cfg)
    res = []
    for i, (w0, m0, g) in enumerate(inputs):
        Wo, Mo, Do, rho_o = po.step_matrix(w0, m0, g[0], 0, oc)
        assert rho_o == 1
        res.append(dict(W=pc.to_host(W[i]), M=pc.to_host(M[i]), D=pc.to_host(D[i]), Wo=Wo, Mo=Mo, Do=Do, W0=w0))
    check(res, 1, cfg, shapes, cfg.lr)


@pytest.mark.parametrize("flag", ["nesterov", "ema_dampening", "gamma_on_refresh", "never_refresh", "ns_plain",
                                  "ns_precise"])
@pytest.mark.parametrize("t", [0, 3])
def test_variants(flag, t):
    shapes = [(96, 320), (300, 88), (64, 64), (33, 130)]
    cfg = prm.config_default(K=3, lr=0.01, wd=0.05, param_dtype=0, grad_dtype=1, **{flag: 1})
    rho, res = run_one_step(shapes, cfg, t, workload_id=91)
    assert rho == (0 if flag == "never_refresh" else (1 if t % 3 == 0 else 0))
    check(res, rho, cfg, shapes, cfg.lr)


@pytest.mark.parametrize("precise", [0, 1])
def test_several_workspace_chunks(precise):
    shapes = [(256, 512), (512, 256), (128, 640), (200, 200), (256, 512)]
    # a budget that holds the largest single matrix but not all of them
    base = prm.config_default(ns_precise=precise)
    one = max(prm.plan_workspace_bytes([s], base) for s in shapes)
    cfg = prm.config_default(K=2, lr=0.01, wd=0.01, workspace_budget_bytes=one, ns_precise=precise)
    assert prm.plan_workspace_bytes(shapes, cfg) < prm.plan_workspace_bytes(shapes, base)
    rho, res = run_one_step(shapes, cfg, 0, workload_id=92)
    check(res, rho, cfg, shapes, cfg.lr)


def test_zero_and_tiny_rows_rownorm_eps():
    # eq. (rownorm): a zero oriented row gives a zero direction, a row whose
    # norm is below eps is divided by eps.
    shapes = [(6, 40), (48, 5)]
    cfg = prm.config_default(K=5, lr=0.1, wd=0.0, param_dtype=0, grad_dtype=0, beta=0.0,
                             eps_rownorm=1e-3)
    rng = np.random.default_rng(3)
    inputs = []
    for (m, n) in shapes:
        G = rng.standard_normal((m, n)).astype(np.float32).astype(np.float64)
        if m <= n:
            G[1] = 0.0
            G[2] = 1e-5
        else:
            G[:, 1] = 0.0
            G[:, 2] = 1e-5
        inputs.append((np.ones((m, n)), np.zeros((m, n)), {1: G}))
    rho, res = run_one_step(shapes, cfg, 1, inputs=inputs)
    assert rho == 0
    check(res, rho, cfg, shapes, cfg.lr)
    r0 = res[0]
    np.testing.assert_array_equal(r0["D"][1], 0.0)
    np.testing.assert_allclose(r0["D"][2], 0.15 * 1e-5 / pc.f32(1e-3), rtol=1e-5)


def test_zero_momentum_refresh_gives_pure_decay():
    shapes = [(64, 192), (192, 64)]
    cfg = prm.config_default(K=1, lr=0.5, wd=0.1, param_dtype=0, grad_dtype=0)
    inputs = [(np.full((m, n), 0.25), np.zeros((m, n)), {0: np.zeros((m, n))}) for m, n in shapes]
    rho, res = run_one_step(shapes, cfg, 0, inputs=inputs)
    assert rho == 1
    for r in res:
        np.testing.assert_array_equal(r["D"], 0.0)
        np.testing.assert_allclose(r["W"], np.float32(0.25) * np.float32(1 - np.float32(0.5) * np.float32(0.1)))


def test_tiny_workload_trajectory():
    """The tiny workload: 6 fp32 matrices, K = 4, eight steps t = 0..7 (two
    refreshes), lr 0.02, wd 0.1; every step compared with the oracle's own
    trajectory from the same initial state and gradients."""
    wl = synth.WORKLOADS[0]
    shapes = list(wl.shapes)
    cfg = prm.config_default(K=wl.K, lr=wl.lr, wd=wl.wd, param_dtype=0, grad_dtype=0)
    steps = range(8)
    inputs = synth.host_workload(0, steps=steps)
    W = [pc.to_device(w, 0) for w, _, _ in inputs]
    M = [pc.to_device(m, 0) for _, m, _ in inputs]
    D = [torch.zeros(s, dtype=torch.float32, device="cuda") for s in shapes]
    Wo = [w for w, _, _ in inputs]
    Mo = [m for _, m, _ in inputs]
    oc = pc.oracle_config(cfg)
    with prm.Optimizer(shapes, cfg) as opt:
        werr_budget = np.zeros(len(shapes))
        for t in steps:
            G = [pc.to_device(g[t], 0) for _, _, g in inputs]
            rho = opt.step(W, G, M, t, directions=D)
            torch.cuda.synchronize()
            Wo, Mo, Do, rho_o = po.step(Wo, Mo, [g[t] for _, _, g in inputs], t, oc)
            assert rho == rho_o == (1 if t % 4 == 0 else 0)
            tol = pc.TOL_NS5 if rho else pc.TOL_ROWWISE
            for i in range(len(shapes)):
                d = pc.to_host(D[i])
                eD = pc.rel(d, Do[i])
                assert eD <= tol, f"t={t} mat {i} {shapes[i]}: D err {eD:.3e}"
                assert pc.rel(pc.to_host(M[i]), Mo[i]) <= pc.TOL_M
                werr_budget[i] += pc.f32(cfg.lr) * np.linalg.norm(d - Do[i]) * 1.01
                werr = np.linalg.norm(pc.to_host(W[i]) - Wo[i])
                assert werr <= werr_budget[i] + 1e-6 * np.linalg.norm(Wo[i]), f"t={t} mat {i}: W"


def _state(shapes, cfg, seed):
    inputs = pc.host_inputs(shapes, cfg, seed, steps=range(8))
    W = [pc.to_device(w, cfg.param_dtype) for w, _, _ in inputs]
    M = [pc.to_device(m, 0) for _, m, _ in inputs]
    Gs = {t: [pc.to_device(g[t], cfg.grad_dtype) for _, _, g in inputs] for t in range(8)}
    return W, M, Gs


def test_bitwise_deterministic_and_resumable():
    shapes = [(130, 390), (390, 130), (64, 64), (8, 4104)]
    cfg = prm.config_default(K=3, lr=0.01)
    W1, M1, Gs = _state(shapes, cfg, 93)
    W2, M2, _ = _state(shapes, cfg, 93)
    with prm.Optimizer(shapes, cfg) as opt:
        for t in range(8):
            opt.step(W1, Gs[t], M1, t)
    # same trajectory in two contexts: 4 steps, destroy, re-init, 4 more
    with prm.Optimizer(shapes, cfg) as opt:
        for t in range(4):
            opt.step(W2, Gs[t], M2, t)
    torch.cuda.synchronize()
    with prm.Optimizer(shapes, cfg) as opt:
        for t in range(4, 8):
            opt.step(W2, Gs[t], M2, t)
    torch.cuda.synchronize()
    for a, b in zip(W1 + M1, W2 + M2):
        assert torch.equal(a, b)


def test_empty_matrix_list_and_pointer_changes():
    cfg = prm.config_default()
    with prm.Optimizer([], cfg) as opt:
        assert opt.step([], [], [], 0) == 1
        assert opt.step([], [], [], 1) == 0
    # new tensors every call: the pointer table is re-uploaded
    shapes = [(16, 48)]
    with prm.Optimizer(shapes, cfg) as opt:
        for t in range(4):
            W, M, Gs = _state(shapes, cfg, 94)
            opt.step(W, Gs[t], M, t)
    torch.cuda.synchronize()


def test_misaligned_pointer_rejected_without_side_effects():
    shapes = [(8, 16)]
    cfg = prm.config_default(param_dtype=0, grad_dtype=0)
    base = torch.zeros(8 * 16 + 4, dtype=torch.float32, device="cuda")
    W = base[1:1 + 128].view(8, 16)
    G = torch.ones(8, 16, device="cuda")
    M = torch.ones(8, 16, device="cuda")
    with prm.Optimizer(shapes, cfg) as opt:
        with pytest.raises(prm.PRMError) as e:
            opt.step([W], [G], [M], 0)
        assert e.value.code == prm.PRM_EALIGN
        with pytest.raises(prm.PRMError) as e:
            opt.step([G], [G], [M], -1)
        assert e.value.code == prm.PRM_EINVAL
    torch.cuda.synchronize()
    assert torch.equal(M, torch.ones_like(M))


def test_host_pointers_rejected_before_any_launch():
    # host memory (pageable or pinned) where device memory is required: the
    # library refuses it before enqueuing anything (a kernel would fault)
    import numpy as np
    shapes = [(8, 16)]
    cfg = prm.config_default(param_dtype=0, grad_dtype=0)
    G = torch.ones(8, 16, device="cuda")
    M = torch.ones(8, 16, device="cuda")
    W = torch.zeros(8, 16, device="cuda")
    pageable = np.zeros(8 * 16 + 16, dtype=np.float32)
    addr = pageable.ctypes.data
    addr += (-addr) % 16  # aligned, so only the memory kind is wrong
    pinned = torch.zeros(8, 16, dtype=torch.float32).pin_memory()
    with prm.Optimizer(shapes, cfg) as opt:
        for bad in (addr, pinned.data_ptr()):
            with pytest.raises(prm.PRMError) as e:
                opt.step([W], [G], [bad], 0)
            assert e.value.code == prm.PRM_EINVAL and "host memory" in str(e.value), str(e.value)
        with pytest.raises(ValueError):
            opt.step([W.cpu()], [G], [M], 0)  # the binding refuses a CPU tensor itself
        opt.step([W], [G], [M], 1)  # valid pointers after the refusals
    torch.cuda.synchronize()
    assert torch.equal(G, torch.ones_like(G))
    with prm.AuxAdamW([128], prm.adamw_config_default(param_dtype=0, grad_dtype=0)) as aux:
        flat = [t.view(-1) for t in (W, G, M)]
        with pytest.raises(prm.PRMError) as e:
            aux.step([flat[0]], [flat[1]], [flat[2]], [pinned.data_ptr()], 1)
        assert e.value.code == prm.PRM_EINVAL


@pytest.mark.parametrize("t", [0, 1])
def test_debug_step_with_some_directions_skipped(t):
    # NULL direction entries: those matrices' D is not written; W, M and the
    # other directions are bitwise those of a debug step with every output
    shapes = [(64, 192), (192, 64), (130, 130), (40, 4104)]
    cfg = prm.config_default(K=2, lr=0.02, wd=0.1, param_dtype=prm.BF16, grad_dtype=prm.BF16)
    inputs = pc.host_inputs(shapes, cfg, 97, steps=(t,))
    outs = []
    for skip in (False, True):
        W = [pc.to_device(w, cfg.param_dtype) for w, _, _ in inputs]
        M = [pc.to_device(m, 0) for _, m, _ in inputs]
        G = [pc.to_device(g[t], cfg.grad_dtype) for _, _, g in inputs]
        D = [torch.full(s, 7.0, dtype=torch.float32, device="cuda") for s in shapes]
        Dp = [None if (skip and i % 2 == 1) else x for i, x in enumerate(D)]
        with prm.Optimizer(shapes, cfg) as opt:
            opt.step(W, G, M, t, directions=Dp)
            torch.cuda.synchronize()
        outs.append((W, M, D))
    (W0, M0, D0), (W1, M1, D1) = outs
    for i in range(len(shapes)):
        assert torch.equal(W0[i], W1[i]) and torch.equal(M0[i], M1[i])
        if i % 2 == 1:
            assert bool((D1[i] == 7.0).all()), "skipped direction was written"
        else:
            assert torch.equal(D0[i], D1[i])


@pytest.mark.parametrize("t", [0, 1])
def test_long_rows_and_columns(t):
    # extreme aspect ratios: a 4 M-element row (the two-sweep generic row-wise
    # kernel; a Gram whose K streams 65536 stages through one tile) and a
    # 2 M-row matrix of width 3 (scalar tall path, 65536 row tiles of partials)
    shapes = [(2, 1 << 22), (1 << 21, 3)]
    cfg = prm.config_default(K=4, lr=0.02, wd=0.1, param_dtype=prm.BF16, grad_dtype=prm.BF16)
    rho, res = run_one_step(shapes, cfg, t, workload_id=98)
    assert rho == (1 if t == 0 else 0)
    check(res, rho, cfg, shapes, cfg.lr)


@pytest.mark.parametrize("t", [0, 1])
def test_largest_dimension(t):
    # the largest dimension the ABI accepts (2^24) on both sides: a 1 x 2^24
    # row (generic row-wise kernel; a Gram whose one tile streams 262144 K
    # stages; 65536 apply tiles) and a 2^24 x 1 column (scalar tall path with
    # 524288 row blocks of partial sums)
    n = 1 << 24
    shapes = [(1, n), (n, 1)]
    cfg = prm.config_default(K=4, lr=0.02, wd=0.1, param_dtype=prm.BF16, grad_dtype=prm.BF16)
    rho, res = run_one_step(shapes, cfg, t, workload_id=99)
    assert rho == (1 if t == 0 else 0)
    check(res, rho, cfg, shapes, cfg.lr)
    torch.cuda.empty_cache()


@pytest.mark.parametrize("flag", [None, "never_refresh"])
def test_context_schedule_and_workspace_queries(flag):
    # prm_is_refresh on a context reports what prm_step returns in did_refresh
    # (the schedule of eq. periodic-direction, or none for the RowNorm-every-step
    # ablation); prm_workspace_bytes reports what the planner said prm_init
    # would allocate
    shapes = [(96, 320), (300, 88)]
    kw = {flag: 1} if flag else {}
    cfg = prm.config_default(K=3, param_dtype=0, grad_dtype=0, **kw)
    inputs = pc.host_inputs(shapes, cfg, 94, steps=tuple(range(7)))
    W = [pc.to_device(w, 0) for w, _, _ in inputs]
    M = [pc.to_device(m, 0) for _, m, _ in inputs]
    oc = pc.oracle_config(cfg)
    with prm.Optimizer(shapes, cfg) as opt:
        assert opt.workspace_bytes() == prm.plan_workspace_bytes(shapes, cfg)
        for t in range(7):
            G = [pc.to_device(g[t], 0) for _, _, g in inputs]
            want = 0 if flag else po.refresh_indicator(t, cfg.K)
            assert opt.is_refresh(t) == want
            assert opt.step(W, G, M, t) == want
        for t in (2 ** 40, 2 ** 40 + 1):
            assert opt.is_refresh(t) == (0 if flag else po.refresh_indicator(t, cfg.K))
        with pytest.raises(prm.PRMError):
            opt.is_refresh(-1)
        torch.cuda.synchronize()
