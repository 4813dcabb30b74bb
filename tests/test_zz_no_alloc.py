"""The allocation-free entry point prm_step_noalloc (one matrix, no context,
scratch in a static device array) against prm_step on a context holding the
same matrix alone: bitwise equal W and M, and both within the oracle's
tolerances.  Two calls in a row, the second on a smaller matrix, so the second
call finds the scratch array holding the first call's data."""
import ctypes
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

# (shape of the first call, shape of the second, smaller call): wide, tall,
# square and ragged; tall row-wise steps use the scratch's column statistics
PAIRS = [((700, 2000), (301, 77)), ((1536, 520), (130, 390)), ((600, 600), (37, 333)),
         ((2048, 6144), (1, 64))]


def run_pair(pair, t, wdt, gdt, workload_id):
    cfg = prm.config_default(K=4, lr=0.02, wd=0.1, param_dtype=wdt, grad_dtype=gdt)
    oc = pc.oracle_config(cfg)
    stream = torch.cuda.current_stream()
    for shape in pair:
        (w0, m0, g), = pc.host_inputs([shape], cfg, workload_id, steps=(t,))
        print(f"  no-alloc {shape} t={t} W {pc.dtype_name(wdt)} G {pc.dtype_name(gdt)}", flush=True)
        Wa, Ma = pc.to_device(w0, wdt), pc.to_device(m0, 0)
        Wb, Mb = Wa.clone(), Ma.clone()
        G = pc.to_device(g[t], gdt)
        D = torch.zeros(shape, dtype=torch.float32, device="cuda")
        with prm.Optimizer([shape], cfg, stream=stream) as opt:
            rho_a = opt.step([Wa], [G], [Ma], t, directions=[D])
            torch.cuda.synchronize()
        rho_b = prm.step_noalloc(cfg, Wb, G, Mb, t, stream=stream)
        torch.cuda.synchronize()
        Wo, Mo, Do, rho_o = po.step_matrix(w0, m0, g[t], t, oc)
        assert rho_a == rho_b == rho_o
        assert torch.equal(Wb, Wa), f"{shape}: W differs from prm_step"
        assert torch.equal(Mb, Ma), f"{shape}: M differs from prm_step"
        # and the shared result is the oracle's, to the parity bar
        tol = pc.TOL_NS5 if rho_o else pc.TOL_ROWWISE
        eD = pc.rel(pc.to_host(D), Do)
        assert eD <= tol, f"{shape}: D err {eD:.3e}"
        assert pc.rel(pc.to_host(Mb), Mo) <= pc.TOL_M
        if wdt == prm.BF16:
            assert pc.bf16_write_bound(pc.to_host(Wb), Wo, pc.to_host(D), Do, cfg.lr) <= 1.0


@pytest.mark.parametrize("t", [0, 1])
@pytest.mark.parametrize("pair", PAIRS, ids=[f"{a[0]}x{a[1]}-then-{b[0]}x{b[1]}" for a, b in PAIRS])
def test_noalloc_matches_prm_step(pair, t):
    run_pair(pair, t, prm.BF16, prm.BF16, 95)


@pytest.mark.parametrize("t", [0, 3])
def test_noalloc_fp32_and_variants(t):
    run_pair(((520, 136), (64, 1)), t, prm.F32, prm.F32, 96)


def test_noalloc_rejects_before_enqueueing():
    cfg = prm.config_default(K=2)
    W = torch.zeros((8, 16), dtype=torch.bfloat16, device="cuda")
    G = torch.zeros_like(W)
    M = torch.zeros((8, 16), dtype=torch.float32, device="cuda")
    L = prm.load()
    # a refresh whose NS5 workspace exceeds the scratch array (4096 x 16384:
    # 4 rp cp + 4 rp^2 bytes = 335 MB); the pointers are never touched
    r = ctypes.c_int32(-1)
    rc = L.prm_step_noalloc(ctypes.byref(cfg), 4096, 16384, W.data_ptr(), G.data_ptr(), M.data_ptr(), 0,
                            -1.0, ctypes.byref(r), None)
    assert rc == prm.PRM_ENOMEM and r.value == -1
    assert "scratch" in L.prm_last_error().decode()
    # its row-wise step (wide: no workspace) is within the limit, but a bad
    # argument is still refused first
    rc = L.prm_step_noalloc(ctypes.byref(cfg), 4096, 16384, W.data_ptr(), None, M.data_ptr(), 1, -1.0, None, None)
    assert rc == prm.PRM_EINVAL
    rc = L.prm_step_noalloc(ctypes.byref(cfg), 8, 16, W.data_ptr() + 2, G.data_ptr(), M.data_ptr(), 1, -1.0,
                            None, None)
    assert rc == prm.PRM_EALIGN
    rc = L.prm_step_noalloc(ctypes.byref(cfg), 8, 16, W.data_ptr(), G.data_ptr(), M.data_ptr(), -1, -1.0,
                            None, None)
    assert rc == prm.PRM_EINVAL
    host = np.zeros(64, dtype=np.float32)
    rc = L.prm_step_noalloc(ctypes.byref(cfg), 8, 16, W.data_ptr(), G.data_ptr(), host.ctypes.data, 1, -1.0,
                            None, None)
    assert rc == prm.PRM_EINVAL
    torch.cuda.synchronize()
    assert torch.count_nonzero(W) == 0 and torch.count_nonzero(M) == 0
