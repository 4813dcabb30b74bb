"""HIP graph capture of prm_step: a refresh step and a row-wise step captured
once each (torch.cuda.graph over the context's stream) and replayed along the
schedule, each replay checked bitwise against an eager context that takes the
same steps on copies of the same state.  The step path allocates nothing,
records no memset and, with unchanged pointers, uploads nothing, so its
kernels are all a graph holds."""
import os
import sys

import pytest
import torch

sys.path.insert(0, os.path.dirname(os.path.abspath(__file__)))
import paper_2608_20818_amd as prm  # noqa: E402
import prm_case as pc  # noqa: E402

pytestmark = [pytest.mark.gpu,
              pytest.mark.skipif(not torch.cuda.is_available(), reason="needs a GPU")]

SHAPES = [(256, 768), (768, 256), (300, 300), (64, 4100)]


@pytest.mark.parametrize("wdt,gdt", [(1, 1), (0, 0)])
def test_captured_steps_replay_bitwise(wdt, gdt):
    K = 2
    cfg = prm.config_default(K=K, lr=0.01, wd=0.05, param_dtype=wdt, grad_dtype=gdt)
    inputs = pc.host_inputs(SHAPES, cfg, 96, steps=(0,))
    G = [pc.to_device(g[0], gdt) for _, _, g in inputs]
    W_e = [pc.to_device(w, wdt) for w, _, _ in inputs]
    M_e = [pc.to_device(m, 0) for _, m, _ in inputs]
    W_g = [w.clone() for w in W_e]
    M_g = [m.clone() for m in M_e]
    side = torch.cuda.Stream()
    eager = prm.Optimizer(SHAPES, cfg)
    graphed = prm.Optimizer(SHAPES, cfg, stream=side)
    try:
        # step 0 on both, eagerly: the graphed context uploads its pointer table
        # here, so that the captured steps hold kernels only
        assert eager.step(W_e, G, M_e, 0) == 1
        with torch.cuda.stream(side):
            assert graphed.step(W_g, G, M_g, 0) == 1
        torch.cuda.synchronize()
        graphs = {}
        for rho, t in ((0, 1), (1, 2)):  # a row-wise and a refresh step
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=side):
                assert graphed.step(W_g, G, M_g, t) == rho
            graphs[rho] = g
        torch.cuda.synchronize()
        # capturing runs nothing: the graphed state is still that after step 0
        for t in range(1, 9):
            rho = 1 if t % K == 0 else 0
            assert eager.step(W_e, G, M_e, t) == rho
            graphs[rho].replay()
            torch.cuda.synchronize()
            for i, s in enumerate(SHAPES):
                assert torch.equal(W_g[i], W_e[i]), f"t={t} W {s}"
                assert torch.equal(M_g[i], M_e[i]), f"t={t} M {s}"
            print(f"  t={t} rho={rho}: replay == eager", flush=True)
    finally:
        eager.close()
        graphed.close()
