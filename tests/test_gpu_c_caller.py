"""GPU parity through a plain-C caller: ``tests/c_caller.c`` (HIP runtime for
memory and a stream, the C ABI for the optimizer, no PyTorch) runs the steps on
inputs written as raw files, and its outputs are compared with the oracle."""
import ctypes
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

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "libc_caller.so")


def caller():
    if not os.path.exists(LIB):
        pytest.fail(f"{LIB} is not built: run __graft_entry__.build()")
    prm.load()  # libprm first, so the caller binds to the same copy
    L = ctypes.CDLL(LIB)
    L.prm_c_run_case.argtypes = [ctypes.c_char_p, ctypes.c_char_p, ctypes.c_int]
    L.prm_c_run_case.restype = ctypes.c_int
    return L


def raw(a, code):
    """float64 array of values exact in the storage type -> raw bytes."""
    f = np.ascontiguousarray(a, dtype=np.float32)
    if code == prm.BF16:
        return (f.view(np.uint32) >> 16).astype(np.uint16).tobytes()
    return f.tobytes()


def unraw(path, shape, code):
    if code == prm.BF16:
        bits = np.fromfile(path, dtype=np.uint16).astype(np.uint32) << 16
        return bits.view(np.float32).astype(np.float64).reshape(shape)
    return np.fromfile(path, dtype=np.float32).astype(np.float64).reshape(shape)


def run_case(tmp, shapes, cfg, inputs, t0, steps):
    with open(os.path.join(tmp, "case.txt"), "w") as f:
        f.write(f"{len(shapes)} {cfg.K} {steps} {t0} {cfg.param_dtype} {cfg.grad_dtype}\n")
        f.write(f"{cfg.beta!r} {cfg.lr!r} {cfg.wd!r} {cfg.gamma!r}\n")
        for m, n in shapes:
            f.write(f"{m} {n}\n")
    for i, (w0, m0, g) in enumerate(inputs):
        open(os.path.join(tmp, f"W{i}.bin"), "wb").write(raw(w0, cfg.param_dtype))
        open(os.path.join(tmp, f"M{i}.bin"), "wb").write(raw(m0, prm.F32))
        for s in range(steps):
            open(os.path.join(tmp, f"G{i}_{s}.bin"), "wb").write(raw(g[t0 + s], cfg.grad_dtype))
    msg = ctypes.create_string_buffer(512)
    print(f"  C caller: {len(shapes)} matrices, t = {t0} .. {t0 + steps - 1}", flush=True)
    rc = caller().prm_c_run_case(str(tmp).encode(), msg, len(msg))
    assert rc == 0, msg.value.decode()
    out = []
    for i, (m, n) in enumerate(shapes):
        out.append({k: unraw(os.path.join(tmp, f"{k}{i}.out"), (m, n), code)
                    for k, code in (("W", cfg.param_dtype), ("M", prm.F32), ("D", prm.F32))})
    rho = [tuple(int(x) for x in line.split()) for line in open(os.path.join(tmp, "rho.txt"))]
    return out, rho


def test_c_caller_tiny_trajectory(tmp_path):
    """The tiny workload (6 fp32 matrices, K = 4) for eight steps t = 0..7 from
    C: rho_t of every step, the final M and W, and the last step's direction."""
    wl = synth.WORKLOADS[0]
    shapes = list(wl.shapes)
    cfg = prm.config_default(K=wl.K, lr=wl.lr, wd=wl.wd, param_dtype=prm.F32, grad_dtype=prm.F32)
    steps = 8
    inputs = synth.host_workload(0, steps=range(steps))
    out, rho = run_case(tmp_path, shapes, cfg, inputs, 0, steps)
    oc = pc.oracle_config(cfg)
    Wo = [w for w, _, _ in inputs]
    Mo = [m for _, m, _ in inputs]
    wbudget = np.zeros(len(shapes))
    for t in range(steps):
        Wo, Mo, Do, rho_o = po.step(Wo, Mo, [g[t] for _, _, g in inputs], t, oc)
        assert rho[t] == (t, rho_o, rho_o, rho_o), rho[t]
        tol = pc.TOL_NS5 if rho_o else pc.TOL_ROWWISE
        # each step moves W by eta D; the GPU direction is within tol of the oracle's
        wbudget += [pc.f32(cfg.lr) * tol * np.linalg.norm(d) * 1.01 for d in Do]
    for i, r in enumerate(out):
        eD = pc.rel(r["D"], Do[i])
        eM = pc.rel(r["M"], Mo[i])
        print(f"  {shapes[i]}: last D err {eD:.3e}, M err {eM:.3e}", flush=True)
        assert eD <= pc.TOL_ROWWISE, f"{shapes[i]}: D err {eD:.3e}"
        assert eM <= pc.TOL_M, f"{shapes[i]}: M err {eM:.3e}"
        assert np.linalg.norm(r["W"] - Wo[i]) <= wbudget[i] + 1e-6 * np.linalg.norm(Wo[i]), shapes[i]


@pytest.mark.parametrize("t0", [5, 6])
def test_c_caller_bf16_one_step(tmp_path, t0):
    """bf16 W and G as raw bytes from C, wide / tall / padded shapes: one refresh
    (t = 5) or one row-wise step (t = 6) with K = 5."""
    shapes = [(256, 768), (1024, 256), (130, 390), (301, 77), (8, 4104)]
    cfg = prm.config_default(K=5, lr=3e-3, wd=0.01, param_dtype=prm.BF16, grad_dtype=prm.BF16)
    inputs = pc.host_inputs(shapes, cfg, 93, steps=(t0,))
    out, rho = run_case(tmp_path, shapes, cfg, inputs, t0, 1)
    oc = pc.oracle_config(cfg)
    for i, (w0, m0, g) in enumerate(inputs):
        Wo, Mo, Do, rho_o = po.step_matrix(w0, m0, g[t0], t0, oc)
        assert rho == [(t0, rho_o, rho_o, rho_o)]
        tol = pc.TOL_NS5 if rho_o else pc.TOL_ROWWISE
        r = out[i]
        eD = pc.rel(r["D"], Do)
        print(f"  {shapes[i]} rho={rho_o}: D err {eD:.3e}", flush=True)
        assert eD <= tol, f"{shapes[i]}: D err {eD:.3e} > {tol}"
        assert pc.rel(r["M"], Mo) <= pc.TOL_M
        assert pc.bf16_write_bound(r["W"], Wo, r["D"], Do, cfg.lr) <= 1.0, shapes[i]
