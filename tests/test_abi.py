"""The C ABI on the CPU: exported symbols, pure host entry points, argument
validation.  Nothing here launches a kernel (no GPU in this environment)."""
import ctypes
import os
import re
import subprocess
import sys

import numpy as np
import pytest

import paper_2608_20818_amd as prm
import synth
from oracle import prm_oracle as po

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "prm.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(prm_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = prm.load()
    names = declared_functions()
    assert {"prm_init", "prm_step", "prm_step_debug", "prm_is_refresh", "prm_workspace_bytes",
            "prm_destroy", "prm_last_error", "prm_config_default", "prm_schedule_is_refresh",
            "prm_plan_workspace_bytes"} <= set(names)
    out = subprocess.run(["nm", "-D", "--defined-only", prm.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r" T (prm_\w+)", out))
    for n in names:
        assert n in exported, n
        assert hasattr(lib, n)


def test_config_struct_layout_matches_header():
    # prm_config: 10 x 4-byte scalars, 9 int32 flags, padding, then a uint64
    assert ctypes.sizeof(prm.Config) == 88
    assert prm.Config.ns_precise.offset == 72
    assert prm.Config.workspace_budget_bytes.offset == 80


def test_config_defaults_are_paper_values():
    cfg = prm.config_default()
    assert cfg.K == 3 and abs(cfg.beta - 0.95) < 1e-7 and abs(cfg.gamma - 0.15) < 1e-7
    assert abs(cfg.wd - 0.01) < 1e-9
    for got, want in zip((cfg.ns_a, cfg.ns_b, cfg.ns_c), po.NS_COEFFS):
        assert abs(got - want) < 1e-6
    assert cfg.param_dtype == prm.BF16 and cfg.grad_dtype == prm.BF16


def _prototypes():
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    return {m.group(1): re.sub(r"\s+", " ", m.group(0)) for m in re.finditer(r"\bint (prm_\w+)\([^;]*\);", text)}


def test_boundary_signatures_follow_the_scope_table():
    # the context-taking schedule and workspace queries of the boundary, and
    # the context-free planners beside them
    p = _prototypes()
    assert p["prm_is_refresh"] == "int prm_is_refresh(const prm_ctx* ctx, int64_t step);"
    assert p["prm_workspace_bytes"] == "int prm_workspace_bytes(const prm_ctx* ctx, size_t* out_bytes);"
    assert p["prm_schedule_is_refresh"] == "int prm_schedule_is_refresh(int64_t step, int32_t K);"
    assert p["prm_init"].startswith("int prm_init(prm_ctx** out, int32_t n_mats, const int64_t* rows, "
                                    "const int64_t* cols, const prm_config* cfg, void* hip_stream)")
    assert p["prm_step"].startswith("int prm_step(prm_ctx* ctx, void* const* params, const void* const* grads, "
                                    "float* const* momentum, int64_t step, float lr, int32_t* did_refresh)")
    assert p["prm_destroy"] == "int prm_destroy(prm_ctx* ctx);"
    L = prm.load()
    out = ctypes.c_size_t(7)
    assert L.prm_is_refresh(None, 0) == prm.PRM_EINVAL
    assert L.prm_workspace_bytes(None, ctypes.byref(out)) == prm.PRM_EINVAL and out.value == 7
    assert L.prm_last_error().decode() != ""


def test_declarations_cite_the_paper():
    # every step entry point names the passage that defines it
    text = open(HEADER).read()
    for name in ("prm_init", "prm_step", "prm_step_debug", "prm_is_refresh", "prm_workspace_bytes"):
        i = text.index(f"int {name}(")
        comment = re.sub(r"\s+\*?\s*", " ", text[text.rindex("/*", 0, i):i])
        assert re.search(r"Alg\. 1|eq\. \(?periodic-direction|Sec\. 3\.3", comment), name


@pytest.mark.parametrize("K", [1, 2, 3, 4, 5, 7, 10, 12])
def test_is_refresh_matches_oracle_exhaustively(K):
    for t in range(0, 600):
        assert prm.schedule_is_refresh(t, K) == po.refresh_indicator(t, K)
    for t in (2 ** 40, 2 ** 40 + 1, 2 ** 62):
        assert prm.schedule_is_refresh(t, K) == po.refresh_indicator(t, K)


def test_is_refresh_rejects_bad_args():
    with pytest.raises(prm.PRMError) as e:
        prm.schedule_is_refresh(0, 0)
    assert e.value.code == prm.PRM_EINVAL
    with pytest.raises(prm.PRMError):
        prm.schedule_is_refresh(-1, 3)


def test_workspace_planning():
    cfg = prm.config_default()
    tiny = synth.WORKLOADS[0].shapes
    b = prm.plan_workspace_bytes(tiny, cfg)
    assert b > 0
    # NS5 region of one matrix: 4 rp cp + 4 rp^2 + 8 rp bytes (the transposed
    # iterate and the next one in bf16, off-diagonal A and B in bf16, their
    # diagonals in fp32)
    one = prm.plan_workspace_bytes([(256, 1024)], cfg)
    assert one >= 4 * 256 * 1024 + 4 * 256 * 256 + 8 * 256
    # a budget smaller than one matrix is refused; a small budget forces chunking
    small = prm.config_default(workspace_budget_bytes=1000)
    with pytest.raises(prm.PRMError) as e:
        prm.plan_workspace_bytes(tiny, small)
    assert e.value.code == prm.PRM_ENOMEM
    chunked = prm.config_default(workspace_budget_bytes=8 * 256 * 1024 + 6 * 256 * 256 + 4096)
    assert prm.plan_workspace_bytes(tiny, chunked) < b
    assert prm.plan_workspace_bytes([], cfg) == 0


def test_workspace_fits_dit_configs():
    cfg = prm.config_default()
    for wl in synth.WORKLOADS[1:]:
        ws = prm.plan_workspace_bytes(wl.shapes, cfg)
        state = sum(m * n for m, n in wl.shapes) * (2 + 2 + 4)
        assert ws <= (48 << 30) + (1 << 30)
        assert state + ws < 288e9 * 0.95, wl.name


@pytest.mark.parametrize("field,value,code", [
    ("K", 0, prm.PRM_EINVAL), ("beta", 1.0, prm.PRM_EINVAL), ("beta", -0.1, prm.PRM_EINVAL),
    ("gamma", 0.0, prm.PRM_EINVAL), ("eps_rownorm", 0.0, prm.PRM_EINVAL),
    ("lr", -1.0, prm.PRM_EINVAL), ("wd", -0.5, prm.PRM_EINVAL), ("scale_mode", 7, prm.PRM_EINVAL),
    ("eps_rownorm", float("inf"), prm.PRM_EINVAL), ("eps_ns", float("nan"), prm.PRM_EINVAL),
    ("eps_ns", 0.0, prm.PRM_EINVAL), ("eps_ns", -1e-7, prm.PRM_EINVAL),
    ("param_dtype", 5, prm.PRM_EDTYPE), ("grad_dtype", -1, prm.PRM_EDTYPE),
    ("nesterov", 2, prm.PRM_EINVAL), ("ns_plain", 2, prm.PRM_EINVAL), ("ns_precise", 2, prm.PRM_EINVAL),
])
def test_init_validates_before_touching_the_device(field, value, code):
    cfg = prm.config_default(**{field: value})
    L = prm.load()
    rows = (ctypes.c_int64 * 1)(4)
    cols = (ctypes.c_int64 * 1)(8)
    ctx = ctypes.c_void_p(123)
    rc = L.prm_init(ctypes.byref(ctx), 1, rows, cols, ctypes.byref(cfg), None)
    assert rc == code
    assert ctx.value is None
    assert L.prm_last_error().decode() != ""


def test_bad_shapes_rejected():
    L = prm.load()
    cfg = prm.config_default()
    for r, c in [(0, 4), (4, 0), (-3, 4), (1 << 25, 2)]:
        rows = (ctypes.c_int64 * 1)(r)
        cols = (ctypes.c_int64 * 1)(c)
        out = ctypes.c_uint64()
        assert L.prm_plan_workspace_bytes(1, rows, cols, ctypes.byref(cfg), ctypes.byref(out)) == prm.PRM_EINVAL
    assert L.prm_plan_workspace_bytes(-1, None, None, ctypes.byref(cfg), ctypes.byref(ctypes.c_uint64())) == prm.PRM_EINVAL
    assert L.prm_plan_workspace_bytes(2, None, None, ctypes.byref(cfg), ctypes.byref(ctypes.c_uint64())) == prm.PRM_EINVAL


def test_null_context_calls_fail_cleanly():
    L = prm.load()
    rho = ctypes.c_int32(-7)
    assert L.prm_step(None, None, None, None, 0, -1.0, ctypes.byref(rho)) == prm.PRM_EINVAL
    assert L.prm_step_debug(None, None, None, None, 0, -1.0, None, None) == prm.PRM_EINVAL
    assert L.prm_profile_enable(None, 1) == prm.PRM_EINVAL
    assert L.prm_profile_read(None, None, 0) == prm.PRM_EINVAL
    assert L.prm_destroy(None) == prm.PRM_OK
    assert L.prm_init(None, 0, None, None, None, None) == prm.PRM_EINVAL


def test_calibration_probes_validate_before_touching_the_device():
    L = prm.load()
    d = ctypes.c_double()
    assert L.prm_peak_mfma(None, 100, None, ctypes.byref(d)) == prm.PRM_EINVAL
    assert L.prm_peak_mfma(None, 0, ctypes.byref(d), ctypes.byref(d)) == prm.PRM_EINVAL
    assert L.prm_peak_hbm(None, 1 << 30, None, ctypes.byref(d), ctypes.byref(d), ctypes.byref(d)) == prm.PRM_EINVAL
    assert L.prm_peak_hbm(None, 1 << 30, ctypes.byref(d), ctypes.byref(d), ctypes.byref(d), None) == prm.PRM_EINVAL
    assert L.prm_peak_hbm(None, 1000, ctypes.byref(d), ctypes.byref(d), ctypes.byref(d), ctypes.byref(d)) == prm.PRM_EINVAL
    assert L.prm_last_error().decode() != ""


def test_adamw_config_layout_and_defaults_are_paper_values():
    # prm_adamw_config: 5 floats, 3 int32
    assert ctypes.sizeof(prm.AdamWConfig) == 32
    c = prm.adamw_config_default()
    gold = po.AdamWConfig()
    for got, want in ((c.lr, gold.lr), (c.beta1, gold.beta1), (c.beta2, gold.beta2), (c.eps, gold.eps),
                      (c.wd, gold.wd)):
        assert got == np.float32(want)
    assert c.param_dtype == prm.BF16 and c.grad_dtype == prm.BF16


@pytest.mark.parametrize("field,value,code", [
    ("lr", -1.0, prm.PRM_EINVAL), ("beta1", 1.0, prm.PRM_EINVAL), ("beta2", -0.1, prm.PRM_EINVAL),
    ("eps", 0.0, prm.PRM_EINVAL), ("wd", float("nan"), prm.PRM_EINVAL),
    ("param_dtype", 3, prm.PRM_EDTYPE), ("grad_dtype", 9, prm.PRM_EDTYPE),
])
def test_adamw_init_validates_before_touching_the_device(field, value, code):
    cfg = prm.adamw_config_default(**{field: value})
    L = prm.load()
    numel = (ctypes.c_int64 * 2)(10, 4096)
    ctx = ctypes.c_void_p(123)
    assert L.prm_adamw_init(ctypes.byref(ctx), 2, numel, ctypes.byref(cfg), None) == code
    assert ctx.value is None
    assert L.prm_last_error().decode() != ""


def test_adamw_bad_sizes_and_null_context():
    L = prm.load()
    cfg = prm.adamw_config_default()
    ctx = ctypes.c_void_p()
    assert L.prm_adamw_init(ctypes.byref(ctx), -1, None, ctypes.byref(cfg), None) == prm.PRM_EINVAL
    assert L.prm_adamw_init(ctypes.byref(ctx), 2, None, ctypes.byref(cfg), None) == prm.PRM_EINVAL
    bad = (ctypes.c_int64 * 2)(5, -1)
    assert L.prm_adamw_init(ctypes.byref(ctx), 2, bad, ctypes.byref(cfg), None) == prm.PRM_EINVAL
    assert L.prm_adamw_init(None, 0, None, ctypes.byref(cfg), None) == prm.PRM_EINVAL
    assert L.prm_adamw_step(None, None, None, None, None, 1, -1.0) == prm.PRM_EINVAL
    assert L.prm_adamw_destroy(None) == prm.PRM_OK


def test_bench_refuses_more_than_one_gpu():
    # one GPU only: the multi-GPU path is a design note, and the bench says so
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_c_caller_reports_bad_cases_before_touching_the_device(tmp_path):
    # the plain-C caller the GPU tests use: it builds, binds to libprm and
    # rejects unreadable or malformed cases before any HIP call
    lib = os.path.join(ROOT, "tests", "libc_caller.so")
    assert os.path.exists(lib), "run __graft_entry__.build()"
    prm.load()
    L = ctypes.CDLL(lib)
    L.prm_c_run_case.argtypes = [ctypes.c_char_p, ctypes.c_char_p, ctypes.c_int]
    L.prm_c_run_case.restype = ctypes.c_int
    msg = ctypes.create_string_buffer(256)
    assert L.prm_c_run_case(str(tmp_path / "absent").encode(), msg, len(msg)) == -1
    assert "cannot open" in msg.value.decode()
    (tmp_path / "case.txt").write_text("2 5 1\n")
    assert L.prm_c_run_case(str(tmp_path).encode(), msg, len(msg)) == -1
    assert "malformed" in msg.value.decode()
    needed = subprocess.run(["readelf", "-d", lib], capture_output=True, text=True, check=True).stdout
    assert "libprm.so" in needed and "libamdhip64" in needed
    assert "libtorch" not in needed and "python" not in needed


def _m0_check(asm_text):
    """(compiler LDS DMAs, inline-asm LDS DMAs, violations): a violation is an
    M0 read the compiler emitted without its own M0 write before it in the
    same basic block with no inline asm in between, or any other M0 reader."""
    other_m0_readers = re.compile(r"^(s_movrel|v_movrel|s_sendmsg|ds_gws|v_interp|s_set_gpr_idx)")
    compiler_m0 = False  # M0 holds a value the compiler wrote, with no asm since
    in_asm = False
    readers = asm_dma = 0
    bad = []
    for line in asm_text.splitlines():
        s = line.strip()
        if s.startswith(";;#ASMSTART"):
            in_asm = True
            continue
        if s.startswith(";;#ASMEND"):
            in_asm = False
            continue
        if re.match(r"^(\.LBB\w*|_Z\w+):", s):
            compiler_m0 = False  # a new basic block or function: nothing is known
            continue
        if not s or s.startswith(";") or s.startswith("."):
            continue
        writes_m0 = re.match(r"^s_\w+\s+m0,", s) is not None
        if in_asm:
            asm_dma += "global_load_lds" in s
            if writes_m0:
                compiler_m0 = False
            continue
        if other_m0_readers.match(s):
            bad.append(s)
        if "global_load_lds" in s or re.search(r"buffer_load\w*.*\blds\b", s):
            readers += 1
            if not compiler_m0:
                bad.append(s)
        if writes_m0:
            compiler_m0 = True
    return readers, asm_dma, bad


def test_m0_check_flags_a_planted_violation():
    ok = "_Zk:\n s_mov_b32 m0, s1\n global_load_lds_dwordx4 v[0:1], off\n"
    assert _m0_check(ok) == (1, 0, [])
    planted = ("_Zk:\n s_mov_b32 m0, s1\n ;;#ASMSTART\n s_mov_b32 m0, s2\n global_load_lds_dwordx4 v1, s[2:3]\n"
               " ;;#ASMEND\n global_load_lds_dwordx4 v[0:1], off\n")
    assert len(_m0_check(planted)[2]) == 1
    assert len(_m0_check("_Zk:\n s_mov_b32 m0, s1\n.LBB0_1:\n global_load_lds_dwordx4 v[0:1], off\n")[2]) == 1
    assert len(_m0_check("_Zk:\n s_sendmsg sendmsg(MSG_DEALLOC_VGPRS)\n")[2]) == 1


def test_gemm_inline_dma_leaves_m0_to_the_compiler(tmp_path):
    # The NS5 GEMM issues its stage loads through inline assembly that writes
    # M0, a register the compiler reserves and does not save around asm.  That
    # is sound only while every M0 read the compiler emits itself follows its
    # own M0 write in the same basic block with no asm in between.
    from paper_2608_20818_amd import build as b
    out = tmp_path / "ns5.s"
    r = subprocess.run([b.hipcc(), f"--offload-arch={b.ARCH}", "-O3", "-std=c++17", "-Xclang", "-target-feature",
                        "-Xclang", "-packed-fp32-ops", "-I", os.path.join(ROOT, "include"), "-I", b.CSRC,
                        "--cuda-device-only", "-S", os.path.join(b.CSRC, "ns5.hip"), "-o", str(out)],
                       capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stderr[-2000:]
    readers, asm_dma, bad = _m0_check(out.read_text())
    assert asm_dma > 0 and readers > 0
    assert not bad, bad[:5]


def test_fullsize_sample_covers_every_chunk():
    # the test's replica of the chunk packing agrees with the library's planner
    # (largest chunk + per-matrix scalars + tall statistics = its total), and the
    # DiT-15B refresh sample reaches every chunk and every matrix kind
    sys.path.insert(0, os.path.join(ROOT, "tests"))
    import prm_case as pc
    import test_gpu_fullsize as fs
    cfg = prm.config_default()
    for wi in (1, 2, 3, 4):
        shapes = synth.WORKLOADS[wi].shapes
        chunk, biggest = pc.ns_chunks(shapes)
        assert prm.plan_workspace_bytes(shapes, cfg) == (biggest + 255) // 256 * 256 + sum(
            prm.plan_workspace_bytes([s], cfg) - pc.ns_chunks([s])[1] for s in shapes), wi
        sample = fs.REFRESH_SAMPLE[wi]
        assert {chunk[i] for i in sample} == set(chunk), wi
        assert {i % 5 for i in sample} == set(range(5)), wi
    assert len(set(pc.ns_chunks(synth.WORKLOADS[4].shapes)[0])) == 3


def test_precise_mode_plans_the_plain_path_with_hi_lo_iterates():
    """ns_precise: a wide matrix (c >= 2r) takes the plain path (two split
    matrices instead of four) and its two iterates gain low parts: the plan
    grows by 2 rp cp bf16 and shrinks by two split matrices."""
    L = prm.load()
    rows = (ctypes.c_int64 * 1)(256)
    cols = (ctypes.c_int64 * 1)(768)
    sizes = {}
    for precise in (0, 1):
        cfg = prm.config_default(ns_precise=precise)
        out = ctypes.c_uint64()
        assert L.prm_plan_workspace_bytes(1, rows, cols, ctypes.byref(cfg), ctypes.byref(out)) == prm.PRM_OK
        sizes[precise] = out.value
    xs, gs, vs = 256 * 768 * 2, 256 * 256 * 2, 256 * 4
    assert sizes[1] - sizes[0] == 2 * xs - 2 * (gs + vs)


def test_precise_mode_refused_by_the_allocation_free_step():
    L = prm.load()
    cfg = prm.config_default(ns_precise=1)
    rho = ctypes.c_int32(-1)
    fake = ctypes.c_void_p(1 << 20)  # never dereferenced: the config is refused first
    rc = L.prm_step_noalloc(ctypes.byref(cfg), 4, 8, fake, fake, fake, 0, -1.0, ctypes.byref(rho), None)
    assert rc == prm.PRM_EINVAL and "ns_precise" in L.prm_last_error().decode()
