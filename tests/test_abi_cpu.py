"""The C-ABI library loads, exports every declared entry point, and rejects
bad arguments on the host before any GPU work (no GPU needed)."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "wino.h")


@pytest.fixture(scope="module")
def abi():
    lib_path = os.path.join(ROOT, "paper_2605_16941_amd", "libwino.so")
    if not os.path.exists(lib_path):
        import __graft_entry__
        __graft_entry__._load_build_module().build()
    from paper_2605_16941_amd import _abi
    return _abi


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(wino_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(abi):
    names = declared_functions()
    assert "wino_step" in names and "wino_decode" in names and "wino_decode_block" in names
    for n in names:
        assert hasattr(abi.lib, n), f"{n} declared in wino.h but not exported"
    assert set(names) == set(abi.EXPORTED)


def test_struct_sizes_match_header_layout(abi):
    assert C.sizeof(abi.wino_model_config) == 36
    assert C.sizeof(abi.wino_params) == 40
    assert C.sizeof(abi.wino_row_stats) == 24
    assert C.sizeof(abi.wino_row_loss) == 16
    assert C.sizeof(abi.wino_weights) == 10 * C.sizeof(C.c_void_p)


def test_status_strings(abi):
    for code in abi.STATUS:
        assert abi.status_string(code)
    assert abi.status_string(0) == "ok"
    assert abi.wino_kernel_class_name(2) == "gemm_qkv_rope"
    assert abi.wino_kernel_class_name(99) == ""


def tiny_cfg(abi, **kw):
    base = dict(n_layers=2, d_model=256, n_heads=4, head_dim=64, d_ff=704, vocab=4096,
                rope_theta=10000.0, rms_eps=1e-5)
    base.update(kw)
    return abi.wino_model_config(*base.values())


def test_workspace_bytes(abi):
    cfg = tiny_cfg(abi)
    a = abi.wino_workspace_bytes(cfg, 1, 112)
    b = abi.wino_workspace_bytes(cfg, 2, 112)
    assert 0 < a < b
    assert abi.lib.wino_workspace_bytes(None, 1, 112) == 0
    assert abi.wino_workspace_bytes(cfg, 0, 112) == 0
    assert abi.wino_epilogue_workspace_bytes(8, 32, 126464) >= 8 * 32 * 8 * 20
    assert abi.wino_epilogue_workspace_bytes(0, 32, 126464) == 0


def test_create_rejects_bad_arguments_before_gpu_work(abi):
    out = C.c_void_p()
    w = abi.wino_weights()
    cfg = tiny_cfg(abi)
    assert abi.lib.wino_create(None, C.byref(w), 1, 112, C.byref(out)) == -1
    assert abi.lib.wino_create(C.byref(cfg), C.byref(w), 0, 112, C.byref(out)) == -2
    bad = tiny_cfg(abi, head_dim=96, d_model=384)
    assert abi.lib.wino_create(C.byref(bad), C.byref(w), 1, 112, C.byref(out)) == -6
    bad = tiny_cfg(abi, vocab=4000)
    assert abi.lib.wino_create(C.byref(bad), C.byref(w), 1, 112, C.byref(out)) == -6
    assert abi.lib.wino_last_error(None) == b"model shape"
    # supported shape, but null weight pointers
    assert abi.lib.wino_create(C.byref(cfg), C.byref(w), 1, 112, C.byref(out)) == -1
    assert abi.lib.wino_last_error(None) == b"null weight pointer"
    assert out.value is None


def test_entry_points_reject_null_context_and_bad_params(abi):
    p = abi.make_params(1, 32, 64, 16, 4095)
    assert abi.lib.wino_step(None, C.byref(p), None, None, None, None, None, None, None) == -1
    assert abi.lib.wino_decode(None, C.byref(p), None, None, None, None, 0, None, None, None) == -1
    assert abi.lib.wino_decode_block(None, C.byref(p), None, None, None, None, None) == -1
    assert abi.lib.wino_destroy(None) == -1
    assert abi.lib.wino_profile(None, 1) == -1
    # standalone epilogue: host-side validation
    ws = C.c_void_p(1)
    bad = abi.make_params(1, 0, 16, 16, 4095, float("nan"), 0.9)
    assert abi.lib.wino_epilogue(C.byref(bad), 4096, ws, ws, ws, None, None, ws, 1 << 20, None) == -1
    bad = abi.make_params(1, 0, 16, 16, 5000, 0.7, 0.9)
    assert abi.lib.wino_epilogue(C.byref(bad), 4096, ws, ws, ws, None, None, ws, 1 << 20, None) == -1
    ok = abi.make_params(1, 0, 16, 16, 4095, 0.7, 0.9)
    assert abi.lib.wino_epilogue(C.byref(ok), 4100, ws, ws, ws, None, None, ws, 1 << 20, None) == -2
    assert abi.lib.wino_epilogue(C.byref(ok), 4096, ws, ws, ws, None, None, ws, 16, None) == -2
    assert abi.lib.wino_epilogue(C.byref(ok), 4096, None, ws, ws, None, None, ws, 1 << 20, None) == -1


def fake_weights(abi, n_layers):
    """A weights struct of non-null placeholder pointers: wino_create stores
    them and never dereferences them before its workspace check."""
    keep = []

    def arr():
        a = (C.c_void_p * n_layers)(*([0x1000] * n_layers))
        keep.append(a)
        return a

    w = abi.wino_weights(0x1000, arr(), arr(), arr(), arr(), arr(), arr(), 0x1000, 0x1000, None)
    return w, keep


def test_workspace_limit_is_enforced_before_any_hip_call(abi, monkeypatch):
    """WINO_WORKSPACE_LIMIT (bytes) below what the context needs makes
    wino_create return WINO_ERR_NO_MEMORY before it touches the HIP runtime,
    so the out-of-memory path is exercised without a GPU."""
    cfg = tiny_cfg(abi)
    need = abi.wino_workspace_bytes(cfg, 2, 112)
    w, keep = fake_weights(abi, cfg.n_layers)
    out = C.c_void_p()
    for limit in (0, need // 2, need - 1):
        monkeypatch.setenv("WINO_WORKSPACE_LIMIT", str(limit))
        assert abi.lib.wino_create(C.byref(cfg), C.byref(w), 2, 112, C.byref(out)) == -4
        assert out.value is None
    # a larger batch needs more than a limit sized for batch 2
    monkeypatch.setenv("WINO_WORKSPACE_LIMIT", str(need))
    assert abi.lib.wino_create(C.byref(cfg), C.byref(w), 3, 112, C.byref(out)) == -4



SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined"]


def _hipcc():
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    pytest.skip("hipcc not available")


def test_host_code_under_address_and_undefined_behaviour_sanitizers():
    """The library's host code (argument validation, sizing, the GEMM tile
    planner's rejections, the workspace limit, status strings) built with
    AddressSanitizer and UndefinedBehaviorSanitizer on the host pass only,
    linked with tests/host_checks.cpp and run without a GPU: every check
    passes and no sanitizer reports anything."""
    import subprocess
    hipcc = _hipcc()
    csrc = os.path.join(ROOT, "paper_2605_16941_amd", "csrc")
    out = os.path.join(ROOT, "_build", "host_sanitize")
    os.makedirs(out, exist_ok=True)
    flags = ["-x", "hip", "--offload-arch=gfx950", "-O1", "-g", "-fno-omit-frame-pointer", "-std=c++17",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", *SANITIZE,
             "-I", os.path.join(ROOT, "include"), "-I", csrc]
    headers = [os.path.join(ROOT, "include", "wino.h")] + [os.path.join(csrc, h) for h in ("common.h", "kernels.h")]
    newest_header = max(os.path.getmtime(h) for h in headers)
    procs, objs = [], []
    for src in ("k_norm.hip", "k_gemm.hip", "k_attn.hip", "k_decide.hip", "wino.cpp"):
        path = os.path.join(csrc, src)
        obj = os.path.join(out, os.path.splitext(src)[0] + ".o")
        objs.append(obj)
        if os.path.exists(obj) and os.path.getmtime(obj) > max(os.path.getmtime(path), newest_header):
            continue
        procs.append(subprocess.Popen([hipcc, *flags, "-c", path, "-o", obj], stdout=subprocess.PIPE,
                                      stderr=subprocess.STDOUT, text=True))
    for p in procs:
        log = p.communicate()[0]
        assert p.returncode == 0, log
    exe = os.path.join(out, "host_checks")
    drv = os.path.join(ROOT, "tests", "host_checks.cpp")
    r = subprocess.run([hipcc, "-x", "c++", "-O1", "-g", "-std=c++17", *SANITIZE, "-I", os.path.join(ROOT, "include"),
                        "-c", drv, "-o", exe + ".o"], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([hipcc, "--offload-arch=gfx950", *SANITIZE, *objs, exe + ".o", "-o", exe],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    env.pop("WINO_WORKSPACE_LIMIT", None)
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0 and "host checks ok" in r.stdout, r.stdout + r.stderr
    assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr


def test_readme_c_example_compiles(tmp_path):
    """The C usage example of README.md compiles against include/wino.h."""
    import shutil
    import subprocess
    text = open(os.path.join(ROOT, "README.md")).read()
    blocks = re.findall(r"```c\n(.*?)```", text, flags=re.S)
    assert len(blocks) == 1
    src = tmp_path / "example.c"
    src.write_text(blocks[0])
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    r = subprocess.run([cc, "-std=c99", "-Wall", "-Werror", "-fsyntax-only", "-I", os.path.join(ROOT, "include"),
                        str(src)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
