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
    assert C.sizeof(abi.wino_model_config) == 32
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
    # supported shape, but null weight pointers
    assert abi.lib.wino_create(C.byref(cfg), C.byref(w), 1, 112, C.byref(out)) == -1
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

