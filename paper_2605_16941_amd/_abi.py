"""ctypes binding of libwino.so - argument marshalling only.

Every function here has the name of the C entry point it calls and forwards
plain pointers, sizes and a stream handle.  torch tensors are accepted where a
device pointer is expected (their data_ptr() is passed after a device / dtype /
contiguity check).  All computation happens in the HIP library; if it is not
built, importing this module fails loudly.
"""
from __future__ import annotations

import ctypes as C
import os

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libwino.so")


class WinoError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str = ""):
        self.status = status
        msg = f"{where}: {status_string(status)} ({status})"
        if detail:
            msg += f": {detail}"
        super().__init__(msg)


def _load():
    if not os.path.exists(_LIB_PATH):
        raise ImportError(
            f"libwino.so not found at {_LIB_PATH}; build it with "
            "`python paper_2605_16941_amd/build.py` (hipcc, gfx950)")
    # The library must run on the HIP runtime that allocates the device memory
    # it is handed.  torch ships its own copy of that runtime: loaded first,
    # it satisfies the library's runtime dependency; loaded after the library,
    # it joins the system copy the library pulled in, and pointers of one copy
    # are unknown to the other (wino_create then fails with WINO_ERR_HIP).
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    return C.CDLL(_LIB_PATH)


lib = _load()

N_KERNEL_CLASSES = 13
WINO_FLAG_NO_FORCE_TOP1 = 0x1
WINO_FLAG_NO_CAP_FILL = 0x2
KEEP, DRAFT, REMASK, FORCED, CAPFILL = 0, 1, 2, 3, 4
STATUS = {0: "WINO_OK", -1: "WINO_ERR_INVALID_ARG", -2: "WINO_ERR_SHAPE", -3: "WINO_ERR_HIP",
          -4: "WINO_ERR_NO_MEMORY", -5: "WINO_ERR_STEP_CAP", -6: "WINO_ERR_UNSUPPORTED"}


class wino_model_config(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d_model", C.c_int32), ("n_heads", C.c_int32),
                ("head_dim", C.c_int32), ("d_ff", C.c_int32), ("vocab", C.c_int32),
                ("rope_theta", C.c_float), ("rms_eps", C.c_float), ("act_precision", C.c_int32)]


ACT_BF16, ACT_FP16 = 0, 1


class wino_weights(C.Structure):
    _fields_ = [("tok_emb", C.c_void_p), ("attn_norm", C.POINTER(C.c_void_p)),
                ("w_qkv", C.POINTER(C.c_void_p)), ("w_o", C.POINTER(C.c_void_p)),
                ("ffn_norm", C.POINTER(C.c_void_p)), ("w_gate_up", C.POINTER(C.c_void_p)),
                ("w_down", C.POINTER(C.c_void_p)), ("final_norm", C.c_void_p),
                ("lm_head", C.c_void_p), ("lm_bias", C.c_void_p)]


class wino_params(C.Structure):
    _fields_ = [("batch", C.c_int32), ("prompt_len", C.c_int32), ("gen_len", C.c_int32),
                ("block_len", C.c_int32), ("mask_id", C.c_int32), ("tau1", C.c_float),
                ("tau2", C.c_float), ("max_steps", C.c_int32), ("flags", C.c_uint32),
                ("tokens_per_step", C.c_int32)]


class wino_row_stats(C.Structure):
    _fields_ = [("m_all", C.c_float), ("sumexp", C.c_float), ("z_best", C.c_float),
                ("z_target", C.c_float), ("argmax", C.c_int32), ("row_kind", C.c_int32)]


ROW_STATS_BYTES = C.sizeof(wino_row_stats)


class wino_row_loss(C.Structure):
    _fields_ = [("entropy", C.c_float), ("nll", C.c_float), ("conf", C.c_float), ("argmax", C.c_int32)]


ROW_LOSS_BYTES = C.sizeof(wino_row_loss)

_vp, _i32, _u32, _sz = C.c_void_p, C.c_int32, C.c_uint32, C.c_size_t
_P = C.POINTER
_protos = {
    "wino_create": (_i32, [_P(wino_model_config), _P(wino_weights), _i32, _i32, _P(_vp)]),
    "wino_destroy": (_i32, [_vp]),
    "wino_workspace_bytes": (_sz, [_P(wino_model_config), _i32, _i32]),
    "wino_step": (_i32, [_vp, _P(wino_params), _vp, _vp, _vp, _vp, _vp, _vp, _vp]),
    "wino_decode_block": (_i32, [_vp, _P(wino_params), _vp, _vp, _vp, _P(_i32), _vp]),
    "wino_decode": (_i32, [_vp, _P(wino_params), _vp, _vp, _vp, _vp, _i32, _P(_i32), _P(_i32), _vp]),
    "wino_epilogue_workspace_bytes": (_sz, [_i32, _i32, _i32]),
    "wino_epilogue": (_i32, [_P(wino_params), _i32, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "wino_epilogue_noalloc": (_i32, [_P(wino_params), _i32, _vp, _vp, _vp, _vp, _vp, _vp]),
    "wino_row_losses": (_i32, [_vp, _P(wino_params), _vp, _vp, _vp, _vp]),
    "wino_debug_logits": (_i32, [_vp, _P(wino_params), _vp, _vp, _vp, _vp]),
    "wino_debug_forward": (_i32, [_vp, _P(wino_params), _vp, _vp, _i32, _vp, _vp]),
    "wino_debug_gemm": (_i32, [_vp, _vp, _i32, _i32, _i32, _vp, _vp]),
    "wino_profile": (_i32, [_vp, _u32]),
    "wino_profile_read": (_i32, [_vp, _P(C.c_int64), _P(C.c_double), _P(C.c_double), _P(C.c_double)]),
    "wino_kernel_class_name": (C.c_char_p, [_i32]),
    "wino_status_string": (C.c_char_p, [_i32]),
    "wino_last_error": (C.c_char_p, [_vp]),
}
for _name, (_res, _args) in _protos.items():
    _f = getattr(lib, _name)
    _f.restype = _res
    _f.argtypes = _args

EXPORTED = tuple(_protos)


# ------------------------------------------------------------------ helpers
def _ptr(x, dtype=None, name="tensor"):
    """Device pointer of a torch tensor (checked), an int, or None."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    import torch
    if not isinstance(x, torch.Tensor):
        raise TypeError(f"{name}: expected a torch tensor, int pointer or None")
    if not x.is_cuda:
        raise ValueError(f"{name}: must be a device tensor")
    if dtype is not None and x.dtype != dtype:
        raise TypeError(f"{name}: dtype {x.dtype}, expected {dtype}")
    if not x.is_contiguous():
        raise ValueError(f"{name}: must be contiguous")
    return x.data_ptr()


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def status_string(s: int) -> str:
    return lib.wino_status_string(int(s)).decode()


def _check(status, where, ctx=None):
    if status != 0:
        detail = lib.wino_last_error(ctx).decode() if ctx else ""
        raise WinoError(status, where, detail)


def make_params(batch, prompt_len, gen_len, block_len, mask_id, tau1=0.7, tau2=0.9,
                max_steps=0, flags=0, tokens_per_step=0) -> wino_params:
    return wino_params(batch, prompt_len, gen_len, block_len, mask_id, tau1, tau2, max_steps, flags,
                       tokens_per_step)


# ------------------------------------------------------------------ entry points
def wino_workspace_bytes(cfg: wino_model_config, max_batch: int, max_seq: int) -> int:
    return int(lib.wino_workspace_bytes(C.byref(cfg), max_batch, max_seq))


def wino_create(cfg: wino_model_config, weights: wino_weights, max_batch: int, max_seq: int) -> int:
    out = C.c_void_p()
    s = lib.wino_create(C.byref(cfg), C.byref(weights), max_batch, max_seq, C.byref(out))
    if s != 0:
        raise WinoError(s, "wino_create", lib.wino_last_error(None).decode())
    return out.value


def wino_destroy(ctx: int) -> None:
    _check(lib.wino_destroy(ctx), "wino_destroy")


def wino_step(ctx, p: wino_params, tokens, block_start, block_steps=None, flags=None,
              n_masked=None, stats=None, stream=None) -> None:
    import torch
    _check(lib.wino_step(ctx, C.byref(p), _ptr(tokens, torch.int32, "tokens"),
                         _ptr(block_start, torch.int32, "block_start"),
                         _ptr(block_steps, torch.int32, "block_steps"),
                         _ptr(flags, torch.uint8, "flags"), _ptr(n_masked, torch.int32, "n_masked"),
                         _ptr(stats, None, "stats"), _stream(stream)), "wino_step", ctx)


def wino_decode_block(ctx, p: wino_params, tokens, block_start, final_step=None, stream=None):
    """Returns the per-sequence steps.  final_step as in wino_decode."""
    import torch
    steps = (C.c_int32 * p.batch)()
    fs = _ptr(final_step, torch.int32, "final_step") if final_step is not None else None
    _check(lib.wino_decode_block(ctx, C.byref(p), _ptr(tokens, torch.int32, "tokens"),
                                 _ptr(block_start, torch.int32, "block_start"), fs, steps,
                                 _stream(stream)), "wino_decode_block", ctx)
    return list(steps)


def wino_decode(ctx, p: wino_params, tokens, block_start, final_step=None, stream=None,
                block_steps=None, max_forwards=0):
    """Returns (per-sequence steps, batched forward passes).  final_step: int32
    [batch, gen_len] device tensor for the finalization steps, or None;
    block_steps: int32 [batch] device tensor (in/out) of steps already taken
    in each current block, or None; max_forwards > 0 stops early with a
    resumable state."""
    import torch
    steps = (C.c_int32 * p.batch)()
    fw = C.c_int32(0)
    fs = _ptr(final_step, torch.int32, "final_step") if final_step is not None else None
    _check(lib.wino_decode(ctx, C.byref(p), _ptr(tokens, torch.int32, "tokens"),
                           _ptr(block_start, torch.int32, "block_start"),
                           _ptr(block_steps, torch.int32, "block_steps"), fs, int(max_forwards), steps,
                           C.byref(fw), _stream(stream)), "wino_decode", ctx)
    return list(steps), fw.value


def wino_row_losses(ctx, p: wino_params, tokens, targets, out, stream=None) -> None:
    """WINO+ per-row quantities of training states (Sec. 5.2-5.3).  tokens int32
    [B, P+G], targets int32 [B, G], out: device buffer of B*G wino_row_loss
    (16 bytes each: entropy, nll, conf float32; argmax int32)."""
    import torch
    _check(lib.wino_row_losses(ctx, C.byref(p), _ptr(tokens, torch.int32, "tokens"),
                               _ptr(targets, torch.int32, "targets"), _ptr(out, None, "out"),
                               _stream(stream)), "wino_row_losses", ctx)


def wino_epilogue_workspace_bytes(batch: int, block_len: int, vocab: int) -> int:
    return int(lib.wino_epilogue_workspace_bytes(batch, block_len, vocab))


def wino_epilogue(p: wino_params, vocab: int, logits, cur_tokens, mask_bitmap, flags=None,
                  stats=None, workspace=None, workspace_bytes=None, stream=None) -> None:
    import torch
    if workspace_bytes is None:
        workspace_bytes = workspace.numel() * workspace.element_size()
    _check(lib.wino_epilogue(C.byref(p), vocab, _ptr(logits, torch.bfloat16, "logits"),
                             _ptr(cur_tokens, torch.int32, "cur_tokens"),
                             _ptr(mask_bitmap, torch.uint8, "mask_bitmap"),
                             _ptr(flags, torch.uint8, "flags"), _ptr(stats, None, "stats"),
                             _ptr(workspace, None, "workspace"), workspace_bytes,
                             _stream(stream)), "wino_epilogue")


EPILOGUE_NOALLOC_MAX_BYTES = 2 << 20


def wino_epilogue_noalloc(p: wino_params, vocab: int, logits, cur_tokens, mask_bitmap, flags=None,
                          stats=None, stream=None) -> None:
    """wino_epilogue with the library's own per-GPU scratch (no workspace)."""
    import torch
    _check(lib.wino_epilogue_noalloc(C.byref(p), vocab, _ptr(logits, torch.bfloat16, "logits"),
                                     _ptr(cur_tokens, torch.int32, "cur_tokens"),
                                     _ptr(mask_bitmap, torch.uint8, "mask_bitmap"),
                                     _ptr(flags, torch.uint8, "flags"), _ptr(stats, None, "stats"),
                                     _stream(stream)), "wino_epilogue_noalloc")


def wino_debug_logits(ctx, p: wino_params, tokens, block_start, logits, stream=None) -> None:
    import torch
    _check(lib.wino_debug_logits(ctx, C.byref(p), _ptr(tokens, torch.int32, "tokens"),
                                 _ptr(block_start, torch.int32, "block_start"),
                                 _ptr(logits, torch.float32, "logits"), _stream(stream)),
           "wino_debug_logits", ctx)


def wino_debug_forward(ctx, p: wino_params, tokens, block_start, n_sublayers, out, stream=None) -> None:
    import torch
    _check(lib.wino_debug_forward(ctx, C.byref(p), _ptr(tokens, torch.int32, "tokens"),
                                  _ptr(block_start, torch.int32, "block_start"), n_sublayers,
                                  _ptr(out, torch.float32, "out"), _stream(stream)),
           "wino_debug_forward", ctx)


def wino_debug_gemm(A, W, out, stream=None) -> None:
    """out = A W^T (fp32) with the backbone GEMM kernel; A [M,K], W [N,K] bf16."""
    import torch
    M, K = A.shape
    N = W.shape[0]
    if W.shape[1] != K or tuple(out.shape) != (M, N):
        raise ValueError("wino_debug_gemm: shape mismatch")
    _check(lib.wino_debug_gemm(_ptr(A, torch.bfloat16, "A"), _ptr(W, torch.bfloat16, "W"), M, N, K,
                               _ptr(out, torch.float32, "out"), _stream(stream)), "wino_debug_gemm")


def wino_profile(ctx, class_mask: int) -> None:
    _check(lib.wino_profile(ctx, class_mask), "wino_profile", ctx)


def wino_profile_read(ctx) -> dict:
    n = N_KERNEL_CLASSES
    la, ms, fl, by = (C.c_int64 * n)(), (C.c_double * n)(), (C.c_double * n)(), (C.c_double * n)()
    _check(lib.wino_profile_read(ctx, la, ms, fl, by), "wino_profile_read", ctx)
    return {wino_kernel_class_name(i): {"launches": la[i], "ms": ms[i], "flops": fl[i], "bytes": by[i]}
            for i in range(n)}


def wino_kernel_class_name(cls: int) -> str:
    return lib.wino_kernel_class_name(cls).decode()


def wino_status_string(s: int) -> str:
    return status_string(s)


def wino_last_error(ctx) -> str:
    return lib.wino_last_error(ctx).decode()
