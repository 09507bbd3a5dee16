"""WINO (Wide-In, Narrow-Out) revokable decoding on MI355X (gfx950).

The decoding step - a bidirectional transformer forward over the prompt, the
response and the shadow verification block, the fused LM-head softmax
statistics and the draft / verify update - runs in the hand-written HIP
library ``libwino.so`` behind the C ABI of ``include/wino.h``.  This package is
the thin binding (``_abi``, same names as the C entry points) plus ``WinoModel``,
which holds a model's device weights and a library context.
"""
from __future__ import annotations

import ctypes as C

from . import _abi
from ._abi import (WinoError, make_params, wino_create, wino_debug_forward, wino_debug_logits,
                   wino_debug_gemm, wino_decode, wino_decode_block, wino_destroy, wino_epilogue,
                   wino_epilogue_noalloc,
                   wino_epilogue_workspace_bytes, wino_kernel_class_name, wino_last_error,
                   wino_profile, wino_profile_read, wino_row_losses, wino_status_string, wino_step,
                   wino_workspace_bytes)

ACT_BF16, ACT_FP16 = _abi.ACT_BF16, _abi.ACT_FP16

__all__ = ["WinoModel", "WinoError", "make_params", "ACT_BF16", "ACT_FP16", "wino_create", "wino_destroy", "wino_step",
           "wino_decode_block", "wino_decode", "wino_epilogue", "wino_epilogue_noalloc", "wino_epilogue_workspace_bytes",
           "wino_debug_logits", "wino_debug_forward", "wino_debug_gemm", "wino_profile", "wino_profile_read",
           "wino_kernel_class_name", "wino_status_string", "wino_last_error",
           "wino_row_losses", "wino_workspace_bytes"]


def model_config(cfg, act_precision: int = _abi.ACT_BF16) -> _abi.wino_model_config:
    """C config from any object with the backbone fields (e.g. a preset)."""
    return _abi.wino_model_config(cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.head_dim, cfg.d_ff,
                                  cfg.vocab, float(cfg.rope_theta), float(cfg.rms_eps), act_precision)


class WinoModel:
    """Device weights (bf16 torch tensors on one GPU) and a library context.

    ``weights`` is a dict: tok_emb [V,d], layers (list of dicts with attn_norm,
    w_qkv, w_o, ffn_norm, w_gate_up, w_down), final_norm, lm_head [V,d] and
    lm_bias (fp32 [V] or None).  The tensors must stay alive with the model.
    ``act_precision``: ACT_BF16 (default) or ACT_FP16 (fp16 activations; the
    context then also holds fp16 copies of the weight matrices).
    """

    def __init__(self, cfg, weights: dict, max_batch: int, max_seq: int,
                 act_precision: int = _abi.ACT_BF16):
        import torch
        self.cfg = cfg
        self.ccfg = model_config(cfg, act_precision)
        self.weights = weights
        n = cfg.n_layers

        def arr(key):
            a = (C.c_void_p * n)()
            for i, lw in enumerate(weights["layers"]):
                a[i] = _abi._ptr(lw[key], torch.bfloat16, key)
            return a

        self._arrays = {k: arr(k) for k in ("attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate_up",
                                            "w_down")}
        bias = weights.get("lm_bias")
        self.cweights = _abi.wino_weights(
            _abi._ptr(weights["tok_emb"], torch.bfloat16, "tok_emb"),
            self._arrays["attn_norm"], self._arrays["w_qkv"], self._arrays["w_o"],
            self._arrays["ffn_norm"], self._arrays["w_gate_up"], self._arrays["w_down"],
            _abi._ptr(weights["final_norm"], torch.bfloat16, "final_norm"),
            _abi._ptr(weights["lm_head"], torch.bfloat16, "lm_head"),
            _abi._ptr(bias, torch.float32, "lm_bias") if bias is not None else None)
        self.ctx = wino_create(self.ccfg, self.cweights, max_batch, max_seq)
        self.max_batch, self.max_seq = max_batch, max_seq

    def close(self):
        if getattr(self, "ctx", None):
            wino_destroy(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
