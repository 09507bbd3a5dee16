"""Backbone forward over the WINO extended sequence, in float64.

Test infrastructure only (see the package docstring).

The paper treats the mask predictor p_theta(. | X, Y) as a black box (Sec. 3;
LLaDA-8B and MMaDA-8B in Sec. 6.1).  The architecture here is the synthetic
LLaDA-shaped transformer the workloads use: token embedding, per layer
pre-RMSNorm bidirectional multi-head attention with rotate-half RoPE and a
pre-RMSNorm SwiGLU feed-forward, both with residual adds, then a final RMSNorm
and the LM head (+ an optional per-vocab bias).  No causal mask, no KV cache
(the paper keeps caching out of scope, Sec. 2.2).

What WINO itself changes in the forward (Sec. 4.2.2):
* the shadow block Y_shad of L_b mask tokens is appended after Y_right;
* shadow position j takes the position id of y_cur,j;
* rows of Y_left / Y_cur / Y_right never attend to Y_shad;
* shadow row j attends to every row except y_cur,j (it does see all of Y_shad,
  including itself - the paper excludes only the corresponding Y_cur position).

Optional ``act_round`` rounds activations at the points where a bf16 pipeline
materialises them: the normed inputs of the backbone's matrix products, q/k/v
after RoPE, the unnormalised attention probabilities that multiply v (relative
to the row maximum; the normalising sum is taken before rounding), the
attention output and the SwiGLU product.  The final normed
hidden state feeding the LM head is not rounded (a pipeline that keeps it as a
hi+lo pair of bf16 values carries 16 mantissa bits there).  With
``act_round=None`` everything stays in float64.
"""
from __future__ import annotations

import numpy as np
import torch


def f64(t) -> np.ndarray:
    """float64 numpy copy of a torch tensor (any dtype, any device) or array."""
    if isinstance(t, torch.Tensor):
        return t.detach().to("cpu", torch.float64).numpy()
    return np.asarray(t, dtype=np.float64)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round to bfloat16 (via float32), round-to-nearest-even, back to float64."""
    x32 = np.ascontiguousarray(x, dtype=np.float32)
    bits = x32.view(np.uint32).astype(np.uint64)
    bits = (bits + 0x7FFF + ((bits >> 16) & 1)) & 0xFFFF0000
    return bits.astype(np.uint32).view(np.float32).astype(np.float64)


def rmsnorm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """y = x / sqrt(mean(x^2) + eps) * g over the last axis."""
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * g


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def rope_cos_sin(pos: np.ndarray, head_dim: int, theta: float):
    """Angles pos * theta^(-2i/hd) for the hd/2 frequency pairs."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    inv_freq = theta ** (-2.0 * i / head_dim)
    ang = np.outer(np.asarray(pos, dtype=np.float64), inv_freq)
    return np.cos(ang), np.sin(ang)


def apply_rope(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """Rotate-half RoPE on x [T, H, hd]: pair (i, i+hd/2) rotated by angle_i."""
    half = x.shape[-1] // 2
    x1, x2 = x[..., :half], x[..., half:]
    c, s = cos[:, None, :], sin[:, None, :]
    return np.concatenate([x1 * c - x2 * s, x2 * c + x1 * s], axis=-1)


def wino_positions(seq_len: int, block_len: int, c0: int) -> np.ndarray:
    """Position ids of the extended sequence (Sec. 4.2.2, "Position IDs").

    Rows 0..S-1 keep their index; shadow row j reuses the id of y_cur,j = c0+j.
    """
    return np.concatenate([np.arange(seq_len), c0 + np.arange(block_len)]).astype(np.int64)


def wino_allowed(seq_len: int, block_len: int, c0: int) -> np.ndarray:
    """Boolean [T, T] attention mask, allowed[i, k] = row i may attend key k.

    Sec. 4.2.2, "Attention Mask": non-shadow rows see all non-shadow rows and no
    shadow row; shadow row j sees every row except y_cur,j (index c0+j).
    """
    t = seq_len + block_len
    a = np.zeros((t, t), dtype=bool)
    a[:seq_len, :seq_len] = True
    a[seq_len:, :] = True
    j = np.arange(block_len)
    a[seq_len + j, c0 + j] = False
    return a


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, allowed: np.ndarray,
              p_round=None) -> np.ndarray:
    """softmax(q k^T / sqrt(hd), restricted to allowed keys) v, per head.

    q, k, v: [T, H, hd]; allowed: [T, T] bool.  Returns [T, H, hd].  With
    p_round, the unnormalised probabilities exp(s - max) are rounded before
    they multiply v (the sum that normalises them is not).
    """
    hd = q.shape[-1]
    qh = np.ascontiguousarray(q.transpose(1, 0, 2))
    kh = np.ascontiguousarray(k.transpose(1, 2, 0))
    vh = np.ascontiguousarray(v.transpose(1, 0, 2))
    s = np.matmul(qh, kh) / np.sqrt(hd)
    s = np.where(allowed[None, :, :], s, -np.inf)
    s = s - np.max(s, axis=-1, keepdims=True)
    p = np.exp(s)
    l = np.sum(p, axis=-1, keepdims=True)
    if p_round is not None:
        p = p_round(p)
    return (np.matmul(p, vh) / l).transpose(1, 0, 2)


def attention_sublayer(x: np.ndarray, lw: dict, cfg, cos, sin, allowed, act_round=None) -> np.ndarray:
    """x + Attn(RMSNorm(x)) W_o^T on the residual stream x [T, d] (float64)."""
    rnd = act_round or (lambda a: a)
    t, d = x.shape
    nh, hd = cfg.n_heads, cfg.head_dim
    h = rnd(rmsnorm(x, f64(lw["attn_norm"]), cfg.rms_eps))
    qkv = h @ f64(lw["w_qkv"]).T
    q = qkv[:, :d].reshape(t, nh, hd)
    k = qkv[:, d:2 * d].reshape(t, nh, hd)
    v = qkv[:, 2 * d:].reshape(t, nh, hd)
    q = rnd(apply_rope(q, cos, sin))
    k = rnd(apply_rope(k, cos, sin))
    v = rnd(v)
    o = rnd(attention(q, k, v, allowed, act_round).reshape(t, d))
    return x + o @ f64(lw["w_o"]).T


def ffn_sublayer(x: np.ndarray, lw: dict, cfg, act_round=None) -> np.ndarray:
    """x + (SiLU(h W_g^T) * h W_u^T) W_d^T with h = RMSNorm(x)."""
    rnd = act_round or (lambda a: a)
    ff = cfg.d_ff
    h = rnd(rmsnorm(x, f64(lw["ffn_norm"]), cfg.rms_eps))
    gu = h @ f64(lw["w_gate_up"]).T
    a = rnd(silu(gu[:, :ff]) * gu[:, ff:])
    return x + a @ f64(lw["w_down"]).T


def layer_forward(x: np.ndarray, lw: dict, cfg, cos, sin, allowed, act_round=None) -> np.ndarray:
    """One transformer layer: attention sublayer then FFN sublayer."""
    x = attention_sublayer(x, lw, cfg, cos, sin, allowed, act_round)
    return ffn_sublayer(x, lw, cfg, act_round)


def forward_residual(weights: dict, cfg, tokens, pos, allowed, act_round=None,
                     n_layers: int | None = None, n_sublayers: int | None = None) -> np.ndarray:
    """Residual stream [T, d] after the embedding and the first n_layers layers
    (or the first n_sublayers sublayers: attention and FFN of each layer)."""
    tokens = np.asarray(tokens, dtype=np.int64)
    x = f64(weights["tok_emb"][torch.as_tensor(tokens)])
    cos, sin = rope_cos_sin(pos, cfg.head_dim, cfg.rope_theta)
    if n_sublayers is None:
        n_sublayers = 2 * (cfg.n_layers if n_layers is None else n_layers)
    for i in range(n_sublayers):
        lw = weights["layers"][i // 2]
        if i % 2 == 0:
            x = attention_sublayer(x, lw, cfg, cos, sin, allowed, act_round)
        else:
            x = ffn_sublayer(x, lw, cfg, act_round)
    return x


def forward_hidden(weights: dict, cfg, tokens, pos, allowed, act_round=None,
                   n_layers: int | None = None) -> np.ndarray:
    """Final-normed hidden states [T, d] for token ids ``tokens`` [T]."""
    x = forward_residual(weights, cfg, tokens, pos, allowed, act_round, n_layers)
    return rmsnorm(x, f64(weights["final_norm"]), cfg.rms_eps)


def lm_logits(weights: dict, h_rows: np.ndarray) -> np.ndarray:
    """z = h W_lm^T (+ bias) for the given hidden rows [R, d] -> [R, V]."""
    z = h_rows @ f64(weights["lm_head"]).T
    if weights.get("lm_bias") is not None:
        z = z + f64(weights["lm_bias"])
    return z


def extended_inputs(tokens, prompt_len: int, gen_len: int, block_len: int,
                    block_start: int, mask_id: int):
    """Extended sequence [Y_left, Y_cur, Y_right, Y_shad] of one sequence.

    ``tokens`` holds prompt + generation (S = P + G ids); ``block_start`` is the
    generation-relative start of Y_cur.  Returns (ext_tokens [T], pos [T],
    allowed [T,T], c0) with c0 the absolute index of y_cur,1.
    """
    s = prompt_len + gen_len
    c0 = prompt_len + block_start
    ext = np.concatenate([np.asarray(tokens, dtype=np.int64)[:s],
                          np.full(block_len, mask_id, dtype=np.int64)])
    return ext, wino_positions(s, block_len, c0), wino_allowed(s, block_len, c0), c0
