"""Seeded synthetic inputs for WINO decoding (weights, prompts, epilogue logits).

This module is shared by the CPU oracle, the tests and the benchmark.  It holds
no arithmetic of the decoding method itself: only model-shape presets and a
counter-based random generator that produces the same bytes on any torch device.

Generator
---------
Every tensor has an integer stream id.  Element ``c`` of stream ``s`` under seed
``seed`` is derived from ``hash32`` (the "lowbias32" integer finaliser:
xorshift-multiply rounds with constants 0x7feb352d and 0x846ca68b), applied to
the counter xor a per-stream key.  Two hashes give a 53-bit uniform in (0, 1);
normals use the Box-Muller cosine branch in float64, then round to the target
dtype (bf16 by round-to-nearest-even).  Integer steps are exact on every device,
so a slice of any tensor can be regenerated independently of the rest.

Model presets follow the workloads the WINO evaluation is scaled to: a tiny
2-layer model, an 8B-parameter LLaDA-shaped model and an MMaDA-shaped model
whose vocabulary is extended by 8192 image-code ids.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, asdict, replace

import torch

_M32 = 0xFFFFFFFF


# --------------------------------------------------------------------------
# model presets
# --------------------------------------------------------------------------
@dataclass(frozen=True)
class ModelConfig:
    n_layers: int
    d_model: int
    n_heads: int
    head_dim: int
    d_ff: int
    vocab: int
    mask_id: int
    rope_theta: float
    rms_eps: float = 1e-5
    text_vocab: int = 0  # ids below this are text ids (0 = all of vocab)

    def as_dict(self):
        return asdict(self)


PRESETS = {
    # 2 layers, d=256, 4 heads of 64, SwiGLU 704, vocab 4096, mask id 4095
    "tiny": ModelConfig(2, 256, 4, 64, 704, 4096, 4095, 10000.0),
    # LLaDA-8B shape: 32 layers, d=4096, 32x128 heads, FFN 12288, vocab 126464
    "llada8b": ModelConfig(32, 4096, 32, 128, 12288, 126464, 126463, 500000.0),
    # same backbone, vocab extended by 8192 image-code ids; text mask id kept
    "mmada8b": ModelConfig(32, 4096, 32, 128, 12288, 134656, 126463, 500000.0,
                           text_vocab=126464),
}


def preset(name: str, **overrides) -> ModelConfig:
    cfg = PRESETS[name]
    return replace(cfg, **overrides) if overrides else cfg


# --------------------------------------------------------------------------
# counter-based generator
# --------------------------------------------------------------------------
def _hash32_int(x: int) -> int:
    x &= _M32
    x ^= x >> 16
    x = (x * 0x7FEB352D) & _M32
    x ^= x >> 15
    x = (x * 0x846CA68B) & _M32
    x ^= x >> 16
    return x


def _hash32(x: torch.Tensor) -> torch.Tensor:
    """lowbias32 on int64 tensors holding values in [0, 2^32)."""
    x = x ^ (x >> 16)
    x = (x * 0x7FEB352D) & _M32
    x = x ^ (x >> 15)
    x = (x * 0x846CA68B) & _M32
    x = x ^ (x >> 16)
    return x


def _stream_keys(seed: int, stream: int):
    k1 = _hash32_int((seed * 0x9E3779B1 + stream * 0x85EBCA77 + 0x27D4EB2F) & _M32)
    k2 = _hash32_int(k1 ^ 0x68E31DA4)
    return k1, k2


_CHUNK = 1 << 26


def uniform(seed: int, stream: int, n: int, device="cpu", offset: int = 0) -> torch.Tensor:
    """float64 uniforms in (0,1) for counters offset..offset+n-1 of a stream."""
    if offset + n > (1 << 32):
        raise ValueError("counter range exceeds 2^32")
    k1, k2 = _stream_keys(seed, stream)
    out = torch.empty(n, dtype=torch.float64, device=device)
    for s in range(0, n, _CHUNK):
        e = min(n, s + _CHUNK)
        c = torch.arange(offset + s, offset + e, dtype=torch.int64, device=device)
        a = _hash32(c ^ k1)
        b = _hash32(a ^ k2)
        hi = (a >> 5).to(torch.float64)
        lo = (b >> 6).to(torch.float64)
        out[s:e] = (hi * 67108864.0 + lo + 0.5) * (1.0 / 9007199254740992.0)
    return out


def normal(seed: int, stream: int, n: int, device="cpu", offset: int = 0) -> torch.Tensor:
    """float64 standard normals (Box-Muller, cosine branch)."""
    out = torch.empty(n, dtype=torch.float64, device=device)
    for s in range(0, n, _CHUNK):
        e = min(n, s + _CHUNK)
        u1 = uniform(seed, 2 * stream, e - s, device, offset + s)
        u2 = uniform(seed, 2 * stream + 1, e - s, device, offset + s)
        out[s:e] = torch.sqrt(-2.0 * torch.log(u1)) * torch.cos((2.0 * math.pi) * u2)
    return out


def randint(seed: int, stream: int, n: int, lo: int, hi: int, device="cpu") -> torch.Tensor:
    """int64 uniform in [lo, hi)."""
    u = uniform(seed, stream, n, device)
    return (torch.floor(u * (hi - lo)).to(torch.int64) + lo).clamp_(lo, hi - 1)


def _normal_bf16(seed, stream, shape, std, device, chunk_rows=None):
    n = math.prod(shape)
    out = torch.empty(n, dtype=torch.bfloat16, device=device)
    step = _CHUNK
    for s in range(0, n, step):
        e = min(n, s + step)
        out[s:e] = (normal(seed, stream, e - s, device, s) * std).to(torch.bfloat16)
    return out.view(*shape)


# --------------------------------------------------------------------------
# weights
# --------------------------------------------------------------------------
STREAM_TOK_EMB = 1
STREAM_LM_HEAD = 2
STREAM_ZIPF_PERM = 3
STREAM_FINAL_NORM = 4


def _layer_stream(layer: int, which: int) -> int:
    return 100 + 10 * layer + which


LAYER_TENSORS = ("attn_norm", "w_qkv", "w_o", "ffn_norm", "w_gate_up", "w_down")


def zipf_bias(vocab: int, seed: int = 0, s: float = 1.1, scale: float = 4.0,
              device="cpu") -> torch.Tensor:
    """Per-vocab fp32 bias: scale * log of a Zipf(s) probability of a seeded rank.

    The rank of id v is pi(v), a seeded permutation of 1..V (argsort of uniforms).
    bias_v = scale * (-s*ln(pi_v) - ln(H_{V,s})).
    """
    u = uniform(seed, STREAM_ZIPF_PERM, vocab, device)
    order = torch.argsort(u, stable=True)
    rank = torch.empty(vocab, dtype=torch.float64, device=device)
    rank[order] = torch.arange(1, vocab + 1, dtype=torch.float64, device=device)
    ks = torch.arange(1, vocab + 1, dtype=torch.float64)
    log_h = math.log(float(torch.sum(ks ** (-s))))
    return (scale * (-s * torch.log(rank) - log_h)).to(torch.float32)


def layer_weights(cfg: ModelConfig, layer: int, seed: int = 0, device="cpu",
                  std: float = 0.02, gain_std: float = 0.0) -> dict:
    d, f = cfg.d_model, cfg.d_ff

    def gain(which):
        if gain_std == 0.0:
            return torch.ones(d, dtype=torch.bfloat16, device=device)
        g = 1.0 + gain_std * normal(seed, _layer_stream(layer, which), d, device)
        return g.to(torch.bfloat16)

    return {
        "attn_norm": gain(0),
        # rows: q (d) | k (d) | v (d); each row is one output feature
        "w_qkv": _normal_bf16(seed, _layer_stream(layer, 1), (3 * d, d), std, device),
        "w_o": _normal_bf16(seed, _layer_stream(layer, 2), (d, d), std, device),
        "ffn_norm": gain(3),
        # rows: gate (F) | up (F)
        "w_gate_up": _normal_bf16(seed, _layer_stream(layer, 4), (2 * f, d), std, device),
        "w_down": _normal_bf16(seed, _layer_stream(layer, 5), (d, f), std, device),
    }


def model_weights(cfg: ModelConfig, seed: int = 0, device="cpu", std: float = 0.02,
                  lm_head_std: float | None = None, gain_std: float = 0.0,
                  zipf_scale: float = 4.0, layers=None) -> dict:
    """All weights of a model preset.

    lm_head_std defaults to 0.5/sqrt(d) ("literal" init); the "wide" variant
    passes sqrt(0.5/sqrt(d)).  ``layers`` restricts which layers are generated
    (others are None), for tests that need a single layer of a large model.
    """
    d, v = cfg.d_model, cfg.vocab
    if lm_head_std is None:
        lm_head_std = 0.5 / math.sqrt(d)
    if layers is None:
        layers = range(cfg.n_layers)
    layers = set(layers)
    w = {
        "tok_emb": _normal_bf16(seed, STREAM_TOK_EMB, (v, d), std, device),
        "layers": [layer_weights(cfg, l, seed, device, std, gain_std) if l in layers else None
                   for l in range(cfg.n_layers)],
        "final_norm": (torch.ones(d, dtype=torch.bfloat16, device=device) if gain_std == 0.0
                       else (1.0 + gain_std * normal(seed, STREAM_FINAL_NORM, d, device))
                       .to(torch.bfloat16)),
        "lm_head": _normal_bf16(seed, STREAM_LM_HEAD, (v, d), lm_head_std, device),
        "lm_bias": zipf_bias(v, seed, scale=zipf_scale, device=device) if zipf_scale else None,
    }
    return w


def wide_lm_head_std(cfg: ModelConfig) -> float:
    return math.sqrt(0.5 / math.sqrt(cfg.d_model))


# --------------------------------------------------------------------------
# prompts and decode state
# --------------------------------------------------------------------------
STREAM_PROMPT = 1000


def prompts(cfg: ModelConfig, batch: int, prompt_len: int, seed: int = 0,
            image_prefix: int = 0, device="cpu") -> torch.Tensor:
    """int32 [batch, prompt_len] token ids; sequence b uses stream 1000+b.

    Text ids are uniform in [0, mask_id) when the mask id closes the text range,
    otherwise uniform over text ids other than the mask id.  The first
    ``image_prefix`` ids of each prompt are uniform image-code ids
    [text_vocab, vocab).
    """
    text_hi = cfg.text_vocab if cfg.text_vocab else cfg.vocab
    out = torch.empty(batch, prompt_len, dtype=torch.int64, device=device)
    for b in range(batch):
        ids = randint(seed, STREAM_PROMPT + b, prompt_len, 0, text_hi - 1, device)
        ids = ids + (ids >= cfg.mask_id).to(torch.int64)  # skip the mask id
        if image_prefix:
            img = randint(seed, STREAM_PROMPT + 500 + b, image_prefix, text_hi, cfg.vocab, device)
            ids[:image_prefix] = img
        out[b] = ids
    return out.to(torch.int32)


def initial_tokens(prompt: torch.Tensor, gen_len: int, mask_id: int) -> torch.Tensor:
    """[batch, prompt_len + gen_len] int32: prompt followed by gen_len mask ids."""
    b = prompt.shape[0]
    gen = torch.full((b, gen_len), mask_id, dtype=torch.int32, device=prompt.device)
    return torch.cat([prompt.to(torch.int32), gen], dim=1).contiguous()


# --------------------------------------------------------------------------
# standalone epilogue inputs: bf16 logits [B, 2*Lb, V] and the current block
# --------------------------------------------------------------------------
STREAM_EPI_NOISE = 2000
STREAM_EPI_PEAK_ID = 2001
STREAM_EPI_PEAK_H = 2002
STREAM_EPI_STATE = 2003
STREAM_EPI_RANDTOK = 2004


def epilogue_inputs(batch: int, block_len: int, vocab: int, mask_id: int, seed: int = 2,
                    heights=(0.0, 12.0), device="cpu"):
    """Logits rows 0..Lb-1 are the current block, rows Lb..2Lb-1 the shadow block.

    Each row is N(0,1) noise plus one planted peak (uniform non-mask id, height
    uniform in ``heights``), rounded to bf16.  The block state per position is
    drawn u ~ U(0,1): u < 0.5 -> mask id; 0.5 <= u < 0.75 -> the shadow row's
    planted id; otherwise a uniform id that is neither the mask nor the planted id.
    Returns (logits bf16 [B,2Lb,V], cur_tokens int32 [B,Lb], peak_ids int64 [B,2Lb]).
    """
    rows = batch * 2 * block_len
    n = rows * vocab
    logits = torch.empty(n, dtype=torch.bfloat16, device=device)
    for s in range(0, n, _CHUNK):
        e = min(n, s + _CHUNK)
        logits[s:e] = normal(seed, STREAM_EPI_NOISE, e - s, device, s).to(torch.float32).to(torch.bfloat16)
    logits = logits.view(batch, 2 * block_len, vocab)
    pid = randint(seed, STREAM_EPI_PEAK_ID, rows, 0, vocab - 1, device)
    pid = pid + (pid >= mask_id).to(torch.int64)
    h = uniform(seed, STREAM_EPI_PEAK_H, rows, device) * (heights[1] - heights[0]) + heights[0]
    flat = logits.view(rows, vocab)
    r = torch.arange(rows, device=device)
    flat[r, pid] = (flat[r, pid].to(torch.float64) + h).to(torch.float32).to(torch.bfloat16)
    pid = pid.view(batch, 2 * block_len)

    u = uniform(seed, STREAM_EPI_STATE, batch * block_len, device).view(batch, block_len)
    rnd = randint(seed, STREAM_EPI_RANDTOK, batch * block_len, 0, vocab - 2, device).view(batch, block_len)
    shadow_pid = pid[:, block_len:]
    # random id avoiding mask id and the planted id of the shadow row
    lo_excl = torch.minimum(shadow_pid, torch.full_like(shadow_pid, mask_id))
    hi_excl = torch.maximum(shadow_pid, torch.full_like(shadow_pid, mask_id))
    rnd = rnd + (rnd >= lo_excl).to(torch.int64)
    rnd = rnd + (rnd >= hi_excl).to(torch.int64)
    cur = torch.where(u < 0.5, torch.full_like(rnd, mask_id),
                      torch.where(u < 0.75, shadow_pid, rnd))
    return logits, cur.to(torch.int32), pid


__all__ = [
    "ModelConfig", "PRESETS", "preset", "uniform", "normal", "randint", "zipf_bias",
    "layer_weights", "model_weights", "wide_lm_head_std", "prompts", "initial_tokens",
    "epilogue_inputs", "LAYER_TENSORS",
]
