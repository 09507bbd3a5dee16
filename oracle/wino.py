"""WINO draft / verify decision, block loop and semi-autoregressive decode.

Test infrastructure only (see the package docstring).

Paper passages followed:
* Sec. 3 (Preliminary), Eq. 1: high-confidence greedy decoding - unmask the
  most confident masked position.  Used here as the forced draft when no
  masked position clears tau1.
* Sec. 3, semi-autoregressive decoding: split the response into blocks and
  decode them left to right.
* Sec. 4.2.1, Eq. 2 (draft): a masked y_cur,l becomes argmax_v p(y_cur,l = v)
  when max_v p(y_cur,l = v) > tau1.
* Sec. 4.2.2, Eq. 3 (verify): an unmasked y_cur,l is re-masked when the shadow
  row's probability of the current token, p(y_shad,l = y_cur,l), is < tau2.
* Sec. 4.2.3, Eq. 4: both rules read the previous state y^(k-1) and act in one
  forward; iterate until Y_cur has no mask token.
* Sec. 5.1: a position's finalization step is the first step from which its
  token no longer changes (the WINO+ trajectory data).
* Sec. 3 and the comparison with naive parallel sampling (Sec. 6.3): the
  baselines unmask a fixed number M of tokens per step - the M most confident
  masked positions of the block, M = 1 being Eq. 1 - with no threshold and no
  verification (``tokens_per_step`` > 0 selects this mode; it needs no step
  cap, a block takes ceil(L_b / M) steps).

Readings of points the paper leaves open (each is a parameter or flag):
* decoding is greedy (argmax, temperature 1, no sampling noise);
* the draft's max / argmax run over ids other than the mask id (the mask id
  stays in the softmax normaliser); argmax ties go to the lowest id;
* comparisons are strict, as printed (> tau1, < tau2);
* forced draft: when a mask remains in Y_cur but no position clears tau1, the
  most confident masked position is drafted (Eq. 1; ties -> lowest position);
* step cap: a block may take at most ``max_steps`` forwards (default L_b); on
  the last allowed step verification is skipped and every remaining mask is
  drafted, so a draft / re-mask cycle cannot run forever;
* the block ends as soon as Y_cur has no mask after a step (no extra
  verify-only forward); Y_left and Y_right are never modified;
* a batch is a set of independent sequences, each with its own block cursor.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import model as M

KEEP, DRAFT, REMASK, FORCED, CAPFILL = 0, 1, 2, 3, 4


@dataclass
class Params:
    prompt_len: int
    gen_len: int
    block_len: int
    mask_id: int
    tau1: float = 0.7
    tau2: float = 0.9
    max_steps: int = 0        # per block; 0 -> block_len
    force_top1: bool = True
    cap_fill: bool = True
    tokens_per_step: int = 0  # > 0: baseline decoding, M tokens per step (Sec. 3)

    @property
    def cap(self) -> int:
        return self.max_steps if self.max_steps > 0 else self.block_len


def softmax_rows(z: np.ndarray) -> np.ndarray:
    z = np.asarray(z, dtype=np.float64)
    e = np.exp(z - np.max(z, axis=-1, keepdims=True))
    return e / np.sum(e, axis=-1, keepdims=True)


def draft_stats(z_cur: np.ndarray, mask_id: int):
    """Eq. 2 quantities per row: (confidence, argmax id) over ids != mask id."""
    p = softmax_rows(z_cur)
    p_ex = p.copy()
    p_ex[:, mask_id] = -1.0
    yhat = np.argmax(p_ex, axis=-1)           # first maximum = lowest id
    conf = p_ex[np.arange(p.shape[0]), yhat]
    return conf, yhat.astype(np.int64)


def verify_stats(z_shad: np.ndarray, cur_tokens: np.ndarray) -> np.ndarray:
    """Eq. 3 quantity per row: p_shad,l evaluated at the current token y_cur,l."""
    p = softmax_rows(z_shad)
    return p[np.arange(p.shape[0]), np.asarray(cur_tokens, dtype=np.int64)]


def wino_update(cur, conf, yhat, s, mask_id, tau1, tau2, force_top1=True, cap_now=False):
    """Eq. 4 on one block.  Returns (new block tokens, per-position flags).

    ``conf``/``yhat`` are read only at masked positions, ``s`` only at unmasked
    ones (both from the previous state, Eq. 4).
    """
    cur = np.asarray(cur, dtype=np.int64)
    masked = cur == mask_id
    flags = np.full(cur.shape, KEEP, dtype=np.int64)
    if cap_now:
        draft = masked.copy()
        remask = np.zeros_like(masked)
        flags[draft] = CAPFILL
    else:
        draft = masked & (np.asarray(conf) > tau1)
        remask = (~masked) & (np.asarray(s) < tau2)
        flags[draft] = DRAFT
        flags[remask] = REMASK
        if force_top1 and masked.any() and not draft.any():
            cand = np.where(masked, np.asarray(conf, dtype=np.float64), -np.inf)
            l_star = int(np.argmax(cand))     # lowest position on ties
            draft[l_star] = True
            flags[l_star] = FORCED
    new = cur.copy()
    new[draft] = np.asarray(yhat)[draft]
    new[remask] = mask_id
    return new, flags


def topm_update(cur, conf, yhat, mask_id, m):
    """Baseline step (Sec. 3): unmask the m most confident masked positions of
    the block (Eq. 1 for m = 1, naive parallel sampling for m > 1); equal
    confidences go to the lower position.  Returns (new block, flags)."""
    cur = np.asarray(cur, dtype=np.int64)
    masked = np.flatnonzero(cur == mask_id)
    order = masked[np.argsort(-np.asarray(conf, dtype=np.float64)[masked], kind="stable")]
    pick = order[:m]
    flags = np.full(cur.shape, KEEP, dtype=np.int64)
    flags[pick] = DRAFT
    new = cur.copy()
    new[pick] = np.asarray(yhat)[pick]
    return new, flags


class ModelProvider:
    """Probabilities for Eq. 4 from the synthetic backbone (one sequence)."""

    def __init__(self, weights, cfg, act_round=None):
        self.w, self.cfg, self.act_round = weights, cfg, act_round

    def __call__(self, tokens, prm: Params, block_start: int):
        ext, pos, allowed, c0 = M.extended_inputs(tokens, prm.prompt_len, prm.gen_len,
                                                  prm.block_len, block_start, prm.mask_id)
        h = M.forward_hidden(self.w, self.cfg, ext, pos, allowed, self.act_round)
        s_len = prm.prompt_len + prm.gen_len
        z_cur = M.lm_logits(self.w, h[c0:c0 + prm.block_len])
        z_sh = M.lm_logits(self.w, h[s_len:s_len + prm.block_len])
        return z_cur, z_sh


@dataclass
class StepResult:
    tokens: np.ndarray        # [P+G] after the step
    flags: np.ndarray         # [Lb]
    conf: np.ndarray          # [Lb] draft confidence (cur rows)
    yhat: np.ndarray          # [Lb] draft argmax
    s: np.ndarray             # [Lb] verify probability (shadow rows at current token)
    margin: np.ndarray        # [Lb] distance of the deciding quantity from its threshold
    top2_gap: np.ndarray      # [Lb] p(top1) - p(top2) over ids != mask, cur rows
    z_cur: np.ndarray
    z_shad: np.ndarray


def step(provider, tokens, prm: Params, block_start: int, block_steps: int) -> StepResult:
    """One WINO step (Eq. 4) for one sequence."""
    tokens = np.asarray(tokens, dtype=np.int64).copy()
    c0 = prm.prompt_len + block_start
    cur = tokens[c0:c0 + prm.block_len].copy()
    z_cur, z_sh = provider(tokens, prm, block_start)
    conf, yhat = draft_stats(z_cur, prm.mask_id)
    cur_for_verify = np.where(cur == prm.mask_id, 0, cur)
    s = verify_stats(z_sh, cur_for_verify)
    cap_now = prm.cap_fill and (block_steps + 1 >= prm.cap)
    masked = cur == prm.mask_id
    if prm.tokens_per_step > 0:
        # the fixed schedule ends a block in ceil(L_b / M) <= L_b steps: no cap
        new, flags = topm_update(cur, conf, yhat, prm.mask_id, prm.tokens_per_step)
        # the selection flips only if the M-th and (M+1)-th confidences swap
        c = np.sort(conf[masked])[::-1]
        m = prm.tokens_per_step
        half_gap = (c[m - 1] - c[m]) / 2 if len(c) > m else np.inf
        margin = np.where(masked, half_gap, np.inf)
    else:
        new, flags = wino_update(cur, conf, yhat, s, prm.mask_id, prm.tau1, prm.tau2,
                                 prm.force_top1, cap_now)
        margin = np.where(masked, np.abs(conf - prm.tau1), np.abs(s - prm.tau2))
    tokens[c0:c0 + prm.block_len] = new
    p = softmax_rows(z_cur)
    p[:, prm.mask_id] = -1.0
    top = np.sort(p, axis=-1)
    gap = top[:, -1] - top[:, -2]
    return StepResult(tokens, flags, conf, yhat, s, margin, gap, z_cur, z_sh)


def decode_block(provider, tokens, prm: Params, block_start: int, trace=None):
    """Iterate Eq. 4 on the block at ``block_start`` until it holds no mask."""
    tokens = np.asarray(tokens, dtype=np.int64).copy()
    c0 = prm.prompt_len + block_start
    steps = 0
    while True:
        r = step(provider, tokens, prm, block_start, steps)
        tokens = r.tokens
        steps += 1
        if trace is not None:
            trace.append(r)
        if not np.any(tokens[c0:c0 + prm.block_len] == prm.mask_id):
            return tokens, steps
        if prm.cap_fill is False and steps >= prm.cap:
            return tokens, steps


def finalization_steps(states, prompt_len: int) -> np.ndarray:
    """Sec. 5.1 (verified trajectories): for the states Y^(0..K) of one
    sequence's decode, t_l = min{t : y_l^(j) = y_l^(K) for every j >= t};
    prompt positions get 0.  Written from the definition: scan t upward."""
    Y = np.asarray(states, dtype=np.int64)          # [K + 1, P + G]
    K = Y.shape[0] - 1
    final = Y[K]
    t = np.zeros(Y.shape[1], dtype=np.int64)
    for l in range(prompt_len, Y.shape[1]):
        for cand in range(K + 1):
            if np.all(Y[cand:, l] == final[l]):
                t[l] = cand
                break
    return t


def decode(provider, tokens, prm: Params, trace=None):
    """Semi-autoregressive decode of the whole generation (Sec. 3).

    Returns (tokens [P+G], per-block step counts).
    """
    if prm.gen_len % prm.block_len:
        raise ValueError("gen_len must be a multiple of block_len")
    tokens = np.asarray(tokens, dtype=np.int64).copy()
    steps = []
    for b in range(prm.gen_len // prm.block_len):
        tokens, n = decode_block(provider, tokens, prm, b * prm.block_len, trace)
        steps.append(n)
    return tokens, steps
