"""Per-row quantities of the WINO+ trajectory-consistency objective.

Test infrastructure only (see the package docstring).

Sec. 5.3 (trajectory consistency objective): for a training state (Sec. 5.2, Eq. 5) - the
response with only the tokens finalized before step t revealed, everything
else the mask token - the model's prediction p at each response position
enters the losses through
* the negative log-likelihood of the target token, -log p(y_dagger) (the
  token term, Eq. 6),
* the Shannon entropy H(p) = -sum_v p(v) log p(v) over the vocabulary (the
  defer term, Eq. 6, and the sharpening term, Eq. 7),
* the greedy prediction y_hat and its confidence c, which select the sets R_t
  and C_t.  The prediction is read as in the draft rule: argmax over ids other
  than the mask id (lowest id on ties), the mask id kept in the normaliser.

The training state is a plain sequence (no shadow block): WINO+ replaces the
draft-and-verify rule, so this forward is the ordinary bidirectional one.
"""
from __future__ import annotations

import numpy as np

from . import model as M
from . import wino as W


def row_quantities(z: np.ndarray, target, mask_id: int):
    """From logits z [R, V]: (entropy [R], nll of target [R], conf [R], yhat [R]),
    each straight from its definition on p = softmax(z)."""
    p = W.softmax_rows(z)
    with np.errstate(divide="ignore", invalid="ignore"):
        plogp = np.where(p > 0, p * np.log(p), 0.0)
    entropy = -plogp.sum(axis=-1)
    target = np.asarray(target, dtype=np.int64)
    nll = -np.log(p[np.arange(p.shape[0]), target])
    conf, yhat = W.draft_stats(z, mask_id)
    return entropy, nll, conf, yhat


def state_logits(weights, cfg, tokens, prompt_len: int, act_round=None):
    """LM-head logits of the response rows of one sequence [G, V] under a plain
    bidirectional forward over prompt + response (positions 0..S-1)."""
    tokens = np.asarray(tokens, dtype=np.int64)
    s = tokens.shape[0]
    h = M.forward_hidden(weights, cfg, tokens, np.arange(s), np.ones((s, s), bool), act_round)
    return M.lm_logits(weights, h[prompt_len:])


def training_state(final, t_fin, t: int, prompt_len: int, mask_id: int):
    """Sec. 5.2, Eq. 5: the state before step t reveals exactly the response tokens
    with finalization step t_l < t (the prompt always); the rest are masks."""
    final = np.asarray(final, dtype=np.int64)
    t_fin = np.asarray(t_fin, dtype=np.int64)
    y = final.copy()
    resp = np.arange(final.shape[0]) >= prompt_len
    y[resp & (t_fin >= t)] = mask_id
    return y
