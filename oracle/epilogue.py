"""WINO decision straight from given logits of the current and shadow blocks.

Test infrastructure only (see the package docstring).

Input logits [B, 2*L_b, V]: rows 0..L_b-1 are the current block Y_cur, rows
L_b..2*L_b-1 the shadow block Y_shad (Sec. 4.2.2).  Per position l of
sequence b the decision of Eq. 4 reads the current row when y_cur,l is the mask
(Eq. 2: max probability and argmax over ids other than the mask id) and the
shadow row at the current token otherwise (Eq. 3).  The forced draft of the
most confident masked position applies when nothing clears tau1 (Eq. 1).
"""
from __future__ import annotations

import numpy as np

from . import model as M
from . import wino as W


def decide(logits, cur_tokens, mask_id: int, tau1: float, tau2: float, force_top1: bool = True):
    """Returns dict with new tokens [B,Lb], mask bitmap [B,Lb] (1 = mask after
    the step), flags, conf, yhat, s and the margin of the deciding quantity."""
    cur_tokens = np.asarray(cur_tokens, dtype=np.int64)
    b_n, lb = cur_tokens.shape
    out = {k: [] for k in ("tokens", "bitmap", "flags", "conf", "yhat", "s", "margin", "gap")}
    for b in range(b_n):
        z = M.f64(logits[b])
        z_cur, z_sh = z[:lb], z[lb:]
        conf, yhat = W.draft_stats(z_cur, mask_id)
        cur = cur_tokens[b]
        s = W.verify_stats(z_sh, np.where(cur == mask_id, 0, cur))
        new, flags = W.wino_update(cur, conf, yhat, s, mask_id, tau1, tau2, force_top1)
        masked = cur == mask_id
        p = W.softmax_rows(z_cur)
        p[:, mask_id] = -1.0
        top = np.sort(p, axis=-1)
        out["tokens"].append(new)
        out["bitmap"].append((new == mask_id).astype(np.int64))
        out["flags"].append(flags)
        out["conf"].append(conf)
        out["yhat"].append(yhat)
        out["s"].append(s)
        out["margin"].append(np.where(masked, np.abs(conf - tau1), np.abs(s - tau2)))
        out["gap"].append(top[:, -1] - top[:, -2])
    return {k: np.stack(v) for k, v in out.items()}
