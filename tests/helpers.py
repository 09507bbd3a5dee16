"""Shared test helpers: weights on the device, oracle runs on the same inputs,
and the comparison rules (logits tolerance, decision margin)."""
from __future__ import annotations

import numpy as np
import torch

import wino_inputs as wi

# Tolerances fixed by the parity contract: logits to 2e-2 max relative error
# (infinity-norm ratio per row, bf16 path vs float64 oracle); decisions and ids
# bit-exact wherever the deciding probability is more than 1e-3 away from its
# threshold (and, for ids, the top-2 probability gap exceeds 1e-3).
LOGIT_TOL = 2e-2
MARGIN = 1e-3


def to_device(w: dict, device="cuda") -> dict:
    out = {k: (v.to(device) if isinstance(v, torch.Tensor) else v) for k, v in w.items() if k != "layers"}
    out["layers"] = [None if lw is None else {k: v.to(device) for k, v in lw.items()} for lw in w["layers"]]
    return out


def to_cpu(w: dict) -> dict:
    return to_device(w, "cpu")


def rowwise_rel_err(got: np.ndarray, ref: np.ndarray) -> float:
    """max over rows of max|g - r| / max|r|."""
    got = np.asarray(got, dtype=np.float64).reshape(-1, ref.shape[-1])
    ref = np.asarray(ref, dtype=np.float64).reshape(-1, ref.shape[-1])
    num = np.max(np.abs(got - ref), axis=-1)
    den = np.maximum(np.max(np.abs(ref), axis=-1), 1e-30)
    return float(np.max(num / den))


def decided_mask(margin: np.ndarray, gap: np.ndarray | None, masked: np.ndarray) -> np.ndarray:
    """Positions whose decision (and drafted id) the oracle fixes robustly."""
    ok = margin > MARGIN
    if gap is not None:
        ok &= ~(masked & (gap <= MARGIN))
    return ok


def forced_is_robust(conf: np.ndarray, masked: np.ndarray) -> bool:
    """A forced draft picks the top conf among masked positions; robust if the
    top-2 gap exceeds the margin."""
    c = np.sort(conf[masked])
    return len(c) < 2 or (c[-1] - c[-2]) > MARGIN
