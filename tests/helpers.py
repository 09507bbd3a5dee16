"""Shared test helpers: weights on the device, oracle runs on the same inputs,
and the comparison rules (logits tolerance, decision margin)."""
from __future__ import annotations

import numpy as np
import torch

import wino_inputs as wi
from oracle import model as M
from oracle import wino as W

# Tolerances fixed by the parity contract: logits to 2e-2 max relative error
# (infinity-norm ratio per row, bf16 path vs float64 oracle); decisions and ids
# bit-exact wherever the deciding probability is more than 1e-3 away from its
# threshold (and, for ids, the top-2 probability gap exceeds 1e-3).
LOGIT_TOL = 2e-2
MARGIN = 1e-3

STATS_DT = np.dtype([("m_all", "<f4"), ("sumexp", "<f4"), ("z_best", "<f4"), ("z_target", "<f4"),
                     ("argmax", "<i4"), ("row_kind", "<i4")])


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


def decided_mask(margin: np.ndarray, gap: np.ndarray | None, masked: np.ndarray, m: float = MARGIN) -> np.ndarray:
    """Positions whose decision (and drafted id) the oracle fixes robustly."""
    ok = margin > m
    if gap is not None:
        ok &= ~(masked & (gap <= m))
    return ok


def forced_is_robust(conf: np.ndarray, masked: np.ndarray, m: float = MARGIN) -> bool:
    """A forced draft picks the top conf among masked positions; robust if the
    top-2 gap exceeds the margin."""
    c = np.sort(conf[masked])
    return len(c) < 2 or (c[-1] - c[-2]) > m


# ------------------------------------------------------------------ workloads
def tiny(variant="wide", seed=0, gain_std=0.1, **kw):
    """The tiny model's weights.  'literal': LM head std 0.5/sqrt(d) with the
    Zipf bias (every block drafts in one step at tau1 = 0.7); 'wide': LM head
    std sqrt(0.5/sqrt(d)); 'sharp': backbone std 0.1 (position-dependent
    attention), wide LM head and a Zipf bias of scale 2, on which WINO drafts,
    re-masks and re-drafts within a block (the iterating workload); 'midmask':
    the wide model with mask id 1000 and the largest LM-head bias on it."""
    if variant == "midmask":
        # the mask id inside the vocabulary, with the largest LM-head bias:
        # it holds the maximum of most logits rows, which counts in every
        # normaliser but never as a draft
        cfg = wi.preset("tiny", mask_id=1000, **kw)
        w = wi.model_weights(cfg, seed=seed, lm_head_std=wi.wide_lm_head_std(cfg), gain_std=gain_std)
        w["lm_bias"] = w["lm_bias"].clone()
        w["lm_bias"][cfg.mask_id] = float(w["lm_bias"].max()) + 2.0
        return cfg, w
    cfg = wi.preset("tiny", **kw)
    if variant == "sharp":
        return cfg, wi.model_weights(cfg, seed=seed, std=0.1, lm_head_std=wi.wide_lm_head_std(cfg),
                                     gain_std=gain_std, zipf_scale=2.0)
    lhs = wi.wide_lm_head_std(cfg) if variant == "wide" else None
    return cfg, wi.model_weights(cfg, seed=seed, lm_head_std=lhs, gain_std=gain_std)


def fp64_provider(w, cfg):
    """The oracle that judges decisions: everything in float64."""
    return W.ModelProvider(w, cfg)


def kernel_precision_provider(w, cfg):
    """Diagnostic only: the float64 oracle with bf16 rounding at the points
    where the kernels hold bf16 activations.  Its distance to the float64
    oracle (delta) measures what precision that arithmetic has."""
    return W.ModelProvider(w, cfg, act_round=M.round_bf16)


def oracle_params(prm_c, **kw):
    return W.Params(prm_c.prompt_len, prm_c.gen_len, prm_c.block_len, prm_c.mask_id,
                    float(np.float32(prm_c.tau1)), float(np.float32(prm_c.tau2)), prm_c.max_steps, **kw)


def deciding(r, cur, mask_id):
    """The probability each position's decision reads: the draft confidence
    (Eq. 2) where the token is the mask, else the verify probability (Eq. 3)."""
    masked = cur == mask_id
    return np.where(masked, r.conf, r.s)


# The bf16-activation pipeline's probability error on the tiny literal and
# wide models (measured up to 5.4e-3 on the wide one; test_contract_teacher_forced
# asserts the bound).  A forced draft (and a baseline decoder's top-M choice)
# ranks the confidences of different positions, each carrying that error, so a
# ranking is fixed only by gaps above twice the bound.
PROB_ERR = 1e-2
RANK_GAP = 2 * PROB_ERR


def robust_positions(r, cur, mask_id, tau1, margin=MARGIN, rank_gap=RANK_GAP):
    """Positions whose flag and token the oracle step r fixes at `margin`:
    the deciding probability lies more than `margin` from its threshold and,
    for drafted ids, the top-2 gap exceeds it; under the cap fill only the
    drafted ids matter.  When no masked confidence clears tau1 the forced draft
    (Eq. 1) picks one masked position by rank: masked positions count only if
    every masked confidence is more than `margin` below tau1 and the top one
    leads the next by more than max(margin, rank_gap)."""
    masked = cur == mask_id
    ok = (r.margin > margin) & ~(masked & (r.top2_gap <= margin))
    if np.any(r.flags == W.CAPFILL):
        return ~masked | (r.top2_gap > margin)
    confm = r.conf[masked]
    if masked.any() and not np.any(confm > tau1 + margin):
        c = np.sort(confm)
        gap_ok = len(c) < 2 or c[-1] - c[-2] > max(margin, rank_gap)
        if not (np.all(confm < tau1 - margin) and gap_ok):
            ok &= ~masked
    return ok


def check_forced_choice(gpu_tok, gpu_flags, r, cur, mask_id, tau1, c0, lb, label, margin=MARGIN,
                        rank_gap=RANK_GAP):
    """Where the oracle forced a draft whose position is not fixed by rank,
    the GPU's choice must still be valid: nothing cleared tau1 on either side
    (every masked confidence is more than `margin` below tau1), exactly one
    masked position was forced, its oracle confidence is within rank_gap of
    the top one, and its id is the oracle's argmax where that is robust."""
    masked = cur == mask_id
    forced = np.flatnonzero(r.flags == W.FORCED)
    if len(forced) == 0 or not np.all(r.conf[masked] < tau1 - margin):
        return 0
    g = np.flatnonzero(gpu_flags[:lb] == W.FORCED)
    assert len(g) == 1 and masked[g[0]], f"{label}: GPU forced {g.tolist()}"
    j = int(g[0])
    assert r.conf[j] >= r.conf[masked].max() - rank_gap, f"{label}: forced position {j} ranks too low"
    if r.top2_gap[j] > margin:
        assert gpu_tok[c0 + j] == r.yhat[j], f"{label}: forced id differs"
    return 1


def compare_step(gpu_tok, gpu_flags, r, cur, mask_id, tau1, c0, lb, label="", margin=MARGIN, verifying=True):
    """Assert GPU decisions equal the oracle's at every robust position (see
    robust_positions), and that a forced draft the ranking does not fix is a
    valid one.  Returns {flag: compared count} with flag the oracle's
    decision, plus 'verify_keep' for unmasked positions that went through
    Eq. 3 and were kept (verifying: tau2 > 0; never on a cap-fill step) and
    'forced_valid' for forced drafts checked for validity only."""
    ok = robust_positions(r, cur, mask_id, tau1, margin)
    masked = cur == mask_id
    verifying = verifying and not np.any(r.flags == W.CAPFILL)
    counts = {f: 0 for f in ("keep", "draft", "remask", "forced", "capfill", "verify_keep", "forced_valid")}
    names = {W.KEEP: "keep", W.DRAFT: "draft", W.REMASK: "remask", W.FORCED: "forced", W.CAPFILL: "capfill"}
    for l in range(lb):
        if not ok[l]:
            continue
        assert gpu_flags[l] == r.flags[l], f"{label} pos {l}: flag {gpu_flags[l]} != {r.flags[l]}"
        assert gpu_tok[c0 + l] == r.tokens[c0 + l], f"{label} pos {l}: token differs"
        counts[names[int(r.flags[l])]] += 1
        if verifying and not masked[l] and r.flags[l] == W.KEEP:
            counts["verify_keep"] += 1
    if masked.any() and not ok[masked].any():
        counts["forced_valid"] += check_forced_choice(gpu_tok, gpu_flags, r, cur, mask_id, tau1, c0, lb, label,
                                                      margin)
    return counts


def add_counts(total, c):
    for k, v in c.items():
        total[k] = total.get(k, 0) + v
    return total


def batch_tokens(cfg, B, p, g, seed=0, fill=None):
    pr = wi.prompts(cfg, B, p, seed=seed)
    tok = wi.initial_tokens(pr, g, cfg.mask_id).numpy().astype(np.int64)
    if fill:
        rng = np.random.default_rng(seed)
        for b in range(B):
            for (lo, hi, frac) in fill:
                idx = np.arange(p + lo, p + hi)
                sel = idx[rng.random(len(idx)) < frac]
                tok[b, sel] = rng.integers(0, cfg.mask_id, len(sel))
    return tok


def gpu_step(P, model, prm, tokens, block_start, block_steps):
    """One wino_step on the given state; returns (tokens, flags, n_masked,
    block_steps, stats) on the host."""
    B, lb = tokens.shape[0], prm.block_len
    tok = torch.tensor(tokens, dtype=torch.int32, device="cuda")
    bs = torch.tensor(block_start, dtype=torch.int32, device="cuda")
    st = torch.tensor(block_steps, dtype=torch.int32, device="cuda")
    flags = torch.full((B, lb), 255, dtype=torch.uint8, device="cuda")
    nm = torch.full((B,), -7, dtype=torch.int32, device="cuda")
    stats = torch.zeros(B * lb * STATS_DT.itemsize, dtype=torch.uint8, device="cuda")
    P.wino_step(model.ctx, prm, tok, bs, st, flags, nm, stats)
    torch.cuda.synchronize()
    return (tok.cpu().numpy(), flags.cpu().numpy(), nm.cpu().numpy(), st.cpu().numpy(),
            stats.cpu().numpy().view(STATS_DT).reshape(B, lb))


def oracle_trajectory(prov, tokens0, prm):
    """[(tokens before, block_start, block_steps, StepResult)] of a full
    decode of one sequence, and its final tokens."""
    out = []
    tok = np.asarray(tokens0, dtype=np.int64).copy()
    for blk in range(prm.gen_len // prm.block_len):
        bs, steps = blk * prm.block_len, 0
        c0 = prm.prompt_len + bs
        if not np.any(tok[c0:c0 + prm.block_len] == prm.mask_id):
            continue
        while True:
            r = W.step(prov, tok, prm, bs, steps)
            out.append((tok.copy(), bs, steps, r))
            tok = r.tokens
            steps += 1
            if not np.any(tok[c0:c0 + prm.block_len] == prm.mask_id):
                break
    return out, tok


def step_is_robust(t, bs, r, prm, margin=MARGIN):
    """Every position of the oracle step is fixed at `margin` (the whole new
    state is determined), including a forced draft's position."""
    c0 = prm.prompt_len + bs
    cur = t[c0:c0 + prm.block_len]
    ok = robust_positions(r, cur, prm.mask_id, prm.tau1, margin)
    return bool(np.all(ok))


def decode_prefix_compare(P, model, prm_c, prm, prov, tok0, label="", margin_of=None, teacher_forced=False):
    """Semi-autoregressive decode through wino_decode one batched forward at a
    time (max_forwards = 1, the state carried in tokens / block_start /
    block_steps), compared with the oracle's trajectory of each sequence.

    Free-running (default): while the oracle's steps are robust, the GPU
    state after every forward must equal the oracle's; the first non-robust
    oracle step is where the two may legitimately part (the divergence step),
    and comparison of that sequence stops there.  Teacher-forced: before
    every forward the GPU state is set to the oracle's, and the robust
    positions of each step are compared (compare_step).
    margin_of(t, bs, steps, r) gives the margin per step (default 1e-3).
    Returns (compared steps per sequence, divergence step per sequence or
    None, GPU forwards, oracle trajectories)."""
    B = tok0.shape[0]
    trajs = [oracle_trajectory(prov, tok0[b], prm)[0] for b in range(B)]
    tok = torch.tensor(tok0, dtype=torch.int32, device="cuda")
    bs = torch.zeros(B, dtype=torch.int32, device="cuda")
    bsteps = torch.zeros(B, dtype=torch.int32, device="cuda")
    compared = [0] * B
    diverged = [None] * B
    forwards = 0
    lb = prm.block_len
    while True:
        k = forwards
        if teacher_forced:
            if all(k >= len(t) for t in trajs):
                break
            for b in range(B):
                if k < len(trajs[b]):
                    t, bs_o, st_o, _ = trajs[b][k]
                    tok[b] = torch.from_numpy(t.astype(np.int32))
                    bs[b], bsteps[b] = bs_o, st_o
                else:
                    bs[b] = prm_c.gen_len
        elif torch.all(bs >= prm_c.gen_len):
            break
        _, fw = P.wino_decode(model.ctx, prm_c, tok, bs, block_steps=bsteps, max_forwards=1)
        torch.cuda.synchronize()
        assert fw == 1
        forwards += 1
        got = tok.cpu().numpy()
        for b in range(B):
            if diverged[b] is not None or k >= len(trajs[b]):
                continue
            t, bs_o, st_o, r = trajs[b][k]
            m = margin_of(t, bs_o, st_o, r) if margin_of else MARGIN
            if teacher_forced:
                c0 = prm.prompt_len + bs_o
                ok = robust_positions(r, t[c0:c0 + lb], prm.mask_id, prm.tau1, m)
                assert np.array_equal(got[b][c0:c0 + lb][ok], r.tokens[c0:c0 + lb][ok]), \
                    f"{label} seq {b} step {k}: tokens differ at robust positions"
                outside = np.ones(len(t), bool)
                outside[c0:c0 + lb] = False
                assert np.array_equal(got[b][outside], t[outside])
                compared[b] += int(ok.sum())
                continue
            if not step_is_robust(t, bs_o, r, prm, m):
                diverged[b] = k
                continue
            assert np.array_equal(got[b], r.tokens), f"{label} seq {b} step {k}: state differs from the oracle"
            compared[b] += 1
        assert forwards <= prm_c.gen_len * 4, "decode did not finish"
    if not teacher_forced:
        for b in range(B):
            if diverged[b] is None:
                assert compared[b] == len(trajs[b]), f"{label} seq {b}: {compared[b]} of {len(trajs[b])} steps"
    return compared, diverged, forwards, trajs
