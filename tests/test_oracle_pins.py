"""Pins of the CPU oracle against facts fixed by the paper and by mathematics.

None of these re-derives an oracle formula: each check uses a closed form, a
property the paper states for the shadow block (Sec. 4.2.2), a special case
that reduces to another algorithm (Eq. 1 greedy decoding, full-parallel
decoding), an independent library routine, or hand-worked decision cases.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import wino_inputs as wi
from oracle import model as M
from oracle import wino as W
from oracle import epilogue as E

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def tiny_cfg(**kw):
    return wi.preset("tiny", **kw)


@pytest.fixture(scope="module")
def tiny_weights():
    return wi.model_weights(tiny_cfg(), seed=0, gain_std=0.1)


# ---------------------------------------------------------------- primitives
def test_round_bf16_matches_torch_and_ties_to_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5e-3, 3.14159, 65504.0, 1e-30])
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(M.round_bf16(x), ref)
    assert M.round_bf16(np.array([1.0 + 2 ** -8]))[0] == 1.0          # tie -> even
    assert M.round_bf16(np.array([1.0 + 3 * 2 ** -8]))[0] == 1.0 + 2 ** -6


def test_rmsnorm_constant_vector_closed_form():
    d, c, eps = 64, -0.37, 1e-5
    g = np.linspace(0.5, 1.5, d)
    y = M.rmsnorm(np.full((1, d), c), g, eps)
    np.testing.assert_allclose(y[0], g * c / math.sqrt(c * c + eps), rtol=1e-14)


def test_silu_known_values():
    x = np.array([0.0, 1.0, -1.0, 30.0, -30.0])
    want = np.array([0.0, 0.7310585786300049, -0.2689414213699951, 30.0, -30.0 * math.exp(-30.0)])
    np.testing.assert_allclose(M.silu(x), want, rtol=1e-12, atol=1e-300)


def test_rope_is_complex_rotation():
    rng = np.random.default_rng(1)
    t, h, hd, theta = 7, 3, 16, 500000.0
    x = rng.standard_normal((t, h, hd))
    pos = np.array([0, 1, 5, 100, 543, 2047, 9])
    cos, sin = M.rope_cos_sin(pos, hd, theta)
    y = M.apply_rope(x, cos, sin)
    z = x[..., :hd // 2] + 1j * x[..., hd // 2:]
    freq = np.array([theta ** (-(2.0 * i) / hd) for i in range(hd // 2)])
    rot = np.exp(1j * pos[:, None] * freq[None, :])[:, None, :]
    zr = z * rot
    np.testing.assert_allclose(y[..., :hd // 2], zr.real, atol=1e-12)
    np.testing.assert_allclose(y[..., hd // 2:], zr.imag, atol=1e-12)


def test_rope_scores_depend_on_position_difference_only():
    rng = np.random.default_rng(2)
    hd = 32
    q = rng.standard_normal((1, 1, hd))
    k = rng.standard_normal((1, 1, hd))
    def score(pq, pk):
        cq, sq = M.rope_cos_sin(np.array([pq]), hd, 10000.0)
        ck, sk = M.rope_cos_sin(np.array([pk]), hd, 10000.0)
        return float(np.sum(M.apply_rope(q, cq, sq) * M.apply_rope(k, ck, sk)))
    assert abs(score(3, 10) - score(103, 110)) < 1e-10
    assert abs(score(3, 10) - score(10, 3)) > 1e-6


# ---------------------------------------------------------------- attention mask
def test_wino_mask_structure():
    s, lb, c0 = 10, 3, 6
    a = M.wino_allowed(s, lb, c0)
    assert a.shape == (13, 13)
    assert a[:s, :s].all() and not a[:s, s:].any()          # never see the shadow
    for j in range(lb):
        row = a[s + j]
        assert not row[c0 + j]                               # excluded: y_cur,j
        assert row.sum() == s + lb - 1                       # everything else
        assert row[s:].all()                                 # all shadow rows, itself too
    pos = M.wino_positions(s, lb, c0)
    np.testing.assert_array_equal(pos[s:], [6, 7, 8])


def test_attention_with_zero_query_averages_allowed_values():
    """q = 0 makes every allowed score equal: the output is the plain mean of
    the allowed value rows - a closed form that pins which keys are visible."""
    rng = np.random.default_rng(3)
    s, lb, c0, h, hd = 9, 3, 4, 2, 8
    t = s + lb
    a = M.wino_allowed(s, lb, c0)
    q = np.zeros((t, h, hd))
    k = rng.standard_normal((t, h, hd))
    v = rng.standard_normal((t, h, hd))
    o = M.attention(q, k, v, a)
    np.testing.assert_allclose(o[:s], np.broadcast_to(v[:s].mean(0), (s, h, hd)), atol=1e-13)
    for j in range(lb):
        keep = [i for i in range(t) if i != c0 + j]
        np.testing.assert_allclose(o[s + j], v[keep].mean(0), atol=1e-13)


def test_attention_matches_torch_sdpa_float64():
    rng = np.random.default_rng(4)
    s, lb, c0, h, hd = 20, 4, 12, 3, 16
    t = s + lb
    a = M.wino_allowed(s, lb, c0)
    q, k, v = (rng.standard_normal((t, h, hd)) for _ in range(3))
    o = M.attention(q, k, v, a)
    tq, tk, tv = (torch.from_numpy(x.transpose(1, 0, 2).copy()) for x in (q, k, v))
    ref = torch.nn.functional.scaled_dot_product_attention(
        tq, tk, tv, attn_mask=torch.from_numpy(a)).numpy().transpose(1, 0, 2)
    np.testing.assert_allclose(o, ref, atol=1e-12)


# ---------------------------------------------------------------- whole-model properties (Sec. 4.2.2)
def _ext_hidden(w, cfg, tokens, p, g, lb, bs, n_layers=None):
    ext, pos, allowed, c0 = M.extended_inputs(tokens, p, g, lb, bs, cfg.mask_id)
    return M.forward_hidden(w, cfg, ext, pos, allowed, n_layers=n_layers), c0


def _tiny_tokens(cfg, p=12, g=16, seed=0, filled=6):
    pr = wi.prompts(cfg, 1, p, seed=seed)[0].numpy().astype(np.int64)
    gen = np.full(g, cfg.mask_id, dtype=np.int64)
    rng = np.random.default_rng(seed)
    gen[:filled] = rng.integers(0, cfg.mask_id, filled)
    return np.concatenate([pr, gen])


def test_shadow_block_does_not_change_other_rows(tiny_weights):
    """Appending Y_shad leaves every non-shadow output unchanged (Sec. 4.2.2)."""
    cfg = tiny_cfg()
    p, g, lb = 12, 16, 4
    tok = _tiny_tokens(cfg, p, g)
    tok[p + 4: p + 6] = [5, 6]                     # partially decoded block
    h_ext, _ = _ext_hidden(tiny_weights, cfg, tok, p, g, lb, 4)
    s = p + g
    h_plain = M.forward_hidden(tiny_weights, cfg, tok, np.arange(s), np.ones((s, s), bool))
    np.testing.assert_allclose(h_ext[:s], h_plain, atol=1e-12, rtol=1e-12)


def test_single_shadow_row_of_masked_position_equals_current_row(tiny_weights):
    """L_b = 1 and y_cur masked: the shadow row sees the same (token, position)
    multiset as y_cur itself, so its output must equal y_cur's in every layer.
    Pins the shadow position id and the shadow row seeing itself."""
    cfg = tiny_cfg()
    p, g, lb = 12, 16, 1
    tok = _tiny_tokens(cfg, p, g)
    bs = 7
    tok[p + bs] = cfg.mask_id
    h, c0 = _ext_hidden(tiny_weights, cfg, tok, p, g, lb, bs)
    np.testing.assert_allclose(h[p + g], h[c0], atol=1e-12)


def test_shadow_row_blind_to_its_own_position_with_one_layer(tiny_weights):
    """One layer: shadow row l cannot see y_cur,l (no leakage, Sec. 4.2.2) but
    does see every other y_cur,j."""
    cfg = tiny_cfg()
    p, g, lb, bs = 12, 16, 4, 4
    tok = _tiny_tokens(cfg, p, g, filled=8)
    s = p + g
    h0, c0 = _ext_hidden(tiny_weights, cfg, tok, p, g, lb, bs, n_layers=1)
    tok2 = tok.copy()
    tok2[c0 + 2] = (tok2[c0 + 2] + 17) % cfg.mask_id
    h1, _ = _ext_hidden(tiny_weights, cfg, tok2, p, g, lb, bs, n_layers=1)
    np.testing.assert_allclose(h1[s + 2], h0[s + 2], atol=1e-13)
    for j in (0, 1, 3):
        assert np.max(np.abs(h1[s + j] - h0[s + j])) > 1e-6


def test_constant_position_offset_leaves_outputs_unchanged(tiny_weights):
    cfg = tiny_cfg()
    p, g, lb, bs = 12, 16, 4, 8
    tok = _tiny_tokens(cfg, p, g)
    ext, pos, allowed, _ = M.extended_inputs(tok, p, g, lb, bs, cfg.mask_id)
    h0 = M.forward_hidden(tiny_weights, cfg, ext, pos, allowed)
    h1 = M.forward_hidden(tiny_weights, cfg, ext, pos + 1000, allowed)
    np.testing.assert_allclose(h1, h0, atol=1e-8)


def test_zeroed_branches_reduce_to_embedding_head():
    """With W_o = W_down = 0 every layer is the identity, so the logits are
    rmsnorm(E[tok]) * g_f @ W_lm^T + bias."""
    cfg = tiny_cfg()
    w = wi.model_weights(cfg, seed=5, gain_std=0.2)
    for lw in w["layers"]:
        lw["w_o"] = torch.zeros_like(lw["w_o"])
        lw["w_down"] = torch.zeros_like(lw["w_down"])
    tok = _tiny_tokens(cfg, 8, 8)
    ext, pos, allowed, c0 = M.extended_inputs(tok, 8, 8, 4, 0, cfg.mask_id)
    h = M.forward_hidden(w, cfg, ext, pos, allowed)
    z = M.lm_logits(w, h)
    e = w["tok_emb"].double()[torch.from_numpy(ext)]
    hn = e / torch.sqrt((e * e).mean(-1, keepdim=True) + cfg.rms_eps) * w["final_norm"].double()
    zref = hn @ w["lm_head"].double().T + w["lm_bias"].double()
    np.testing.assert_allclose(z, zref.numpy(), rtol=1e-10, atol=1e-10)


# ---------------------------------------------------------------- confidences
def test_draft_stats_exclude_mask_and_break_ties_low():
    z = np.zeros((3, 8))
    z[0, 7] = 5.0; z[0, 2] = 4.0            # mask id 7 is the top logit
    z[1, 3] = 2.0; z[1, 5] = 2.0            # tie -> lowest id
    conf, yhat = W.draft_stats(z, mask_id=7)
    assert yhat[0] == 2 and yhat[1] == 3 and yhat[2] == 0
    p0 = math.exp(4.0) / (math.exp(5.0) + math.exp(4.0) + 6)   # mask stays in the normaliser
    assert abs(conf[0] - p0) < 1e-15
    assert abs(conf[2] - 1 / 8) < 1e-15


def test_softmax_rows_sum_to_one_and_confidence_bounds():
    rng = np.random.default_rng(6)
    z = rng.standard_normal((5, 1000)) * 4
    p = W.softmax_rows(z)
    np.testing.assert_allclose(p.sum(-1), 1.0, atol=1e-13)
    conf, _ = W.draft_stats(z, mask_id=999)
    assert np.all(conf >= 1 / 1000) and np.all(conf <= 1)


# ---------------------------------------------------------------- decision rule
def test_golden_decision_cases():
    g = json.load(open(os.path.join(GOLDEN, "decision_cases.json")))
    for c in g["cases"]:
        new, flags = W.wino_update(c["cur"], c["conf"], c["yhat"], c["s"], g["mask_id"],
                                   c["tau1"], c["tau2"])
        assert new.tolist() == c["new"], c["name"]
        assert flags.tolist() == c["flags"], c["name"]
    for c in g["cap_cases"]:
        new, flags = W.wino_update(c["cur"], c["conf"], c["yhat"], c["s"], g["mask_id"],
                                   c["tau1"], c["tau2"], cap_now=True)
        assert new.tolist() == c["new"], c["name"]
        assert flags.tolist() == c["flags"], c["name"]


class Scripted:
    """Probability provider from a function of (tokens, block_start)."""

    def __init__(self, fn):
        self.fn = fn

    def __call__(self, tokens, prm, block_start):
        return self.fn(np.asarray(tokens), prm, block_start)


def test_livelock_ends_at_the_step_cap():
    """A block where verification always fails would cycle forever: position 0
    never clears tau1 (so it is forced in when it is the only mask left), the
    others always clear it, and every unmasked token is re-masked.  The cap
    fills the remaining masks on the last allowed step (L_b = 4)."""
    v, mask = 6, 5
    prm = W.Params(prompt_len=2, gen_len=4, block_len=4, mask_id=mask, tau1=0.5, tau2=0.9)
    def fn(tok, prm, bs):
        zc = np.zeros((4, v)); zc[1:, 1] = 20.0           # rows 1-3 confident in id 1
        zs = np.zeros((4, v))                             # s = 1/6 -> always re-masked
        return zc, zs
    tok = np.array([0, 2, mask, mask, mask, mask])
    trace = []
    out, steps = W.decode(Scripted(fn), tok, prm, trace)
    assert steps == [4]
    assert [r.flags.tolist() for r in trace] == [[0, 1, 1, 1], [3, 2, 2, 2],
                                                 [2, 1, 1, 1], [4, 0, 0, 0]]
    assert out.tolist() == [0, 2, 0, 1, 1, 1]


@pytest.mark.parametrize("variant", ["literal", "wide"])
def test_greedy_special_case_equals_eq1_decoding(variant):
    """tau1 >= 1 and tau2 = 0: no position ever clears tau1 and nothing is
    re-masked, so each step unmasks exactly the most confident masked position:
    Eq. 1 high-confidence greedy decoding, one token per step."""
    cfg = tiny_cfg()
    lhs = None if variant == "literal" else wi.wide_lm_head_std(cfg)
    w = wi.model_weights(cfg, seed=1, lm_head_std=lhs)
    p, g, lb = 8, 8, 4
    prompt = wi.prompts(cfg, 1, p, seed=3)[0].numpy()
    tok0 = np.concatenate([prompt, np.full(g, cfg.mask_id)]).astype(np.int64)
    prm = W.Params(p, g, lb, cfg.mask_id, tau1=1.0, tau2=0.0)
    out, steps = W.decode(W.ModelProvider(w, cfg), tok0, prm)
    assert steps == [lb] * (g // lb)

    # Eq. 1 written independently: plain bidirectional forward over Y only
    # (no shadow block is needed when nothing is verified)
    tok = tok0.copy()
    s = p + g
    for b in range(g // lb):
        for _ in range(lb):
            h = M.forward_hidden(w, cfg, tok, np.arange(s), np.ones((s, s), bool))
            z = M.lm_logits(w, h[p + b * lb: p + (b + 1) * lb])
            pr = np.exp(z - z.max(-1, keepdims=True))
            pr /= pr.sum(-1, keepdims=True)
            pr[:, cfg.mask_id] = 0.0          # the mask id is never a prediction
            best = pr.max(-1)
            cand = [l for l in range(lb) if tok[p + b * lb + l] == cfg.mask_id]
            l_star = max(cand, key=lambda l: (best[l], -l))
            tok[p + b * lb + l_star] = int(np.argmax(pr[l_star]))
    assert out.tolist() == tok.tolist()


def naive_parallel_reference(w, cfg, tok0, p, g, lb, m):
    """Sec. 3 baseline written out independently: per step, a plain
    bidirectional forward over Y (no shadow block), then the m masked
    positions of the block with the highest top probability (over ids other
    than the mask; equal values -> lower position) take their argmax id."""
    tok = np.asarray(tok0, dtype=np.int64).copy()
    s = p + g
    steps = []
    for b in range(g // lb):
        n = 0
        while any(tok[p + b * lb + l] == cfg.mask_id for l in range(lb)):
            h = M.forward_hidden(w, cfg, tok, np.arange(s), np.ones((s, s), bool))
            z = M.lm_logits(w, h[p + b * lb: p + (b + 1) * lb])
            pr = np.exp(z - z.max(-1, keepdims=True))
            pr /= pr.sum(-1, keepdims=True)
            pr[:, cfg.mask_id] = 0.0
            best = pr.max(-1)
            cand = [l for l in range(lb) if tok[p + b * lb + l] == cfg.mask_id]
            for l in sorted(cand, key=lambda l: (-best[l], l))[:m]:
                tok[p + b * lb + l] = int(np.argmax(pr[l]))
            n += 1
        steps.append(n)
    return tok, steps


@pytest.mark.parametrize("m", [1, 3, 4, 9])
def test_fixed_tokens_per_step_baseline(m):
    """tokens_per_step = m: ceil(lb / m) steps per block, tokens equal to the
    independently written baseline (m = 1 is Eq. 1 greedy decoding; m >= lb
    is the full-parallel special case)."""
    cfg = tiny_cfg()
    w = wi.model_weights(cfg, seed=1, lm_head_std=wi.wide_lm_head_std(cfg))
    p, g, lb = 8, 16, 8
    prompt = wi.prompts(cfg, 1, p, seed=5)[0].numpy()
    tok0 = np.concatenate([prompt, np.full(g, cfg.mask_id)]).astype(np.int64)
    prm = W.Params(p, g, lb, cfg.mask_id, tokens_per_step=m)
    trace = []
    out, steps = W.decode(W.ModelProvider(w, cfg), tok0, prm, trace)
    assert steps == [-(-lb // m)] * (g // lb)
    # every step drafts exactly min(m, masks left in the block)
    left = lb
    for r in trace:
        assert int((r.flags == W.DRAFT).sum()) == min(m, left)
        left -= min(m, left)
        left = left or lb
    ref, ref_steps = naive_parallel_reference(w, cfg, tok0, p, g, lb, m)
    assert steps == ref_steps
    assert out.tolist() == ref.tolist()
    # no position is ever re-masked or forced in this mode
    assert all(not np.any((r.flags == W.REMASK) | (r.flags == W.FORCED)) for r in trace)


def test_topm_selection_hand_worked():
    """Five positions, mask id 9: masked 0, 2, 3, 4 with confidences 0.3, 0.9,
    0.3, 0.5.  m = 2 drafts positions 2 and 4; m = 3 adds position 0 (tied
    with 3, the lower position wins); m = 9 drafts every mask."""
    cur = np.array([9, 5, 9, 9, 9])
    conf = np.array([0.3, 0.99, 0.9, 0.3, 0.5])
    yhat = np.array([10, 11, 12, 13, 14])
    new, fl = W.topm_update(cur, conf, yhat, 9, 2)
    assert fl.tolist() == [0, 0, 1, 0, 1] and new.tolist() == [9, 5, 12, 9, 14]
    new, fl = W.topm_update(cur, conf, yhat, 9, 3)
    assert fl.tolist() == [1, 0, 1, 0, 1] and new.tolist() == [10, 5, 12, 9, 14]
    new, fl = W.topm_update(cur, conf, yhat, 9, 9)
    assert fl.tolist() == [1, 0, 1, 1, 1] and new.tolist() == [10, 5, 12, 13, 14]


def test_finalization_steps_hand_worked():
    """Prompt of 1 and 4 response positions (mask 9) over K = 4 steps:
    position 1 drafted at step 1 and kept (t = 1); position 2 drafted at 1,
    re-masked at 2, drafted again with the same id at 3 (t = 3); position 3
    drafted 7 at 2, re-masked at 3, drafted 6 at 4 (t = 4); position 4
    drafted at 4 (t = 4)."""
    Y = [[5, 9, 9, 9, 9],
         [5, 1, 2, 9, 9],
         [5, 1, 9, 7, 9],
         [5, 1, 2, 9, 9],
         [5, 1, 2, 6, 4]]
    assert W.finalization_steps(Y, 1).tolist() == [0, 1, 3, 4, 4]


def test_finalization_steps_of_a_decode(tiny_weights):
    """Along a real decode: t_l is the last step at which position l changed,
    every response position gets 1 <= t_l <= K, and each block's positions
    finalise within that block's steps."""
    cfg = tiny_cfg()
    p, g, lb = 8, 16, 8
    tok0 = np.concatenate([wi.prompts(cfg, 1, p, seed=4)[0].numpy(), np.full(g, cfg.mask_id)])
    prm = W.Params(p, g, lb, cfg.mask_id, tau1=0.3, tau2=0.9)
    trace = []
    out, steps = W.decode(W.ModelProvider(tiny_weights, cfg), tok0, prm, trace)
    states = [tok0] + [r.tokens for r in trace]
    t = W.finalization_steps(states, p)
    K = len(trace)
    assert np.all(t[:p] == 0) and np.all((t[p:] >= 1) & (t[p:] <= K))
    for l in range(p, p + g):
        changes = [k for k in range(1, K + 1) if states[k][l] != states[k - 1][l]]
        assert t[l] == changes[-1]
    ends = np.cumsum(steps)
    for b in range(g // lb):
        lo = ends[b - 1] if b else 0
        assert np.all((t[p + b * lb:p + (b + 1) * lb] > lo) & (t[p + b * lb:p + (b + 1) * lb] <= ends[b]))


def test_full_parallel_special_case_one_step_per_block(tiny_weights):
    """tau1 < 0 and tau2 = 0: every masked position clears tau1 at once."""
    cfg = tiny_cfg()
    p, g, lb = 8, 16, 4
    tok0 = np.concatenate([wi.prompts(cfg, 1, p, seed=4)[0].numpy(), np.full(g, cfg.mask_id)])
    prm = W.Params(p, g, lb, cfg.mask_id, tau1=-1.0, tau2=0.0)
    trace = []
    out, steps = W.decode(W.ModelProvider(tiny_weights, cfg), tok0, prm, trace)
    assert steps == [1] * (g // lb)
    assert all((r.flags == W.DRAFT).all() for r in trace)
    # each block's tokens are the argmax of its first (all-masked) forward
    for b, r in enumerate(trace):
        np.testing.assert_array_equal(out[p + b * lb: p + (b + 1) * lb], r.yhat)


@pytest.mark.parametrize("variant,tau1,tau2", [("literal", 0.7, 0.9), ("wide", 0.7, 0.9),
                                               ("wide", 0.5, 0.9), ("wide", 0.9, 0.0)])
def test_decode_invariants(variant, tau1, tau2):
    cfg = tiny_cfg()
    lhs = None if variant == "literal" else wi.wide_lm_head_std(cfg)
    w = wi.model_weights(cfg, seed=0, lm_head_std=lhs)
    p, g, lb = 16, 32, 8
    tok0 = np.concatenate([wi.prompts(cfg, 1, p, seed=7)[0].numpy(), np.full(g, cfg.mask_id)])
    prm = W.Params(p, g, lb, cfg.mask_id, tau1=tau1, tau2=tau2)
    trace = []
    out, steps = W.decode(W.ModelProvider(w, cfg), tok0, prm, trace)
    assert out[:p].tolist() == tok0[:p].tolist()             # prompt untouched
    assert not np.any(out == cfg.mask_id)                    # fully decoded
    assert all(1 <= n <= lb for n in steps)                  # cap = L_b
    assert sum(steps) <= g
    # revealed tokens stay inside the current block
    prev = tok0
    k = 0
    for b, n in enumerate(steps):
        lo, hi = p + b * lb, p + (b + 1) * lb
        for _ in range(n):
            cur = trace[k].tokens
            changed = np.nonzero(cur != prev)[0]
            assert np.all((changed >= lo) & (changed < hi))
            prev = cur
            k += 1
    if tau2 == 0.0:
        assert all((r.flags != W.REMASK).all() for r in trace)


def test_full_diffusion_is_a_single_block(tiny_weights):
    cfg = tiny_cfg()
    p, g = 8, 16
    tok0 = np.concatenate([wi.prompts(cfg, 1, p, seed=8)[0].numpy(), np.full(g, cfg.mask_id)])
    prm = W.Params(p, g, g, cfg.mask_id, tau1=0.7, tau2=0.9)
    out, steps = W.decode(W.ModelProvider(tiny_weights, cfg), tok0, prm)
    assert len(steps) == 1 and 1 <= steps[0] <= g
    assert not np.any(out == cfg.mask_id)


def test_margins_and_top2_gap_closed_forms():
    """The quantities that choose which positions a parity test compares
    (Eq. 2-4): on logits whose softmax is known in closed form, the draft
    confidence, the verify probability, the margin of each from its threshold
    and the top-2 gap over ids other than the mask equal their closed forms.
    The mask id's logit enters every normaliser but never the gap, and the
    decisions follow: nothing clears tau1, so the most confident masked
    position is drafted (Eq. 1); s < tau2 re-masks (Eq. 3)."""
    V, mask, lb = 16, 15, 2
    z = np.zeros((1, 2 * lb, V))
    z[0, 0, 3], z[0, 0, 7], z[0, 0, mask] = 2.0, 1.0, 5.0   # position 0 (masked): current row
    z[0, 1, 9] = 1.5                                         # position 1: current row
    z[0, lb + 1, 4] = 3.0                                    # position 1 holds id 4: shadow row
    cur = np.array([[mask, 4]])
    tau1, tau2 = 0.05, 0.9
    r = E.decide(z, cur, mask, tau1, tau2)
    e = math.exp
    s0 = e(2) + e(1) + e(5) + (V - 3)          # three non-zero logits, the rest e^0
    conf0, gap0 = e(2) / s0, (e(2) - e(1)) / s0
    s1 = e(3) / (e(3) + V - 1)
    gap1 = (e(1.5) - 1.0) / (e(1.5) + V - 1)
    assert r["yhat"][0, 0] == 3
    assert math.isclose(r["conf"][0, 0], conf0, rel_tol=1e-12)
    assert math.isclose(r["margin"][0, 0], abs(conf0 - tau1), rel_tol=1e-12)
    assert math.isclose(r["gap"][0, 0], gap0, rel_tol=1e-12)
    assert math.isclose(r["s"][0, 1], s1, rel_tol=1e-12)
    assert math.isclose(r["margin"][0, 1], abs(s1 - tau2), rel_tol=1e-12)
    assert math.isclose(r["gap"][0, 1], gap1, rel_tol=1e-12)
    assert r["flags"][0].tolist() == [W.FORCED, W.REMASK]
    assert r["tokens"][0].tolist() == [3, mask]
    # a confidence exactly at tau1 has margin 0: never robust at any margin
    r2 = E.decide(z, cur, mask, float(r["conf"][0, 0]), tau2)
    assert r2["margin"][0, 0] == 0.0


def test_step_margins_equal_the_epilogue_on_its_own_logits(tiny_weights):
    """The model-driven step reports the same confidences, verify
    probabilities, margins, top-2 gaps and decisions as the epilogue oracle
    (pinned above by closed forms) applied to that step's current and shadow
    logits: one definition of the compared positions for every parity test."""
    cfg = tiny_cfg()
    p, g, lb = 8, 16, 8
    rng = np.random.default_rng(3)
    tok = np.concatenate([wi.prompts(cfg, 1, p, seed=5)[0].numpy(), np.full(g, cfg.mask_id)])
    tok[p + rng.choice(lb, 3, replace=False)] = rng.integers(0, cfg.mask_id, 3)   # some drafted ids
    for tau1, tau2 in ((0.7, 0.9), (0.05, 0.5)):
        prm = W.Params(p, g, lb, cfg.mask_id, tau1=tau1, tau2=tau2)
        r = W.step(W.ModelProvider(tiny_weights, cfg), tok, prm, 0, 0)
        z = np.concatenate([r.z_cur, r.z_shad])[None]
        e = E.decide(z, tok[None, p:p + lb], cfg.mask_id, tau1, tau2)
        masked = tok[p:p + lb] == cfg.mask_id
        np.testing.assert_array_equal(r.flags, e["flags"][0])
        np.testing.assert_array_equal(r.tokens[p:p + lb], e["tokens"][0])
        np.testing.assert_allclose(r.margin, e["margin"][0], rtol=0, atol=1e-15)
        np.testing.assert_allclose(r.top2_gap, e["gap"][0], rtol=0, atol=1e-15)
        np.testing.assert_allclose(r.conf[masked], e["conf"][0][masked], rtol=0, atol=1e-15)
        np.testing.assert_allclose(r.s[~masked], e["s"][0][~masked], rtol=0, atol=1e-15)


def test_epilogue_single_peak_closed_form():
    """Rows that are zero except one peak of height h have p(peak) =
    e^h / (e^h + V - 1): the draft reads the current row, the verify the
    shadow row at the current token."""
    v, lb, mask = 16, 3, 15
    h_cur = [3.0, 1.0, 5.0]
    h_sh = [2.0, 4.0, 0.5]
    logits = np.zeros((1, 2 * lb, v))
    peak = [4, 9, 2, 6, 7, 11]
    for r in range(lb):
        logits[0, r, peak[r]] = h_cur[r]
        logits[0, lb + r, peak[lb + r]] = h_sh[r]
    cur = np.array([[mask, 7, 12]])          # pos 1 holds the shadow peak id, pos 2 not
    out = E.decide(logits, cur, mask, tau1=0.7, tau2=0.9)
    pk = lambda h: math.exp(h) / (math.exp(h) + v - 1)
    assert abs(out["conf"][0, 0] - pk(3.0)) < 1e-15 and out["yhat"][0, 0] == 4
    assert abs(out["s"][0, 1] - pk(4.0)) < 1e-15
    assert abs(out["s"][0, 2] - 1.0 / (math.exp(0.5) + v - 1)) < 1e-15
    # pk(3) = 0.573 < 0.7 -> forced draft; pk(4) = 0.785 < 0.9 -> re-mask; pos 2 re-mask
    assert out["tokens"][0].tolist() == [4, mask, mask]
    assert out["bitmap"][0].tolist() == [0, 1, 1]


def test_epilogue_planted_peaks_recovered():
    v, mask = 4096, 4095
    logits, cur, pid = wi.epilogue_inputs(2, 8, v, mask, seed=11, heights=(10.0, 16.0))
    out = E.decide(logits, cur.numpy(), mask, tau1=0.7, tau2=0.9)
    z = logits.double().numpy()
    for b in range(2):
        for l in range(8):
            second = np.sort(np.delete(z[b, l], [mask]))[-2]
            if z[b, l, pid[b, l]] > second:
                assert out["yhat"][b, l] == pid[b, l]


@pytest.mark.parametrize("norm,mat", [("attn_norm", "w_qkv"), ("ffn_norm", "w_gate_up")])
def test_norm_gain_scales_like_the_following_matrix(norm, mat):
    """RMSNorm's gain multiplies the normalised row before the next matrix
    product, so doubling the gain must equal doubling that matrix (both exact
    in bf16), and must differ from leaving both alone."""
    cfg = tiny_cfg(n_layers=1)
    w = wi.model_weights(cfg, seed=9, gain_std=0.1)
    tok = _tiny_tokens(cfg, 8, 8)
    ext, pos, allowed, _ = M.extended_inputs(tok, 8, 8, 4, 0, cfg.mask_id)
    base = M.forward_hidden(w, cfg, ext, pos, allowed)
    lw = w["layers"][0]
    g0, m0 = lw[norm], lw[mat]
    lw[norm] = g0 * 2
    h_gain = M.forward_hidden(w, cfg, ext, pos, allowed)
    lw[norm], lw[mat] = g0, m0 * 2
    h_mat = M.forward_hidden(w, cfg, ext, pos, allowed)
    np.testing.assert_allclose(h_gain, h_mat, atol=1e-12)
    assert np.max(np.abs(h_gain - base)) > 1e-4


# ---------------------------------------------------------------- WINO+ per-row quantities (Sec. 5.3)
from oracle import losses as L  # noqa: E402


def test_losses_uniform_and_two_point_closed_forms():
    V = 50
    e, nll, conf, yhat = L.row_quantities(np.zeros((1, V)), [7], mask_id=V - 1)
    assert abs(e[0] - math.log(V)) < 1e-12 and abs(nll[0] - math.log(V)) < 1e-12
    assert abs(conf[0] - 1.0 / V) < 1e-15 and yhat[0] == 0   # lowest id among ties
    # two live ids (a, b), the rest at -1e4: binary entropy of q = sigmoid(a - b)
    a, b = 1.3, -0.4
    z = np.full((1, V), -1e4)
    z[0, 3], z[0, 11] = a, b
    q = 1.0 / (1.0 + math.exp(b - a))
    e, nll, conf, yhat = L.row_quantities(z, [11], mask_id=V - 1)
    assert abs(e[0] - (-q * math.log(q) - (1 - q) * math.log(1 - q))) < 1e-12
    assert abs(nll[0] + math.log(1 - q)) < 1e-12
    assert yhat[0] == 3 and abs(conf[0] - q) < 1e-12


def test_losses_peaked_row_and_mask_excluded_from_prediction():
    V = 40
    z = np.zeros((2, V))
    z[0, 5] = 60.0
    z[1, V - 1] = 60.0          # the mask id dominates row 1
    z[1, 9] = 3.0
    e, nll, conf, yhat = L.row_quantities(z, [5, V - 1], mask_id=V - 1)
    assert e[0] < 1e-20 and nll[0] < 1e-20 and yhat[0] == 5
    assert yhat[1] == 9 and conf[1] < 1e-20 and nll[1] < 1e-20


def test_losses_entropy_is_expected_nll_and_bounded():
    rng = np.random.default_rng(3)
    V = 64
    z = rng.normal(0, 3, (4, V))
    e, _, _, _ = L.row_quantities(z, np.zeros(4, dtype=int), mask_id=V - 1)
    assert np.all(e >= 0) and np.all(e <= math.log(V) + 1e-12)
    p = W.softmax_rows(z)
    for r in range(4):
        nll_all = L.row_quantities(np.repeat(z[r:r + 1], V, 0), np.arange(V), mask_id=V - 1)[1]
        assert abs(float(p[r] @ nll_all) - e[r]) < 1e-10


def test_training_state_reveals_tokens_finalized_before_t():
    final = np.array([4, 4, 10, 11, 12, 13])
    t_fin = np.array([0, 0, 2, 1, 3, 2])
    assert L.training_state(final, t_fin, 1, 2, 99).tolist() == [4, 4, 99, 99, 99, 99]
    assert L.training_state(final, t_fin, 2, 2, 99).tolist() == [4, 4, 99, 11, 99, 99]
    assert L.training_state(final, t_fin, 3, 2, 99).tolist() == [4, 4, 10, 11, 99, 13]
    assert L.training_state(final, t_fin, 4, 2, 99).tolist() == [4, 4, 10, 11, 12, 13]
