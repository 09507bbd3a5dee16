"""Parity of the HIP path (through the C ABI) against the float64 oracle:
forward pieces (embedding, residual stream per sublayer, logits), the block
and baseline decoders, the step cap, the WINO+ per-row quantities, argument
checks, determinism and the GEMM tiles.

Every input is seeded and synthetic; oracle inputs are the same bytes the GPU
receives.  Logits must lie within 2e-2 max relative error per row of the
float64 oracle.  Decisions are judged by the float64 oracle (see
test_gpu_decisions.py for the contract tests); the oracle with bf16 rounding
at the kernels' rounding points serves only to size the tolerance of the
residual-stream checks (how far float32-level noise moves a bf16 pipeline).
"""
import numpy as np
import pytest
import torch

import wino_inputs as wi
from oracle import model as M
from oracle import wino as W
from helpers import (LOGIT_TOL, RANK_GAP, batch_tokens, decided_mask, decode_prefix_compare, forced_is_robust, fp64_provider,
                     gpu_step, oracle_params, oracle_trajectory, rowwise_rel_err, tiny, to_cpu, to_device)

pytestmark = pytest.mark.gpu

@pytest.fixture(scope="module")
def P():
    import paper_2605_16941_amd as pkg
    return pkg


# ---------------------------------------------------------------- forward pieces
def test_embedding_rows_are_exact(P):
    cfg, w = tiny()
    wd = to_device(w)
    p, g, lb, B = 32, 64, 16, 2
    model = P.WinoModel(cfg, wd, B, p + g + lb)
    tok = batch_tokens(cfg, B, p, g, fill=[(0, 16, 0.5)])
    prm = P.make_params(B, p, g, lb, cfg.mask_id)
    out = torch.empty(B, p + g + lb, cfg.d_model, dtype=torch.float32, device="cuda")
    P.wino_debug_forward(model.ctx, prm, torch.tensor(tok, dtype=torch.int32, device="cuda"),
                         torch.tensor([0, 16], dtype=torch.int32, device="cuda"), 0, out)
    torch.cuda.synchronize()
    ext = np.concatenate([tok, np.full((B, lb), cfg.mask_id)], axis=1)
    want = w["tok_emb"].float()[torch.from_numpy(ext)]
    assert torch.equal(out.cpu(), want)
    model.close()


@pytest.mark.parametrize("n_sub", [1, 2, 3, 4])
def test_residual_stream_matches_oracle(P, n_sub):
    """Residual stream after each sublayer: close to float64, and as close to
    the oracle run at the kernel's bf16 rounding points as that oracle is to
    itself under float32-level input noise (its rounding points make it
    sensitive: a 1e-7 input change moves it by up to ~3e-3 here)."""
    cfg, w = tiny()
    wd = to_device(w)
    p, g, lb, B = 32, 64, 16, 2
    model = P.WinoModel(cfg, wd, B, p + g + lb)
    tok = batch_tokens(cfg, B, p, g, fill=[(0, 16, 0.5), (16, 48, 1.0)])
    bstart = [16, 0]
    prm = P.make_params(B, p, g, lb, cfg.mask_id)
    out = torch.empty(B, p + g + lb, cfg.d_model, dtype=torch.float32, device="cuda")
    P.wino_debug_forward(model.ctx, prm, torch.tensor(tok, dtype=torch.int32, device="cuda"),
                         torch.tensor(bstart, dtype=torch.int32, device="cuda"), n_sub, out)
    torch.cuda.synchronize()
    model.close()
    got = out.cpu().numpy()
    errs, errs16, chaos = [], [], 0.0
    for b in range(B):
        ext, pos, allowed, _ = M.extended_inputs(tok[b], p, g, lb, bstart[b], cfg.mask_id)
        ref = oracle_rows(w, cfg, ext, pos, allowed, n_sub)
        ref16 = oracle_rows(w, cfg, ext, pos, allowed, n_sub, M.round_bf16)
        for seed in (1, 2):
            ref16p = oracle_rows(w, cfg, ext, pos, allowed, n_sub, M.round_bf16, perturb=1e-7, seed=seed)
            chaos = max(chaos, rowwise_rel_err(ref16p, ref16))
        errs.append(rowwise_rel_err(got[b], ref))
        errs16.append(rowwise_rel_err(got[b], ref16))
    print(f"sublayers {n_sub}: rel err vs fp64 {max(errs):.2e}, vs bf16-point {max(errs16):.2e}, "
          f"oracle self-sensitivity {chaos:.2e}")
    assert max(errs) < 1e-2
    assert max(errs16) < 3 * chaos + 1e-4


@pytest.mark.parametrize("p,g,lb,B", [(0, 21, 7, 3), (6, 24, 3, 2), (13, 20, 20, 1)])
def test_ragged_shapes_fp16_activations(P, p, g, lb, B):
    """The fp16 kernel instances at the ragged shapes: the full-depth residual
    stream moves from float64 less than with bf16 activations, and little."""
    cfg, w = tiny("wide", seed=2)
    wd = to_device(w)
    T = p + g + lb
    rng = np.random.default_rng(4)
    tok = batch_tokens(cfg, B, p, g, seed=4, fill=[(0, lb, 0.5)]) if p > 0 else \
        np.where(rng.random((B, g)) < 0.5, rng.integers(0, cfg.mask_id, (B, g)), cfg.mask_id)
    bstart = [0] * B
    prm = P.make_params(B, p, g, lb, cfg.mask_id)
    n_sub = 2 * cfg.n_layers
    errs = {}
    for act in (P.ACT_BF16, P.ACT_FP16):
        model = P.WinoModel(cfg, wd, B, T, act_precision=act)
        out = torch.empty(B, T, cfg.d_model, dtype=torch.float32, device="cuda")
        P.wino_debug_forward(model.ctx, prm, torch.tensor(tok, dtype=torch.int32, device="cuda"),
                             torch.tensor(bstart, dtype=torch.int32, device="cuda"), n_sub, out)
        torch.cuda.synchronize()
        got = out.cpu().numpy()
        model.close()
        e = 0.0
        for b in range(B):
            ext, pos, allowed, _ = M.extended_inputs(tok[b], p, g, lb, bstart[b], cfg.mask_id)
            e = max(e, rowwise_rel_err(got[b], oracle_rows(w, cfg, ext, pos, allowed, n_sub)))
        errs[act] = e
    print(f"T={T}: residual rel err vs float64: bf16 {errs[P.ACT_BF16]:.2e}, fp16 {errs[P.ACT_FP16]:.2e}")
    assert errs[P.ACT_FP16] < errs[P.ACT_BF16] and errs[P.ACT_FP16] < 2e-3


def test_package_imported_before_torch(P):
    """A process that imports the package before torch still runs the library
    on torch's HIP runtime: one copy of the runtime is loaded, and a context
    created on torch's device memory works (with the system copy loaded
    beside torch's, wino_create failed with WINO_ERR_HIP)."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    code = ("import paper_2605_16941_amd as P\n"
            "import torch\n"
            "import wino_inputs as wi\n"
            "cfg = wi.preset('tiny')\n"
            "P.WinoModel(cfg, wi.model_weights(cfg, seed=0, device='cuda'), 1, 112).close()\n"
            "print('runtimes', len({l.split()[-1] for l in open('/proc/self/maps') if 'libamdhip64' in l}))\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=root, capture_output=True, text=True, timeout=240)
    assert r.returncode == 0, r.stderr[-2000:]
    assert "runtimes 1" in r.stdout, r.stdout


def test_fp16_copies_reject_weights_beyond_fp16_range(P):
    """wino_create in fp16 mode refuses weights with no finite fp16 copy (a
    value beyond 65504 in any multiplied matrix) and accepts the largest bf16
    value inside that range (65280)."""
    cfg, w = tiny("literal", seed=2)
    for key, layer, val, ok in (("w_down", 1, 65280.0, True), ("w_down", 1, 66000.0, False),
                                ("w_qkv", 0, -1.0e5, False), ("lm_head", None, 7.0e4, False)):
        wd = to_device(w)
        tgt = wd["lm_head"] if layer is None else wd["layers"][layer][key]
        tgt.view(-1)[12345 % tgt.numel()] = val
        torch.cuda.synchronize()
        if ok:
            P.WinoModel(cfg, wd, 1, 64, act_precision=P.ACT_FP16).close()
            continue
        with pytest.raises(P.WinoError) as e:
            P.WinoModel(cfg, wd, 1, 64, act_precision=P.ACT_FP16)
        assert e.value.status == -6 and "no finite fp16 copy" in str(e.value), (key, val, str(e.value))
        # the same weights are accepted with bf16 activations
        P.WinoModel(cfg, wd, 1, 64).close()


@pytest.mark.parametrize("p,g,lb,B", [(0, 21, 7, 3), (6, 24, 3, 2), (13, 20, 20, 1)])
def test_ragged_shapes_forward_and_decode(P, p, g, lb, B):
    """Ragged edge cases: no prompt, T = P + G + L_b not a multiple of 8 (the
    QKV epilogue's element stores for v^T runs that cross a sequence end), an
    odd block length, and a single block spanning the whole response.  The
    full-depth residual stream must match the oracle as closely as the
    oracle's own sensitivity to float32-level noise allows, and a decode must agree
    with the oracle's wherever its decisions are robust."""
    cfg, w = tiny("wide", seed=2)
    wd = to_device(w)
    T = p + g + lb
    model = P.WinoModel(cfg, wd, B, T)
    tok = batch_tokens(cfg, B, p, g, seed=4, fill=[(0, lb, 0.5)]) if p > 0 else \
        np.full((B, g), cfg.mask_id, dtype=np.int64)
    if p == 0:
        rng = np.random.default_rng(4)
        first = rng.random((B, lb)) < 0.5
        tok[:, :lb][first] = rng.integers(0, cfg.mask_id, int(first.sum()))
    bstart = [0] * B
    prm = P.make_params(B, p, g, lb, cfg.mask_id)
    n_sub = 2 * cfg.n_layers
    out = torch.empty(B, T, cfg.d_model, dtype=torch.float32, device="cuda")
    P.wino_debug_forward(model.ctx, prm, torch.tensor(tok, dtype=torch.int32, device="cuda"),
                         torch.tensor(bstart, dtype=torch.int32, device="cuda"), n_sub, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    # The bf16-point oracle's sensitivity is a step function: an input change
    # either flips no bf16 rounding (error ~ the change) or flips one (~1e-3).
    # Float32 accumulation-order differences over a K-long dot product reach
    # ~sqrt(K) * 2^-24 ~ 1e-6 relative, so the noise is probed at 1e-7 and 1e-6.
    chaos, errs16 = 0.0, []
    for b in range(B):
        ext, pos, allowed, _ = M.extended_inputs(tok[b], p, g, lb, bstart[b], cfg.mask_id)
        ref = oracle_rows(w, cfg, ext, pos, allowed, n_sub)
        ref16 = oracle_rows(w, cfg, ext, pos, allowed, n_sub, M.round_bf16)
        for eps in (1e-7, 1e-6):
            for seed in (1, 2):
                chaos = max(chaos, rowwise_rel_err(oracle_rows(w, cfg, ext, pos, allowed, n_sub, M.round_bf16,
                                                               perturb=eps, seed=seed), ref16))
        assert rowwise_rel_err(got[b], ref) < 1e-2
        errs16.append(rowwise_rel_err(got[b], ref16))
    print(f"T={T}: vs bf16-point {max(errs16):.2e}, oracle self-sensitivity {chaos:.2e}")
    assert max(errs16) < 3 * chaos + 1e-4
    # decode from all-mask responses with the same prompts, one forward per
    # call, against the float64 oracle up to its first non-robust step
    tok0 = tok.copy()
    tok0[:, p:] = cfg.mask_id
    compared, diverged, forwards, trajs = decode_prefix_compare(P, model, prm, oracle_params(prm),
                                                                fp64_provider(w, cfg), tok0, f"T={T}")
    print(f"T={T}: decode steps compared {compared} of {[len(t) for t in trajs]}, divergence {diverged}")
    assert sum(compared) >= 1
    model.close()


def oracle_rows(w, cfg, ext, pos, allowed, n_sub, act_round=None, perturb=0.0, seed=0):
    """Oracle residual after n_sub sublayers, optionally with the embedding
    rows scaled by (1 + perturb * N(0,1)) to expose float32-level sensitivity."""
    rows = M.f64(w["tok_emb"][torch.as_tensor(ext)])
    if perturb:
        rows = rows * (1.0 + perturb * np.random.default_rng(seed).standard_normal(rows.shape))
    ws = dict(w, tok_emb=torch.from_numpy(rows))
    return M.forward_residual(ws, cfg, np.arange(len(ext)), pos, allowed, act_round=act_round,
                              n_sublayers=n_sub)


@pytest.mark.slow
@pytest.mark.parametrize("n_sub", [1, 2])
def test_full_shape_residual_per_sublayer(P, n_sub):
    """At the 8B shape the bf16 rounding points make the forward sensitive:
    float32-level input noise (1e-7) already moves the kernel-precision oracle
    by ~1e-3.  The GPU must agree with that oracle as well as the oracle
    agrees with itself under such noise, and stay within 1.5e-2 of float64."""
    cfg, wd = big_one_layer("llada8b")
    B, p, g, lb = 1, 256, 256, 32
    model = P.WinoModel(cfg, wd, B, p + g + lb)
    pr = wi.prompts(cfg, B, p, seed=1).numpy()
    tok = np.concatenate([pr, np.full((B, g), cfg.mask_id)], axis=1).astype(np.int64)
    tok[0, p:p + 48] = np.random.default_rng(0).integers(0, cfg.mask_id, 48)
    prm = P.make_params(B, p, g, lb, cfg.mask_id)
    out = torch.empty(B, p + g + lb, cfg.d_model, dtype=torch.float32, device="cuda")
    P.wino_debug_forward(model.ctx, prm, torch.tensor(tok, dtype=torch.int32, device="cuda"),
                         torch.tensor([32], dtype=torch.int32, device="cuda"), n_sub, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy()[0]
    model.close()
    w = to_cpu(wd)
    del wd
    ext, pos, allowed, _ = M.extended_inputs(tok[0], p, g, lb, 32, cfg.mask_id)
    ref = oracle_rows(w, cfg, ext, pos, allowed, n_sub)
    ref16 = oracle_rows(w, cfg, ext, pos, allowed, n_sub, M.round_bf16)
    ref16p = oracle_rows(w, cfg, ext, pos, allowed, n_sub, M.round_bf16, perturb=1e-7)
    err, err16, chaos = (rowwise_rel_err(got, ref), rowwise_rel_err(got, ref16),
                         rowwise_rel_err(ref16p, ref16))
    print(f"8B shape, sublayers {n_sub}: vs fp64 {err:.2e}, vs bf16-point {err16:.2e}, "
          f"oracle self-sensitivity {chaos:.2e}")
    assert err < 1.5e-2
    assert err16 < 3 * chaos + 1e-4


@pytest.mark.parametrize("variant", ["literal", "wide"])
def test_logits_match_oracle(P, variant):
    cfg, w = tiny(variant)
    wd = to_device(w)
    p, g, lb, B = 32, 64, 16, 2
    model = P.WinoModel(cfg, wd, B, p + g + lb)
    tok = batch_tokens(cfg, B, p, g, seed=3, fill=[(0, 32, 1.0), (32, 48, 0.4)])
    bstart = [32, 32]
    prm = P.make_params(B, p, g, lb, cfg.mask_id)
    logits = torch.empty(B, 2 * lb, cfg.vocab, dtype=torch.float32, device="cuda")
    P.wino_debug_logits(model.ctx, prm, torch.tensor(tok, dtype=torch.int32, device="cuda"),
                        torch.tensor(bstart, dtype=torch.int32, device="cuda"), logits)
    torch.cuda.synchronize()
    got = logits.cpu().numpy()
    for b in range(B):
        ext, pos, allowed, c0 = M.extended_inputs(tok[b], p, g, lb, bstart[b], cfg.mask_id)
        s = p + g
        for rnd, tol in ((None, LOGIT_TOL), (M.round_bf16, LOGIT_TOL)):
            h = M.forward_hidden(w, cfg, ext, pos, allowed, act_round=rnd)
            ref = np.concatenate([M.lm_logits(w, h[c0:c0 + lb]), M.lm_logits(w, h[s:s + lb])])
            err = rowwise_rel_err(got[b], ref)
            assert err < tol, f"seq {b} ({'bf16' if rnd else 'fp64'} oracle): logits rel err {err}"
    model.close()


@pytest.mark.parametrize("variant", ["literal", "wide", "midmask"])
def test_logits_fp16_activations(P, variant):
    """fp16 activations (and fp16 copies of the weight matrices): the logits
    move from float64 several times less than with bf16 activations, and
    the fp16 GEMM, attention and norm paths agree with the float64 oracle."""
    cfg, w = tiny(variant)
    wd = to_device(w)
    p, g, lb, B = 32, 64, 16, 2
    tok = batch_tokens(cfg, B, p, g, seed=3, fill=[(0, 32, 1.0), (32, 48, 0.4)])
    bstart = [32, 32]
    prm = P.make_params(B, p, g, lb, cfg.mask_id)
    errs = {}
    for act in (P.ACT_BF16, P.ACT_FP16):
        model = P.WinoModel(cfg, wd, B, p + g + lb, act_precision=act)
        logits = torch.empty(B, 2 * lb, cfg.vocab, dtype=torch.float32, device="cuda")
        P.wino_debug_logits(model.ctx, prm, torch.tensor(tok, dtype=torch.int32, device="cuda"),
                            torch.tensor(bstart, dtype=torch.int32, device="cuda"), logits)
        torch.cuda.synchronize()
        got = logits.cpu().numpy()
        model.close()
        e = 0.0
        for b in range(B):
            ext, pos, allowed, c0 = M.extended_inputs(tok[b], p, g, lb, bstart[b], cfg.mask_id)
            s = p + g
            h = M.forward_hidden(w, cfg, ext, pos, allowed)
            ref = np.concatenate([M.lm_logits(w, h[c0:c0 + lb]), M.lm_logits(w, h[s:s + lb])])
            e = max(e, rowwise_rel_err(got[b], ref))
        errs[act] = e
    print(f"{variant}: logits rel err vs float64: bf16 {errs[P.ACT_BF16]:.2e}, fp16 {errs[P.ACT_FP16]:.2e}")
    assert errs[P.ACT_FP16] < LOGIT_TOL / 4
    assert errs[P.ACT_FP16] < errs[P.ACT_BF16] / 3


# ---------------------------------------------------------------- block and baseline decoders
def test_decode_block_and_idle_sequences(P):
    cfg, w = tiny("wide", seed=4)
    wd = to_device(w)
    p, g, lb, B = 16, 32, 16, 3
    model = P.WinoModel(cfg, wd, B, p + g + lb)
    prm_c = P.make_params(B, p, g, lb, cfg.mask_id, 0.7, 0.9)
    tok0 = batch_tokens(cfg, B, p, g, seed=2)
    tok0[1, p:p + lb] = 7              # sequence 1: current block already complete
    tok = torch.tensor(tok0, dtype=torch.int32, device="cuda")
    bs = torch.tensor([0, 0, g], dtype=torch.int32, device="cuda")  # sequence 2 finished
    steps = P.wino_decode_block(model.ctx, prm_c, tok, bs)
    torch.cuda.synchronize()
    got = tok.cpu().numpy()
    assert steps[1] == 0 and steps[2] == 0 and 1 <= steps[0] <= lb
    assert np.array_equal(got[1], tok0[1]) and np.array_equal(got[2], tok0[2])
    assert not np.any(got[0, p:p + lb] == cfg.mask_id)
    assert np.array_equal(got[0, p + lb:], tok0[0, p + lb:])
    model.close()


def block_trajectory(prov, tokens0, prm, bs):
    """[(tokens before, block_start, block_steps, StepResult)] of one block."""
    out = []
    tok = np.asarray(tokens0, dtype=np.int64).copy()
    c0, steps = prm.prompt_len + bs, 0
    while np.any(tok[c0:c0 + prm.block_len] == prm.mask_id):
        r = W.step(prov, tok, prm, bs, steps)
        out.append((tok.copy(), bs, steps, r))
        tok = r.tokens
        steps += 1
    return out, tok


def robust_trajectory(traj, p, lb, mask_id):
    return all(np.all(decided_mask(r.margin, r.top2_gap, t[c0:c0 + lb] == mask_id))
               and (not np.any(r.flags == W.FORCED) or forced_is_robust(r.conf, t[c0:c0 + lb] == mask_id))
               for (t, bs_, _, r) in traj for c0 in [p + bs_])


@pytest.mark.parametrize("mixed", [False, True])
def test_decode_block_matches_oracle(P, mixed):
    """wino_decode_block from a fresh block (first step without the shadow
    block) and from a mixed batch (one sequence holds drafts: shadow kept)."""
    cfg, w = tiny("wide", seed=2)
    wd = to_device(w)
    p, g, lb, B = 32, 64, 16, 2
    model = P.WinoModel(cfg, wd, B, p + g + lb)
    prm_c = P.make_params(B, p, g, lb, cfg.mask_id, 0.7, 0.9)
    prm = oracle_params(prm_c)
    # sequence 0 starts block 1 fresh (block 0 filled when mixed); sequence 1
    # starts block 0, half drafted when mixed (its trajectory re-masks 7)
    tok0 = batch_tokens(cfg, B, p, g, seed=3, fill=[(0, 16, 1.0)] if mixed else None)
    starts = [16, 0] if mixed else [0, 16]
    if mixed:
        rng = np.random.default_rng(11)
        tok0[1, p:p + lb][rng.random(lb) < 0.5] = cfg.mask_id
    tok = torch.tensor(tok0, dtype=torch.int32, device="cuda")
    bs = torch.tensor(starts, dtype=torch.int32, device="cuda")
    fin = torch.zeros(B, g, dtype=torch.int32, device="cuda")
    steps = P.wino_decode_block(model.ctx, prm_c, tok, bs, fin)
    torch.cuda.synchronize()
    got = tok.cpu().numpy()
    fin = fin.cpu().numpy()
    prov = fp64_provider(w, cfg)
    n_cmp = 0
    for b in range(B):
        traj, final = block_trajectory(prov, tok0[b], prm, starts[b])
        c0 = p + starts[b]
        assert not np.any(got[b, c0:c0 + lb] == cfg.mask_id)
        outside = np.ones(p + g, bool)
        outside[c0:c0 + lb] = False
        assert np.array_equal(got[b][outside], tok0[b][outside])
        if robust_trajectory(traj, p, lb, cfg.mask_id):
            assert np.array_equal(got[b], final), f"seq {b}: block differs from the oracle"
            assert steps[b] == len(traj)
            # Sec. 5.1 finalization steps relative to this call (0: never changed,
            # e.g. a kept pre-filled draft); re-masked drafts finalise later
            t = W.finalization_steps([tok0[b]] + [r.tokens for (_, _, _, r) in traj], p)
            assert np.array_equal(fin[b], t[p:]), f"seq {b}: finalization steps differ"
            n_cmp += 1
    assert n_cmp > 0
    # the same blocks again: none holds a mask, so the call runs no forward
    P.wino_profile(model.ctx, 1)  # class 0: the embedding, once per forward
    P.wino_profile_read(model.ctx)
    tok_done = tok.clone()
    assert P.wino_decode_block(model.ctx, prm_c, tok, bs) == [0] * B
    torch.cuda.synchronize()
    assert P.wino_profile_read(model.ctx)[P.wino_kernel_class_name(0)]["launches"] == 0
    assert torch.equal(tok, tok_done)
    P.wino_profile(model.ctx, 0)
    model.close()


@pytest.mark.parametrize("m", [1, 4])
def test_baseline_decoders_match_oracle(P, m):
    """tokens_per_step = m (Sec. 3 baselines: Eq. 1 greedy for 1, naive
    parallel sampling for 4), teacher-forced along the oracle's trajectory.
    The synthetic model's masked positions often have confidences within
    1e-3 of each other, so the rank decision is compared exactly only where
    the oracle's m-th / (m+1)-th gap is robust; everywhere else the GPU's
    choice must be a valid top-m set: no undrafted mask more confident than a
    drafted one by more than the tolerance.  A rank or an id compares two
    probabilities, each within PROB_ERR of the float64 oracle (the bound the
    contract tests hold on this model), so both are fixed only by gaps above
    RANK_GAP = 2 * PROB_ERR."""
    tol = RANK_GAP
    cfg, w = tiny("wide", seed=4)
    wd = to_device(w)
    p, g, lb, B = 32, 64, 16, 2
    model = P.WinoModel(cfg, wd, B, p + g + lb)
    prm_c = P.make_params(B, p, g, lb, cfg.mask_id, tokens_per_step=m)
    prm = oracle_params(prm_c, tokens_per_step=m)
    tok0 = batch_tokens(cfg, B, p, g, seed=9)
    prov = fp64_provider(w, cfg)
    trajs = [oracle_trajectory(prov, tok0[b], prm)[0] for b in range(B)]
    n_exact = 0
    for k in range(max(len(t) for t in trajs)):
        states = [t[min(k, len(t) - 1)] for t in trajs]
        tokens = np.stack([st_[0] for st_ in states])
        gt, gf, gnm, gst, _ = gpu_step(P, model, prm_c, tokens, [st_[1] for st_ in states],
                                       [st_[2] for st_ in states])
        for b, (tb, bs_, steps_, r) in enumerate(states):
            c0 = p + bs_
            cur = tb[c0:c0 + lb]
            new = gt[b][c0:c0 + lb]
            masked = cur == cfg.mask_id
            drafted = gf[b] == W.DRAFT
            assert int(drafted.sum()) == min(m, int(masked.sum()))
            assert not np.any(gf[b][~masked]) and np.array_equal(new[~masked], cur[~masked])
            assert np.all(drafted <= masked) and gst[b] == steps_ + 1
            assert gnm[b] == int(masked.sum()) - int(drafted.sum())
            rest = masked & ~drafted
            if drafted.any() and rest.any():
                assert r.conf[drafted].min() >= r.conf[rest].max() - tol
            sure = drafted & (r.top2_gap > tol)
            assert np.array_equal(new[sure], r.yhat[sure])
            ok = masked & (r.margin > tol / 2) & (r.top2_gap > tol)
            assert np.array_equal(gf[b][ok], r.flags[ok])
            n_exact += int(ok.sum())
    assert n_exact > 0
    # full decode: the fixed schedule of ceil(lb / m) steps per block
    tok = torch.tensor(tok0, dtype=torch.int32, device="cuda")
    bs = torch.zeros(B, dtype=torch.int32, device="cuda")
    steps, forwards = P.wino_decode(model.ctx, prm_c, tok, bs)
    torch.cuda.synchronize()
    got = tok.cpu().numpy()
    assert forwards == (g // lb) * -(-lb // m) and all(s_ == forwards for s_ in steps)
    assert not np.any(got[:, p:] == cfg.mask_id) and np.array_equal(got[:, :p], tok0[:, :p])
    model.close()


@pytest.mark.parametrize("tau1,m", [(1.0, 1), (-1.0, 16)])
def test_threshold_special_cases_equal_baselines(P, tau1, m):
    """Special cases on the same kernels (the tau2 = 0 ablation of Sec. 6.3): with tau2 = 0 nothing is
    re-masked; tau1 >= 1 then drafts only the forced top-1 position (Eq. 2 can
    never exceed 1), which is Eq. 1 greedy decoding, one token per step; tau1 < 0
    drafts every masked position at once, one step per block.  Both must equal
    the fixed-schedule baselines (tokens_per_step 1 and L_b) bit for bit: the
    same forward (no shadow block in either) and the same confidence ranking,
    ties to the lowest position."""
    cfg, w = tiny("wide", seed=4)
    wd = to_device(w)
    p, g, lb, B = 32, 64, 16, 2
    model = P.WinoModel(cfg, wd, B, p + g + lb)
    tok0 = batch_tokens(cfg, B, p, g, seed=12)
    outs = []
    for prm_c in (P.make_params(B, p, g, lb, cfg.mask_id, tau1, 0.0),
                  P.make_params(B, p, g, lb, cfg.mask_id, tokens_per_step=m)):
        tok = torch.tensor(tok0, dtype=torch.int32, device="cuda")
        bs = torch.zeros(B, dtype=torch.int32, device="cuda")
        steps, forwards = P.wino_decode(model.ctx, prm_c, tok, bs)
        torch.cuda.synchronize()
        outs.append((tok.cpu().numpy(), list(steps), forwards))
    (wt, ws, wf), (bt, bsteps, bf) = outs
    assert wf == bf == (g // lb) * -(-lb // m)
    assert ws == bsteps == [wf] * B
    assert not np.any(wt[:, p:] == cfg.mask_id) and np.array_equal(wt[:, :p], tok0[:, :p])
    assert np.array_equal(wt, bt)
    model.close()


LOSS_DT = np.dtype([("entropy", "<f4"), ("nll", "<f4"), ("conf", "<f4"), ("argmax", "<i4")])


@pytest.mark.parametrize("variant", ["literal", "wide"])
def test_row_losses_match_oracle(P, variant):
    """WINO+ per-row quantities (Sec. 5.3) of training states (Sec. 5.2): entropy, target
    NLL and greedy prediction of every response row, fused into the LM head.
    Two sequences whose training states reveal the tokens finalized before
    different steps; 128 response rows in chunks of the workspace's rows."""
    from oracle import losses as LS
    cfg, w = tiny(variant, seed=3)
    wd = to_device(w)
    p, g, lb, B = 32, 64, 16, 2
    model = P.WinoModel(cfg, wd, B, p + g + lb)
    prm_c = P.make_params(B, p, g, lb, cfg.mask_id)
    rng = np.random.default_rng(5)
    final = batch_tokens(cfg, B, p, g, seed=6, fill=[(0, g, 1.0)])
    t_fin = np.concatenate([np.zeros((B, p), int), rng.integers(1, 9, (B, g))], axis=1)
    states = np.stack([LS.training_state(final[b], t_fin[b], t, p, cfg.mask_id)
                       for b, t in enumerate([3, 6])])
    targets = final[:, p:]
    out = torch.zeros(B * g * LOSS_DT.itemsize, dtype=torch.uint8, device="cuda")
    P.wino_row_losses(model.ctx, prm_c, torch.tensor(states, dtype=torch.int32, device="cuda"),
                      torch.tensor(targets, dtype=torch.int32, device="cuda"), out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(LOSS_DT).reshape(B, g)
    for b in range(B):
        for act_round, tol in ((M.round_bf16, 5e-3), (None, 2e-2)):
            z = LS.state_logits(w, cfg, states[b], p, act_round)
            e, nll, conf, yhat = LS.row_quantities(z, targets[b], cfg.mask_id)
            assert np.max(np.abs(got[b]["entropy"] - e)) < 2 * tol
            assert np.max(np.abs(got[b]["nll"] - nll) / (1 + nll)) < 2 * tol
            assert np.max(np.abs(got[b]["conf"] - conf)) < tol
            if act_round is None:
                pr = W.softmax_rows(z)
                pr[:, cfg.mask_id] = -1.0
                top = np.sort(pr, axis=-1)
                sure = top[:, -1] - top[:, -2] > 1e-2
                assert sure.any() and np.array_equal(got[b]["argmax"][sure], yhat[sure])
    model.close()


@pytest.mark.parametrize("cap_fill", [True, False])
def test_step_cap_without_forced_draft(P, cap_fill):
    """An unreachable draft threshold (tau1 = 1.5), no forced draft (Eq. 1
    off) and max_steps = 3: no step drafts until the cap.  With cap fill the
    third step drafts every remaining mask with its argmax, so each block
    takes exactly 3 steps and the decode equals the oracle's wherever that is
    robust; without it the decode stops with WINO_ERR_STEP_CAP and the
    tokens untouched."""
    cfg, w = tiny("wide", seed=2)
    wd = to_device(w)
    p, g, lb, B = 32, 64, 16, 2
    model = P.WinoModel(cfg, wd, B, p + g + lb)
    flags = P._abi.WINO_FLAG_NO_FORCE_TOP1 | (0 if cap_fill else P._abi.WINO_FLAG_NO_CAP_FILL)
    prm_c = P.make_params(B, p, g, lb, cfg.mask_id, 1.5, 0.9, max_steps=3, flags=flags)
    tok0 = batch_tokens(cfg, B, p, g, seed=5)
    tok = torch.tensor(tok0, dtype=torch.int32, device="cuda")
    bs = torch.zeros(B, dtype=torch.int32, device="cuda")
    if not cap_fill:
        with pytest.raises(P.WinoError) as e:
            P.wino_decode(model.ctx, prm_c, tok, bs)
        assert e.value.status == -5
        torch.cuda.synchronize()
        assert np.array_equal(tok.cpu().numpy(), tok0) and torch.all(bs == 0)
        model.close()
        return
    steps, forwards = P.wino_decode(model.ctx, prm_c, tok, bs)
    torch.cuda.synchronize()
    assert steps == [3 * (g // lb)] * B and forwards == 3 * (g // lb)
    got = tok.cpu().numpy()
    assert not np.any(got[:, p:] == cfg.mask_id)
    prm = oracle_params(prm_c, force_top1=False, cap_fill=True)
    prov = fp64_provider(w, cfg)
    compared = 0
    for b in range(B):
        traj, final = oracle_trajectory(prov, tok0[b], prm)
        assert len(traj) == 3 * (g // lb)
        if robust_trajectory(traj, p, lb, cfg.mask_id):
            assert np.array_equal(got[b], final), f"seq {b}: decode differs from the oracle"
            compared += 1
    assert compared >= 1
    model.close()


def test_params_rejected_against_the_context(P):
    """With a live context, parameters the context cannot serve are rejected on
    the host with the documented status before any device work (batch above
    max_batch, P + G + L_b above max_seq, L_b not dividing G, a mask id outside
    the vocabulary, a NaN threshold, a negative tokens_per_step), and the
    context is unharmed: a valid step afterwards equals a fresh context's."""
    cfg, w = tiny()
    wd = to_device(w)
    p, g, lb, B = 32, 64, 16, 2
    model = P.WinoModel(cfg, wd, B, p + g + lb)
    tok = torch.tensor(batch_tokens(cfg, B, p, g, fill=[(0, 16, 0.5)]), dtype=torch.int32, device="cuda")
    bs = torch.zeros(B, dtype=torch.int32, device="cuda")
    invalid, shape = -1, -2
    cases = [(P.make_params(B + 1, p, g, lb, cfg.mask_id), shape),
             (P.make_params(B, p + 1, g, lb, cfg.mask_id), shape),
             (P.make_params(B, p, g, 12, cfg.mask_id), shape),
             (P.make_params(B, p, g, lb, cfg.vocab), invalid),
             (P.make_params(B, p, g, lb, cfg.mask_id, float("nan")), invalid),
             (P.make_params(B, p, g, lb, cfg.mask_id, tokens_per_step=-1), invalid)]
    for prm, want in cases:
        t = tok.clone()
        with pytest.raises(P.WinoError) as e:
            P.wino_step(model.ctx, prm, t, bs)
        assert e.value.status == want
        with pytest.raises(P.WinoError) as e:
            P.wino_decode(model.ctx, prm, t, bs.clone())
        assert e.value.status == want
        torch.cuda.synchronize()
        assert torch.equal(t, tok)
    prm = P.make_params(B, p, g, lb, cfg.mask_id)
    t1 = tok.clone()
    P.wino_step(model.ctx, prm, t1, bs)
    fresh = P.WinoModel(cfg, wd, B, p + g + lb)
    t2 = tok.clone()
    P.wino_step(fresh.ctx, prm, t2, bs)
    torch.cuda.synchronize()
    assert torch.equal(t1, t2) and not torch.equal(t1, tok)
    model.close()
    fresh.close()


def test_step_is_deterministic(P):
    cfg, w = tiny("wide", seed=6)
    wd = to_device(w)
    p, g, lb, B = 32, 64, 16, 2
    model = P.WinoModel(cfg, wd, B, p + g + lb)
    prm_c = P.make_params(B, p, g, lb, cfg.mask_id)
    tok0 = batch_tokens(cfg, B, p, g, seed=1, fill=[(0, 16, 0.5)])
    a = gpu_step(P, model, prm_c, tok0, [0, 0], [1, 1])
    b = gpu_step(P, model, prm_c, tok0, [0, 0], [1, 1])
    for x, y in zip(a, b):
        assert np.array_equal(x.view(np.uint8), y.view(np.uint8))
    model.close()


# ---------------------------------------------------------------- GEMM tiles
@pytest.mark.parametrize("M,N,K", [(544, 512, 4096), (100, 512, 1024), (1, 256, 256)])
def test_gemm_tiles_within_exact_product_bound(P, M, N, K, monkeypatch):
    """Each entry of the GEMM tile table, forced through WINO_GEMM_TILE (an
    entry that cannot serve the call falls back to the planner's choice),
    against the float64 sum of the same bf16 products.  Products of bf16
    values are exact in fp32, so any order of fp32 additions stays within
    (K-1)*2^-24 * sum|a*w| of that sum.  Ragged M (544 = 2*256 + 32, 100, 1)
    covers the partial row tiles whose waves skip rows past M.  The tiles
    with a third W stage change only when the copies land: they reproduce
    their two-stage twins (entries 6 and 9) bit for bit."""
    gen = torch.Generator().manual_seed(M * 7 + K)
    A = torch.randn(M, K, generator=gen).bfloat16()
    Wt = (torch.randn(N, K, generator=gen) * 0.02).bfloat16()
    ref = A.double() @ Wt.double().T
    bound = (K - 1) * 2.0 ** -24 * (A.double().abs() @ Wt.double().abs().T)
    Ad, Wd = A.cuda(), Wt.cuda()
    outs = {}
    for t in range(16):
        monkeypatch.setenv("WINO_GEMM_TILE", str(t))
        out = torch.full((M, N), float("nan"), device="cuda")
        P.wino_debug_gemm(Ad, Wd, out)
        torch.cuda.synchronize()
        outs[t] = out.cpu()
        err = (outs[t].double() - ref).abs()
        assert bool((err <= bound).all()), (t, float((err / bound.clamp_min(1e-300)).max()))
    assert torch.equal(outs[6], outs[11]) and torch.equal(outs[9], outs[12])




def big_one_layer(name, seed=0, wide=True):
    cfg = wi.preset(name, n_layers=1)
    lhs = wi.wide_lm_head_std(cfg) if wide else None
    w = wi.model_weights(cfg, seed=seed, device="cuda", lm_head_std=lhs, gain_std=0.1)
    return cfg, w
