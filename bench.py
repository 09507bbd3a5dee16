"""Benchmark of one WINO decoding step at the LLaDA-8B shape on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config bs16|bs1|mmada|tiny]
                    [--parts step,bs1,epilogue,baselines,wide,fp16,configs,cpu]

A "step" is one pass of the whole hot path through the C ABI (wino_step):
embedding, 32 layers of bidirectional attention with the shadow block and
SwiGLU FFN, the final norm of the rows the decision reads, the LM head with its
fused softmax statistics and the draft / verify update, for every sequence of
the batch.  Inputs (random-init bf16 weights of the 8B architecture, seeded
prompts) are resident in HBM before timing starts; each timed step starts from
the same mid-block decoding state (a 32 KB device copy restores it).

One JSON line is printed.  `value` is steps/s over K steps timed with no
profiling; the dominant kernel's roofline figures come from HIP events around
its launches in a second timed pass of K steps.  The line also carries
generated tokens/s of full decodes (literal init, and a labelled wide-init
decode with its re-masks), the HBM-bound kernels' bandwidth, the same steps
with fp16 activations, the other workloads, and the float64 CPU oracle timed
per workload on this host.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "WINO denoise steps/s + gen tokens/s, LLaDA-8B shape bs1/bs16; MFMA util %"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0

CONFIGS = {
    # name: (preset, batch, prompt, gen, block, tau1, tau2, image_prefix)
    "bs16": ("llada8b", 16, 256, 256, 32, 0.7, 0.9, 0),
    "bs1": ("llada8b", 1, 256, 256, 32, 0.7, 0.9, 0),
    "mmada": ("mmada8b", 4, 1024, 1024, 64, 0.6, 0.9, 576),
    "tiny": ("tiny", 1, 32, 64, 16, 0.7, 0.9, 0),
}
DOMINANT = "gemm_gateup_swiglu"


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def resident_weights(wi, cfg, **kw):
    """The synthetic weights, generated on the GPU and then placed the way a
    checkpoint load places them: copied to the host, the generator's device
    memory released, and copied back into allocations of their own.  (Tensors
    left where the generator put them, among its recycled temporaries, made
    the batch-1 LM head ~10% slower: 205 against 186 us per launch.)"""
    import torch
    w = wi.model_weights(cfg, device="cuda", **kw)
    host = {k: (v.cpu() if isinstance(v, torch.Tensor) else v) for k, v in w.items() if k != "layers"}
    host["layers"] = [None if lw is None else {k: v.cpu() for k, v in lw.items()} for lw in w["layers"]]
    del w
    torch.cuda.empty_cache()
    out = {k: (v.cuda() if isinstance(v, torch.Tensor) else v) for k, v in host.items() if k != "layers"}
    out["layers"] = [None if lw is None else {k: v.cuda() for k, v in lw.items()} for lw in host["layers"]]
    torch.cuda.synchronize()
    return out


def make_state(wi, cfg, B, p, g, lb, image_prefix, seed=1000):
    """Prompt ids, then a decoded first block and a half-drafted second block."""
    import torch
    pr = wi.prompts(cfg, B, p, seed=seed, image_prefix=image_prefix)
    tok = wi.initial_tokens(pr, g, cfg.mask_id)
    u = wi.uniform(seed, 77, B * g).view(B, g)
    rnd = wi.randint(seed, 78, B * g, 0, cfg.mask_id).view(B, g).to(torch.int32)
    gen = tok[:, p:]
    filled = torch.zeros(B, g, dtype=torch.bool)
    filled[:, :lb] = True
    filled[:, lb:2 * lb] = u[:, lb:2 * lb] < 0.5
    gen[filled] = rnd[filled]
    block_start = torch.full((B,), lb, dtype=torch.int32)
    return tok.contiguous(), block_start


def decode_counts(P, model, prm, tok0, mask_id, max_forwards=4096):
    """The same decode as wino_decode in one call, replayed one batched forward
    per call (the state carried in tokens / block_start / block_steps, which
    reproduces the one-call decode exactly) to count what each forward did:
    drafts (mask -> token, forced drafts and cap fills included) and re-masks
    (token -> mask, Eq. 3).  Not timed."""
    import torch
    B = tok0.shape[0]
    tok = tok0.clone()
    bs = torch.zeros(B, dtype=torch.int32, device="cuda")
    bst = torch.zeros(B, dtype=torch.int32, device="cuda")
    drafts = remasks = forwards = 0
    while not bool(torch.all(bs >= prm.gen_len)) and forwards < max_forwards:
        prev = tok.clone()
        P.wino_decode(model.ctx, prm, tok, bs, block_steps=bst, max_forwards=1)
        drafts += int(((prev == mask_id) & (tok != mask_id)).sum())
        remasks += int(((prev != mask_id) & (tok == mask_id)).sum())
        forwards += 1
    return {"forwards": forwards, "drafts": drafts, "remasks": remasks}


def timed_steps(model, P, one_step, steps, profile_mask=0):
    """steps wino_step calls between two synchronisations; returns seconds
    and, with profile_mask, the per-class event totals of that region."""
    import torch
    P.wino_profile(model.ctx, profile_mask)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        one_step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    prof = P.wino_profile_read(model.ctx) if profile_mask else None
    P.wino_profile(model.ctx, 0)
    return elapsed, prof


def run_workload(P, wi, cfg, weights, name, steps, warmup, profile_dominant=True, decode=True, act=0):
    """The WINO step of workload `name` from a fixed mid-block state: warmup,
    then `steps` timed steps with no profiling (the reported rate), then the
    same number of steps with HIP events around every launch of the dominant
    kernel (its average launch time for the roofline), then two steps with
    events around every launch (the per-kernel breakdown), then a full decode
    from the prompt (tokens/s) and its replay with counts."""
    import torch
    preset, B, p, g, lb, tau1, tau2, img = CONFIGS[name]
    model = P.WinoModel(cfg, weights, B, p + g + lb, act_precision=act)
    prm = P.make_params(B, p, g, lb, cfg.mask_id, tau1, tau2)
    tok0, bs0 = make_state(wi, cfg, B, p, g, lb, img)
    tok0, bs0 = tok0.cuda(), bs0.cuda()
    tok = tok0.clone()
    bs = bs0.clone()
    st0 = torch.ones(B, dtype=torch.int32, device="cuda")
    st = st0.clone()
    flags = torch.empty(B, lb, dtype=torch.uint8, device="cuda")
    nm = torch.empty(B, dtype=torch.int32, device="cuda")

    def one_step():
        tok.copy_(tok0)
        st.copy_(st0)
        P.wino_step(model.ctx, prm, tok, bs, st, flags, nm)

    for _ in range(warmup):
        one_step()
    torch.cuda.synchronize()
    classes = {P.wino_kernel_class_name(i): i for i in range(P._abi.N_KERNEL_CLASSES)}
    elapsed, _ = timed_steps(model, P, one_step, steps)
    dom, elapsed_ev = None, None
    if profile_dominant:
        elapsed_ev, prof = timed_steps(model, P, one_step, steps, 1 << classes[DOMINANT])
        dom = prof[DOMINANT]
    # per-kernel breakdown (separate pass, not part of the timed value)
    _, per = timed_steps(model, P, one_step, 2, (1 << P._abi.N_KERNEL_CLASSES) - 1)
    kernels = {}
    step_flops = sum(v["flops"] for v in per.values()) / 2
    step_bytes = sum(v["bytes"] for v in per.values()) / 2
    for k, v in per.items():
        if v["launches"] == 0:
            continue
        ms = v["ms"] / 2
        kernels[k] = {"ms_per_step": round(ms, 4), "launches_per_step": v["launches"] // 2,
                      "tflops": round(v["flops"] / 2 / (ms * 1e-3) / 1e12, 2) if v["flops"] else None,
                      "gbs": round(v["bytes"] / 2 / (ms * 1e-3) / 1e9, 1) if v["bytes"] else None,
                      "bytes_per_launch": v["bytes"] / max(v["launches"], 1) if v["bytes"] else None,
                      "ms_per_launch": round(v["ms"] / max(v["launches"], 1), 5)}
    out = {"elapsed": elapsed, "elapsed_with_events": elapsed_ev, "dominant": dom, "kernels": kernels,
           "step_flops": step_flops, "step_bytes": step_bytes, "decode": None}
    if decode:
        out["decode"] = timed_decode(P, wi, cfg, model, prm, B, p, g, img)
    model.close()
    return out


def timed_decode(P, wi, cfg, model, prm, B, p, g, img):
    """Full semi-autoregressive decode from the seeded prompts (all response
    positions masked), timed; then its replay with counts."""
    import torch
    pr_tok = wi.initial_tokens(wi.prompts(cfg, B, p, seed=1000, image_prefix=img), g, cfg.mask_id).cuda()
    tok = pr_tok.clone()
    dbs = torch.zeros(B, dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    seq_steps, forwards = P.wino_decode(model.ctx, prm, tok, dbs)
    torch.cuda.synchronize()
    dec_s = time.perf_counter() - t1
    counts = decode_counts(P, model, prm, pr_tok, cfg.mask_id)
    return {"forwards": forwards, "seconds": round(dec_s, 4), "tokens_per_s": round(B * g / dec_s, 2),
            "steps_per_seq_mean": sum(seq_steps) / len(seq_steps), "drafts": counts["drafts"],
            "remasks": counts["remasks"], "replay_forwards": counts["forwards"]}


def run_baselines(P, wi, cfg, weights, name, ms=(1, 4)):
    """Full decodes from the prompt with the Sec. 3 baselines (tokens_per_step
    m: 1 = Eq. 1 greedy, m > 1 naive parallel sampling) and the single-threshold
    rule of WINO+ inference (tau2 = 0: draft only, no shadow block) on the same
    kernels, next to WINO: forwards, tokens/s and WINO's step reduction /
    speedup.  Synthetic weights: the ratios show the mechanism, not accuracy."""
    import torch
    preset, B, p, g, lb, tau1, tau2, img = CONFIGS[name]
    model = P.WinoModel(cfg, weights, B, p + g + lb)
    out = {}
    runs = [("wino", 0, tau2), ("single_threshold", 0, 0.0)] + [(f"tokens_per_step_{m}", m, tau2) for m in ms]
    for label, m, t2 in runs:
        prm = P.make_params(B, p, g, lb, cfg.mask_id, tau1, t2, tokens_per_step=m)
        tok = wi.initial_tokens(wi.prompts(cfg, B, p, seed=1000, image_prefix=img), g, cfg.mask_id).cuda()
        bs = torch.zeros(B, dtype=torch.int32, device="cuda")
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        _, forwards = P.wino_decode(model.ctx, prm, tok, bs)
        torch.cuda.synchronize()
        sec = time.perf_counter() - t0
        out[label] = {"forwards": forwards, "seconds": round(sec, 4), "tokens_per_s": round(B * g / sec, 2)}
    model.close()
    w = out["wino"]
    for m in ms:
        b = out[f"tokens_per_step_{m}"]
        b["wino_step_reduction"] = round(b["forwards"] / w["forwards"], 3)
        b["wino_tps_speedup"] = round(w["tokens_per_s"] / b["tokens_per_s"], 3)
    out["workload"] = f"{preset} decode, batch {B}, prompt {p}, gen {g}, block {lb}, tau1 {tau1}, tau2 {tau2}"
    return out


def run_epilogue(P, wi, n_calls=20, n_buf=4):
    """Standalone WINO epilogue on given bf16 logits [8, 64, 126464] (the
    decision of Eq. 2-4 read from materialised logits), timed with HIP events
    over n_calls calls rotating n_buf logit buffers (more bytes than the 256 MB
    Infinity Cache holds), each call on a fresh copy of the block state, all
    queued behind a spin kernel so the host's per-call overhead is not timed."""
    import torch
    B, lb, V, mask = 8, 32, 126464, 126463
    bufs, curs = [], []
    for i in range(n_buf):
        lg, cur, _ = wi.epilogue_inputs(B, lb, V, mask, seed=2 + 100 * i, device="cuda")
        bufs.append(lg)
        curs.append(cur)
    states = [curs[i % n_buf].clone() for i in range(n_calls)]
    prm = P.make_params(B, 1, lb, lb, mask, 0.7, 0.9)
    ws_bytes = P.wino_epilogue_workspace_bytes(B, lb, V)
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device="cuda")
    bitmap = torch.empty(B, lb, dtype=torch.uint8, device="cuda")
    for i in range(2):
        P.wino_epilogue(prm, V, bufs[i % n_buf], curs[i % n_buf].clone(), bitmap, workspace=ws)
    torch.cuda.synchronize()
    # a spin kernel first, so every call below is queued before the GPU gets to
    # them: the events then time the device work, not the host's call overhead
    torch.cuda._sleep(20_000_000)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for i in range(n_calls):
        P.wino_epilogue(prm, V, bufs[i % n_buf], states[i], bitmap, workspace=ws)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / n_calls
    algo = B * lb * V * 2  # one bf16 row per position is read (Eq. 4)
    out = {"workload": f"standalone epilogue, logits [{B}, {2 * lb}, {V}] bf16, {n_buf} rotating buffers",
           "ms_per_call": round(ms, 4), "algorithmic_bytes": algo,
           "gbs": round(algo / (ms * 1e-3) / 1e9, 1),
           "hbm_frac": round(algo / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4), "traffic": None}
    rec = _summary(MEMBOUND_FILE, MEMBOUND_SOURCES)
    try:
        t = float(rec["epilogue.epilogue_stats.bytes_per_launch"]) + float(rec["epilogue.decide.bytes_per_launch"])
        out.update({"traffic": round(t), "traffic_gbs": round(t / (ms * 1e-3) / 1e9, 1),
                    "traffic_hbm_frac": round(t / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)})
    except (TypeError, KeyError, ValueError):
        pass
    return out


def mmada_cpu_sample(wi, cfg, weights, name):
    """The float64 oracle on one layer of one sequence of the MMaDA workload
    (its weights copied from the device), plus the LM head of that
    sequence's block rows, extrapolated to 32 layers x the batch."""
    import numpy as np
    import torch
    from oracle import model as M
    preset, B, p, g, lb, tau1, tau2, img = CONFIGS[name]
    tok, bs = make_state(wi, cfg, B, p, g, lb, img)
    ext, pos, allowed, c0 = M.extended_inputs(tok[0].numpy(), p, g, lb, int(bs[0]), cfg.mask_id)
    w1 = {"tok_emb": weights["tok_emb"][torch.as_tensor(ext).cuda()].cpu(),
          "layers": [{k: v.cpu() for k, v in weights["layers"][0].items()}],
          "final_norm": weights["final_norm"].cpu(), "lm_head": weights["lm_head"].cpu(),
          "lm_bias": weights["lm_bias"].cpu()}
    cfg1 = wi.preset(preset, n_layers=1)
    t0 = time.perf_counter()
    x = M.forward_residual(w1, cfg1, np.arange(len(ext)), pos, allowed)
    t_layer = time.perf_counter() - t0
    t0 = time.perf_counter()
    M.lm_logits(w1, M.rmsnorm(x[c0:c0 + lb], M.f64(w1["final_norm"]), cfg.rms_eps))
    t_head = time.perf_counter() - t0
    step_s = B * (cfg.n_layers * t_layer + t_head)
    return {"value": round(1.0 / step_s, 6), "unit": "steps/s", "seconds_per_step": round(step_s, 1),
            "kind": "oracle", "sample": f"1 layer of 1 sequence (T={len(ext)}) {t_layer:.1f}s + LM head of "
                                        f"{lb} rows {t_head:.1f}s, extrapolated to {cfg.n_layers} layers x {B} sequences"}


def run_other_configs(P, wi, steps, warmup, names=("mmada", "tiny"), cpu_sample=True):
    """The remaining workload configurations on their own weights: the
    MMaDA-shaped long step (vocabulary 134656, batch 4, prompt and response
    1024, block 64) and the tiny model; step rate, step floors and full-decode
    tokens/s for each."""
    import torch
    out = {}
    for name in names:
        preset, B, p, g, lb, tau1, tau2, img = CONFIGS[name]
        cfg = wi.preset(preset)
        weights = resident_weights(wi, cfg, seed=0)
        n = steps if cfg.n_layers > 2 else 10 * steps
        r = run_workload(P, wi, cfg, weights, name, n, warmup, profile_dominant=False)
        cpu = mmada_cpu_sample(wi, cfg, weights, name) if (cpu_sample and name == "mmada") else None
        ms = r["elapsed"] / n * 1e3
        out[name] = {"workload": f"{preset} WINO step, batch {B}, prompt {p}"
                                 + (f" ({img} image-code ids)" if img else "")
                                 + f", gen {g}, block {lb}, tau1 {tau1}, tau2 {tau2}, vocab {cfg.vocab}",
                     "steps_per_s": round(1e3 / ms, 3), "ms_per_step": round(ms, 3),
                     "tflops": round(r["step_flops"] / (ms * 1e-3) / 1e12, 1),
                     "step_floor": {"mfma_ms": round(r["step_flops"] / (PEAK_BF16_TFLOPS * 1e12) * 1e3, 3),
                                    "hbm_ms": round(r["step_bytes"] / (PEAK_HBM_GBS * 1e9) * 1e3, 3)},
                     "tokens_per_s": r["decode"]["tokens_per_s"], "decode": r["decode"],
                     "attention_ms_per_step": r["kernels"].get("attention", {}).get("ms_per_step"),
                     "kernels": r["kernels"]}
        if cpu:
            out[name]["cpu_baseline"] = cpu
        del weights
        torch.cuda.empty_cache()
    return out


def run_wide(P, wi, cfg, weights, name="bs1", ms=(1, 4)):
    """The labelled wide-init decode: the same backbone with the LM head drawn
    with std sqrt(0.5/sqrt(d)) instead of 0.5/sqrt(d) (wider confidence
    spread), decoded from the prompt; forwards, drafts, re-masks, tokens/s and
    the step reduction against the fixed-schedule baselines (G/M forwards for
    M tokens per step, Sec. 3; their time per forward does not depend on the
    weights, so their tokens/s is taken on this model too)."""
    import torch
    preset, B, p, g, lb, tau1, tau2, img = CONFIGS[name]
    head = wi.model_weights(cfg, seed=0, device="cuda", lm_head_std=wi.wide_lm_head_std(cfg), layers=[])
    wide = dict(weights, lm_head=head["lm_head"])
    model = P.WinoModel(cfg, wide, B, p + g + lb)
    out = {"workload": f"{preset} decode, batch {B}, prompt {p}, gen {g}, block {lb}, tau1 {tau1}, tau2 {tau2}, "
                       f"wide LM head (std {wi.wide_lm_head_std(cfg):.4f}) + Zipf bias"}
    prm = P.make_params(B, p, g, lb, cfg.mask_id, tau1, tau2)
    out["wino"] = timed_decode(P, wi, cfg, model, prm, B, p, g, img)
    for m in ms:
        prm_m = P.make_params(B, p, g, lb, cfg.mask_id, tokens_per_step=m)
        tok = wi.initial_tokens(wi.prompts(cfg, B, p, seed=1000, image_prefix=img), g, cfg.mask_id).cuda()
        bs = torch.zeros(B, dtype=torch.int32, device="cuda")
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        _, fw = P.wino_decode(model.ctx, prm_m, tok, bs)
        torch.cuda.synchronize()
        sec = time.perf_counter() - t0
        out[f"tokens_per_step_{m}"] = {"forwards": fw, "seconds": round(sec, 4),
                                       "tokens_per_s": round(B * g / sec, 2),
                                       "wino_step_reduction": round(fw / out["wino"]["forwards"], 3),
                                       "wino_tps_speedup": round(out["wino"]["tokens_per_s"] * sec / (B * g), 3)}
    model.close()
    del head, wide
    torch.cuda.empty_cache()
    return out


def host_cores():
    """Host threads the oracle's BLAS uses, the cores this process may run
    on, and the CPU model."""
    try:
        from threadpoolctl import threadpool_info
        blas = max([i.get("num_threads", 1) for i in threadpool_info()] or [0])
    except Exception:  # pragma: no cover
        blas = 0
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        avail = os.cpu_count()
    model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:  # pragma: no cover
        pass
    return {"blas_threads": blas or avail, "cpus_available": avail, "cpu_model": model}


def cpu_baselines(wi, weights):
    """The float64 oracle, unchanged, timed on this host per workload:
    the tiny model's full decode and the standalone epilogue in full, and one
    whole step of the LLaDA-8B batch-1 workload (all 32 layers and the LM
    head of the block rows), which batch 16 repeats for 16 independent
    sequences (extrapolated).  The MMaDA workload's sample is taken in
    run_other_configs, where its weights exist."""
    import numpy as np
    import torch
    from oracle import epilogue as E
    from oracle import model as M
    from oracle import wino as W
    hc = host_cores()
    out = {"host": hc}
    # tiny model: full decode
    preset, B, p, g, lb, tau1, tau2, img = CONFIGS["tiny"]
    cfg_t = wi.preset(preset)
    wt = wi.model_weights(cfg_t, seed=0)
    prm = W.Params(p, g, lb, cfg_t.mask_id, float(np.float32(tau1)), float(np.float32(tau2)))
    tok = wi.initial_tokens(wi.prompts(cfg_t, B, p, seed=1000), g, cfg_t.mask_id)[0].numpy()
    t0 = time.perf_counter()
    _, steps = W.decode(W.ModelProvider(wt, cfg_t), tok, prm)
    sec = time.perf_counter() - t0
    out["tiny"] = {"tokens_per_s": round(B * g / sec, 2), "steps_per_s": round(sum(steps) / sec, 3),
                   "seconds": round(sec, 3), "sample": f"full decode of {g} positions ({sum(steps)} steps)"}
    # standalone epilogue: one call in full
    Bq, lbq, V, mask = 8, 32, 126464, 126463
    logits, cur, _ = wi.epilogue_inputs(Bq, lbq, V, mask, seed=2, device="cuda")
    logits, cur = logits.cpu(), cur.cpu()
    t0 = time.perf_counter()
    E.decide(logits, cur.numpy(), mask, float(np.float32(0.7)), float(np.float32(0.9)))
    sec = time.perf_counter() - t0
    out["epilogue"] = {"ms_per_call": round(sec * 1e3, 1), "seconds": round(sec, 3),
                       "sample": f"one call on logits [{Bq}, {2 * lbq}, {V}]"}
    del logits
    # LLaDA-8B shape, batch 1: one whole step
    preset, B, p, g, lb, tau1, tau2, img = CONFIGS["bs1"]
    cfg = wi.preset(preset)
    prm = W.Params(p, g, lb, cfg.mask_id, float(np.float32(tau1)), float(np.float32(tau2)))
    tok, bs = make_state(wi, cfg, B, p, g, lb, img)
    wc = {k: (v.cpu() if isinstance(v, torch.Tensor) else v) for k, v in weights.items() if k != "layers"}
    wc["layers"] = [{k: v.cpu() for k, v in lw.items()} for lw in weights["layers"]]
    t0 = time.perf_counter()
    W.step(W.ModelProvider(wc, cfg), tok[0].numpy(), prm, int(bs[0]), 1)
    step_s = time.perf_counter() - t0
    del wc
    out["bs1"] = {"steps_per_s": round(1.0 / step_s, 5), "seconds_per_step": round(step_s, 2),
                  "sample": f"one whole step ({cfg.n_layers} layers, T={p + g + lb}, LM head of {lb} rows)"}
    out["bs16"] = {"steps_per_s": round(1.0 / (16 * step_s), 6), "seconds_per_step": round(16 * step_s, 1),
                   "sample": "extrapolated: 16 x the batch-1 step (sequences are independent)"}
    return out


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_gateup_swiglu_llada8b_bs16_traffic.txt")
CSRC = os.path.join(ROOT, "paper_2605_16941_amd", "csrc")
GEMM_SOURCES = [os.path.join(CSRC, f) for f in ("common.h", "kernels.h", "k_gemm.hip")]
MEMBOUND_FILE = os.path.join(ROOT, "profiles", "memory_bound_kernels_hbm_traffic.txt")
MEMBOUND_SOURCES = [os.path.join(CSRC, f) for f in ("common.h", "kernels.h", "k_gemm.hip", "k_norm.hip",
                                                    "k_decide.hip")]
# kernel classes whose roofline is HBM bandwidth, per workload
MEMBOUND = {"bs16": ("rmsnorm", "embed_norm", "select_norm", "decide"),
            "bs1": ("lm_head_stats", "rmsnorm", "embed_norm", "select_norm", "decide")}


def _summary(path, sources):
    """key=value records of a committed counter summary, or None when it is
    missing or the kernel sources have changed since the counters were taken."""
    import hashlib
    try:
        lines = open(path).read().splitlines()
        rec = dict(l.split("=", 1) for l in lines if "=" in l and not l.startswith("#"))
        h = hashlib.sha256()
        for f in sources:
            h.update(open(f, "rb").read())
        if rec.get("source_sha256", "").strip() != h.hexdigest():
            return None
        return rec
    except (OSError, ValueError):
        return None


def measured_traffic():
    """HBM bytes per launch of the dominant kernel (calibrated FETCH_SIZE +
    WRITE_SIZE), from the committed counter summary; None when that summary is
    missing or the GEMM sources have changed since the counters were taken."""
    rec = _summary(TRAFFIC_FILE, GEMM_SOURCES)
    try:
        return float(rec["bytes_per_launch"]) if rec else None
    except (KeyError, ValueError):
        return None


def memory_bound(kernels, name):
    """Per HBM-bound kernel class of a workload: algorithmic bytes per launch,
    event-timed GB/s and fraction of the 8 TB/s peak, and, where the committed
    counter summary is current, the measured HBM bytes per launch
    (FETCH_SIZE + WRITE_SIZE, calibrated) and the bandwidth they give."""
    rec = _summary(MEMBOUND_FILE, MEMBOUND_SOURCES) or {}
    out = {}
    for k in MEMBOUND.get(name, ()):
        v = kernels.get(k)
        if not v or not v.get("bytes_per_launch"):
            continue
        ms = v["ms_per_launch"]
        algo = v["bytes_per_launch"]
        e = {"bytes_per_launch": round(algo), "us_per_launch": round(ms * 1e3, 2),
             "gbs": round(algo / (ms * 1e-3) / 1e9, 1),
             "hbm_frac": round(algo / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4), "traffic": None}
        t = rec.get(f"{name}.{k}.bytes_per_launch")
        if t is not None:
            e["traffic"] = float(t)
            e["traffic_gbs"] = round(float(t) / (ms * 1e-3) / 1e9, 1)
            e["traffic_hbm_frac"] = round(float(t) / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)
        out[k] = e
    return out


def step_floor(r, ms):
    return {"flops": r["step_flops"], "bytes": r["step_bytes"],
            "mfma_ms": round(r["step_flops"] / (PEAK_BF16_TFLOPS * 1e12) * 1e3, 3),
            "hbm_ms": round(r["step_bytes"] / (PEAK_HBM_GBS * 1e9) * 1e3, 3),
            "frac_of_mfma_floor": round(r["step_flops"] / (PEAK_BF16_TFLOPS * 1e12) * 1e3 / ms, 4)}


PARTS = ("step", "bs1", "epilogue", "baselines", "wide", "fp16", "configs", "cpu")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="bs16", choices=sorted(CONFIGS))
    ap.add_argument("--parts", default=",".join(PARTS),
                    help="comma list of " + ", ".join(PARTS) + " (the headline step always runs "
                         "unless 'step' is left out and another part is named)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-bs1", action="store_true", help="only the headline workload (and the CPU baseline)")
    ap.add_argument("--no-decode", action="store_true",
                    help="skip the full decodes (kernel profiles of the step shape only)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run plain device copies of known size (HBM counter calibration)")
    a = ap.parse_args()
    if a.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the WINO step is benchmarked on a single MI355X; "
              "sharding across GPUs is described, not implemented.", file=sys.stderr)
        sys.exit(2)
    parts = set(x.strip() for x in a.parts.split(",") if x.strip())
    if a.no_cpu_baseline:
        parts.discard("cpu")
    if a.no_bs1 or a.config != "bs16":
        parts -= {"bs1", "epilogue", "baselines", "wide", "configs"}

    import torch
    import paper_2605_16941_amd as P
    import wino_inputs as wi

    preset = CONFIGS[a.config][0]
    cfg = wi.preset(preset)
    log(f"generating {preset} weights on the GPU")
    t0 = time.perf_counter()
    weights = resident_weights(wi, cfg, seed=0)
    log(f"weights ready in {time.perf_counter() - t0:.1f}s")

    if a.copy_calibration:
        # 3 copies of 512 MiB: each reads and writes exactly 512 MiB of HBM
        src = torch.empty(1 << 28, dtype=torch.int16, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log("copy calibration done (3 x 512 MiB)")

    _, B, p, g, lb, tau1, tau2, img = CONFIGS[a.config]
    line = {"metric": METRIC, "value": None, "unit": "steps/s", "n_gpus": 1, "steps": a.steps,
            "warmup": a.warmup, "ms_per_step": None, "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic (seeded random-init weights of the architecture, seeded prompts)",
            "config": {"workload": f"{preset} WINO step, batch {B}, prompt {p}, gen {g}, block {lb}",
                       "batch": B, "prompt_len": p, "gen_len": g, "block_len": lb, "tau1": tau1,
                       "tau2": tau2, "init": "literal (LM head std 0.5/sqrt(d), Zipf bias)"}}
    if "step" in parts or not (parts - {"cpu"}):
        log(f"{a.config} step")
        res = run_workload(P, wi, cfg, weights, a.config, a.steps, a.warmup, decode=not a.no_decode)
        ms = res["elapsed"] / a.steps * 1e3
        dom = res["dominant"]
        dom_ms = dom["ms"] / max(dom["launches"], 1)
        dom_flops = dom["flops"] / max(dom["launches"], 1)
        achieved = dom_flops / (dom_ms * 1e-3) / 1e12
        line.update({
            "value": round(1e3 / ms, 4), "ms_per_step": round(ms, 3),
            "tokens_per_s": res["decode"]["tokens_per_s"] if res["decode"] else None,
            "decode": res["decode"],
            "roofline": {"bound": "mfma", "kernel": DOMINANT, "achieved": round(achieved, 2),
                         "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                         "traffic": measured_traffic(), "avg_launch_ms": round(dom_ms, 4),
                         "flops_per_launch": dom_flops, "launches": dom["launches"],
                         # the events around each launch of the dominant kernel
                         # ran in a second timed pass of the same steps
                         "ms_per_step_with_events": round(res["elapsed_with_events"] / a.steps * 1e3, 3)},
            "kernels": res["kernels"],
            "memory_bound": memory_bound(res["kernels"], a.config),
            # algorithmic work of one step (sum over its kernels) at the MI355X
            # peaks: the step's floor time, and how far the measured step is from it
            "step_floor": step_floor(res, ms)})
    if "bs1" in parts:
        log("bs1 workload")
        r1 = run_workload(P, wi, cfg, weights, "bs1", a.steps, a.warmup, decode=not a.no_decode)
        ms1 = r1["elapsed"] / a.steps * 1e3
        line["bs1"] = {"steps_per_s": round(1e3 / ms1, 3), "ms_per_step": round(ms1, 3),
                       "step_floor": step_floor(r1, ms1),
                       "tokens_per_s": r1["decode"]["tokens_per_s"] if r1["decode"] else None,
                       "decode": r1["decode"], "kernels": r1["kernels"],
                       "memory_bound": memory_bound(r1["kernels"], "bs1")}
    if "epilogue" in parts:
        log("standalone epilogue")
        line["epilogue"] = run_epilogue(P, wi)
    if "baselines" in parts:
        log("baseline decoders (bs1)")
        line["baselines"] = run_baselines(P, wi, cfg, weights, "bs1")
    if "wide" in parts:
        log("wide-init decode (bs1)")
        line["wide_decode"] = run_wide(P, wi, cfg, weights, "bs1")
    if "fp16" in parts:
        log("fp16 activations (bs16, bs1)")
        f16 = {"note": "the same steps with fp16 activations and fp16 copies of the weight matrices "
                       "(act_precision = WINO_ACT_FP16); the headline value is bf16"}
        for name in ("bs16", "bs1"):
            r = run_workload(P, wi, cfg, weights, name, a.steps, a.warmup, decode=False, act=P.ACT_FP16)
            ms_f = r["elapsed"] / a.steps * 1e3
            gu = r["kernels"].get(DOMINANT, {})
            f16[name] = {"ms_per_step": round(ms_f, 3), "steps_per_s": round(1e3 / ms_f, 4),
                         "gemm_gateup_tflops": gu.get("tflops"),
                         "attention_ms_per_step": r["kernels"].get("attention", {}).get("ms_per_step")}
        line["fp16"] = f16
    if "cpu" in parts:
        log("cpu baselines (oracle)")
        cb = cpu_baselines(wi, weights)
        hc = cb["host"]
        head = cb[a.config] if a.config in cb else cb["bs1"]
        line["cpu_baseline"] = {"value": head["steps_per_s"], "unit": "steps/s", "cores": hc["blas_threads"],
                                "kind": "oracle", "sample": head["sample"],
                                "cpus_available": hc["cpus_available"], "cpu_model": hc["cpu_model"]}
        # oracle tokens/s at the GPU decode's step counts (extrapolated: the
        # oracle ran one step, not the decode)
        for key, dec in (("bs16", (line.get("decode") if a.config == "bs16" else None)),
                         ("bs1", (line.get("bs1") or {}).get("decode"))):
            if dec and key in cb and dec.get("forwards"):
                _, Bk, _, gk, _, _, _, _ = CONFIGS[key]
                cb[key]["tokens_per_s_extrapolated"] = round(Bk * gk / (dec["forwards"] / cb[key]["steps_per_s"]), 5)
        line["cpu_baselines"] = cb
    if "configs" in parts:
        del weights
        torch.cuda.empty_cache()
        log("other configurations (mmada, tiny)")
        line["configs"] = run_other_configs(P, wi, a.steps, a.warmup, cpu_sample="cpu" in parts)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
