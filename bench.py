"""Benchmark of one WINO decoding step at the LLaDA-8B shape on one MI355X.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--config bs16|bs1|mmada|tiny]

A "step" is one pass of the whole hot path through the C ABI (wino_step):
embedding, 32 layers of bidirectional attention with the shadow block and
SwiGLU FFN, the final norm of the rows the decision reads, the LM head with its
fused softmax statistics and the draft / verify update, for every sequence of
the batch.  Inputs (random-init bf16 weights of the 8B architecture, seeded
prompts) are resident in HBM before timing starts; each timed step starts from
the same mid-block decoding state (a 32 KB device copy restores it).

One JSON line is printed.  `value` is steps/s; the line also carries
generated tokens/s from a full semi-autoregressive decode, the dominant
kernel's roofline figures measured with HIP events during the timed region,
and the CPU oracle timed on a bounded sample of the same workload.
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


def run_workload(P, wi, cfg, weights, name, steps, warmup, profile_dominant=True, decode=True):
    import torch
    preset, B, p, g, lb, tau1, tau2, img = CONFIGS[name]
    model = P.WinoModel(cfg, weights, B, p + g + lb)
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
    if profile_dominant:
        P.wino_profile(model.ctx, 1 << classes[DOMINANT])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        one_step()
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    dom = P.wino_profile_read(model.ctx)[DOMINANT] if profile_dominant else None
    P.wino_profile(model.ctx, 0)

    # per-kernel breakdown (separate pass, not part of the timed value)
    P.wino_profile(model.ctx, (1 << P._abi.N_KERNEL_CLASSES) - 1)
    for _ in range(2):
        one_step()
    torch.cuda.synchronize()
    per = P.wino_profile_read(model.ctx)
    P.wino_profile(model.ctx, 0)
    kernels = {}
    step_flops = sum(v["flops"] for v in per.values()) / 2
    step_bytes = sum(v["bytes"] for v in per.values()) / 2
    for k, v in per.items():
        if v["launches"] == 0:
            continue
        ms = v["ms"] / 2
        kernels[k] = {"ms_per_step": round(ms, 4), "launches_per_step": v["launches"] // 2,
                      "tflops": round(v["flops"] / 2 / (ms * 1e-3) / 1e12, 2) if v["flops"] else None,
                      "gbs": round(v["bytes"] / 2 / (ms * 1e-3) / 1e9, 1) if v["bytes"] else None}

    if not decode:
        model.close()
        return {"elapsed": elapsed, "dominant": dom, "kernels": kernels,
                "step_flops": step_flops, "step_bytes": step_bytes, "decode": None}
    # full decode from the prompt: generated tokens per second
    pr_tok = wi.initial_tokens(wi.prompts(cfg, B, p, seed=1000, image_prefix=img), g, cfg.mask_id).cuda()
    dbs = torch.zeros(B, dtype=torch.int32, device="cuda")
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    seq_steps, forwards = P.wino_decode(model.ctx, prm, pr_tok, dbs)
    torch.cuda.synchronize()
    dec_s = time.perf_counter() - t1
    model.close()
    return {"elapsed": elapsed, "dominant": dom, "kernels": kernels,
            "step_flops": step_flops, "step_bytes": step_bytes,
            "decode": {"forwards": forwards, "seconds": round(dec_s, 4),
                       "tokens_per_s": round(B * g / dec_s, 2),
                       "steps_per_seq_mean": sum(seq_steps) / len(seq_steps)}}


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
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
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
    return {"workload": f"standalone epilogue, logits [{B}, {2 * lb}, {V}] bf16, {n_buf} rotating buffers",
            "ms_per_call": round(ms, 4), "algorithmic_bytes": algo,
            "gbs": round(algo / (ms * 1e-3) / 1e9, 1),
            "hbm_frac": round(algo / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}


def run_other_configs(P, wi, steps, warmup, names=("mmada", "tiny")):
    """The remaining workload configurations on their own weights: the
    MMaDA-shaped long step (vocabulary 134656, batch 4, prompt and response
    1024, block 64) and the tiny model; step rate, step floors and full-decode
    tokens/s for each."""
    import torch
    out = {}
    for name in names:
        preset, B, p, g, lb, tau1, tau2, img = CONFIGS[name]
        cfg = wi.preset(preset)
        weights = wi.model_weights(cfg, seed=0, device="cuda")
        torch.cuda.synchronize()
        n = steps if cfg.n_layers > 2 else 10 * steps
        r = run_workload(P, wi, cfg, weights, name, n, warmup, profile_dominant=False)
        ms = r["elapsed"] / n * 1e3
        out[name] = {"workload": f"{preset} WINO step, batch {B}, prompt {p}"
                                 + (f" ({img} image-code ids)" if img else "")
                                 + f", gen {g}, block {lb}, tau1 {tau1}, tau2 {tau2}, vocab {cfg.vocab}",
                     "steps_per_s": round(1e3 / ms, 3), "ms_per_step": round(ms, 3),
                     "tflops": round(r["step_flops"] / (ms * 1e-3) / 1e12, 1),
                     "step_floor": {"mfma_ms": round(r["step_flops"] / (PEAK_BF16_TFLOPS * 1e12) * 1e3, 3),
                                    "hbm_ms": round(r["step_bytes"] / (PEAK_HBM_GBS * 1e9) * 1e3, 3)},
                     "tokens_per_s": r["decode"]["tokens_per_s"], "decode": r["decode"],
                     "attention_ms_per_step": r["kernels"].get("attention", {}).get("ms_per_step")}
        del weights
        torch.cuda.empty_cache()
    return out


def cpu_baseline(wi, cfg, weights, name, n_seq=4, n_layers=4):
    """The float64 oracle on a bounded sample of the same step (about 10 s on
    16 host threads): the first n_layers layers for n_seq of the batch's
    sequences, plus the LM head of each one's block rows, extrapolated to
    every layer and every sequence of one batched step."""
    import numpy as np
    import torch
    from oracle import model as M
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info()] or [os.cpu_count()])
    except Exception:  # pragma: no cover
        cores = os.cpu_count()
    preset, B, p, g, lb, tau1, tau2, img = CONFIGS[name]
    n_seq, n_layers = min(n_seq, B), min(n_layers, cfg.n_layers)
    layers = [{k: v.cpu() for k, v in weights["layers"][l].items()} for l in range(n_layers)]
    head = {"final_norm": weights["final_norm"].cpu(), "lm_head": weights["lm_head"].cpu(),
            "lm_bias": weights["lm_bias"].cpu()}
    tok, bs = make_state(wi, cfg, B, p, g, lb, img)
    t_layers = t_head = 0.0
    T = 0
    for s_ in range(n_seq):
        ext, pos, allowed, c0 = M.extended_inputs(tok[s_].numpy(), p, g, lb, int(bs[s_]), cfg.mask_id)
        T = len(ext)
        w1 = dict(head, tok_emb=weights["tok_emb"][torch.as_tensor(ext).cuda()].cpu(), layers=layers)
        t0 = time.perf_counter()
        x = M.forward_residual(w1, cfg, np.arange(len(ext)), pos, allowed, n_layers=n_layers)
        t_layers += time.perf_counter() - t0
        t0 = time.perf_counter()
        h = M.rmsnorm(x[c0:c0 + lb], M.f64(head["final_norm"]), cfg.rms_eps)
        M.lm_logits(w1, h)
        t_head += time.perf_counter() - t0
    per_layer = t_layers / (n_seq * n_layers)
    step_s = B * (cfg.n_layers * per_layer + t_head / n_seq)
    return {"value": round(1.0 / step_s, 6), "unit": "steps/s", "cores": int(cores), "kind": "oracle",
            "seconds_per_step": round(step_s, 2),
            "sample": (f"float64 numpy oracle: {n_layers} of {cfg.n_layers} layers for {n_seq} of {B} "
                       f"sequences (T={T}) took {t_layers:.1f}s ({per_layer:.2f}s per layer and sequence), "
                       f"LM head of their {lb} block rows {t_head:.1f}s; extrapolated to "
                       f"{cfg.n_layers} layers x {B} sequences")}


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "gemm_gateup_swiglu_llada8b_bs16_traffic.txt")
GEMM_SOURCES = [os.path.join(ROOT, "paper_2605_16941_amd", "csrc", f)
                for f in ("common.h", "kernels.h", "k_gemm.hip")]


def measured_traffic():
    """HBM bytes per launch of the dominant kernel (calibrated FETCH_SIZE +
    WRITE_SIZE), from the committed counter summary; None when that summary is
    missing or the GEMM sources have changed since the counters were taken."""
    import hashlib
    try:
        lines = open(TRAFFIC_FILE).read().splitlines()
        rec = dict(l.split("=", 1) for l in lines if "=" in l and not l.startswith("#"))
        h = hashlib.sha256()
        for f in GEMM_SOURCES:
            h.update(open(f, "rb").read())
        if rec.get("source_sha256", "").strip() != h.hexdigest():
            return None
        return float(rec["bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="bs16", choices=sorted(CONFIGS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-bs1", action="store_true")
    ap.add_argument("--no-decode", action="store_true",
                    help="skip the full decode (kernel profiles of the step shape only)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run plain device copies of known size (HBM counter calibration)")
    a = ap.parse_args()
    if a.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the WINO step is benchmarked on a single MI355X; "
              "sharding across GPUs is described, not implemented.", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2605_16941_amd as P
    import wino_inputs as wi

    preset = CONFIGS[a.config][0]
    cfg = wi.preset(preset)
    log(f"generating {preset} weights on the GPU")
    t0 = time.perf_counter()
    weights = wi.model_weights(cfg, seed=0, device="cuda")
    torch.cuda.synchronize()
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

    res = run_workload(P, wi, cfg, weights, a.config, a.steps, a.warmup, decode=not a.no_decode)
    _, B, p, g, lb, tau1, tau2, img = CONFIGS[a.config]
    ms = res["elapsed"] / a.steps * 1e3
    dom = res["dominant"]
    dom_ms = dom["ms"] / max(dom["launches"], 1)
    dom_flops = dom["flops"] / max(dom["launches"], 1)
    achieved = dom_flops / (dom_ms * 1e-3) / 1e12
    line = {
        "metric": METRIC, "value": round(1e3 / ms, 4), "unit": "steps/s", "n_gpus": 1,
        "steps": a.steps, "warmup": a.warmup, "ms_per_step": round(ms, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded random-init weights of the architecture, seeded prompts)",
        "config": {"workload": f"{preset} WINO step, batch {B}, prompt {p}, gen {g}, block {lb}",
                   "batch": B, "prompt_len": p, "gen_len": g, "block_len": lb, "tau1": tau1,
                   "tau2": tau2, "init": "literal (LM head std 0.5/sqrt(d), Zipf bias)"},
        "tokens_per_s": res["decode"]["tokens_per_s"] if res["decode"] else None,
        "decode": res["decode"],
        "roofline": {"bound": "mfma", "kernel": DOMINANT, "achieved": round(achieved, 2),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": measured_traffic(), "avg_launch_ms": round(dom_ms, 4),
                     "flops_per_launch": dom_flops, "launches": dom["launches"]},
        "kernels": res["kernels"],
        # algorithmic work of one step (sum over its kernels) at the MI355X
        # peaks: the step's floor time, and how far the measured step is from it
        "step_floor": {"flops": res["step_flops"], "bytes": res["step_bytes"],
                       "mfma_ms": round(res["step_flops"] / (PEAK_BF16_TFLOPS * 1e12) * 1e3, 3),
                       "hbm_ms": round(res["step_bytes"] / (PEAK_HBM_GBS * 1e9) * 1e3, 3),
                       "frac_of_mfma_floor": round(res["step_flops"] / (PEAK_BF16_TFLOPS * 1e12) * 1e3 / ms, 4)},
    }
    if a.config == "bs16" and not a.no_bs1:
        log("bs1 workload")
        r1 = run_workload(P, wi, cfg, weights, "bs1", a.steps, a.warmup)
        ms1 = r1["elapsed"] / a.steps * 1e3
        line["bs1"] = {"steps_per_s": round(1e3 / ms1, 3), "ms_per_step": round(ms1, 3),
                       "step_floor": {"mfma_ms": round(r1["step_flops"] / (PEAK_BF16_TFLOPS * 1e12) * 1e3, 3),
                                      "hbm_ms": round(r1["step_bytes"] / (PEAK_HBM_GBS * 1e9) * 1e3, 3)},
                       "tokens_per_s": r1["decode"]["tokens_per_s"], "decode": r1["decode"],
                       "kernels": r1["kernels"]}
    if a.config == "bs16" and not a.no_bs1:
        log("standalone epilogue")
        line["epilogue"] = run_epilogue(P, wi)
        log("baseline decoders (bs1)")
        line["baselines"] = run_baselines(P, wi, cfg, weights, "bs1")
        log("other configurations (mmada, tiny)")
        line["configs"] = run_other_configs(P, wi, a.steps, a.warmup)
    if not a.no_cpu_baseline:
        log("cpu baseline (oracle sample)")
        line["cpu_baseline"] = cpu_baseline(wi, cfg, weights, a.config)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
