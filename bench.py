#!/usr/bin/env python3
"""Throughput of the early-exit hot path on one MI355X.

One step = one generation pass of a Llama-7B-shaped decoder (32 layers,
width 4096, 32 heads x 128, SwiGLU 11008, vocab 32000; bf16, random-init
weights): prefill of 64 prompts of 4096 uniform-random tokens, then 256
greedy decode steps, with token-level exit throughout -- per layer the
regular layer for the active rows, the exit test (Eq. 7-8), compaction of
the active list and the decoupled KV generation (Eq. 9) of the rows that
exit; attention runs over the cache of computed and generated entries.
Inputs, weights and the cache are resident in HBM before timing.  The value
is (prefill + decode) tokens/s of the whole pass.

Printed: one JSON line with that value, the roofline of the pass's dominant
kernel (timed live with HIP events inside the timed passes), the 8 x 2048
prefill section (threshold sweep, calibrated thresholds, the no-exit and
fixed-schedule variants, per-kernel MFMA figures), the standalone KV
generation, mapper, exit test and compaction, the fixed-schedule generation,
the GPT2-XL-shaped generation, the BERT-base classification, the tiny f32 decoder, and the CPU oracle on a
bounded sample.

    python bench.py [--steps K] [--warmup W] [--delta D | --budget 0.2] [--metric global]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

PEAK_BF16 = 2.5e15      # dense bf16 MFMA, FLOP/s
PEAK_HBM = 8.0e12       # HBM3E, B/s
HERE = os.path.dirname(os.path.abspath(__file__))
# rocprofv3 traffic summaries: the generation headline (decode attention) and
# the 8 x 2048 prefill section (GEMMs, prefill attention, exit test, compaction)
TRAFFIC_FILES = (os.path.join(HERE, "profiles", "llama7b_generation_64x4096_hbm_traffic.json"),
                 os.path.join(HERE, "profiles", "llama7b_prefill_8x2048_hbm_traffic.json"),
                 os.path.join(HERE, "profiles", "kvgen_4096tok_32layers_mfma_traffic.json"))


# HIP sources each kernel family is built from (its traffic figure is void
# once any of them changes)
FAMILY_SOURCES = {
    "gemm": ("gemm.hip", "common.h"), "kv_generate": ("gemm.hip", "kvgen.hip", "common.h"),
    "attention": ("attention.hip", "common.h"), "attention_decode": ("attention.hip", "common.h"),
    "exit_test": ("exit_test.hip", "common.h"),
    "compact_single": ("compact.hip", "common.h"),
}


def family_sources(fam):
    return FAMILY_SOURCES["gemm" if fam.startswith("gemm_") else fam]


def sources_sha256(files):
    """Hash of the given HIP sources, the same way the traffic summary records it."""
    import hashlib
    h = hashlib.sha256()
    d = os.path.join(HERE, "paper_2601_03700_amd", "csrc")
    for f in sorted(files):
        with open(os.path.join(d, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(fam):
    """HBM bytes per launch of a kernel family from the committed rocprofv3
    FETCH_SIZE / WRITE_SIZE summary (each scaled by what it reads for a
    device copy of known size), or None when the sources of that kernel
    changed after the counters were taken."""
    if fam not in FAMILY_SOURCES and not fam.startswith("gemm_"):
        return None
    for path in TRAFFIC_FILES:
        try:
            with open(path) as fh:
                d = json.load(fh)
        except OSError:
            continue
        k = d.get("kernels", {}).get(fam)
        if k is None:
            continue
        if k.get("source_sha256") != sources_sha256(family_sources(fam)):
            return None
        return k["traffic_bytes"]
    return None


def measured_traffic_ratio(fam):
    """HBM bytes per algorithmic byte of a kernel family from the committed
    summaries (for a kernel whose bytes per launch vary with the workload,
    such as the decode attention with the context length), or None."""
    for path in TRAFFIC_FILES:
        try:
            with open(path) as fh:
                k = json.load(fh).get("kernels", {}).get(fam)
        except OSError:
            continue
        if k is None:
            continue
        if k.get("source_sha256") != sources_sha256(family_sources(fam)):
            return None
        return k.get("traffic_per_algorithmic_byte")
    return None


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2,
                    help="timed generation passes (prefill + decode steps) of the headline")
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--prefill-steps", type=int, default=5,
                    help="timed steps of the 8 x 2048 prefill section")
    ap.add_argument("--delta", type=float, default=None,
                    help="exit threshold of the headline generation; default: calibrated on a "
                         "no-exit pass of the same workload to skip --budget of the token-layers")
    ap.add_argument("--budget", type=float, default=0.20,
                    help="skipped fraction of (token, layer) pairs the headline threshold is "
                         "calibrated to (the paper's operating points are 5-25%%)")
    ap.add_argument("--prefill-delta", type=float, default=0.95,
                    help="threshold of the 8 x 2048 prefill section, the classification and "
                         "the CPU baseline (the prefill configuration's 0.90/0.95/0.99 sweep)")
    ap.add_argument("--metric", choices=("global", "local"), default="global")
    ap.add_argument("--batch", type=int, default=8)
    ap.add_argument("--seq", type=int, default=2048)
    ap.add_argument("--no-extras", action="store_true", help="skip the variant and kernel runs")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-generation", action="store_true",
                    help="skip the generation run (batch 64, 4096-token context, decode steps)")
    ap.add_argument("--no-classification", action="store_true",
                    help="skip the BERT-base classification run (64 x 512 tokens)")
    ap.add_argument("--gen-batch", type=int, default=64)
    ap.add_argument("--gen-context", type=int, default=4096)
    ap.add_argument("--gen-steps", type=int, default=256)
    ap.add_argument("--cpu-tokens", type=int, default=2048)
    ap.add_argument("--cpu-layers", type=int, default=4)
    ap.add_argument("--sections", default="all",
                    help="comma list of the parts to run (profiling runs): headline, prefill, "
                         "variants (prefill no-exit / fixed schedule / sweep), kvgen, hsm, exit, "
                         "generation, gpt2, classification, tiny, cpu; default all")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="copy 256 MiB device to device first (a kernel of known traffic "
                         "for scaling hardware byte counters)")
    args = ap.parse_args()
    every = {"headline", "prefill", "variants", "kvgen", "hsm", "exit", "generation", "gpt2",
             "classification", "tiny", "cpu"}
    sec = every if args.sections == "all" else set(args.sections.split(","))
    if sec - every:
        ap.error(f"unknown sections {sorted(sec - every)}")
    if args.no_extras:
        sec -= {"variants", "kvgen", "hsm", "exit", "tiny"}
    if args.no_cpu_baseline:
        sec.discard("cpu")
    if args.no_generation:
        sec.discard("generation")
    if args.no_classification:
        sec.discard("classification")
    if "variants" in sec:
        sec.add("prefill")
    args.sec = sec
    return args


def layer_counts(exit_layer, n_layers):
    """Active rows entering each layer i = 1..N: tokens with exit layer >= i."""
    import torch
    el = exit_layer.to(torch.int64)
    return [int((el >= i).sum()) for i in range(1, n_layers + 1)]


def step_work(shape, exit_layer, pos):
    """Algorithmic FLOPs / bytes of one prefill step, per kernel family."""
    import torch
    N, D, Dq, F = shape.n_layers, shape.d_model, shape.d_q, shape.d_ff
    el = exit_layer.to(torch.int64).cpu()
    p1 = (pos.to(torch.int64).cpu() + 1).double()
    cnt = layer_counts(el, N)
    w = {
        "gemm_qkv": sum(2.0 * m * D * 3 * Dq for m in cnt),
        "gemm_o": sum(2.0 * m * Dq * D for m in cnt),
        "gemm_gate_up": sum(2.0 * m * D * 2 * F for m in cnt),
        "gemm_down": sum(2.0 * m * F * D for m in cnt),
        # causal attention: QK^T and PV, 2 * 2 * (p+1) * Dq per active query
        "attention": sum(float(4.0 * Dq * p1[el >= i].sum()) for i in range(1, N + 1)),
        # skipped-layer K/V of exited tokens: 2 * D * 2Dq per (token, layer)
        "kv_generate": float(4.0 * D * Dq * (N - el).clamp(min=0).sum()),
    }
    return w, cnt


def family(kernel_name):
    """Work family of a timed kernel name (template arguments ignored), or None."""
    base = kernel_name.strip("()").split("<")[0]
    return {"gemm_qkv": "gemm_qkv", "gemm_o": "gemm_o", "gemm_gate_up": "gemm_gate_up",
            "gemm_down": "gemm_down", "attend_prefill_kernel": "attention",
            "gemm_kv_grouped_kernel": "kv_generate", "gemm_kv_flat_kernel": "kv_generate"}.get(base)


def kernel_table(kern, work, ms, steps):
    """Per-kernel launches, average duration, share of the timed region and,
    for the matrix kernels, achieved TFLOP/s from the algorithmic work."""
    out = {}
    for name, (n_launch, tot) in sorted(kern.items(), key=lambda kv: -kv[1][1]):
        out[name] = {"launches": n_launch, "avg_us": 1e3 * tot / max(n_launch, 1),
                     "share": tot / (ms * steps)}
        f = family(name)
        if f and tot > 0:
            out[name]["tflops"] = work[f] * steps / (tot / 1e3) / 1e12
    return out


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the early-exit hot path is built for a single "
              "MI355X (no sharding, no collectives); run it with --gpus 1.", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import adept_inputs as ai
    from paper_2601_03700_amd import binding as B
    from paper_2601_03700_amd.model import DecoderModel

    B.lib()  # fails loudly when the HIP library is missing
    if not torch.cuda.is_available():
        raise SystemExit("bench.py needs a GPU")
    shape = ai.LLAMA7B
    N, D, Dq = shape.n_layers, shape.d_model, shape.d_q
    Bn, T = args.batch, args.seq
    n_tok = Bn * T
    t0 = time.time()
    weights = ai.decoder_weights_torch(shape, seed=7, device="cuda")
    rope_pos = max(T, args.gen_context + args.gen_steps)
    model = DecoderModel(shape, weights, dtype="bf16", rope_max_pos=rope_pos)
    del weights
    torch.cuda.empty_cache()
    if args.copy_calibration:
        src = torch.ones(1 << 27, dtype=torch.int16, device="cuda")   # 256 MiB
        dst = torch.empty_like(src)
        dst.copy_(src)
        del src, dst
    torch.cuda.synchronize()
    log(f"weights ready in {time.time() - t0:.1f}s; "
        f"{torch.cuda.memory_allocated() / 2**30:.1f} GiB allocated")

    # ---- headline: generation (prefill + decode) with the policy's decisions
    out = {"metric": "tokens/s (prefill+decode) at Llama-7B shape; KV-gen MFMA util %",
           "value": None, "unit": "tokens/s", "n_gpus": 1, "sections": sorted(args.sec)}
    if "headline" in args.sec:
        out = headline(args, model, shape, ai, B, torch, np)
    run_sections(args, out, model, shape, ai, B, torch, np, Bn, T, n_tok)


def headline(args, model, shape, ai, B, torch, np):
    log(f"headline: generation, batch {args.gen_batch}, {args.gen_context}-token prompts, "
        f"{args.gen_steps} decode steps, metric={args.metric}, delta "
        f"{args.delta if args.delta is not None else f'calibrated to skip {args.budget:.0%}'}; "
        f"{args.warmup} warmup + {args.steps} timed passes")
    head = generation_policy(args, model, shape, ai, B, torch, np)
    if args.delta is None:
        how = (f"delta {head['delta']:.6f}, calibrated on a no-exit pass of the same workload "
               f"to skip {args.budget:.0%} of the token-layers")
    else:
        how = f"delta {head['delta']}"
    out = {
        "metric": "tokens/s (prefill+decode) at Llama-7B shape; KV-gen MFMA util %",
        "value": head["tokens_per_s"], "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": head["ms_per_pass"], "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded uniform token ids, random-init N(0,0.02) weights)",
        "config": {"workload": (f"Llama-7B-shaped decoder generation: batch {args.gen_batch}, "
                                f"{args.gen_context}-token prompts prefilled, then "
                                f"{args.gen_steps} greedy decode steps; token-level exit "
                                f"with the policy's own decisions ({args.metric} metric, {how})"),
                   "global_batch": args.gen_batch, "seq_len": args.gen_context + args.gen_steps,
                   "parallelism": "none (one GPU)"},
        "roofline": head.pop("roofline"),
        "generation_policy": head,
    }
    return out


def run_sections(args, out, model, shape, ai, B, torch, np, Bn, T, n_tok):
    N = shape.n_layers
    # ---- prefill 8 x 2048 with the threshold sweep and the per-kernel figures
    ids = torch.from_numpy(ai.token_ids(8, shape.vocab, Bn, T)).cuda()
    cache = model.new_cache(Bn, T)

    def run(cfg, force=None, steps=args.prefill_steps, warmup=2, timing=False):
        for _ in range(warmup):
            res, _ = model.prefill(ids, cfg, cache=cache, logits="last", force_layer=force)
        torch.cuda.synchronize()
        if timing:
            B.timing_reset()
            B.timing_enable(True)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            res, _ = model.prefill(ids, cfg, cache=cache, logits="last", force_layer=force)
        e1.record()
        torch.cuda.synchronize()
        kern = None
        if timing:
            B.timing_enable(False)
            kern = B.timing_read()
        return e0.elapsed_time(e1) / steps, res, kern

    cfg = B.exit_cfg(args.prefill_delta, N, args.metric)
    psteps = args.prefill_steps
    if "prefill" in args.sec:
        prefill_section(args, out, run, cfg, model, shape, ai, B, torch, np, Bn, T, n_tok, ids,
                        cache)
    if "kvgen" in args.sec:
        out["kv_generate_standalone"] = kv_generate_standalone(model, shape, ai, B, torch, np)
    if "hsm" in args.sec:
        out["hsm_standalone"] = hsm_standalone(shape, B, torch, np)
        log(f"hsm (mapper) 4096 rows: {out['hsm_standalone']['call_ms']:.2f} ms, "
            f"{out['hsm_standalone']['tflops']:.0f} TFLOP/s")
    if "exit" in args.sec:
        out["exit_test_standalone"] = exit_test_standalone(shape, ai, B, torch, np, n_tok)

    del cache, ids
    torch.cuda.empty_cache()
    if "generation" in args.sec:
        out["generation_fixed_schedule"] = generation(args, model, shape, ai, B, torch, np)

    if "gpt2" in args.sec:
        out["gpt2_xl_generation"] = gpt2_generation(args, ai, B, torch, np)

    if "classification" in args.sec:
        del model
        torch.cuda.empty_cache()
        out["classification"] = classification(args, ai, B, torch, np)

    if "tiny" in args.sec:
        out["tiny_f32"] = tiny_decoder(ai, B, torch, np)

    if "cpu" in args.sec:
        out["cpu_baseline"] = cpu_baseline(args, shape, ai, np)
    print(json.dumps(out), flush=True)


def prefill_section(args, out, run, cfg, model, shape, ai, B, torch, np, Bn, T, n_tok, ids,
                    cache):
    N = shape.n_layers
    psteps = args.prefill_steps
    ms, res, kern = run(cfg, timing=True, warmup=0 if psteps <= 1 else 2)
    tok_s = n_tok / (ms / 1e3)
    pos = torch.arange(T, dtype=torch.int32).repeat(Bn)
    work, cnt = step_work(shape, res.exit_layer, pos)
    exit_frac = 1.0 - cnt[-1] / n_tok
    log(f"prefill {Bn}x{T}: {ms:.1f} ms/step, {tok_s:.0f} tokens/s, exited {exit_frac:.3%}")
    per_kernel = kernel_table(kern, work, ms, psteps)
    dom = max((k for k in kern if family(k)), key=lambda k: kern[k][1])
    d_launch, d_ms = kern[dom]
    d_flops_launch = work[family(dom)] * psteps / d_launch
    d_avg_s = d_ms / d_launch / 1e3
    achieved = d_flops_launch / d_avg_s
    pre = {
        "workload": (f"Llama-7B-shaped decoder prefill, batch {Bn} x {T}, token-level exit "
                     f"({args.metric} metric, delta {args.prefill_delta})"),
        "tokens_per_s": tok_s, "ms_per_step": ms, "steps": psteps,
        "dominant_kernel": {"bound": "mfma", "kernel": dom, "achieved": achieved / 1e12,
                            "peak": PEAK_BF16 / 1e12, "unit": "TFLOP/s",
                            "frac": achieved / PEAK_BF16,
                            "traffic": measured_traffic(family(dom)),
                            "flops_per_launch": d_flops_launch, "avg_launch_us": d_avg_s * 1e6,
                            "launches": d_launch},
        "exit_fraction": exit_frac,
        "rdc": reduction(res.exit_layer, shape),
        "active_rows_per_layer": cnt,
        "kernels": per_kernel,
    }
    out["prefill_8x2048"] = pre

    if "variants" in args.sec:
        # no-exit reference (delta = +inf) and a fixed exit schedule (i* ~ U{8..31})
        ms_inf, _, _ = run(B.exit_cfg(math.inf, N, args.metric), steps=max(2, psteps // 2),
                           warmup=1)
        sched = torch.from_numpy(ai.forced_exit_layers(3, n_tok, 8, 31)).cuda()
        ms_f, res_f, kern_f = run(cfg, force=sched, steps=max(2, psteps // 2), warmup=1,
                                  timing=True)
        work_f, cnt_f = step_work(shape, res_f.exit_layer, pos)
        pre["no_exit"] = {"tokens_per_s": n_tok / (ms_inf / 1e3), "ms_per_step": ms_inf}
        steps_f = max(2, psteps // 2)
        pre["fixed_schedule"] = {
            "schedule": "exit layer uniform in 8..31 per token (seeded)",
            "tokens_per_s": n_tok / (ms_f / 1e3), "ms_per_step": ms_f,
            "speedup_vs_no_exit": ms_inf / ms_f,
            "rdc": reduction(res_f.exit_layer, shape),
            "active_rows_per_layer": cnt_f,
            "kernels": kernel_table(kern_f, work_f, ms_f, steps_f),
        }
        log(f"prefill no-exit {ms_inf:.1f} ms/step; fixed schedule {ms_f:.1f} ms/step")
        # similarities of a no-exit pass, for the thresholds calibrated to a budget
        from paper_2601_03700_amd.calibrate import SimRecorder
        rec = SimRecorder(N, n_tok, "cuda")
        model.prefill(ids, B.exit_cfg(math.inf, N, args.metric), cache=cache, logits="last",
                      on_layer=rec)
        sims = rec.sims.cpu().numpy()
        del rec
        pre["delta_sweep"] = delta_sweep(args, run, B, N, n_tok, pos, shape, ms_inf, sims)


def skipped_fraction(exit_layer, n_layers):
    """Fraction of (token, layer) pairs a run skipped: layers after each exit."""
    el = exit_layer.to("cpu").long()
    return float((n_layers - el).clamp(min=0).sum()) / (n_layers * el.numel())


def reduction(exit_layer, shape):
    """Compute reduction (RDC) of a run's exit layers, three K/V charges
    (none / the paper's / algorithmic); dense projections of a layer (SwiGLU:
    three FFN matrices, the GELU MLP two) plus the LM head once per token."""
    from paper_2601_03700_amd.accounting import rdc
    return rdc(exit_layer.to("cpu").numpy(), shape.n_layers, shape.d_model, shape.d_q,
               shape.d_ff, shape.vocab, ffn_mats=2 if shape.family == "gpt2" else 3)


def exit_histogram(exit_layer, n_layers):
    import torch
    return torch.bincount(exit_layer.to("cpu").long(), minlength=n_layers + 1)[1:].tolist()


def delta_sweep(args, run, B, N, n_tok, pos, shape, ms_inf, sims):
    """The policy's own decisions: the threshold set {0.90, 0.95, 0.99} of
    the prefill configuration, then thresholds calibrated on the no-exit
    pass's similarities (calibrate.calibrate_delta: the largest delta whose
    running-max count skips the budget) so that 10 / 20 / 25 % of the
    (token, layer) pairs are skipped by the exit test itself."""
    from paper_2601_03700_amd.calibrate import calibrate_delta, skipped_fraction_at
    res_out = {"thresholds": {}, "calibrated": {}}
    for d in (0.90, 0.95, 0.99):
        ms, res, _ = run(B.exit_cfg(d, N, args.metric), steps=2, warmup=1)
        res_out["thresholds"][f"{d:.2f}"] = {
            "tokens_per_s": n_tok / (ms / 1e3), "ms_per_step": ms,
            "skipped_fraction": skipped_fraction(res.exit_layer, N),
            "rdc": reduction(res.exit_layer, shape),
            "exit_layer_histogram": exit_histogram(res.exit_layer, N)}
    for target in (0.10, 0.20, 0.25):
        d = calibrate_delta(sims, target, N)
        ms, res, _ = run(B.exit_cfg(d, N, args.metric), steps=2, warmup=1)
        frac = skipped_fraction(res.exit_layer, N)
        # the all-at-once variant (Appendix H.2) at the same threshold: each
        # prompt's last token decides for the whole prompt
        ms_a, res_a, _ = run(B.exit_cfg(d, N, args.metric, prompt_level=True), steps=2, warmup=1)
        res_out["calibrated"][f"{int(round(target * 100))}%"] = {
            "delta": d, "predicted_skipped_fraction": skipped_fraction_at(sims, d, N),
            "tokens_per_s": n_tok / (ms / 1e3), "ms_per_step": ms,
            "skipped_fraction": frac, "speedup_vs_no_exit": ms_inf / ms,
            "rdc": reduction(res.exit_layer, shape),
            "exit_layer_histogram": exit_histogram(res.exit_layer, N),
            "all_at_once": {"tokens_per_s": n_tok / (ms_a / 1e3), "ms_per_step": ms_a,
                            "skipped_fraction": skipped_fraction(res_a.exit_layer, N),
                            "rdc": reduction(res_a.exit_layer, shape),
                            "exit_layer_histogram": exit_histogram(res_a.exit_layer, N)}}
        log(f"calibrated delta {d:.4f}: {frac:.1%} of token-layers skipped, "
            f"{ms:.1f} ms/step ({ms_inf / ms:.2f}x vs no exit)")
    return res_out


def kv_generate_standalone(model, shape, ai, B, torch, np, reps=10):
    """4096 exited tokens, exit layers uniform in 8..31 of 32, hidden N(0,1):
    K/V for every skipped layer into a [32][4096][32][128] cache, one call."""
    N, D, H, hd, Dq = shape.n_layers, shape.d_model, shape.n_heads, shape.head_dim, shape.d_q
    n = 4096
    g = torch.Generator(device="cuda").manual_seed(11)
    s = torch.randn((n, D), generator=g, device="cuda").to(torch.bfloat16)
    el = torch.from_numpy(ai.forced_exit_layers(12, n, 8, 31)).cuda()
    rows = torch.arange(n, dtype=torch.int32, device="cuda")
    cnt = torch.tensor([n], dtype=torch.int32, device="cuda")
    # NaN sentinel: exactly layers i*+1..N of each slot must be written
    kc = torch.full((N, n, H, hd), float("nan"), dtype=torch.bfloat16, device="cuda")
    vc = torch.full_like(kc, float("nan"))
    ws = torch.empty(B.kv_generate_workspace_bytes(N, n), dtype=torch.uint8, device="cuda")
    w_kv = model.w_qkv[:, Dq:]          # K and V rows of each layer's stacked QKV weight
    # positions 0..4095 (token t at position t and slot t)
    cos = torch.empty((n, hd // 2), dtype=torch.float32, device="cuda")
    sin = torch.empty_like(cos)
    B.rope_table(n, hd, shape.rope_theta, cos, sin)

    def call():
        B.kv_generate(N, D, H, hd, shape.rms_eps, s, rows, cnt, n, el, rows, rows, w_kv,
                      3 * Dq * D, None, cos, sin, kc, vc, n, ws)
    call()
    torch.cuda.synchronize()
    layer = torch.arange(1, N + 1, device="cuda").view(N, 1)
    want = layer > el.view(1, n).long()                      # [N][n]: layer r > i*
    written_k = ~torch.isnan(kc).any(dim=(2, 3))
    written_v = ~torch.isnan(vc).any(dim=(2, 3))
    sentinel_ok = bool(torch.equal(written_k, want) and torch.equal(written_v, want))
    # the whole call without per-launch events, then every launch bracketed
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        call()
    e1.record()
    torch.cuda.synchronize()
    call_ms = e0.elapsed_time(e1) / reps
    B.timing_reset()
    B.timing_enable(True)
    for _ in range(reps):
        call()
    torch.cuda.synchronize()
    B.timing_enable(False)
    k = B.timing_read()
    pairs = int((N - el.long()).clamp(min=0).sum())
    flops = 4.0 * D * Dq * pairs
    grouped = [v for kk, v in k.items()
               if kk.strip("()").startswith(("gemm_kv_grouped_kernel", "gemm_kv_flat_kernel"))]
    assert grouped, f"no grouped KV-generation launch timed: {sorted(k)}"
    g_launch, g_ms = grouped[0]
    gemm_ms = g_ms / g_launch
    log(f"kv generation 4096 tokens: call {call_ms:.3f} ms, grouped GEMM {gemm_ms:.3f} ms = "
        f"{flops / (gemm_ms / 1e3) / PEAK_BF16:.3f} of the bf16 peak")
    return {"tokens": n, "pairs": pairs, "tflop": flops / 1e12, "call_ms": call_ms,
            "sentinel_ok": sentinel_ok, "traffic": measured_traffic("kv_generate"),
            "gemm_ms": gemm_ms, "mfma_util": flops / (gemm_ms / 1e3) / PEAK_BF16,
            "mfma_util_whole_call": flops / (call_ms / 1e3) / PEAK_BF16,
            "kernels": {kk: {"launches": v[0], "avg_us": 1e3 * v[1] / max(v[0], 1)}
                        for kk, v in k.items()}}


def hsm_standalone(shape, B, torch, np, n_rows=4096, reps=5):
    """Hidden state mapper (Section 4.2, Table S1) at the decoder's width for
    n_rows exiting tokens: 144 D^2 FLOPs per row in the four fully connected
    layers (MFMA GEMMs), plus the input and norm row kernels."""
    D = shape.d_model
    g = torch.Generator(device="cuda").manual_seed(21)
    std = 1.0 / math.sqrt(4 * D)

    def rnd(*dims, mean=0.0, sd=std):
        return (torch.randn(dims, generator=g, device="cuda") * sd + mean).to(torch.bfloat16)
    # random-init weights of the Table S1 layer list, drawn on the device
    wd = {"g0": rnd(D, mean=1.0, sd=0.1), "w1": rnd(4 * D, D), "b1": rnd(4 * D),
          "w2": rnd(8 * D, 4 * D), "b2": rnd(8 * D), "w3": rnd(4 * D, 8 * D), "b3": rnd(4 * D),
          "g1": rnd(4 * D, mean=1.0, sd=0.1), "w4": rnd(D, 4 * D), "b4": rnd(D),
          "g2": rnd(D, mean=1.0, sd=0.1),
          "conv": np.random.default_rng(21).normal(0.0, 0.5, (3, 3)), "conv_b": 0.05}
    hw = B.hsm_weights(wd)
    h = torch.randn((n_rows, D), generator=g, device="cuda").to(torch.bfloat16)
    hp = torch.randn((n_rows, D), generator=g, device="cuda").to(torch.bfloat16)
    inertia = torch.randn((n_rows, D), generator=g, device="cuda")
    rows = torch.arange(n_rows, dtype=torch.int32, device="cuda")
    cnt = torch.tensor([n_rows], dtype=torch.int32, device="cuda")
    out = torch.empty_like(h)
    ws = torch.empty(B.hsm_workspace_bytes(D, n_rows), dtype=torch.uint8, device="cuda")

    def call():
        B.hsm_forward(D, shape.rms_eps, hw, rows, cnt, n_rows, h, hp, inertia, 0, out, ws)
    call()
    torch.cuda.synchronize()
    B.timing_reset()
    B.timing_enable(True)
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(reps):
        call()
    e1.record()
    torch.cuda.synchronize()
    B.timing_enable(False)
    k = B.timing_read()
    ms = e0.elapsed_time(e1) / reps
    flops = 144.0 * D * D * n_rows
    fc_ms = sum(v[1] for kk, v in k.items() if kk.startswith("hsm_fc")) / reps
    del wd, h, hp, inertia, out, ws
    return {"d_model": D, "rows": n_rows, "gflop_per_row": 144.0 * D * D / 1e9, "call_ms": ms,
            "tflops": flops / (ms / 1e3) / 1e12, "mfma_util": flops / (ms / 1e3) / PEAK_BF16,
            "fc_gemm_ms": fc_ms, "fc_mfma_util": flops / (fc_ms / 1e3) / PEAK_BF16 if fc_ms else None,
            "kernels": {kk: {"launches": v[0], "avg_us": 1e3 * v[1] / max(v[0], 1)}
                        for kk, v in k.items()}}


def exit_test_standalone(shape, ai, B, torch, np, n_tok, reps=20):
    """Exit test at the prefill shape (16384 rows x 4096, bf16, global metric):
    reads h (2 B/elem) and the inertia (4 B/elem), writes the inertia back."""
    D, N = shape.d_model, shape.n_layers
    g = torch.Generator(device="cuda").manual_seed(5)
    h = torch.randn((n_tok, D), generator=g, device="cuda").to(torch.bfloat16)
    inertia = torch.randn((n_tok, D), generator=g, device="cuda")
    rows = torch.arange(n_tok, dtype=torch.int32, device="cuda")
    cnt = torch.tensor([n_tok], dtype=torch.int32, device="cuda")
    flag = torch.empty(n_tok, dtype=torch.uint8, device="cuda")
    cfg = B.exit_cfg(0.95, N, "global")
    nxt = torch.empty_like(rows)
    ext = torch.empty_like(rows)
    cnt2 = torch.empty(2, dtype=torch.int32, device="cuda")
    el = torch.full((n_tok,), N, dtype=torch.int32, device="cuda")

    def call():
        B.exit_test(D, 5, cfg, rows, cnt, n_tok, h, None, inertia, None, flag)
        B.compact(5, N, flag, rows, cnt, n_tok, nxt, cnt2[0:1], ext, cnt2[1:2], el)
    call()
    torch.cuda.synchronize()
    B.timing_reset()
    B.timing_enable(True)
    for _ in range(reps):
        call()
    torch.cuda.synchronize()
    B.timing_enable(False)
    k = B.timing_read()
    name = [x for x in k if x.startswith("(exit_test_kernel")][0]
    et_launch, et_ms = k[name]
    comp_launch, comp_ms = k.get("compact_single", (reps, 0.0))
    bytes_et = n_tok * (2 * D + 4 * D + 4 * D) + n_tok * (4 + 1)
    bytes_comp = n_tok * (1 + 4 + 4)
    et_s = et_ms / et_launch / 1e3
    comp_s = comp_ms / comp_launch / 1e3
    # the combined metric (global and local cosine) also reads h_prev: 12 D + 5 bytes per row
    h_prev = torch.randn((n_tok, D), generator=g, device="cuda").to(torch.bfloat16)
    cfg_b = B.exit_cfg(0.95, N, "both")
    B.exit_test(D, 5, cfg_b, rows, cnt, n_tok, h, h_prev, inertia, None, flag)
    torch.cuda.synchronize()
    B.timing_reset()
    B.timing_enable(True)
    for _ in range(reps):
        B.exit_test(D, 5, cfg_b, rows, cnt, n_tok, h, h_prev, inertia, None, flag)
    torch.cuda.synchronize()
    B.timing_enable(False)
    kb = B.timing_read()
    both_launch, both_ms = kb[[x for x in kb if x.startswith("(exit_test_kernel")][0]]
    both_s = both_ms / both_launch / 1e3
    bytes_both = n_tok * (2 * D + 2 * D + 8 * D) + n_tok * (4 + 1)
    del h, inertia, h_prev
    # compaction of a 2^26-entry list (multi-pass path): reads flags (1 B) and
    # rows (4 B), writes each row once (4 B) -> 9 B per entry, plus the exit
    # layer (4 B) of each exiting row.  Exit fraction 0.3 is the headline;
    # 0 and 1 bracket it (no exit-layer writes / exit-layer writes that cover
    # whole 64-byte lines), since at 0.3 the exit-layer scatter writes part
    # of every line of a dense row range.
    n_big = 1 << 26
    rows_b = torch.arange(n_big, dtype=torch.int32, device="cuda")
    nxt_b, ext_b = torch.empty_like(rows_b), torch.empty_like(rows_b)
    el_b = torch.full_like(rows_b, N)        # every listed row holds "never exited"
    cnt_b = torch.tensor([n_big, 0, 0], dtype=torch.int32, device="cuda")
    ws_b = torch.empty(B.compact_workspace_bytes(n_big), dtype=torch.uint8, device="cuda")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    by_frac = {}
    for frac in (0.3, 0.0, 1.0):
        g2 = torch.Generator(device="cuda").manual_seed(6)
        flags_b = (torch.rand(n_big, generator=g2, device="cuda") < frac).to(torch.uint8)

        def big():
            B.compact(5, N, flags_b, rows_b, cnt_b[0:1], n_big, nxt_b, cnt_b[1:2], ext_b,
                      cnt_b[2:3], el_b, ws_b)
        big()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(5):
            big()
        e1.record()
        torch.cuda.synchronize()
        t_s = e0.elapsed_time(e1) / 5 / 1e3
        nb = 9.0 * n_big + 4.0 * int(cnt_b[2].item())
        by_frac[str(frac)] = {"us": t_s * 1e6, "gbs": nb / t_s / 1e9, "hbm_frac": nb / t_s / PEAK_HBM}
        del flags_b
    big_s = by_frac["0.3"]["us"] / 1e6
    bytes_big = by_frac["0.3"]["gbs"] * 1e9 * big_s
    del rows_b, nxt_b, ext_b, el_b, ws_b
    # attainable bandwidth of a plain device copy (read + write 512 MiB each)
    src = torch.ones(1 << 27, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    e0.record()
    for _ in range(5):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    copy_s = e0.elapsed_time(e1) / 5 / 1e3
    copy_gbs = 2.0 * src.numel() * 4 / copy_s / 1e9
    del src, dst
    return {"rows": n_tok, "d_model": D, "exit_test_us": et_s * 1e6,
            "exit_test_gbs": bytes_et / et_s / 1e9, "exit_test_hbm_frac": bytes_et / et_s / PEAK_HBM,
            "exit_test_both_metric_us": both_s * 1e6, "exit_test_both_metric_gbs": bytes_both / both_s / 1e9,
            "exit_test_both_metric_hbm_frac": bytes_both / both_s / PEAK_HBM,
            "compact_us": comp_s * 1e6, "compact_gbs": bytes_comp / comp_s / 1e9,
            "compact_2p26_us": big_s * 1e6, "compact_2p26_gbs": bytes_big / big_s / 1e9,
            "compact_2p26_hbm_frac": bytes_big / big_s / PEAK_HBM,
            "compact_2p26_by_exit_fraction": by_frac,
            "copy_512MiB_gbs": copy_gbs,
            "note": "exit-test working set 671 MB > 256 MB MALL; per-layer compaction "
                    "(16K entries) is latency-bound, the 2^26 list measures bandwidth"}


def decode_attention_bytes(shape, el_steps, T):
    """Algorithmic bytes of the decode attention over a pass: each active
    (query, layer) streams the K and V rows (bf16) of its whole context.
    el_steps: [S][B] exit layers of the decode steps' tokens."""
    import torch
    N, H, hd = shape.n_layers, shape.n_heads, shape.head_dim
    el = el_steps.to(torch.int64).cpu()
    total = 0.0
    for k in range(el.shape[0]):
        active = sum(int((el[k] >= i).sum()) for i in range(1, N + 1))
        total += active * (T + k + 1) * H * hd * 2 * 2
    return total


def generation_policy(args, model, shape, ai, B, torch, np, tag="headline"):
    """The headline: generation at the 7B shape with the policy's own exit
    decisions.  One step = one pass: prefill of gen_batch prompts of
    gen_context uniform-random tokens, then gen_steps greedy decode steps
    (each new token through the layers with token-level exit, attention over
    the mixed computed / generated cache).  Unless --delta is given, the
    threshold is calibrated first (Section 4.1 budget): one untimed pass that
    never exits records every layer's similarity of every prompt and decode
    token, and delta is the largest threshold that skips --budget of the
    (token, layer) pairs on it.  Timed: `steps` passes after `warmup` untimed
    ones, each decode-attention launch also timed on its stream; one more
    pass times every launch for the per-kernel table; then the same workload
    with no exit (delta = +inf) for comparison."""
    from paper_2601_03700_amd.calibrate import SimRecorder, calibrate_delta, skipped_fraction_at
    N = shape.n_layers
    Bn, T, S = args.gen_batch, args.gen_context, args.gen_steps
    cache = model.new_cache(Bn, T + S)
    ids = torch.from_numpy(ai.token_ids(9, shape.vocab, Bn, T)).cuda()
    cfg_inf = B.exit_cfg(math.inf, N, args.metric)
    pos_dec = [torch.full((Bn,), T + k, dtype=torch.int32, device="cuda") for k in range(S)]

    def one_pass(cfg, ev=None, rec=None):
        if ev is not None:
            ev[0].record()
        res, _ = model.prefill(ids, cfg, cache=cache, logits="last",
                               on_layer=None if rec is None else rec[0])
        nxt = model.greedy(res.logits)
        if ev is not None:
            ev[1].record()
        els = []
        for k in range(S):
            st = model.decode_step(cache, nxt, pos_dec[k], cfg, pos_max=T + k,
                                   on_layer=None if rec is None else rec[1 + k])
            nxt = model.greedy(st.logits)
            els.append(st.exit_layer)
        if ev is not None:
            ev[2].record()
        return res.exit_layer, torch.stack(els) if els else torch.zeros((0, Bn), dtype=torch.int32)

    t0 = time.time()
    calib = None
    if args.delta is None:
        recs = [SimRecorder(N, Bn * T, "cuda")] + [SimRecorder(N, Bn, "cuda") for _ in range(S)]
        one_pass(cfg_inf, rec=recs)
        sims = torch.cat([r.sims for r in recs], dim=1).cpu().numpy()
        delta = calibrate_delta(sims, args.budget, N)
        calib = {"budget": args.budget, "pass_tokens": int(sims.shape[1]),
                 "predicted_skipped_fraction": skipped_fraction_at(sims, delta, N),
                 "method": "largest delta whose running-max similarity count on a no-exit pass "
                           "of the same workload skips the budget (calibrate.calibrate_delta)"}
        del recs, sims
        log(f"{tag}: delta calibrated to {delta:.6f} for a {args.budget:.0%} budget "
            f"({time.time() - t0:.1f}s)")
    else:
        delta = args.delta
    cfg = B.exit_cfg(delta, N, args.metric)
    for _ in range(args.warmup):
        one_pass(cfg)
    torch.cuda.synchronize()
    log(f"{tag}: cache {2 * cache.k.numel() * 2 / 2**30:.0f} GiB, {args.warmup} warmup "
        f"pass(es) in {time.time() - t0:.1f}s")
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    # only the dominant kernel (the decode attention) is bracketed by events
    # in the timed passes; the per-kernel table comes from one more pass with
    # every launch bracketed
    B.timing_reset()
    B.timing_select("attend_split")
    B.timing_enable(True)
    torch.cuda.synchronize()
    e0.record()
    passes = [one_pass(cfg, evs[k]) for k in range(args.steps)]
    e1.record()
    torch.cuda.synchronize()
    B.timing_enable(False)
    kern = B.timing_read()
    B.timing_select(None)
    B.timing_reset()
    B.timing_enable(True)
    i0, i1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    i0.record()
    one_pass(cfg)
    i1.record()
    torch.cuda.synchronize()
    B.timing_enable(False)
    kern_all = B.timing_read()
    ms_instr = i0.elapsed_time(i1)
    ms_pass = e0.elapsed_time(e1) / args.steps
    prefill_ms = sum(e[0].elapsed_time(e[1]) for e in evs) / args.steps
    decode_ms = sum(e[1].elapsed_time(e[2]) for e in evs) / args.steps
    el_prompt, el_dec = passes[-1]
    # the same workload without exits (no event bracketing)
    n_inf = max(1, min(2, args.steps))
    evi = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(n_inf)]
    one_pass(cfg_inf)
    torch.cuda.synchronize()
    for k in range(n_inf):
        one_pass(cfg_inf, evi[k])
    torch.cuda.synchronize()
    inf_ms = sum(e[0].elapsed_time(e[2]) for e in evi) / n_inf
    inf_prefill = sum(e[0].elapsed_time(e[1]) for e in evi) / n_inf
    inf_decode = sum(e[1].elapsed_time(e[2]) for e in evi) / n_inf
    # the dominant kernel over the timed passes and its roofline
    dom = max(kern, key=lambda k: kern[k][1])
    d_launch, d_ms = kern[dom]
    d_avg_s = d_ms / d_launch / 1e3
    if dom.startswith("attend_split"):
        bytes_launch = sum(decode_attention_bytes(shape, p[1], T) for p in passes) / d_launch
        achieved = bytes_launch / d_avg_s
        ratio = measured_traffic_ratio("attention_decode")
        roofline = {"bound": "hbm", "kernel": dom, "achieved": achieved / 1e9,
                    "peak": PEAK_HBM / 1e9, "unit": "GB/s", "frac": achieved / PEAK_HBM,
                    "traffic": ratio * bytes_launch if ratio else None,
                    "bytes_per_launch": bytes_launch, "avg_launch_us": d_avg_s * 1e6,
                    "launches": d_launch}
    else:
        roofline = {"bound": None, "kernel": dom, "achieved": None, "peak": None, "unit": None,
                    "frac": None, "traffic": None, "avg_launch_us": d_avg_s * 1e6,
                    "launches": d_launch}
    tokens = Bn * (T + S)
    el_all = torch.cat([el_prompt.reshape(-1), el_dec.reshape(-1)]).to(torch.int64)
    out = {
        "delta": delta, "calibration": calib,
        "tokens_per_s": tokens / (ms_pass / 1e3), "ms_per_pass": ms_pass,
        "prefill_ms": prefill_ms, "decode_ms": decode_ms,
        "prefill_tokens_per_s": Bn * T / (prefill_ms / 1e3),
        "decode_tokens_per_s": Bn * S / (decode_ms / 1e3) if S else None,
        "decode_ms_per_step": decode_ms / S if S else None,
        "skipped_fraction": float((N - el_all).clamp(min=0).sum()) / (N * el_all.numel()),
        "prompt_exit_fraction": float((el_prompt < N).to(torch.float64).mean()),
        "prompt_rdc": reduction(el_prompt, shape),
        "decode_exit_fraction": float((el_dec < N).to(torch.float64).mean()) if S else None,
        "decode_rdc": reduction(el_dec.reshape(-1), shape) if S else None,
        "exit_layer_histogram": exit_histogram(el_all, N),
        "exited_fraction_by_layer": [float((el_dec <= i).to(torch.float64).mean())
                                     for i in range(1, N + 1)] if S else None,
        "no_exit": {"tokens_per_s": tokens / (inf_ms / 1e3), "ms_per_pass": inf_ms,
                    "prefill_ms": inf_prefill, "decode_ms": inf_decode, "passes": n_inf},
        "speedup_vs_no_exit": inf_ms / ms_pass,
        "roofline": roofline,
        "instrumented_pass_ms": ms_instr,
        "kernels": {k: {"launches": n, "avg_us": ms * 1e3 / n, "share": ms / ms_instr}
                    for k, (n, ms) in sorted(kern_all.items(), key=lambda kv: -kv[1][1])[:16]},
    }
    log(f"{tag}: {ms_pass:.0f} ms per pass = {out['tokens_per_s']:.0f} tokens/s "
        f"(prefill {prefill_ms:.0f} ms, decode {decode_ms / max(S, 1):.1f} ms/step), "
        f"{out['skipped_fraction']:.1%} of token-layers skipped; no exit {inf_ms:.0f} ms "
        f"({out['speedup_vs_no_exit']:.2f}x); {dom} {roofline.get('frac') or 0:.3f} of its roofline")
    del cache, ids
    torch.cuda.empty_cache()
    return out


def generation(args, model, shape, ai, B, torch, np):
    """Generation at the 7B shape: a batch of gen_context-token prompts is
    prefilled with exits (exit layer uniform in 8..31 per token, seeded), so
    the cache mixes computed and generated entries, then gen_steps greedy
    decode steps run with the same per-token schedule.  A no-exit decode run
    (delta = +inf) over the same cache follows for comparison."""
    N, H, hd, Dq = shape.n_layers, shape.n_heads, shape.head_dim, shape.d_q
    Bn, T, S = args.gen_batch, args.gen_context, args.gen_steps
    s_max = T + S
    t0 = time.time()
    cache = model.new_cache(Bn, s_max)
    ids = torch.from_numpy(ai.token_ids(9, shape.vocab, Bn, T)).cuda()
    cfg = B.exit_cfg(args.prefill_delta, N, args.metric)
    sched_p = torch.from_numpy(ai.forced_exit_layers(5, Bn * T, 8, 31)).cuda()
    sched_d = torch.from_numpy(ai.forced_exit_layers(6, S * Bn, 8, 31)).cuda().view(S, Bn)
    torch.cuda.synchronize()
    tp = time.time()
    res, _ = model.prefill(ids, cfg, cache=cache, logits="last", force_layer=sched_p)
    torch.cuda.synchronize()
    prefill_s = time.time() - tp
    first = model.greedy(res.logits)
    gen_frac = float((N - sched_p.to(torch.float64)).mean() / N)
    log(f"generation: cache {2 * cache.k.numel() * 2 / 2**30:.0f} GiB, prefill of {Bn}x{T} "
        f"in {prefill_s:.2f}s ({time.time() - t0:.1f}s with setup)")
    del res
    torch.cuda.empty_cache()

    def decode(n_steps, force, timing=False, cfg_=cfg):
        nxt = first
        el = []
        for k in range(2):      # warmup at the first two positions (rewritten below)
            pos = torch.full((Bn,), T + k, dtype=torch.int32, device="cuda")
            model.decode_step(cache, nxt, pos, cfg_, force_layer=None if force is None else force[k],
                              pos_max=T + k)
        torch.cuda.synchronize()
        if timing:      # the decode attention only: its roofline is reported below
            B.timing_reset()
            B.timing_select("attend_split")
            B.timing_enable(True)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for k in range(n_steps):
            pos = torch.full((Bn,), T + k, dtype=torch.int32, device="cuda")
            st = model.decode_step(cache, nxt, pos, cfg_,
                                   force_layer=None if force is None else force[k], pos_max=T + k)
            nxt = model.greedy(st.logits)
            el.append(st.exit_layer)
        e1.record()
        torch.cuda.synchronize()
        kern = None
        if timing:
            B.timing_enable(False)
            kern = B.timing_read()
            B.timing_select(None)
        return e0.elapsed_time(e1) / 1e3, torch.stack(el), kern

    dec_s, el, kern = decode(S, sched_d, timing=True)
    exited_by_layer = [float((el <= i).to(torch.float64).mean()) for i in range(1, N + 1)]
    # decode attention: each active (query, head) streams its context's K and V rows
    att = {k: v for k, v in kern.items() if k.startswith("attend_split")}
    att_launch, att_ms = att.get("attend_split_kernel<128>", (0, 0.0))
    ctx_keys = sum(T + k + 1 for k in range(S))          # keys per sequence summed over steps
    active_q = int(sum((el >= i).sum() for i in range(1, N + 1)))   # (token, layer) queries
    att_bytes = (active_q / (S * Bn)) * ctx_keys * Bn * H * hd * 2 * 2   # K + V, bf16
    kinf_s, _, _ = decode(max(8, S // 4), None, cfg_=B.exit_cfg(math.inf, N, args.metric))
    n_inf = max(8, S // 4)
    out = {
        "workload": (f"Llama-7B-shaped generation: batch {Bn}, {T}-token prompts prefilled with "
                     f"exit layer uniform in 8..31 per token, then {S} greedy decode steps with "
                     f"the same per-token schedule"),
        "prefill_tokens_per_s": Bn * T / prefill_s,
        "decode_tokens_per_s": Bn * S / dec_s,
        "decode_ms_per_step": dec_s * 1e3 / S,
        "prefill_plus_decode_tokens_per_s": Bn * (T + S) / (prefill_s + dec_s),
        "no_exit_decode_tokens_per_s": Bn * n_inf / kinf_s,
        "no_exit_decode_ms_per_step": kinf_s * 1e3 / n_inf,
        "generated_cache_fraction_prompt": gen_frac,
        "exited_fraction_by_layer": exited_by_layer,
        "decode_attention": {
            "launches": att_launch, "avg_us": att_ms * 1e3 / max(1, att_launch),
            "bytes_per_step": att_bytes / S,
            "gbs": att_bytes / (att_ms / 1e3) / 1e9 if att_ms else None,
            "hbm_frac": att_bytes / (att_ms / 1e3) / PEAK_HBM if att_ms else None},
    }
    log(f"generation: decode {dec_s * 1e3 / S:.1f} ms/step ({Bn * S / dec_s:.0f} tok/s), "
        f"no-exit {kinf_s * 1e3 / n_inf:.1f} ms/step; decode attention "
        f"{out['decode_attention']['gbs'] or 0:.0f} GB/s")
    del cache
    torch.cuda.empty_cache()
    return out


def gpt2_generation(args, ai, B, torch, np, batch=64, context=768, steps=256):
    """GPT2-XL-shaped decoder (48 layers, width 1600, 25 heads of 64, GELU MLP
    6400, learned positions up to 1024, vocab 50304 tied; bf16, random-init
    weights) generating with the policy's own decisions, as the headline:
    batch 64 prompts of 768 uniform-random tokens prefilled, then 256 greedy
    decode steps (1024 positions, the model's limit), the threshold
    calibrated on a no-exit pass to skip --budget of the token-layers, and
    the same workload without exits beside it."""
    from paper_2601_03700_amd.model import DecoderModel
    shape = ai.GPT2_XL
    t0 = time.time()
    w = ai.gpt2_weights_torch(shape, seed=27, device="cuda")
    model = DecoderModel(shape, w, dtype="bf16")
    del w
    torch.cuda.empty_cache()
    log(f"gpt2-xl: weights ready in {time.time() - t0:.1f}s")
    sub = argparse.Namespace(**vars(args))
    sub.gen_batch, sub.gen_context, sub.gen_steps = batch, context, steps
    sub.steps, sub.warmup, sub.delta = 1, 1, None
    out = generation_policy(sub, model, shape, ai, B, torch, np, tag="gpt2-xl")
    out = {"workload": (f"GPT2-XL-shaped decoder generation: batch {batch}, {context}-token "
                        f"prompts prefilled, then {steps} greedy decode steps; token-level exit "
                        f"with the policy's own decisions ({args.metric} metric, delta "
                        f"{out['delta']:.6f} calibrated to skip {args.budget:.0%})"), **out}
    del model
    torch.cuda.empty_cache()
    return out


def classification(args, ai, B, torch, np, reps=5):
    """BERT-base-shaped encoder classification with token-level exit: batch
    64 x 512 uniform-random tokens, global metric at --delta; also the no-exit
    pass (delta = +inf) and a fixed schedule (exit layer uniform in 3..11 of
    12 per token, seeded) that shows the exit path's cost and benefit."""
    from paper_2601_03700_amd.model import EncoderModel
    shape = ai.BERT_BASE
    N = shape.n_layers
    Bn, T = 64, 512
    n = Bn * T
    t0 = time.time()
    model = EncoderModel(shape, ai.encoder_weights(shape, seed=17, dtype="bf16"))
    ids = torch.from_numpy(ai.token_ids(18, shape.vocab, Bn, T)).cuda()
    log(f"classification: weights ready in {time.time() - t0:.1f}s")

    def run(delta, force=None, timing=False, stop=True):
        cfg = B.exit_cfg(delta, N, args.metric)
        out = model.classify(ids, cfg, force_layer=force, stop_at_cls=stop)
        st = out.state
        out = model.classify(ids, cfg, force_layer=force, state=st, stop_at_cls=stop)
        torch.cuda.synchronize()
        if timing:
            B.timing_reset()
            B.timing_enable(True)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            out = model.classify(ids, cfg, force_layer=force, state=st, stop_at_cls=stop)
        e1.record()
        torch.cuda.synchronize()
        kern = None
        if timing:
            B.timing_enable(False)
            kern = B.timing_read()
        return e0.elapsed_time(e1) / reps, out, kern

    ms, out, _ = run(args.prefill_delta)
    _, _, kern = run(args.prefill_delta, timing=True)     # per-kernel HIP events (separate run)
    el = out.exit_layer.to(torch.int64)
    ms_inf, _, _ = run(math.inf)
    sched = torch.from_numpy(ai.forced_exit_layers(19, n, 3, N - 1)).cuda()
    ms_f, out_f, _ = run(math.inf, force=sched)
    el_f = out_f.exit_layer.to(torch.int64)
    cls_f = out_f.cls_exit_layer.cpu().numpy()
    ms_fg, _, _ = run(math.inf, force=sched, stop=False)
    res = {
        "workload": (f"BERT-base-shaped encoder classification (12 layers, width 768, 12x64 heads, "
                     f"GELU FFN 3072, 2-class head on [CLS]), batch {Bn} x {T}, token-level exit "
                     f"({args.metric} metric, delta {args.prefill_delta})"),
        "sequences_per_s": Bn / (ms / 1e3), "tokens_per_s": n / (ms / 1e3), "ms_per_pass": ms,
        "exit_fraction": float((el < N).to(torch.float64).mean()),
        "no_exit": {"sequences_per_s": Bn / (ms_inf / 1e3), "ms_per_pass": ms_inf},
        "fixed_schedule": {
            "schedule": "exit layer uniform in 3..11 per token (seeded); a sequence's rows "
                        "leave when its [CLS] row exits",
            "sequences_per_s": Bn / (ms_f / 1e3), "ms_per_pass": ms_f,
            "speedup_vs_no_exit": ms_inf / ms_f,
            "active_rows_per_layer": [int((el_f >= i).sum()) for i in range(1, N + 1)],
            "cls_exit_layer_histogram": np.bincount(cls_f, minlength=N + 1)[1:].tolist(),
            "without_cls_stop": {"ms_per_pass": ms_fg, "sequences_per_s": Bn / (ms_fg / 1e3)}},
        "kernels": {k: {"launches": c, "avg_us": t * 1e3 / c,
                        "share": t / sum(x[1] for x in kern.values())}
                    for k, (c, t) in sorted(kern.items(), key=lambda kv: -kv[1][1])[:10]},
    }
    log(f"classification: {ms:.2f} ms/pass ({Bn / (ms / 1e3):.0f} seq/s), no-exit {ms_inf:.2f}, "
        f"fixed schedule {ms_f:.2f} ms ({ms_fg:.2f} without the [CLS] stop)")
    del model
    torch.cuda.empty_cache()
    return res


def tiny_decoder(ai, B, torch, np, prompt=128, steps=32, reps=5):
    """The tiny f32 decoder (4 layers, width 256, 4 x 64 heads, FFN 1024,
    vocab 1024): one 128-token prompt, then 32 greedy steps, local metric
    delta 0.95, against delta = +inf.  Launch-latency-bound at this size."""
    from paper_2601_03700_amd.model import DecoderModel
    shape = ai.TINY
    model = DecoderModel(shape, ai.decoder_weights(shape, seed=21, dtype="f32"), dtype="f32",
                         rope_max_pos=prompt + steps)
    ids = ai.token_ids(22, shape.vocab, 1, prompt)
    out = {"workload": f"tiny f32 decoder, 1 x {prompt}-token prompt + {steps} greedy steps, "
                       "local metric"}
    for name, delta in (("delta_0.95", 0.95), ("no_exit", math.inf)):
        cfg = B.exit_cfg(delta, shape.n_layers, "local")
        model.generate(ids, steps, cfg)      # warm-up
        torch.cuda.synchronize()
        tp = td = 0.0
        for _ in range(reps):
            t0 = time.perf_counter()
            res, cache = model.prefill(ids, cfg, s_max=prompt + steps, logits="last")
            nxt = model.greedy(res.logits)
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            for k in range(steps):
                pos = torch.full((1,), prompt + k, dtype=torch.int32, device="cuda")
                st = model.decode_step(cache, nxt, pos, cfg)
                nxt = model.greedy(st.logits)
            torch.cuda.synchronize()
            t2 = time.perf_counter()
            tp += t1 - t0
            td += t2 - t1
        tp, td = tp / reps, td / reps
        out[name] = {"prefill_tokens_per_s": prompt / tp, "decode_tokens_per_s": steps / td,
                     "combined_tokens_per_s": (prompt + steps) / (tp + td),
                     "prefill_ms": 1e3 * tp, "decode_ms_per_step": 1e3 * td / steps,
                     "prefill_skipped_fraction": skipped_fraction(res.exit_layer, shape.n_layers)}
    log(f"tiny f32: prefill {out['delta_0.95']['prefill_ms']:.2f} ms, decode "
        f"{out['delta_0.95']['decode_ms_per_step']:.2f} ms/step")
    return out


def cpu_baseline(args, shape, ai, np):
    """The oracle (numpy fp64) on a bounded sample of the same workload: one
    sequence of --cpu-tokens tokens through --cpu-layers of the 32 layers at
    full width (plus its LM head over all rows), extrapolated per
    (token x layer) to the 32-layer step."""
    import dataclasses
    from oracle import adept_oracle as O
    L = args.cpu_layers
    sub = dataclasses.replace(shape, n_layers=L)
    log(f"cpu baseline: drawing {L}-layer oracle weights")
    w = O.as64(ai.decoder_weights(sub, seed=7, dtype="bf16"))
    ids = ai.token_ids(8, shape.vocab, 1, args.cpu_tokens)
    cfg = O.ExitConfig(delta=args.prefill_delta, metric=args.metric)
    t0 = time.perf_counter()
    O.prefill(w, sub, ids, cfg)
    dt = time.perf_counter() - t0
    scaled = dt * shape.n_layers / L
    cores = len(os.sched_getaffinity(0))
    log(f"cpu baseline: {dt:.1f}s for the sample")
    # one thread, a smaller sample (256 tokens through 2 layers)
    from threadpoolctl import threadpool_limits
    sub1 = dataclasses.replace(shape, n_layers=2)
    w1 = O.as64(ai.decoder_weights(sub1, seed=7, dtype="bf16"))
    ids1 = ai.token_ids(8, shape.vocab, 1, 256)
    with threadpool_limits(limits=1):
        t1 = time.perf_counter()
        O.prefill(w1, sub1, ids1, cfg)
        dt1 = time.perf_counter() - t1
    one_thread = 256 / (dt1 * shape.n_layers / 2)
    cpu_model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    cpu_model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    log(f"cpu baseline (1 thread): {dt1:.1f}s for 256 tokens x 2 layers")
    return {"value": args.cpu_tokens / scaled, "unit": "tokens/s", "cores": cores,
            "kind": "oracle",
            "sample": (f"1 x {args.cpu_tokens} tokens through {L} of 32 layers at full width "
                       f"(numpy fp64, BLAS on {cores} threads), {dt:.1f}s, extrapolated x{shape.n_layers / L:g} "
                       f"to the 32-layer step; includes the oracle's LM head over all rows"),
            "sample_seconds": dt, "cpu_model": cpu_model,
            "one_thread": {"value": one_thread, "unit": "tokens/s",
                           "sample": "1 x 256 tokens through 2 of 32 layers, extrapolated x16",
                           "sample_seconds": dt1}}


if __name__ == "__main__":
    main()
