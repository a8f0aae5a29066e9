#!/usr/bin/env python3
"""Batch-1 greedy decode throughput: self-speculative vs autoregressive.

One step is one generate call of the workload (prefill of the prompt, then
max_new greedy tokens) through the library's C ABI on seeded synthetic
weights and prompts, with every input already resident in HBM.  The
reported value is self-speculative decode tokens/s (prefill excluded, GPU
time from the library's HIP events); the autoregressive rate of the same
library on the same inputs is reported beside it.

Default workload: LLaMA-2-13B shape (40 layers, d 5120, 40 heads x 128,
FFN 13824, vocab 32000, bf16), prompt 1024 uniform-random ids, 512 new
tokens, 20 random sublayers skipped in the draft, K_max 12, gamma 0.6.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import sd_synth as S  # noqa: E402

HBM_PEAK_GBPS = 8000.0


def step_bytes(cfg, skip, ctx: float, rows: int = 1):
    """Algorithmic HBM bytes of one forward: weights of the sublayers run,
    read once whatever the row count, plus the KV read at ctx positions and
    written for `rows` new positions in the attention sublayers run."""
    es = 2 if cfg.dtype == "bf16" else 4
    d, dh, H, KVH, F = cfg.d_model, cfg.head_dim, cfg.n_heads, cfg.n_kv_heads, cfg.ffn_dim
    attn_w = (cfg.qkv_rows * d + d * H * dh + d) * es
    mlp_w = (3 * d * F + d) * es
    kv_read = 2 * ctx * KVH * dh * es
    kv_write = 2 * rows * KVH * dh * es
    total = (cfg.vocab * d + d) * es + d * es  # lm head, final norm, one embedding row
    for l in range(cfg.n_layers):
        if skip is None or not skip[2 * l]:
            total += attn_w + kv_read + kv_write
        if skip is None or not skip[2 * l + 1]:
            total += mlp_w
    return total


def linear_bytes(cfg, kind: str) -> int:
    es = 2 if cfg.dtype == "bf16" else 4
    d, F = cfg.d_model, cfg.ffn_dim
    return {"qkv": cfg.qkv_rows * d, "o": d * cfg.n_heads * cfg.head_dim, "gate_up": 2 * F * d,
            "down": d * F, "head": cfg.vocab * d}[kind] * es


def cpu_baseline(cfg, weights, prompt, wl, skip, sample_prompt=16, sample_new=4):
    import oracle

    om = oracle.Model(cfg, weights)
    pr = prompt[:sample_prompt]
    t0 = time.perf_counter()
    om.generate_sd(pr, sample_new, skip, wl.k_max, wl.gamma)
    dt = time.perf_counter() - t0
    return {
        "value": round(sample_new / dt, 4), "unit": "tokens/s", "cores": oracle.num_threads(), "kind": "oracle",
        "sample": (f"oracle self-speculative decode of {sample_new} tokens after the first {sample_prompt} prompt "
                   f"tokens (prefill included), same model, mask, K_max and gamma; {dt:.1f} s"),
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="13b", choices=sorted(S.WORKLOADS))
    ap.add_argument("--max-new", type=int, default=None, help="override the workload's generated tokens")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-ar", action="store_true", help="skip the autoregressive comparison")
    args = ap.parse_args()

    if args.gpus != 1:
        print(f"bench.py runs on one GPU: --gpus {args.gpus} is not supported (the decode path is "
              "batch-1 on a single MI355X; see DESIGN.md for how it would shard)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2309_08168_amd import binding

    torch.cuda.set_device(0)
    wl = S.WORKLOADS[args.workload]
    cfg = S.MODELS[wl.model]
    max_new = args.max_new or wl.max_new
    t0 = time.perf_counter()
    host = S.make_weights(cfg, args.seed)
    t_gen = time.perf_counter() - t0
    dw = binding.DeviceWeights(cfg, host)
    torch.cuda.synchronize()
    t_up = time.perf_counter() - t0 - t_gen
    print(f"[bench] {cfg.name}: {cfg.param_count() / 1e9:.2f} B params, generated in {t_gen:.1f} s, "
          f"uploaded in {t_up:.1f} s", file=sys.stderr, flush=True)
    model = binding.Model(cfg, dw)
    prompt = S.prompt(cfg, wl.prompt_len, args.seed)
    skip = S.skip_mask(cfg, wl.mask, args.seed)

    def run_sd():
        return model.generate_sd(prompt, max_new, skip, wl.k_max, wl.gamma)

    def run_ar():
        return model.generate_ar(prompt, max_new)

    for i in range(args.warmup):
        run_sd()
        if not args.no_ar:
            run_ar()
        print(f"[bench] warmup {i + 1}/{args.warmup} done", file=sys.stderr, flush=True)

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    sd_stats = []
    sd_tokens = None
    for i in range(args.steps):
        sd_tokens, st = run_sd()
        sd_stats.append(st)
        print(f"[bench] step {i + 1}/{args.steps}: decode {st['decode_ms']:.1f} ms, stages {st['n_stages']}, "
              f"acceptance {st['n_accepted']}/{st['n_drafted']}", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    ar_stats = []
    ar_tokens = None
    if not args.no_ar:
        for i in range(args.steps):
            ar_tokens, st = run_ar()
            ar_stats.append(st)
        torch.cuda.synchronize()

    dec_ms = sum(s["decode_ms"] for s in sd_stats)
    value = args.steps * max_new / (dec_ms / 1e3)
    drafted = sum(s["n_drafted"] for s in sd_stats)
    accepted = sum(s["n_accepted"] for s in sd_stats)
    steps_d = sum(s["n_draft_steps"] for s in sd_stats)
    stages = sum(s["n_stages"] for s in sd_stats)
    draft_ms = sum(s["draft_ms"] for s in sd_stats) / max(steps_d, 1)
    verify_ms = sum(s["verify_ms"] for s in sd_stats) / max(stages, 1)
    ctx = wl.prompt_len + max_new / 2
    b_draft = step_bytes(cfg, skip, ctx, 1)
    mean_rows = 1 + drafted / max(stages, 1)
    b_verify = step_bytes(cfg, None, ctx, mean_rows)
    extra = {
        "acceptance": round(accepted / drafted, 4) if drafted else None,
        "tokens_per_stage": round(args.steps * max_new / max(stages, 1), 4),
        "draft_step_ms": round(draft_ms, 4),
        "draft_step_GBps": round(b_draft / (draft_ms / 1e3) / 1e9, 1),
        "draft_step_frac_hbm": round(b_draft / (draft_ms / 1e3) / 1e9 / HBM_PEAK_GBPS, 4),
        "verify_step_ms": round(verify_ms, 4),
        "verify_mean_rows": round(mean_rows, 3),
        "verify_step_GBps": round(b_verify / (verify_ms / 1e3) / 1e9, 1),
        "verify_step_frac_hbm": round(b_verify / (verify_ms / 1e3) / 1e9 / HBM_PEAK_GBPS, 4),
        "prefill_ms": round(sum(s["prefill_ms"] for s in sd_stats) / args.steps, 2),
    }
    if ar_stats:
        ar_ms = sum(s["decode_ms"] for s in ar_stats)
        ar_tps = args.steps * max_new / (ar_ms / 1e3)
        b_ar = step_bytes(cfg, None, ctx, 1)
        extra.update({
            "ar_tokens_per_s": round(ar_tps, 2),
            "speedup_vs_ar": round(value / ar_tps, 4),
            "ar_step_ms": round(ar_ms / (args.steps * max_new), 4),
            "ar_step_GBps": round(b_ar / (ar_ms / (args.steps * max_new) / 1e3) / 1e9, 1),
            "ar_step_frac_hbm": round(b_ar / (ar_ms / (args.steps * max_new) / 1e3) / 1e9 / HBM_PEAK_GBPS, 4),
            "sd_equals_ar_tokens": int(np.sum(np.asarray(sd_tokens) == np.asarray(ar_tokens))),
        })

    roofline = {
        "bound": "hbm", "achieved": extra["draft_step_GBps"], "peak": HBM_PEAK_GBPS, "unit": "GB/s",
        "frac": extra["draft_step_frac_hbm"], "traffic": None,
        "kernel": "whole draft step (first measurement)",
    }
    cpu = None
    if not args.no_cpu_baseline:
        print("[bench] timing the oracle on a bounded sample", file=sys.stderr, flush=True)
        cpu = cpu_baseline(cfg, host, prompt, wl, skip)

    line = {
        "metric": "bs1 decode tokens/s self-spec vs autoregressive (13B shape); HBM GB/s",
        "value": round(value, 3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / args.steps, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded N(0, 0.02^2) weights, uniform-random prompt)",
        "config": {"workload": f"{cfg.name}: prompt {wl.prompt_len}, generate {max_new}, mask {wl.mask}, "
                               f"K_max {wl.k_max}, gamma {wl.gamma}", "global_batch": 1,
                   "seq_len": wl.prompt_len + max_new, "parallelism": "none (1 GPU)"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        **extra,
    }
    print(json.dumps(line), flush=True)
    model.close()


if __name__ == "__main__":
    main()
