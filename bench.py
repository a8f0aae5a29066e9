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

Other modes:
  --verify-micro        verification-forward latency, GB/s and MFMA use at
                        the 13B shape for M in {1, 4, 8, 13, 16} rows over a
                        KV cache of 512 / 2048 / 4096 N(0, 1) positions
  --supplementary       labelled planted-redundancy runs (skipped sublayers'
                        output projections scaled down, lm-head scaled up),
                        static and adaptive draft exit; --supp-mask picks
                        another skip set (e.g. random36, the paper's 13B
                        skip count); --fp8-draft adds runs whose draft reads
                        FP8 copies of its weights
  --sampling            labelled runs of the sampling variant (temperature and
                        top-p as in the paper's appendix) against autoregressive
                        sampling, static and adaptive exit, random and planted
                        weights
  --calibrate-copy      a plain device copy of known size, for scaling the
                        FETCH_SIZE / WRITE_SIZE profiler counters
  --summarize-stats / --summarize-pmc   write profiles/ summaries from
                        rocprofv3 CSV output
"""

from __future__ import annotations

import argparse
import csv
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import sd_synth as S  # noqa: E402

HBM_PEAK_GBPS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
KERNEL_SOURCE = os.path.join(ROOT, "paper_2309_08168_amd", "csrc", "kernels_linear.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "pmc_verify2_13b.json")


def log(msg: str):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def step_bytes(cfg, skip, ctx: float, rows: float = 1, fp8: bool = False):
    """Algorithmic HBM bytes of one forward: weights of the sublayers run,
    read once whatever the row count, plus the KV read at ctx positions and
    written for `rows` new positions in the attention sublayers run.  fp8:
    the sublayers' four weight matrices are FP8 copies (one byte per weight
    and a 4-byte exponent per output row); norms and the lm-head stay bf16."""
    es = 2 if cfg.dtype == "bf16" else 4
    d, dh, H, KVH, F = cfg.d_model, cfg.head_dim, cfg.n_heads, cfg.n_kv_heads, cfg.ffn_dim
    if fp8:
        attn_w = cfg.qkv_rows * d + d * H * dh + 4 * (cfg.qkv_rows + d) + d * es
        mlp_w = 3 * d * F + 4 * (2 * F + d) + d * es
    else:
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


def gate_up_bytes(n: int, k: int, rows: float, es: int = 2) -> float:
    """Algorithmic bytes of one gate/up launch with the RMSNorm folded in:
    the n x k weights (gate and up rows) and the norm gain once, the float32
    input rows, and the float32 SwiGLU outputs (n / 2 per row)."""
    return n * k * es + k * es + rows * k * 4 + rows * (n // 2) * 4


def source_hash() -> str:
    return hashlib.sha256(open(KERNEL_SOURCE, "rb").read()).hexdigest()[:16]


def traffic_for(kernel: str, workload: str = "13b"):
    """HBM bytes per launch from the committed counter summary, if it was
    taken on the current kernel source and on the same workload's shapes
    (the summary is the 13B verification microbenchmark's)."""
    try:
        t = json.load(open(TRAFFIC_FILE))
    except (OSError, ValueError):
        return None
    e = t.get("kernels", {}).get(kernel)
    if not e or t.get("source_hash") != source_hash() or t.get("workload", "13b") != workload:
        return None
    return e["bytes_per_launch"]


def prefill_flops(cfg, M: int) -> float:
    """Useful flops of the full-model forward of M rows from position 0:
    every linear layer (2 M N K) and causal attention (scores and weighted
    values, 2 head_dim flops per query-key pair each)."""
    hd = cfg.n_heads * cfg.head_dim
    nq = (cfg.n_heads + 2 * cfg.n_kv_heads) * cfg.head_dim
    lin = nq * cfg.d_model + cfg.d_model * hd + 2 * cfg.ffn_dim * cfg.d_model + cfg.d_model * cfg.ffn_dim
    attn = 2 * 2 * cfg.head_dim * cfg.n_heads * M * (M + 1) / 2
    return cfg.n_layers * (2.0 * M * lin + attn)


def prefill_roofline(cfg, M: int, ms: float):
    """The prefill against the bf16 matrix-core peak.  Activations enter the
    matrix cores as three bf16 terms, so the cores issue three times the
    useful flops."""
    if ms <= 0 or M < 1:
        return None
    fl = prefill_flops(cfg, M)
    useful = fl / (ms / 1e3) / 1e12
    return {"bound": "mfma", "rows": M, "ms": round(ms, 2), "useful_tflops": round(useful, 1),
            "issued_tflops": round(3 * useful, 1), "peak_tflops": MFMA_BF16_PEAK_TFLOPS,
            "frac_useful": round(useful / MFMA_BF16_PEAK_TFLOPS, 4),
            "frac_issued": round(3 * useful / MFMA_BF16_PEAK_TFLOPS, 4)}


def host_cpu() -> dict:
    """The host the oracle runs on: CPU model, logical CPUs, OpenMP setting."""
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"cpu_model": model, "nproc": os.cpu_count(), "omp_num_threads_env": os.environ.get("OMP_NUM_THREADS")}


def oracle_decode_rates(cfg, weights, prompt, wl, skip, prefix=8, n_tokens=4) -> dict:
    """The oracle at the workload's model shape, decode separated from prefill.

    The prefill of prompt[:prefix] is timed alone; each generate call
    (prefill + n_tokens) is timed whole and the prefill time subtracted,
    which leaves the decode-only time of n_tokens greedy autoregressive
    tokens and of n_tokens self-speculative tokens (same mask, K_max and
    gamma).  The oracle's per-token cost is its weight passes (one float64
    matrix-vector product per weight), so a short context stands in for the
    workload's: attention over the workload's mean context adds
    2 * ctx * n_kv_heads * head_dim multiply-adds per attention sublayer,
    reported as attn_share_at_workload_ctx."""
    import oracle

    om = oracle.Model(cfg, weights)
    pr = np.asarray(prompt[:prefix], np.int32)
    c = om.cache(prefix)
    t0 = time.perf_counter()
    om.forward(c, pr[:-1], want_logits=False)
    t_pf = time.perf_counter() - t0
    del c
    t0 = time.perf_counter()
    om.generate_ar(pr, n_tokens)
    t_ar = time.perf_counter() - t0 - t_pf
    t0 = time.perf_counter()
    sd = om.generate_sd(pr, n_tokens, skip, wl.k_max, wl.gamma)
    t_sd = time.perf_counter() - t0 - t_pf
    d, L = cfg.d_model, cfg.n_layers
    macs_w = cfg.param_count() - cfg.vocab * d  # the embedding is gathered
    ctx = wl.prompt_len + wl.max_new / 2
    macs_attn = L * 2 * ctx * cfg.n_heads * cfg.head_dim
    return {
        "sd_tokens_per_s": round(n_tokens / t_sd, 4), "ar_tokens_per_s": round(n_tokens / t_ar, 4),
        "prefill_s": round(t_pf, 3), "prefill_rows": int(prefix - 1), "decode_tokens": n_tokens,
        "sd_stages": int(sd["n_stages"]), "sd_drafted": int(sd["n_drafted"]),
        "context": f"{prefix - 1}..{prefix - 2 + n_tokens} positions",
        "attn_share_at_workload_ctx": round(macs_attn / (macs_w + macs_attn), 4),
        "threads": oracle.num_threads(), "seconds": round(t_pf * 3 + t_ar + t_sd, 1),
    }


def cpu_baseline(cfg, weights, prompt, wl, skip):
    r = oracle_decode_rates(cfg, weights, prompt, wl, skip)
    return {
        "value": r["sd_tokens_per_s"], "unit": "tokens/s", "cores": r["threads"], "kind": "oracle",
        "sample": (f"oracle decode-only tokens/s of the {cfg.name} model ({wl.mask}, K_max {wl.k_max}, gamma "
                   f"{wl.gamma}): {r['decode_tokens']} self-speculative and {r['decode_tokens']} autoregressive "
                   f"tokens after a {r['prefill_rows'] + 1}-token prefix of the workload's prompt (context "
                   f"{r['context']}); prefill of {r['prefill_rows']} rows timed alone and reported apart; "
                   f"{r['seconds']} s of CPU work"),
        "ar_value": r["ar_tokens_per_s"], "prefill_s": r["prefill_s"], "prefill_rows": r["prefill_rows"],
        "attn_share_at_workload_ctx": r["attn_share_at_workload_ctx"], **host_cpu(),
    }


def run_cpu_table(args):
    """Oracle decode rates per workload on this host, with every OpenMP
    thread and with one thread (tiny and 7B), each in a child process so
    that OMP_NUM_THREADS takes effect.  One JSON line."""
    import subprocess

    rows = []
    for name, threads in (("tiny", None), ("tiny", 1), ("7b", None), ("7b", 1), ("13b", None)):
        env = dict(os.environ)
        if threads:
            env["OMP_NUM_THREADS"] = str(threads)
        out = subprocess.run([sys.executable, os.path.abspath(__file__), "--cpu-rates-child", name],
                             env=env, capture_output=True, text=True, check=True).stdout
        r = json.loads(out.strip().splitlines()[-1])
        log(f"oracle {name} x {r['threads']} threads: SD {r['sd_tokens_per_s']} tok/s, AR {r['ar_tokens_per_s']} tok/s")
        rows.append({"workload": name, **r})
    print(json.dumps({"mode": "cpu-table", "kind": "oracle", **host_cpu(), "rows": rows}), flush=True)


def run_cpu_rates_child(name):
    wl = S.WORKLOADS[name]
    cfg = S.MODELS[wl.model]
    w = S.make_weights(cfg, 0)
    pr = S.prompt(cfg, wl.prompt_len, 0)
    z = S.skip_mask(cfg, wl.mask, 0)
    kw = {"prefix": 8, "n_tokens": 16} if name == "tiny" else {"prefix": 4, "n_tokens": 2}
    print(json.dumps(oracle_decode_rates(cfg, w, pr, wl, z, **kw)), flush=True)


def load_model(cfg, seed):
    import torch

    from paper_2309_08168_amd import binding

    t0 = time.perf_counter()
    host = S.make_weights(cfg, seed)
    t_gen = time.perf_counter() - t0
    dw = binding.DeviceWeights(cfg, host)
    torch.cuda.synchronize()
    log(f"{cfg.name}: {cfg.param_count() / 1e9:.2f} B params, generated in {t_gen:.1f} s, uploaded in "
        f"{time.perf_counter() - t0 - t_gen:.1f} s")
    return host, binding.Model(cfg, dw)


# ---------------------------------------------------------------------------
# main benchmark


def run_bench(args):
    import torch

    wl = S.WORKLOADS[args.workload]
    cfg = S.MODELS[wl.model]
    max_new = args.max_new or wl.max_new
    host, model = load_model(cfg, args.seed)
    prompt = S.prompt(cfg, wl.prompt_len, args.seed)
    skip = S.skip_mask(cfg, wl.mask, args.seed)

    def run_sd():
        return model.generate_sd(prompt, max_new, skip, wl.k_max, wl.gamma)

    def run_ar():
        return model.generate_ar(prompt, max_new)

    warm = None
    for i in range(args.warmup):
        _, warm = run_sd()
        if not args.no_ar:
            run_ar()
        log(f"warmup {i + 1}/{args.warmup} done")

    # the dominant kernel of the step: the gate/up projection at the row
    # count the verification forwards run at (timed live with HIP events)
    mean_rows = 1 + warm["n_drafted"] / max(warm["n_stages"], 1) if warm else 2.0
    regime = 2 if mean_rows <= 2.0 else 16
    model.time_kernel("gate_up", regime)

    torch.cuda.synchronize()
    t0 = time.perf_counter()
    sd_stats = []
    sd_tokens = None
    for i in range(args.steps):
        sd_tokens, st = run_sd()
        sd_stats.append(st)
        log(f"step {i + 1}/{args.steps}: decode {st['decode_ms']:.1f} ms, stages {st['n_stages']}, "
            f"acceptance {st['n_accepted']}/{st['n_drafted']}")
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kt = model.kernel_time()
    model.time_kernel(None)

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
    vrows = 1 + drafted / max(stages, 1)
    b_verify = step_bytes(cfg, None, ctx, vrows)
    extra = {
        "acceptance": round(accepted / drafted, 4) if drafted else None,
        "tokens_per_stage": round(args.steps * max_new / max(stages, 1), 4),
        "draft_step_ms": round(draft_ms, 4),
        "draft_step_GBps": round(b_draft / (draft_ms / 1e3) / 1e9, 1),
        "draft_step_frac_hbm": round(b_draft / (draft_ms / 1e3) / 1e9 / HBM_PEAK_GBPS, 4),
        "verify_step_ms": round(verify_ms, 4),
        "verify_mean_rows": round(vrows, 3),
        "verify_step_GBps": round(b_verify / (verify_ms / 1e3) / 1e9, 1),
        "verify_step_frac_hbm": round(b_verify / (verify_ms / 1e3) / 1e9 / HBM_PEAK_GBPS, 4),
        "host_gap_us_per_step": round(1e3 * sum(s["decode_ms"] - s["draft_ms"] - s["verify_ms"] - s["noop_ms"]
                                                for s in sd_stats) / max(steps_d + stages, 1), 2),
        "cancelled_steps": sum(s["n_guarded_noop_steps"] for s in sd_stats) / args.steps,
        "prefill_ms": round(sum(s["prefill_ms"] for s in sd_stats) / args.steps, 2),
        "prefill": prefill_roofline(cfg, wl.prompt_len - 1, sum(s["prefill_ms"] for s in sd_stats) / args.steps),
    }
    if ar_stats:
        ar_ms = sum(s["decode_ms"] for s in ar_stats)
        ar_tps = args.steps * max_new / (ar_ms / 1e3)
        b_ar = step_bytes(cfg, None, ctx, 1)
        per = ar_ms / (args.steps * max_new)
        extra.update({
            "ar_tokens_per_s": round(ar_tps, 2),
            "speedup_vs_ar": round(value / ar_tps, 4),
            "ar_step_ms": round(per, 4),
            "ar_step_GBps": round(b_ar / (per / 1e3) / 1e9, 1),
            "ar_step_frac_hbm": round(b_ar / (per / 1e3) / 1e9 / HBM_PEAK_GBPS, 4),
            "sd_tokens_equal_ar": int(np.sum(np.asarray(sd_tokens) == np.asarray(ar_tokens))),
        })
        # break-even acceptance with one draft per stage: a* = c_draft + c_verify - 1
        extra["break_even_acceptance_1draft"] = round(draft_ms / per + verify_ms / per - 1.0, 3)

    roofline = None
    if kt["launches"]:
        avg_ms = kt["total_ms"] / kt["launches"]
        rows = regime if regime == 2 else vrows
        nbytes = gate_up_bytes(kt["n"], kt["k"], rows)
        achieved = nbytes / (avg_ms / 1e3) / 1e9
        roofline = {
            "bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic_for(kt["kernel"], args.workload),
            "kernel": kt["kernel"], "layer": f"gate_up, verification of <= {regime} rows",
            "bytes_per_launch": int(nbytes), "avg_launch_us": round(avg_ms * 1e3, 2), "launches": kt["launches"],
        }
    cpu = None
    if not args.no_cpu_baseline:
        log("timing the oracle on a bounded sample")
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


# ---------------------------------------------------------------------------
# verification-forward microbenchmark (13B stack over an N(0, 1) KV cache)


def run_verify_micro(args):
    import torch

    cfg = S.MODELS["13b"]
    host, model = load_model(cfg, args.seed)
    del host
    es = 2
    rows_list = [int(x) for x in args.micro_rows.split(",")]
    ctx_list = [int(x) for x in args.micro_ctx.split(",")]
    params = cfg.param_count() - cfg.vocab * cfg.d_model  # embedding table is gathered, not streamed
    results = []
    for ctx in ctx_list:
        cap = ctx + max(rows_list)
        buf = torch.empty(model.kv_cache_bytes(cap) // 2, dtype=torch.int16, device="cuda")
        # fill positions [0, ctx) of every (layer, K/V, head) with N(0, 1)
        view = buf.view(cfg.n_layers * 2 * cfg.n_kv_heads, cap, cfg.head_dim)
        fill = S.kv_fill(cfg, cfg.n_layers * 2 * cfg.n_kv_heads * ctx * cfg.head_dim, args.seed)
        view[:, :ctx].copy_(torch.from_numpy(fill.view(np.int16)).view(-1, ctx, cfg.head_dim).to("cuda"))
        del fill
        cache = model.cache(cap, device_buf=buf)
        for M in rows_list:
            toks = S.prompt(cfg, M, args.seed + M)
            logits = torch.empty((M, cfg.vocab), dtype=torch.float32, device="cuda")
            times = []
            for it in range(args.micro_iters + 1):
                cache.set_length(ctx)
                a = torch.cuda.Event(enable_timing=True)
                b = torch.cuda.Event(enable_timing=True)
                a.record()
                model.forward(toks, cache, logits=logits)
                b.record()
                b.synchronize()
                if it:
                    times.append(a.elapsed_time(b))
            ms = float(np.median(times))
            nbytes = step_bytes(cfg, None, ctx, M)
            useful = 2.0 * params * M
            # MFMA path: ceil(3 M / 16) packings of 16 columns (three bf16 terms per row)
            issued = 2.0 * params * 16 * ((3 * M + 15) // 16) if M > 2 else 0.0
            r = {"rows": M, "ctx": ctx, "ms": round(ms, 4), "GBps": round(nbytes / (ms / 1e3) / 1e9, 1),
                 "frac_hbm": round(nbytes / (ms / 1e3) / 1e9 / HBM_PEAK_GBPS, 4),
                 "mfma_useful_frac": round(useful / (ms / 1e3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 5),
                 "mfma_issued_frac": round(issued / (ms / 1e3) / 1e12 / MFMA_BF16_PEAK_TFLOPS, 5)}
            results.append(r)
            log(json.dumps(r))
        cache.close()
        del buf
    print(json.dumps({"mode": "verify-micro", "model": "13b stack (40 layers + lm-head)", "results": results}))


# ---------------------------------------------------------------------------
# supplementary planted-redundancy runs (labelled; not the headline value)


def run_supplementary(args):
    import torch  # noqa: F401

    from paper_2309_08168_amd import binding

    wl = S.WORKLOADS[args.workload]
    cfg = S.MODELS[wl.model]
    max_new = args.max_new or wl.max_new
    host = S.make_weights(cfg, args.seed)
    prompt = S.prompt(cfg, wl.prompt_len, args.seed)
    mask = args.supp_mask or wl.mask
    skip = S.skip_mask(cfg, mask, args.seed)
    out = []
    for rho, gain, gamma in [(float(x.split(":")[0]), float(x.split(":")[1]), float(x.split(":")[2]))
                             for x in args.planted.split(",")]:
        w = S.plant_redundancy(cfg, host, skip, rho, gain)
        model = binding.Model(cfg, binding.DeviceWeights(cfg, w))
        model.generate_sd(prompt, max_new, skip, wl.k_max, gamma)
        model.generate_ar(prompt, max_new)
        sd_tok, sd = model.generate_sd(prompt, max_new, skip, wl.k_max, gamma)
        ar_tok, ar = model.generate_ar(prompt, max_new)
        n_st, n_dr = max(sd["n_stages"], 1), max(sd["n_draft_steps"], 1)
        r = {"rho": rho, "head_gain": gain, "gamma": gamma,
             "sd_tokens_per_s": round(max_new / (sd["decode_ms"] / 1e3), 2),
             "ar_tokens_per_s": round(max_new / (ar["decode_ms"] / 1e3), 2),
             "speedup": round(ar["decode_ms"] / sd["decode_ms"], 4),
             "acceptance": round(sd["n_accepted"] / max(sd["n_drafted"], 1), 4),
             "tokens_per_stage": round(max_new / n_st, 3),
             "draft_steps": sd["n_draft_steps"], "stages": sd["n_stages"],
             "draft_step_ms": round(sd["draft_ms"] / n_dr, 4),
             "verify_step_ms": round(sd["verify_ms"] / n_st, 4),
             "verify_mean_rows": round((sd["n_drafted"] + sd["n_stages"]) / n_st, 3),
             "host_gap_us_per_step": round(1e3 * (sd["decode_ms"] - sd["draft_ms"] - sd["verify_ms"] - sd["noop_ms"]) /
                                           (sd["n_stages"] + sd["n_draft_steps"]), 2),
             "cancelled_steps": sd["n_guarded_noop_steps"], "cancelled_ms": round(sd["noop_ms"], 3),
             "ar_step_ms": round(ar["decode_ms"] / max_new, 4),
             "tokens_equal": int(np.sum(sd_tok == ar_tok))}
        # the same planted model with the adaptive exit (the paper's settings)
        model.generate_sd_adaptive(prompt, max_new, skip, wl.k_max)
        ad_tok, ad = model.generate_sd_adaptive(prompt, max_new, skip, wl.k_max)
        r.update({"adaptive_sd_tokens_per_s": round(max_new / (ad["decode_ms"] / 1e3), 2),
                  "adaptive_speedup": round(ar["decode_ms"] / ad["decode_ms"], 4),
                  "adaptive_acceptance": round(ad["n_accepted"] / max(ad["n_drafted"], 1), 4),
                  "adaptive_tokens_per_stage": round(max_new / max(ad["n_stages"], 1), 3),
                  "adaptive_gamma_last": round(float(ad["gammas"][-1]), 4) if len(ad["gammas"]) else None,
                  "adaptive_tokens_equal": int(np.sum(ad_tok == ar_tok))})
        d = np.nonzero(sd_tok != ar_tok)[0]
        if d.size:
            # the two agree up to d; the GPU's own logits there decide whether
            # the split is a near-tie (the tolerance of the parity tests)
            d = int(d[0])
            seq = np.concatenate([prompt, ar_tok[:d]]).astype(np.int32)
            c = model.cache(len(seq) + 1)
            model.forward(seq[:-1], c)
            lg = torch.empty((1, cfg.vocab), dtype=torch.float32, device="cuda")
            model.forward(seq[-1:], c, logits=lg)
            lg = lg[0].cpu().numpy()
            top2 = np.sort(lg)[-2:]
            c.close()
            r.update({"first_divergence": d, "gpu_top2_margin": round(float(top2[1] - top2[0]), 5),
                      "near_tie_tau": round(float(2 * 3e-2 * lg.std()), 5)})
        if args.fp8_draft:
            r.update(fp8_draft_runs(model, cfg, prompt, max_new, skip, wl, gamma, ar, ar_tok))
        out.append(r)
        log(json.dumps(r))
        model.close()
        del w
    print(json.dumps({"mode": "supplementary (planted redundancy)", "workload": wl.name, "mask": mask,
                      "skipped_sublayers": int(np.sum(skip)), "adaptive": binding.PAPER_ADAPTIVE, "results": out}))


def fp8_draft_runs(model, cfg, prompt, max_new, skip, wl, gamma, ar, ar_tok) -> dict:
    """The same model with FP8 copies of the draft's weights (verification
    keeps bf16): static and adaptive exit, against the bf16 autoregressive
    run `ar`.  The quantization time is wall time of the synchronous call,
    allocation of the copies included."""
    t0 = time.perf_counter()
    model.quantize_draft(skip)
    q_ms = (time.perf_counter() - t0) * 1e3
    model.generate_sd(prompt, max_new, skip, wl.k_max, gamma)
    tok, sd = model.generate_sd(prompt, max_new, skip, wl.k_max, gamma)
    model.generate_sd_adaptive(prompt, max_new, skip, wl.k_max)
    ad_tok, ad = model.generate_sd_adaptive(prompt, max_new, skip, wl.k_max)
    model.quantize_draft(None)
    n_st, n_dr = max(sd["n_stages"], 1), max(sd["n_draft_steps"], 1)
    draft_ms = sd["draft_ms"] / n_dr
    nbytes = step_bytes(cfg, skip, wl.prompt_len + max_new / 2, 1, fp8=True)
    return {"fp8_quantize_ms": round(q_ms, 2),
            "fp8_sd_tokens_per_s": round(max_new / (sd["decode_ms"] / 1e3), 2),
            "fp8_speedup": round(ar["decode_ms"] / sd["decode_ms"], 4),
            "fp8_acceptance": round(sd["n_accepted"] / max(sd["n_drafted"], 1), 4),
            "fp8_tokens_per_stage": round(max_new / n_st, 3),
            "fp8_draft_step_ms": round(draft_ms, 4),
            "fp8_draft_step_GBps": round(nbytes / (draft_ms / 1e3) / 1e9, 1),
            "fp8_draft_step_frac_hbm": round(nbytes / (draft_ms / 1e3) / 1e9 / HBM_PEAK_GBPS, 4),
            "fp8_verify_step_ms": round(sd["verify_ms"] / n_st, 4),
            "fp8_tokens_equal": int(np.sum(tok == ar_tok)),
            "fp8_adaptive_sd_tokens_per_s": round(max_new / (ad["decode_ms"] / 1e3), 2),
            "fp8_adaptive_speedup": round(ar["decode_ms"] / ad["decode_ms"], 4),
            "fp8_adaptive_acceptance": round(ad["n_accepted"] / max(ad["n_drafted"], 1), 4),
            "fp8_adaptive_tokens_equal": int(np.sum(ad_tok == ar_tok))}


# ---------------------------------------------------------------------------
# sampling variant (labelled supplementary runs)


def run_sampling(args):
    import torch  # noqa: F401

    from paper_2309_08168_amd import binding

    wl = S.WORKLOADS[args.workload]
    cfg = S.MODELS[wl.model]
    max_new = args.max_new or wl.max_new
    host = S.make_weights(cfg, args.seed)
    prompt = S.prompt(cfg, wl.prompt_len, args.seed)
    skip = S.skip_mask(cfg, wl.mask, args.seed)
    # (temperature, top_p): the paper's summarisation and code settings
    settings = [(0.2, 0.85), (0.6, 0.95)]
    out = []
    for label, rho, gain in (("random weights", None, None), ("planted, rho 0 / head gain 16", 0.0, 16.0)):
        w = host if rho is None else S.plant_redundancy(cfg, host, skip, rho, gain)
        model = binding.Model(cfg, binding.DeviceWeights(cfg, w))
        _, greedy = model.generate_ar(prompt, max_new)
        for T, top_p in settings:
            seed = 1234
            model.generate_sd_sample(prompt, max_new, skip, wl.k_max, T, top_p, seed, gamma=wl.gamma)
            _, sd = model.generate_sd_sample(prompt, max_new, skip, wl.k_max, T, top_p, seed, gamma=wl.gamma)
            _, ad = model.generate_sd_sample(prompt, max_new, skip, wl.k_max, T, top_p, seed, adaptive={})
            _, ar = model.generate_ar_sample(prompt, max_new, T, top_p, seed)
            n_st, n_dr = max(sd["n_stages"], 1), max(sd["n_draft_steps"], 1)
            r = {"weights": label, "temperature": T, "top_p": top_p,
                 "sd_tokens_per_s": round(max_new / (sd["decode_ms"] / 1e3), 2),
                 "adaptive_sd_tokens_per_s": round(max_new / (ad["decode_ms"] / 1e3), 2),
                 "ar_tokens_per_s": round(max_new / (ar["decode_ms"] / 1e3), 2),
                 "speedup": round(ar["decode_ms"] / sd["decode_ms"], 4),
                 "adaptive_speedup": round(ar["decode_ms"] / ad["decode_ms"], 4),
                 "acceptance": round(sd["n_accepted"] / max(sd["n_drafted"], 1), 4),
                 "adaptive_acceptance": round(ad["n_accepted"] / max(ad["n_drafted"], 1), 4),
                 "tokens_per_stage": round(max_new / n_st, 3),
                 "draft_step_ms": round(sd["draft_ms"] / n_dr, 4),
                 "verify_step_ms": round(sd["verify_ms"] / n_st, 4),
                 "ar_sample_step_ms": round(ar["decode_ms"] / max_new, 4),
                 "ar_greedy_step_ms": round(greedy["decode_ms"] / max_new, 4)}
            out.append(r)
            log(json.dumps(r))
        model.close()
        del w
    print(json.dumps({"mode": "sampling (labelled supplementary)", "workload": wl.name, "mask": wl.mask,
                      "k_max": wl.k_max, "gamma": wl.gamma, "adaptive": binding.PAPER_ADAPTIVE,
                      "results": out}))


# ---------------------------------------------------------------------------
# skip-set search (labelled supplementary runs)


def strategy_mask(cfg, n_att: int, n_mlp: int, where: str, seed: int = 0) -> np.ndarray:
    """A mask skipping n_att attention and n_mlp MLP sublayers at the first,
    middle or last layers, or at random ones (the fixed strategies the
    paper's appendix compares with the searched mask)."""
    L = cfg.n_layers
    z = np.zeros(2 * L, np.uint8)
    g = np.random.default_rng(seed)
    for kind, n in ((0, n_att), (1, n_mlp)):
        if where == "first":
            layers = np.arange(n)
        elif where == "last":
            layers = np.arange(L - n, L)
        elif where == "mid":
            layers = np.arange((L - n) // 2, (L - n) // 2 + n)
        else:
            layers = g.choice(L, size=n, replace=False)
        z[2 * layers + kind] = 1
    return z


def run_search(args):
    import torch  # noqa: F401

    from paper_2309_08168_amd import binding

    wl = S.WORKLOADS[args.workload]
    cfg = S.MODELS[wl.model]
    planted = S.skip_mask(cfg, args.search_mask, args.seed)
    host = S.make_weights(cfg, args.seed)
    w = S.plant_redundancy(cfg, host, planted, 0.0, 16.0)
    model = binding.Model(cfg, binding.DeviceWeights(cfg, w))
    dev = np.stack([S.prompt(cfg, args.search_prompt_len, seed=100 + i) for i in range(args.search_prompts)])
    held = np.stack([S.prompt(cfg, args.search_prompt_len, seed=200 + i) for i in range(args.search_prompts)])
    new_dev, new_held = args.search_new, 4 * args.search_new
    model.generate_sd(dev[0], new_dev, planted, wl.k_max, wl.gamma)  # first-call set-up
    prm = dict(n_init=args.search_init, iterations=args.search_iters, n_candidates=256, length_scale=0.5, noise=1e-3,
               xi=0.01, seed=args.seed)
    log(f"search: {cfg.name}, {2 * cfg.n_layers} sublayers, planted {int(planted.sum())}, "
        f"{prm['n_init'] + prm['iterations']} evaluations of {len(dev)} x {new_dev} tokens")
    t0 = time.perf_counter()
    res = model.search_skip_set(dev, new_dev, wl.k_max, gamma=wl.gamma, objective="measured", **prm)
    wall = time.perf_counter() - t0
    best = res["best_mask"]
    log(f"search done in {wall:.1f} s; best {res['best_value']:.4f} ms/token")

    def decode_ms(prompts, n, mask):
        tot, acc, drafted = 0.0, 0, 0
        for pr in prompts:
            if mask is None:
                _, st = model.generate_ar(pr, n)
            else:
                _, st = model.generate_sd(pr, n, mask, wl.k_max, wl.gamma)
                acc += st["n_accepted"]
                drafted += st["n_drafted"]
            tot += st["decode_ms"]
        return tot / (len(prompts) * n), (acc / drafted if drafted else None)

    n_att, n_mlp = int(best[0::2].sum()), int(best[1::2].sum())
    masks = {"searched": best, "planted": planted, "none": np.zeros_like(best)}
    for where in ("first", "mid", "last", "random"):
        masks[where] = strategy_mask(cfg, n_att, n_mlp, where, args.seed)
    ar_ms, _ = decode_ms(held, new_held, None)
    table = {}
    for name, z in masks.items():
        decode_ms(held[:1], new_held, z)  # warm
        ms, acc = decode_ms(held, new_held, z)
        table[name] = {"ms_per_token": round(ms, 4), "speedup_vs_ar": round(ar_ms / ms, 4),
                       "acceptance": None if acc is None else round(acc, 4),
                       "attention_skipped": int(z[0::2].sum()), "mlp_skipped": int(z[1::2].sum())}
        log(f"{name}: {json.dumps(table[name])}")
    # host cost of the search itself, objective aside: the same steps over a
    # free objective, and the oracle's search on a few of them
    t0 = time.perf_counter()
    binding.search_skip_set_fn(lambda z: float(z.sum()), 2 * cfg.n_layers, **prm)
    native_s = time.perf_counter() - t0
    steps = prm["n_init"] + prm["iterations"]
    cpu = None
    if not args.no_cpu_baseline:
        from oracle import skip_search as O

        k = 12
        t0 = time.perf_counter()
        O.search(lambda z: float(z.sum()), 2 * cfg.n_layers, **{**binding.SEARCH_DEFAULTS, **prm, "iterations": k})
        osec = time.perf_counter() - t0
        cpu = {"value": round(osec / (prm["n_init"] + k) * 1e3, 3), "unit": "ms per evaluation (search host cost)",
               "cores": 1, "kind": "oracle",
               "sample": f"oracle search of {prm['n_init']} + {k} evaluations of a free objective over "
                         f"{2 * cfg.n_layers} sublayers, {prm['n_candidates']} candidates per step; {osec:.1f} s"}
    print(json.dumps({
        "mode": "skip-set search (labelled supplementary)", "workload": wl.name, "weights": "planted rho 0 gain 16",
        "planted_mask": args.search_mask, "planted_sublayers": int(planted.sum()), "k_max": wl.k_max, "gamma": wl.gamma, "params": prm,
        "dev_prompts": [len(dev), args.search_prompt_len, new_dev], "held_out": [len(held), new_held],
        "evaluations": len(res["values"]), "search_wall_s": round(wall, 2),
        "search_best_ms_per_token": round(res["best_value"], 4),
        "initial_best_ms_per_token": round(float(res["values"][:prm["n_init"]].min()), 4),
        "overlap_with_planted": int(np.sum(best & planted)),
        "search_host_ms_per_evaluation": round(native_s / steps * 1e3, 3), "cpu_baseline": cpu,
        "ar_ms_per_token": round(ar_ms, 4), "masks": table}))
    model.close()


# ---------------------------------------------------------------------------
# profiler helpers


def run_stream_probe(args):
    """Achievable HBM read bandwidth: the library's streaming-read probe
    (sd_measure_read_bandwidth) over a 4 GiB device buffer, at the byte
    counts of the 13B decode layers and at 4 GiB, for 1-16 work-groups per
    compute unit.  Consecutive reads of one size start at different offsets,
    so a read never finds its bytes in the 256 MB last-level cache.  Also
    fits t = bytes / B + t0 over the layer sizes at each size's best shape."""
    import torch

    from paper_2309_08168_amd import binding

    total = 4 << 30
    buf = torch.ones(total, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(4, dtype=torch.int32, device="cuda")
    cfg = S.MODELS["13b"]
    d, F = cfg.d_model, cfg.ffn_dim
    sizes = {"o_proj_13b": d * d * 2, "down_13b": d * F * 2, "qkv_13b": cfg.qkv_rows * d * 2,
             "gate_up_13b": 2 * F * d * 2, "lm_head_13b": cfg.vocab * d * 2, "4GiB": total}
    reps = args.probe_reps
    rows, best = [], {}
    for name, n in sizes.items():
        n = n // 256 * 256
        span = max(total - n, 0)
        for wg, lif in [(w_, l_) for w_ in (1, 2, 4, 8, 16) for l_ in (2, 4, 8, 16)]:
            ms = []
            for it in range(reps):
                off = 0 if span == 0 else (it * n) % span // 256 * 256
                ms.append(binding.measure_read_bandwidth(buf, n, wg, 1, sink, offset=off, loads_in_flight=lif))
            med = float(np.median(ms))
            r = {"size": name, "bytes": n, "wg_per_cu": wg, "loads_in_flight": lif, "median_us": round(med * 1e3, 2),
                 "min_us": round(min(ms) * 1e3, 2), "GBps": round(n / (med / 1e3) / 1e9, 1)}
            rows.append(r)
            if name not in best or r["GBps"] > best[name]["GBps"]:
                best[name] = r
            log(json.dumps(r))
    layer = [b for k, b in best.items() if k != "4GiB"]
    x = np.array([b["bytes"] for b in layer], float)
    y = np.array([b["median_us"] for b in layer], float)
    slope, t0 = np.polyfit(x, y, 1)
    out = {"mode": "stream-probe", "kernel": "k_read_probe (16-byte non-temporal loads, 256 threads)",
           "best": best, "fit_layer_sizes": {"GBps": round(1e-3 / slope, 1), "t0_us": round(float(t0), 2)},
           "peak_GBps": HBM_PEAK_GBPS, "rows": rows}
    print(json.dumps(out), flush=True)


def run_calibrate_copy(args):
    import torch

    n = args.copy_bytes
    a = torch.ones(n // 4, dtype=torch.float32, device="cuda")
    b = torch.empty_like(a)
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"mode": "calibrate-copy", "bytes_read": n, "bytes_written": n}))


def _read_csv(path):
    return list(csv.DictReader(open(path)))


def run_summarize_stats(args):
    rows = _read_csv(args.summarize_stats)
    lines = [f"# rocprofv3 --kernel-trace --stats summary", f"# command: {args.command}", "",
             f"{'calls':>7} {'avg_us':>9} {'total_ms':>10} {'pct':>6}  kernel"]
    for r in rows[: args.top]:
        lines.append(f"{int(r['Calls']):7d} {float(r['AverageNs']) / 1e3:9.2f} {float(r['TotalDurationNs']) / 1e6:10.2f} "
                     f"{float(r['Percentage']):6.2f}  {r['Name']}")
    os.makedirs(os.path.dirname(args.out), exist_ok=True)
    open(args.out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def _counter_per_kernel(path, counter):
    per = {}
    for r in _read_csv(path):
        name = r.get("Kernel_Name") or r.get("Kernel-Name")
        if r.get("Counter_Name", counter) != counter:
            continue
        per.setdefault(name, []).append(float(r["Counter_Value"]))
    return per


def run_summarize_pmc(args):
    fetch_csv, write_csv = args.summarize_pmc
    fetch = _counter_per_kernel(fetch_csv, "FETCH_SIZE")
    write = _counter_per_kernel(write_csv, "WRITE_SIZE")
    # calibration: the device-to-device copy of --copy-bytes (--with-copy)
    # runs as the runtime's copy kernel; the largest median among copy kernels
    # (the largest copy dispatch; smaller copies share the kernel name)
    copy_names = [k for k in fetch if "copybuffer" in k.lower()]
    calib_f = calib_w = None
    if copy_names:
        k = copy_names[0]
        calib_f = args.copy_bytes / (max(fetch[k]) * 1024.0)
        if k in write:
            calib_w = args.copy_bytes / (max(write[k]) * 1024.0)
    kernels = {}
    for name in args.kernels.split(";"):
        if name in fetch and name in write:
            f = float(np.median(fetch[name])) * 1024.0 * (calib_f or 1.0)
            w = float(np.median(write[name])) * 1024.0 * (calib_w or 1.0)
            kernels[name] = {"fetch_bytes": f, "write_bytes": w, "bytes_per_launch": f + w}
    out = {"source_hash": source_hash(), "copy_scale_fetch": calib_f, "copy_scale_write": calib_w,
           "commands": args.command, "kernels": kernels}
    json.dump(out, open(TRAFFIC_FILE, "w"), indent=1)
    print(json.dumps(out, indent=1))


def _dispatches(path):
    """Counter values per dispatch, in dispatch order: [(kernel, {counter: value}, ns)]."""
    d = {}
    for r in _read_csv(path):
        i = int(r["Dispatch_Id"])
        e = d.setdefault(i, [r["Kernel_Name"], {}, int(r["End_Timestamp"]) - int(r["Start_Timestamp"])])
        e[1][r["Counter_Name"]] = float(r["Counter_Value"])
    return [tuple(d[i]) for i in sorted(d)]


def _forwards(disp):
    """The dispatches of each sd_forward (a forward of up to 16 rows starts with
    the control-block kernel); runtime copies and torch kernels are left out."""
    out, cur = [], None
    for name, c, ns in disp:
        if "k_set_ctl" in name:
            cur = []
            out.append(cur)
        elif cur is not None and "copyBuffer" not in name and "at::native" not in name:
            cur.append((name, c, ns))
    return out


def run_summarize_step_counters(args):
    """HBM bytes per verification forward from FETCH_SIZE / WRITE_SIZE (all
    kernels of the forward, calibrated by the 1 GiB copy) against the
    algorithmic bytes, and the MFMA use of the forward's matrix-core linear
    layers, for every (context, rows) pair of --micro-ctx x --micro-rows.
    Inputs: the counter CSVs of --verify-micro --micro-iters 1 --with-copy
    with --pmc FETCH_SIZE, --pmc WRITE_SIZE and --pmc
    SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU_MFMA_MOPS_BF16 GRBM_GUI_ACTIVE."""
    fetch_csv, write_csv, mfma_csv = args.summarize_step_counters
    cfg = S.MODELS["13b"]
    fd, wd = _dispatches(fetch_csv), _dispatches(write_csv)

    def calib(disp, counter):
        cp = [c[counter] for name, c, _ in disp if "copybuffer" in name.lower() and counter in c]
        return args.copy_bytes / (max(cp) * 1024.0) if cp else 1.0

    cf, cw = calib(fd, "FETCH_SIZE"), calib(wd, "WRITE_SIZE")
    ff, wf, md = _forwards(fd), _forwards(wd), _forwards(_dispatches(mfma_csv))
    rows_list = [int(x) for x in args.micro_rows.split(",")]
    ctx_list = [int(x) for x in args.micro_ctx.split(",")]
    pairs = [(ctx, M) for ctx in ctx_list for M in rows_list]
    lines = ["# HBM bytes per 13B forward (FETCH_SIZE + WRITE_SIZE over all its kernels) and MFMA use",
             f"# command: {args.command}",
             f"# copy calibration: FETCH_SIZE x{cf:.4f}, WRITE_SIZE x{cw:.4f}", "",
             f"{'rows':>4} {'ctx':>5} {'kernels':>7} {'fetch_GB':>9} {'write_GB':>9} {'total_GB':>9} "
             f"{'algorithmic_GB':>15} {'ratio':>6}"]
    for j, (ctx, M) in enumerate(pairs):
        idx = 2 * j + 1  # the timed forward of each pair (after one warm-up)
        if idx >= len(ff) or idx >= len(wf):
            break
        fb = sum(c.get("FETCH_SIZE", 0.0) for _, c, _ in ff[idx]) * 1024.0 * cf
        wb = sum(c.get("WRITE_SIZE", 0.0) for _, c, _ in wf[idx]) * 1024.0 * cw
        alg = step_bytes(cfg, None, ctx, M)
        lines.append(f"{M:4d} {ctx:5d} {len(ff[idx]):7d} {fb / 1e9:9.3f} {wb / 1e9:9.3f} {(fb + wb) / 1e9:9.3f} "
                     f"{alg / 1e9:15.3f} {(fb + wb) / alg:6.3f}")
    lines += ["", "# MFMA use per forward (rows > 2: matrix-core linear layers).  busy = SQ_VALU_MFMA_BUSY_CYCLES /",
              "# (1024 SIMDs x 2.4 GHz x time); issued = SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 flops (three bf16 terms",
              "# per row, 16 columns per packing); useful = 2 x rows x weights; over the MFMA kernels' time and over",
              "# the whole forward (all its kernels, measured under counter collection)",
              f"{'rows':>4} {'ctx':>5} {'mfma_us':>8} {'busy':>6} {'issued_TF':>9} {'useful_TF':>9} {'fwd_us':>8} "
              f"{'issued_TF_fwd':>13} {'useful_frac_peak':>16}"]
    params = cfg.param_count() - cfg.vocab * cfg.d_model
    for j, (ctx, M) in enumerate(pairs):
        idx = 2 * j + 1
        if M <= 2 or idx >= len(md):
            continue
        ks = [(n, c, ns) for n, c, ns in md[idx] if "k_linear_mfma" in n]
        t_m = sum(ns for _, _, ns in ks)
        t_f = sum(ns for _, _, ns in md[idx])
        busy = sum(c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0) for _, c, _ in ks)
        flops = sum(c.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0) for _, c, _ in ks) * 512.0
        useful = 2.0 * M * params
        if t_m <= 0:
            continue
        lines.append(f"{M:4d} {ctx:5d} {t_m / 1e3:8.1f} {busy / (1024 * t_m * 2.4):6.3f} {flops / t_m / 1e3:9.1f} "
                     f"{useful / t_m / 1e3:9.1f} {t_f / 1e3:8.1f} {flops / t_f / 1e3:13.1f} "
                     f"{useful / t_f / 1e3 / MFMA_BF16_PEAK_TFLOPS:16.4f}")
    # per kernel at the largest row count and the first context
    sel = [j for j, (ctx, M) in enumerate(pairs) if ctx == ctx_list[0] and M == max(rows_list)]
    if sel and 2 * sel[0] + 1 < len(md):
        lines += ["", f"# {max(rows_list)}-row forward at {ctx_list[0]} keys, per MFMA kernel",
                  f"{'calls':>5} {'avg_us':>7} {'busy':>6} {'issued_TFLOPs':>13}  kernel"]
        per = {}
        for name, c, ns in md[2 * sel[0] + 1]:
            if "k_linear_mfma" not in name:
                continue
            e = per.setdefault(name, [0, 0.0, 0.0, 0.0])
            e[0] += 1
            e[1] += ns
            e[2] += c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
            e[3] += c.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0.0) * 512.0
        for name, (n, ns, busy, flops) in sorted(per.items(), key=lambda kv: -kv[1][1]):
            lines.append(f"{n:5d} {ns / n / 1e3:7.2f} {busy / (1024 * ns * 2.4):6.3f} {flops / ns / 1e3:13.1f}  {name}")
    os.makedirs(os.path.dirname(args.out), exist_ok=True)
    open(args.out, "w").write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=3)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="13b", choices=sorted(S.WORKLOADS))
    ap.add_argument("--max-new", type=int, default=None, help="override the workload's generated tokens")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-table", action="store_true",
                    help="oracle decode rates on this host per workload, all threads and one thread")
    ap.add_argument("--cpu-rates-child", default=None, help=argparse.SUPPRESS)
    ap.add_argument("--no-ar", action="store_true", help="skip the autoregressive comparison")
    ap.add_argument("--verify-micro", action="store_true")
    ap.add_argument("--micro-rows", default="1,4,8,13,16")
    ap.add_argument("--micro-ctx", default="512,2048,4096")
    ap.add_argument("--micro-iters", type=int, default=5)
    ap.add_argument("--supplementary", action="store_true")
    ap.add_argument("--supp-mask", default=None,
                    help="skip mask for --supplementary (default: the workload's; e.g. random36)")
    ap.add_argument("--fp8-draft", action="store_true",
                    help="with --supplementary: also decode with FP8 copies of the draft's weights")
    ap.add_argument("--planted", default="0.05:8:0.6,0.05:8:0.0,0.02:16:0.6",
                    help="rho:head_gain:gamma triples for --supplementary")
    ap.add_argument("--sampling", action="store_true",
                    help="labelled runs of the sampling variant (temperature, top-p) against AR sampling")
    ap.add_argument("--search", action="store_true", help="skip-set search on the planted model (supplementary)")
    ap.add_argument("--search-prompts", type=int, default=2)
    ap.add_argument("--search-prompt-len", type=int, default=32)
    ap.add_argument("--search-mask", default="random36", help="the planted redundant sublayers")
    ap.add_argument("--search-new", type=int, default=32)
    ap.add_argument("--search-init", type=int, default=16)
    ap.add_argument("--search-iters", type=int, default=144)
    ap.add_argument("--stream-probe", action="store_true", help="achievable HBM read bandwidth (read probe)")
    ap.add_argument("--probe-reps", type=int, default=10)
    ap.add_argument("--calibrate-copy", action="store_true")
    ap.add_argument("--with-copy", action="store_true", help="also run the calibration copy after the bench")
    ap.add_argument("--copy-bytes", type=int, default=1 << 30)
    ap.add_argument("--summarize-stats", default=None, help="rocprofv3 kernel_stats.csv to summarize")
    ap.add_argument("--summarize-pmc", nargs=2, default=None, metavar=("FETCH_CSV", "WRITE_CSV"))
    ap.add_argument("--kernels", default="", help="';'-separated kernel symbols for --summarize-pmc")
    ap.add_argument("--summarize-step-counters", nargs=3, default=None, metavar=("FETCH_CSV", "WRITE_CSV", "MFMA_CSV"))
    ap.add_argument("--out", default=os.path.join(ROOT, "profiles", "kernel_stats.txt"))
    ap.add_argument("--top", type=int, default=20)
    ap.add_argument("--command", default="", help="the profiling command, recorded in the summary")
    args = ap.parse_args()

    if args.summarize_stats:
        return run_summarize_stats(args)
    if args.summarize_pmc:
        return run_summarize_pmc(args)
    if args.summarize_step_counters:
        return run_summarize_step_counters(args)
    if args.cpu_rates_child:
        return run_cpu_rates_child(args.cpu_rates_child)
    if args.cpu_table:
        return run_cpu_table(args)
    if args.gpus != 1:
        print(f"bench.py runs on one GPU: --gpus {args.gpus} is not supported (the decode path is "
              "batch-1 on a single MI355X; independent requests would run one model copy per GPU)", file=sys.stderr)
        sys.exit(2)
    import torch

    torch.cuda.set_device(0)
    if args.calibrate_copy:
        return run_calibrate_copy(args)
    if args.stream_probe:
        return run_stream_probe(args)
    if args.verify_micro:
        run_verify_micro(args)
    elif args.supplementary:
        run_supplementary(args)
    elif args.sampling:
        run_sampling(args)
    elif args.search:
        run_search(args)
    else:
        run_bench(args)
    if args.with_copy:
        run_calibrate_copy(args)


if __name__ == "__main__":
    main()
