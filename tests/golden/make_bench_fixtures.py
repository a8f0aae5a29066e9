"""Writes tests/golden/bench_<workload>.npz: the oracle's greedy decode of a
LLaMA-2-shaped benchmark workload at its full length.

Only the oracle (oracle/) and the seeded input generators (sd_synth) are
called; nothing here touches the GPU library.  The greedy tokens of Algorithm
1 are, by losslessness (Sec. 3.2), also the tokens self-speculative decoding
must emit, so the GPU's self-speculative and autoregressive outputs are both
compared with them.

Workloads (weights seed 0, prompt seed 0, as the benchmark runs them):
  7b   32 layers, d 4096, prompt 512, 256 new tokens   (~17 min on 8 cores)
  13b  40 layers, d 5120, prompt 1024, 512 new tokens  (~70 min on 8 cores)
The 70B shape (138 GB of bf16 weights) does not fit a 64 GB host.

Stored per generated position i (input token at position prompt_len - 1 + i):
  tokens[i]     the oracle's argmax (lowest id among equal float32 logits)
  margin[i]     top-1 minus top-2 float64 logit
  std[i]        standard deviation of the row's float64 logits
  top1[i]       the top-1 logit; top2_id[i], top2[i] the runner-up
and the full float32 logit rows of the last BLOCK positions (a block of
verification rows over the longest context of the run).

Usage: python tests/golden/make_bench_fixtures.py 7b [13b]
"""

from __future__ import annotations

import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import sd_synth as S  # noqa: E402

BLOCK = 13  # the 13B workload's K_max + 1 verification rows
PREFILL_CHUNK = 64


def weight_digest(w) -> np.ndarray:
    """Sums of the first 4096 stored values of a few tensors (uint64), so a
    test can tell that its regenerated weights are the ones used here."""
    names = ["tok_emb", "layers.0.w_qkv", "layers.0.w_down", "lm_head"]
    return np.array([int(np.asarray(w[n]).reshape(-1)[:4096].view(np.uint16 if w[n].dtype == np.uint16
                                                                  else np.uint32).astype(np.uint64).sum())
                     for n in names], dtype=np.uint64)


def make(name: str) -> str:
    wl = S.WORKLOADS[name]
    cfg = S.MODELS[wl.model]
    t0 = time.time()

    def say(msg):
        print(f"[{name} {time.time() - t0:8.1f}s] {msg}", flush=True)

    w = S.make_weights(cfg, 0)
    pr = S.prompt(cfg, wl.prompt_len, 0)
    om = oracle.Model(cfg, w)
    say(f"weights ready, {oracle.num_threads()} threads")
    c = om.cache(wl.prompt_len + wl.max_new)
    # Algorithm 1 with the prompt split as for decoding: prompt[0..t-2]
    # fills the cache, prompt[t-1] is the first input row.
    for i in range(0, wl.prompt_len - 1, PREFILL_CHUNK):
        om.forward(c, pr[i:min(wl.prompt_len - 1, i + PREFILL_CHUNK)], want_logits=False)
        say(f"prefill {min(wl.prompt_len - 1, i + PREFILL_CHUNK)}/{wl.prompt_len - 1}")
    n = wl.max_new
    tokens = np.empty(n, np.int32)
    margin = np.empty(n, np.float64)
    std = np.empty(n, np.float64)
    top1 = np.empty(n, np.float64)
    top2 = np.empty(n, np.float64)
    top2_id = np.empty(n, np.int32)
    block = np.empty((BLOCK, cfg.vocab), np.float32)
    last = int(pr[-1])
    for i in range(n):
        r = om.forward(c, [last])
        lg = r["logits"][0]
        tokens[i] = r["argmax"][0]
        margin[i] = r["margin"][0]
        std[i] = lg.std()
        top1[i] = lg[tokens[i]]
        rest = lg.copy()
        rest[tokens[i]] = -np.inf
        top2_id[i] = int(np.argmax(rest))
        top2[i] = lg[top2_id[i]]
        if i >= n - BLOCK:
            block[i - (n - BLOCK)] = lg.astype(np.float32)
        last = int(tokens[i])
        if i % 16 == 15 or i == n - 1:
            say(f"token {i + 1}/{n}")
    out = os.path.join(HERE, f"bench_{name}.npz")
    np.savez_compressed(out, workload=name, prompt=pr, tokens=tokens, margin=margin, std=std, top1=top1,
                        top2=top2, top2_id=top2_id, block_start=np.int32(n - BLOCK), block_logits=block,
                        weight_digest=weight_digest(w), threads=np.int32(oracle.num_threads()),
                        seconds=np.float64(time.time() - t0))
    say(f"wrote {out}")
    return out


if __name__ == "__main__":
    for nm in sys.argv[1:] or ["7b"]:
        make(nm)
