"""Writes tests/golden/tiny_decode.json from the oracle only.

Run: python tests/golden/make_golden.py
The fixture records the tiny fp32 workload (4 layers, d 256, prompt 16,
32 new tokens, skip = attention of layer 1 + MLP of layer 2, K_max 4,
gamma 0.6) as the oracle decodes it: greedy AR tokens and the
self-speculative stage trace (k_e, n_e).
"""
import json
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import oracle  # noqa: E402
import sd_synth as S  # noqa: E402


def main():
    cfg = S.MODELS["tiny"]
    wl = S.WORKLOADS["tiny"]
    m = oracle.Model(cfg, S.make_weights(cfg, 0))
    pr = S.prompt(cfg, wl.prompt_len)
    ar, margin = m.generate_ar(pr, wl.max_new)
    sd = m.generate_sd(pr, wl.max_new, S.skip_mask(cfg, wl.mask), wl.k_max, wl.gamma)
    out = {
        "source": "oracle (sd_oracle.c), seed 0",
        "prompt": pr.tolist(),
        "ar_tokens": ar.tolist(),
        "ar_min_margin": float(margin.min()),
        "sd_stages": sd["stages"].tolist(),
    }
    path = os.path.join(os.path.dirname(os.path.abspath(__file__)), "tiny_decode.json")
    with open(path, "w") as f:
        json.dump(out, f, indent=1)
    print("wrote", path)


if __name__ == "__main__":
    main()
