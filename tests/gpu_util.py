"""Helpers shared by the GPU tests: device models over seeded weights, and
the near-tie rules the comparisons with the oracle follow.

Tolerances: float32 models compare logits within 1e-4 absolute; bfloat16
models within 3e-2 * std(oracle logits of the row).  A token may differ from
the oracle's only where the oracle's top-2 margin is below tau = 2 * tol
(each of the two logits may move by tol).
"""

from __future__ import annotations

import numpy as np

import sd_synth as S

FP32_TOL = 1e-4
BF16_REL_TOL = 3e-2


def row_tol(cfg, oracle_logits: np.ndarray) -> np.ndarray:
    """Per-row logit tolerance for a model's dtype."""
    if cfg.dtype == "bf16":
        return BF16_REL_TOL * oracle_logits.std(axis=-1)
    return np.full(oracle_logits.shape[:-1], FP32_TOL)


def device_model(cfg, host_weights):
    from paper_2309_08168_amd import binding

    dw = binding.DeviceWeights(cfg, host_weights)
    return binding.Model(cfg, dw)


def check_logits(cfg, got: np.ndarray, ref: np.ndarray, what: str):
    tol = row_tol(cfg, ref)
    err = np.abs(got.astype(np.float64) - ref).max(axis=-1)
    bad = np.nonzero(~(err <= tol))[0]
    assert bad.size == 0, f"{what}: rows {bad[:8].tolist()} max|d| {err[bad[:8]].tolist()} > tol {tol[bad[:8]].tolist()}"
    return float((err / tol).max())


def check_tokens_teacher_forced(cfg, omodel, prompt, gpu_tokens, what: str):
    """Every GPU token is the oracle's argmax after the GPU's own prefix, or
    within tau of the oracle's top-1 logit there."""
    seq = np.concatenate([np.asarray(prompt, np.int32), np.asarray(gpu_tokens, np.int32)])
    r = omodel.score(seq[:-1])
    lg = r["logits"][len(prompt) - 1:]
    tau = 2 * row_tol(cfg, lg)
    top = lg.max(axis=1)
    mine = lg[np.arange(len(gpu_tokens)), gpu_tokens]
    gap = top - mine
    bad = np.nonzero(gap > tau)[0]
    assert bad.size == 0, f"{what}: tokens at {bad[:8].tolist()} are {gap[bad[:8]].tolist()} below the top logit"
    return int(np.sum(r["argmax"][len(prompt) - 1:] != gpu_tokens))


def check_free_running(cfg, gpu_tokens, ref_tokens, ref_margin, ref_logit_std, what: str):
    """Equal up to the first position whose oracle top-2 margin is below tau;
    returns that position (or len) so callers can report it."""
    tol = BF16_REL_TOL * np.asarray(ref_logit_std) if cfg.dtype == "bf16" else np.full(len(ref_tokens), FP32_TOL)
    tau = 2 * tol
    for i, (g, r) in enumerate(zip(gpu_tokens, ref_tokens)):
        if ref_margin[i] < tau[i]:
            return i
        assert g == r, f"{what}: token {i} differs (gpu {g}, oracle {r}) at margin {ref_margin[i]:.3g} >= tau"
    return len(ref_tokens)


MINI_BF16 = S.ModelConfig("mini_bf16", 2, 256, 4, 2, 64, 512, 1000, "bf16")
MICRO_GQA = S.micro_config(n_layers=2, d_model=64, n_heads=4, n_kv_heads=2, head_dim=16, ffn_dim=96, vocab=97)
