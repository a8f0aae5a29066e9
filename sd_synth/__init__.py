"""Seeded synthetic inputs for the self-speculative decoding hot path.

This module is shared by the CPU oracle side and the GPU side.  It holds the
model and workload shapes, and deterministic generators for weights, prompts,
skip masks and externally filled KV caches.  It contains none of the decoding
method's arithmetic: no norm, no attention, no argmax.

Weights follow the synthetic recipe of the workloads: every linear weight and
the token embedding are N(0, 0.02^2); the two output projections of each
layer (attention output, MLP down) use std 0.02 / sqrt(2 * n_layers); norm
gains are 1.0; the lm-head is untied from the embedding.  Normal draws are
inverse-transform samples: element i of a tensor takes the quantile of a
16-bit hash of (i, tensor key) from a table of the 65536 equiprobable
quantiles of N(0, std^2), rounded to the storage dtype.  The hash is
integer-only, so every machine produces the same bits.
"""

from __future__ import annotations

import ctypes
import dataclasses
import hashlib
import os
import statistics
from typing import Dict, List, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "_fill.so")
_lib = None


def build(verbose: bool = False) -> str:
    """Compile the integer hash filler (plain C, OpenMP) in place."""
    import subprocess

    src = os.path.join(_HERE, "_fill.c")
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", src, "-o", _LIB_PATH]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        lib = ctypes.CDLL(_LIB_PATH)
        for name, ptype in (("sdsynth_fill_u16", ctypes.c_void_p), ("sdsynth_fill_f32", ctypes.c_void_p)):
            fn = getattr(lib, name)
            fn.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint64, ptype]
            fn.restype = None
        _lib = lib
    return _lib


# ----------------------------------------------------------------------------
# shapes


@dataclasses.dataclass(frozen=True)
class ModelConfig:
    name: str
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    dtype: str  # "f32" or "bf16": storage type of weights and KV cache
    rms_eps: float = 1e-6
    rope_base: float = 10000.0

    @property
    def qkv_rows(self) -> int:
        return (self.n_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def n_sublayers(self) -> int:
        return 2 * self.n_layers

    def param_count(self) -> int:
        d, L = self.d_model, self.n_layers
        per_layer = self.qkv_rows * d + d * self.n_heads * self.head_dim + 3 * d * self.ffn_dim + 2 * d
        return L * per_layer + 2 * self.vocab * d + d


MODELS: Dict[str, ModelConfig] = {
    "tiny": ModelConfig("tiny", 4, 256, 4, 4, 64, 688, 1024, "f32"),
    "7b": ModelConfig("7b", 32, 4096, 32, 32, 128, 11008, 32000, "bf16"),
    "13b": ModelConfig("13b", 40, 5120, 40, 40, 128, 13824, 32000, "bf16"),
    "70b": ModelConfig("70b", 80, 8192, 64, 8, 128, 28672, 32000, "bf16"),
}


@dataclasses.dataclass(frozen=True)
class Workload:
    """One decode workload: a model shape plus prompt/generation/draft settings."""

    name: str
    model: str
    prompt_len: int
    max_new: int
    mask: str  # how the skip mask is built, see skip_mask()
    k_max: int
    gamma: float


WORKLOADS: Dict[str, Workload] = {
    # 4 layers, fp32: attention of layer 1 and MLP of layer 2 skipped.
    "tiny": Workload("tiny", "tiny", 16, 32, "tiny", 4, 0.6),
    # LLaMA-2-7B shape: both sublayers of layers 8, 10, ..., 30 skipped.
    "7b": Workload("7b", "7b", 512, 256, "every2nd_8_30", 12, 0.6),
    # LLaMA-2-13B shape, long summarisation-like context: 20 random sublayers.
    "13b": Workload("13b", "13b", 1024, 512, "random20", 12, 0.6),
    # LLaMA-2-70B shape (GQA 64/8): 40 random sublayers.
    "70b": Workload("70b", "70b", 512, 128, "random40", 8, 0.6),
}

# Verify-step microbenchmark at the 13B shape: rows per forward and KV lengths.
VERIFY_MICRO_M = (1, 4, 8, 13, 16)
VERIFY_MICRO_CTX = (512, 2048, 4096)


# ----------------------------------------------------------------------------
# keys and tables


def tensor_key(seed: int, name: str) -> int:
    """64-bit key of one tensor: a digest of (seed, name); stable across runs."""
    h = hashlib.sha256(f"{int(seed)}:{name}".encode()).digest()
    return int.from_bytes(h[:8], "little")


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even float32 -> bfloat16 bit patterns (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


_TABLES: Dict[tuple, np.ndarray] = {}


def normal_table(std: float, dtype: str) -> np.ndarray:
    """The 65536 quantiles std * Phi^-1((i + 0.5) / 65536), in storage dtype."""
    key = (float(std), dtype)
    if key not in _TABLES:
        nd = statistics.NormalDist(0.0, 1.0)
        q = np.array([nd.inv_cdf((i + 0.5) / 65536.0) for i in range(65536)], dtype=np.float64)
        q32 = (q * std).astype(np.float32)
        _TABLES[key] = f32_to_bf16_bits(q32) if dtype == "bf16" else q32
    return _TABLES[key]


def fill_normal(out: np.ndarray, key: int, std: float, dtype: str) -> np.ndarray:
    """Fill a contiguous array (uint16 bf16 bits or float32) with seeded N(0, std^2)."""
    lib = _load()
    tab = normal_table(std, dtype)
    assert out.flags["C_CONTIGUOUS"]
    if dtype == "bf16":
        assert out.dtype == np.uint16
        lib.sdsynth_fill_u16(out.ctypes.data, out.size, key, tab.ctypes.data)
    else:
        assert out.dtype == np.float32
        lib.sdsynth_fill_f32(out.ctypes.data, out.size, key, tab.ctypes.data)
    return out


def _np_dtype(dtype: str):
    return np.uint16 if dtype == "bf16" else np.float32


def _ones(n: int, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return np.full(n, 0x3F80, dtype=np.uint16)
    return np.ones(n, dtype=np.float32)


# ----------------------------------------------------------------------------
# weights


def weight_specs(cfg: ModelConfig):
    """(name, shape, std) of every tensor; std None means a norm gain of 1.0.

    Row-major [out, in] like nn.Linear.  w_qkv stacks the q rows (n_heads *
    head_dim), then k rows, then v rows (n_kv_heads * head_dim each).
    w_gate_up stacks the ffn_dim gate rows, then the ffn_dim up rows.
    """
    d, L, dh = cfg.d_model, cfg.n_layers, cfg.head_dim
    out_std = 0.02 / np.sqrt(2.0 * L)
    specs = [("tok_emb", (cfg.vocab, d), 0.02)]
    for l in range(L):
        specs += [
            (f"layers.{l}.attn_norm", (d,), None),
            (f"layers.{l}.w_qkv", (cfg.qkv_rows, d), 0.02),
            (f"layers.{l}.w_o", (d, cfg.n_heads * dh), out_std),
            (f"layers.{l}.mlp_norm", (d,), None),
            (f"layers.{l}.w_gate_up", (2 * cfg.ffn_dim, d), 0.02),
            (f"layers.{l}.w_down", (d, cfg.ffn_dim), out_std),
        ]
    specs += [("final_norm", (d,), None), ("lm_head", (cfg.vocab, d), 0.02)]
    return specs


def make_tensor(cfg: ModelConfig, name: str, shape, std, seed: int, out: Optional[np.ndarray] = None):
    n = int(np.prod(shape))
    if out is None:
        out = np.empty(n, dtype=_np_dtype(cfg.dtype))
    out = out.reshape(-1)
    if std is None:
        out[:] = _ones(n, cfg.dtype)
    else:
        fill_normal(out, tensor_key(seed, name), float(std), cfg.dtype)
    return out.reshape(shape)


def make_weights(cfg: ModelConfig, seed: int = 0) -> Dict[str, np.ndarray]:
    """All tensors of a model on the host (uint16 bf16 bits or float32)."""
    return {name: make_tensor(cfg, name, shape, std, seed) for name, shape, std in weight_specs(cfg)}


def scale_tensor(w: np.ndarray, factor: float, dtype: str) -> np.ndarray:
    """w * factor in storage dtype (used for labelled planted-redundancy runs)."""
    if dtype == "bf16":
        return f32_to_bf16_bits(bf16_bits_to_f32(w) * np.float32(factor)).reshape(w.shape)
    return (w * np.float32(factor)).astype(np.float32)


def plant_redundancy(cfg: ModelConfig, weights: Dict[str, np.ndarray], skip: np.ndarray,
                     rho: float, head_gain: float) -> Dict[str, np.ndarray]:
    """Scale the output projections of the masked sublayers by rho and the lm-head by head_gain.

    This stands in for a trained model's redundant layers: skipped sublayers
    then contribute little to the residual stream, and a larger head gain
    makes top-1 probabilities large enough to exercise long drafts.
    """
    w = dict(weights)
    for l in range(cfg.n_layers):
        if skip[2 * l]:
            w[f"layers.{l}.w_o"] = scale_tensor(w[f"layers.{l}.w_o"], rho, cfg.dtype)
        if skip[2 * l + 1]:
            w[f"layers.{l}.w_down"] = scale_tensor(w[f"layers.{l}.w_down"], rho, cfg.dtype)
    if head_gain != 1.0:
        w["lm_head"] = scale_tensor(w["lm_head"], head_gain, cfg.dtype)
    return w


# ----------------------------------------------------------------------------
# prompts, masks, KV fill


def prompt(cfg: ModelConfig, length: int, seed: int = 0) -> np.ndarray:
    """length token ids uniform over [0, vocab)."""
    g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(seed) + 1, 0x5D01])))
    return g.integers(0, cfg.vocab, size=length, dtype=np.int64).astype(np.int32)


def skip_mask(cfg: ModelConfig, spec: str, seed: int = 0) -> np.ndarray:
    """uint8[2 * n_layers]; entry 2l is attention of layer l, 2l+1 its MLP; 1 = skip.

    spec: "none", "tiny" (attention of layer 1 and MLP of layer 2),
    "every2nd_A_B" (both sublayers of layers A, A+2, ..., B), "randomS"
    (S distinct sublayers drawn uniformly without replacement), "all",
    or an explicit comma-separated list of sublayer indices "i,j,...".
    """
    z = np.zeros(cfg.n_sublayers, dtype=np.uint8)
    if spec == "none":
        return z
    if spec == "all":
        z[:] = 1
        return z
    if spec == "tiny":
        z[2 * 1] = 1
        z[2 * 2 + 1] = 1
        return z
    if spec.startswith("every2nd_"):
        a, b = (int(v) for v in spec.split("_")[1:3])
        for l in range(a, b + 1, 2):
            z[2 * l] = z[2 * l + 1] = 1
        return z
    if spec.startswith("random"):
        s = int(spec[len("random"):])
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(seed) + 2, 0x5D02])))
        z[g.choice(cfg.n_sublayers, size=s, replace=False)] = 1
        return z
    for tok in spec.split(","):
        z[int(tok)] = 1
    return z


def kv_fill(cfg: ModelConfig, n_elems: int, seed: int = 0) -> np.ndarray:
    """n_elems values N(0, 1) in storage dtype, for an externally filled KV cache."""
    out = np.empty(n_elems, dtype=_np_dtype(cfg.dtype))
    return fill_normal(out, tensor_key(int(seed) + 3, "kv_cache"), 1.0, cfg.dtype)


def micro_config(n_layers=2, d_model=64, n_heads=4, n_kv_heads=2, head_dim=16, ffn_dim=96, vocab=97,
                 dtype="f32", name="micro") -> ModelConfig:
    """Small models for brute-force pins (any GQA ratio, odd sizes)."""
    return ModelConfig(name, n_layers, d_model, n_heads, n_kv_heads, head_dim, ffn_dim, vocab, dtype)


def weights_as_f64(cfg: ModelConfig, weights: Dict[str, np.ndarray]) -> Dict[str, np.ndarray]:
    """Exact float64 view of every tensor (for library-built cross-checks)."""
    if cfg.dtype == "bf16":
        return {k: bf16_bits_to_f32(v).astype(np.float64).reshape(v.shape) for k, v in weights.items()}
    return {k: v.astype(np.float64) for k, v in weights.items()}


__all__: List[str] = [
    "ModelConfig", "Workload", "MODELS", "WORKLOADS", "VERIFY_MICRO_M", "VERIFY_MICRO_CTX",
    "make_weights", "make_tensor", "weight_specs", "prompt", "skip_mask", "kv_fill",
    "plant_redundancy", "scale_tensor", "micro_config", "weights_as_f64", "tensor_key",
    "normal_table", "fill_normal", "f32_to_bf16_bits", "bf16_bits_to_f32", "build",
]
