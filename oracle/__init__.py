"""ctypes wrapper of the plain C oracle (sd_oracle.c).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the CPU
baseline of the benchmark may import this package; the product library
never does.
"""

from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Dict, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "liboracle.so")
_libs: Dict[str, ctypes.CDLL] = {}


def build(verbose: bool = False, src: Optional[str] = None, out: str = LIB_PATH) -> str:
    """Compile the oracle (or, for mutation tests, another source file) to out."""
    src = src or os.path.join(_HERE, "sd_oracle.c")
    cmd = ["gcc", "-std=c11", "-O2", "-fopenmp", "-fPIC", "-shared", "-Wall", "-Wextra", "-I", _HERE, src,
           "-o", out, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.check_call(cmd)
    return out


class _Config(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("ffn_dim", ctypes.c_int32),
        ("vocab", ctypes.c_int32), ("rms_eps", ctypes.c_double), ("rope_base", ctypes.c_double),
        ("wdtype", ctypes.c_int32),
    ]


class _Weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("tok_emb", "final_norm", "lm_head")] + [
        (n, ctypes.POINTER(ctypes.c_void_p))
        for n in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down")
    ]


class Adaptive(ctypes.Structure):
    """Adaptive draft-exit parameters (Sec. 3.4, Eqs. 2-4)."""

    _fields_ = [(n, ctypes.c_double) for n in ("gamma0", "alpha", "epsilon", "beta1", "beta2")]


# The paper's settings (appendix table of hyperparameters): gamma0 0.6,
# epsilon 0.01, beta1 0.5, beta2 0.9; alpha 0.90 for LLaMA-2-13B on CNN/DM.
PAPER_ADAPTIVE = dict(gamma0=0.6, alpha=0.9, epsilon=0.01, beta1=0.5, beta2=0.9)


class Sampling(ctypes.Structure):
    """Sampling parameters of the sampling variant: temperature, top-p, seed."""

    _fields_ = [("temperature", ctypes.c_double), ("top_p", ctypes.c_double), ("seed", ctypes.c_uint64)]


# Purposes of the uniforms (the second counter word): the draw of a draft,
# the acceptance test of a draft, and the draw after the accepted drafts
# (residual or bonus; every draw of autoregressive sampling).
U_DRAFT, U_ACCEPT, U_FINAL = 0, 1, 2


class SDStats(ctypes.Structure):
    _fields_ = [
        ("n_stages", ctypes.c_int64), ("n_drafted", ctypes.c_int64), ("n_accepted", ctypes.c_int64),
        ("n_emitted", ctypes.c_int64), ("n_draft_steps", ctypes.c_int64), ("min_gamma_gap", ctypes.c_double),
        ("min_draft_margin", ctypes.c_double),
    ]


def _load(path: str = LIB_PATH):
    if path not in _libs:
        if path == LIB_PATH and not os.path.exists(LIB_PATH):
            build()
        lib = ctypes.CDLL(path)
        vp, i32, p = ctypes.c_void_p, ctypes.c_int32, ctypes.POINTER
        lib.orc_create.argtypes = [p(_Config), p(_Weights)]
        lib.orc_create.restype = vp
        lib.orc_destroy.argtypes = [vp]
        lib.orc_num_threads.restype = i32
        lib.orc_cache_create.argtypes = [vp, i32]
        lib.orc_cache_create.restype = vp
        lib.orc_cache_destroy.argtypes = [vp]
        lib.orc_cache_length.argtypes = [vp]
        lib.orc_cache_length.restype = i32
        lib.orc_cache_truncate.argtypes = [vp, i32]
        lib.orc_cache_load.argtypes = [vp, vp, i32, i32]
        lib.orc_forward.argtypes = [vp, vp, vp, i32, vp, vp, vp, vp, vp]
        lib.orc_generate_ar.argtypes = [vp, vp, i32, i32, vp, vp]
        lib.orc_generate_sd.argtypes = [vp, vp, i32, i32, vp, i32, ctypes.c_float, vp, vp, p(SDStats), vp, vp]
        lib.orc_generate_sd_adaptive.argtypes = [vp, vp, i32, i32, vp, i32, p(Adaptive), vp, vp, p(SDStats), vp,
                                                 vp, vp]
        u64 = ctypes.c_uint64
        lib.orc_philox4x64.argtypes = [vp, vp, vp]
        lib.orc_philox4x64.restype = None
        lib.orc_uniform.argtypes = [u64, ctypes.c_int64, i32, ctypes.c_int64]
        lib.orc_uniform.restype = ctypes.c_double
        lib.orc_warp.argtypes = [vp, i32, ctypes.c_double, ctypes.c_double, vp, vp]
        lib.orc_warp.restype = i32
        lib.orc_generate_ar_sample.argtypes = [vp, vp, i32, i32, p(Sampling), vp, vp]
        lib.orc_generate_sd_sample.argtypes = [vp, vp, i32, i32, vp, i32, ctypes.c_float, vp, p(Sampling), vp, vp,
                                               p(SDStats), vp, vp, vp]
        lib.orc_fp8_value.argtypes = [ctypes.c_uint8]
        lib.orc_fp8_value.restype = ctypes.c_double
        lib.orc_quantize_fp8_rows.argtypes = [vp, ctypes.c_int64, ctypes.c_int64, vp, vp]
        lib.orc_set_draft_fp8.argtypes = [vp, vp]
        for fn in ("orc_quantize_fp8_rows", "orc_set_draft_fp8"):
            getattr(lib, fn).restype = ctypes.c_int
        for fn in ("orc_cache_truncate", "orc_cache_load", "orc_forward", "orc_generate_ar", "orc_generate_sd",
                   "orc_generate_sd_adaptive", "orc_generate_ar_sample", "orc_generate_sd_sample"):
            getattr(lib, fn).restype = ctypes.c_int
        _libs[path] = lib
    return _libs[path]


def num_threads() -> int:
    return int(_load().orc_num_threads())


def philox4x64(ctr, key, lib_path: str = LIB_PATH) -> np.ndarray:
    """The four 64-bit words of Philox4x64-10 block ctr (4 words) under key (2 words)."""
    c = np.ascontiguousarray(ctr, dtype=np.uint64)
    k = np.ascontiguousarray(key, dtype=np.uint64)
    out = np.empty(4, np.uint64)
    _load(lib_path).orc_philox4x64(c.ctypes.data, k.ctypes.data, out.ctypes.data)
    return out


def uniform(seed: int, index: int, purpose: int, stage: int, lib_path: str = LIB_PATH) -> float:
    return float(_load(lib_path).orc_uniform(seed, index, purpose, stage))


def warp(logits, temperature: float, top_p: float, lib_path: str = LIB_PATH):
    """(pi, kept count, cut margin) of the warped distribution of one logits row."""
    lg = np.ascontiguousarray(logits, dtype=np.float64)
    pi = np.empty_like(lg)
    cm = ctypes.c_double()
    kept = _load(lib_path).orc_warp(lg.ctypes.data, lg.size, temperature, top_p, pi.ctypes.data, ctypes.byref(cm))
    if kept < 0:
        raise OracleError(f"orc_warp failed with status {kept}")
    return pi, int(kept), cm.value


def fp8_value(b: int, lib_path: str = LIB_PATH) -> float:
    """The value of an OCP FP8 E4M3 byte."""
    return float(_load(lib_path).orc_fp8_value(int(b)))


def quantize_fp8_rows(w_bf16: np.ndarray, lib_path: str = LIB_PATH):
    """(bytes uint8 [N][K], exponents int32 [N]) of a bf16 matrix [N][K]: the
    nearest E4M3 value of W[n][k] * 2^-e[n], e[n] the smallest exponent that
    keeps the row's largest magnitude within 448."""
    w = np.ascontiguousarray(w_bf16, dtype=np.uint16)
    n, k = w.shape
    q = np.empty((n, k), np.uint8)
    e = np.empty(n, np.int32)
    _check(_load(lib_path).orc_quantize_fp8_rows(w.ctypes.data, n, k, q.ctypes.data, e.ctypes.data),
           "orc_quantize_fp8_rows")
    return q, e


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


class OracleError(RuntimeError):
    pass


def _check(rc: int, what: str):
    if rc != 0:
        raise OracleError(f"{what} failed with status {rc}")


class Model:
    """The oracle model over host weight arrays (see sd_synth.weight_specs)."""

    def __init__(self, cfg, weights: Dict[str, np.ndarray], lib_path: str = LIB_PATH):
        self._lib = lib = _load(lib_path)
        self._lib_path = lib_path
        self.cfg = cfg
        self._w = weights  # keep arrays alive
        c = _Config(cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.ffn_dim, cfg.vocab,
                    cfg.rms_eps, cfg.rope_base, 1 if cfg.dtype == "bf16" else 0)
        L = cfg.n_layers
        self._arrays = {}
        for key in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down"):
            arr = (ctypes.c_void_p * L)(*[weights[f"layers.{l}.{key}"].ctypes.data for l in range(L)])
            self._arrays[key] = arr
        w = _Weights(weights["tok_emb"].ctypes.data, weights["final_norm"].ctypes.data,
                     weights["lm_head"].ctypes.data,
                     *[ctypes.cast(self._arrays[k], ctypes.POINTER(ctypes.c_void_p))
                       for k in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down")])
        self._h = lib.orc_create(ctypes.byref(c), ctypes.byref(w))
        if not self._h:
            raise OracleError("orc_create rejected the configuration")

    def __del__(self):
        if getattr(self, "_h", None):
            self._lib.orc_destroy(self._h)
            self._h = None

    def set_draft_fp8(self, skip):
        """Quantize the draft's weights (the sublayers skip keeps) to FP8; None removes them."""
        sk = None if skip is None else np.ascontiguousarray(skip, dtype=np.uint8)
        _check(self._lib.orc_set_draft_fp8(self._h, _ptr(sk)), "orc_set_draft_fp8")

    def cache(self, capacity: int) -> "Cache":
        return Cache(self, capacity)

    def forward(self, cache: "Cache", tokens, skip=None, want_logits=True):
        """Forward of len(tokens) rows appended to cache; returns dict of outputs."""
        tok = np.ascontiguousarray(tokens, dtype=np.int32)
        n = tok.size
        sk = None if skip is None else np.ascontiguousarray(skip, dtype=np.uint8)
        logits = np.empty((n, self.cfg.vocab), np.float64) if want_logits else None
        amax = np.empty(n, np.int32)
        pmax = np.empty(n, np.float32)
        margin = np.empty(n, np.float64)
        rc = self._lib.orc_forward(self._h, cache._h, tok.ctypes.data, n, _ptr(sk), _ptr(logits), amax.ctypes.data,
                                 pmax.ctypes.data, margin.ctypes.data)
        _check(rc, "orc_forward")
        return {"logits": logits, "argmax": amax, "pmax": pmax, "margin": margin}

    def score(self, tokens, skip=None):
        """Logits of every row of one from-scratch forward over tokens (fresh cache)."""
        c = self.cache(len(tokens))
        return self.forward(c, tokens, skip)

    def generate_ar(self, prompt, max_new: int):
        pr = np.ascontiguousarray(prompt, dtype=np.int32)
        out = np.empty(max_new, np.int32)
        margin = np.empty(max_new, np.float64)
        _check(self._lib.orc_generate_ar(self._h, pr.ctypes.data, pr.size, max_new, out.ctypes.data,
                                       margin.ctypes.data), "orc_generate_ar")
        return out, margin

    def generate_sd(self, prompt, max_new: int, skip, k_max: int, gamma: float):
        pr = np.ascontiguousarray(prompt, dtype=np.int32)
        sk = None if skip is None else np.ascontiguousarray(skip, dtype=np.uint8)
        out = np.empty(max_new, np.int32)
        margin = np.empty(max_new, np.float64)
        log = np.zeros((max(max_new, 1), 2), np.int32)
        pm = np.zeros(max(max_new * max(k_max, 1), 1), np.float32)
        st = SDStats()
        _check(self._lib.orc_generate_sd(self._h, pr.ctypes.data, pr.size, max_new, _ptr(sk), k_max,
                                       ctypes.c_float(gamma), out.ctypes.data, margin.ctypes.data,
                                       ctypes.byref(st), log.ctypes.data, pm.ctypes.data), "orc_generate_sd")
        return {
            "tokens": out, "margin": margin, "stages": log[: st.n_stages].copy(),
            "draft_pmax": pm[: st.n_draft_steps].copy(), "n_stages": st.n_stages, "n_drafted": st.n_drafted,
            "n_accepted": st.n_accepted, "n_emitted": st.n_emitted, "min_gamma_gap": st.min_gamma_gap,
            "min_draft_margin": st.min_draft_margin,
        }

    def generate_sd_adaptive(self, prompt, max_new: int, skip, k_max: int, **params):
        """Self-speculative decoding with the adaptive threshold; params are
        gamma0, alpha, epsilon, beta1, beta2 (defaults: PAPER_ADAPTIVE)."""
        ad = Adaptive(**{**PAPER_ADAPTIVE, **params})
        pr = np.ascontiguousarray(prompt, dtype=np.int32)
        sk = None if skip is None else np.ascontiguousarray(skip, dtype=np.uint8)
        out = np.empty(max_new, np.int32)
        margin = np.empty(max_new, np.float64)
        log = np.zeros((max(max_new, 1), 2), np.int32)
        pm = np.zeros(max(max_new * max(k_max, 1), 1), np.float32)
        glog = np.zeros(max(max_new, 1), np.float32)
        st = SDStats()
        _check(self._lib.orc_generate_sd_adaptive(self._h, pr.ctypes.data, pr.size, max_new, _ptr(sk), k_max,
                                                ctypes.byref(ad), out.ctypes.data, margin.ctypes.data,
                                                ctypes.byref(st), log.ctypes.data, pm.ctypes.data,
                                                glog.ctypes.data), "orc_generate_sd_adaptive")
        return {
            "tokens": out, "margin": margin, "stages": log[: st.n_stages].copy(),
            "draft_pmax": pm[: st.n_draft_steps].copy(), "gammas": glog[: st.n_stages].copy(),
            "n_stages": st.n_stages, "n_drafted": st.n_drafted, "n_accepted": st.n_accepted,
            "n_emitted": st.n_emitted, "min_gamma_gap": st.min_gamma_gap, "min_draft_margin": st.min_draft_margin,
        }

    def generate_ar_sample(self, prompt, max_new: int, temperature: float, top_p: float, seed: int):
        sp = Sampling(temperature, top_p, seed)
        pr = np.ascontiguousarray(prompt, dtype=np.int32)
        out = np.empty(max_new, np.int32)
        margin = np.empty(max_new, np.float64)
        _check(self._lib.orc_generate_ar_sample(self._h, pr.ctypes.data, pr.size, max_new, ctypes.byref(sp),
                                              out.ctypes.data, margin.ctypes.data), "orc_generate_ar_sample")
        return out, margin

    def generate_sd_sample(self, prompt, max_new: int, skip, k_max: int, temperature: float, top_p: float,
                           seed: int, gamma: Optional[float] = None, adaptive: Optional[dict] = None):
        """Self-speculative sampling with a static gamma, or with the adaptive
        threshold when adaptive is a dict of its parameters (defaults:
        PAPER_ADAPTIVE)."""
        sp = Sampling(temperature, top_p, seed)
        ad = None if adaptive is None else Adaptive(**{**PAPER_ADAPTIVE, **adaptive})
        if ad is None and gamma is None:
            raise ValueError("gamma or adaptive is required")
        pr = np.ascontiguousarray(prompt, dtype=np.int32)
        sk = None if skip is None else np.ascontiguousarray(skip, dtype=np.uint8)
        out = np.empty(max_new, np.int32)
        margin = np.empty(max_new, np.float64)
        log = np.zeros((max(max_new, 1), 2), np.int32)
        qm = np.zeros(max(max_new * max(k_max, 1), 1), np.float32)
        glog = np.zeros(max(max_new, 1), np.float32)
        st = SDStats()
        _check(self._lib.orc_generate_sd_sample(self._h, pr.ctypes.data, pr.size, max_new, _ptr(sk), k_max,
                                              ctypes.c_float(0.0 if gamma is None else gamma),
                                              None if ad is None else ctypes.byref(ad), ctypes.byref(sp),
                                              out.ctypes.data, margin.ctypes.data, ctypes.byref(st),
                                              log.ctypes.data, qm.ctypes.data, glog.ctypes.data),
               "orc_generate_sd_sample")
        return {
            "tokens": out, "margin": margin, "stages": log[: st.n_stages].copy(),
            "draft_qmax": qm[: st.n_draft_steps].copy(), "gammas": glog[: st.n_stages].copy(),
            "n_stages": st.n_stages, "n_drafted": st.n_drafted, "n_accepted": st.n_accepted,
            "n_emitted": st.n_emitted, "min_gamma_gap": st.min_gamma_gap,
        }


class Cache:
    def __init__(self, model: Model, capacity: int):
        self.model = model
        self._lib = model._lib
        self._h = self._lib.orc_cache_create(model._h, capacity)
        if not self._h:
            raise OracleError("orc_cache_create failed")

    def __del__(self):
        if getattr(self, "_h", None):
            self._lib.orc_cache_destroy(self._h)
            self._h = None

    @property
    def length(self) -> int:
        return int(self._lib.orc_cache_length(self._h))

    def truncate(self, n: int):
        _check(self._lib.orc_cache_truncate(self._h, n), "orc_cache_truncate")

    def load(self, kv: np.ndarray, length: int, dtype: str):
        kv = np.ascontiguousarray(kv)
        _check(self._lib.orc_cache_load(self._h, kv.ctypes.data, length, 1 if dtype == "bf16" else 0),
               "orc_cache_load")
