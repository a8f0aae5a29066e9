"""ctypes binding of libsd.so (include/sd.h): argument marshalling only.

Every computation of the decoding path runs in the library's HIP kernels.
PyTorch provides device memory (weight and KV buffers) and the stream.
If the library is not built, loading fails loudly; nothing falls back to
another implementation.
"""

from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional

import numpy as np

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsd.so")

SD_OK, SD_ERR_INVALID_ARG, SD_ERR_CAPACITY, SD_ERR_OOM, SD_ERR_DEVICE, SD_ERR_UNIMPLEMENTED = 0, -1, -2, -3, -4, -5
SD_F32, SD_BF16 = 0, 1

# Every entry point declared in include/sd.h.
EXPORTS = (
    "sd_model_create", "sd_model_destroy", "sd_kv_cache_bytes", "sd_kv_cache_create", "sd_kv_cache_destroy",
    "sd_kv_cache_length", "sd_kv_cache_truncate", "sd_kv_cache_set_length", "sd_forward", "sd_forward_static",
    "sd_self_spec_generate", "sd_self_spec_generate_adaptive", "sd_autoregressive_generate",
    "sd_self_spec_sample", "sd_autoregressive_sample", "sd_search_skip_set_fn", "sd_search_skip_set",
    "sd_model_time_kernel", "sd_model_kernel_time", "sd_measure_read_bandwidth", "sd_model_quantize_draft",
    "sd_model_draft_fp8",
    "sd_last_error", "sd_version",
)


class SDError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"status {status}: {message}")
        self.status = status


class sd_config(ctypes.Structure):
    _fields_ = [
        ("n_layers", ctypes.c_int32), ("d_model", ctypes.c_int32), ("n_heads", ctypes.c_int32),
        ("n_kv_heads", ctypes.c_int32), ("head_dim", ctypes.c_int32), ("ffn_dim", ctypes.c_int32),
        ("vocab", ctypes.c_int32), ("rms_eps", ctypes.c_float), ("rope_base", ctypes.c_float),
        ("dtype", ctypes.c_int32),
    ]


class sd_weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("tok_emb", "final_norm", "lm_head")] + [
        (n, ctypes.POINTER(ctypes.c_void_p))
        for n in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down")
    ]


class sd_stats(ctypes.Structure):
    _fields_ = [
        ("n_stages", ctypes.c_int64), ("n_drafted", ctypes.c_int64), ("n_accepted", ctypes.c_int64),
        ("n_emitted", ctypes.c_int64), ("n_draft_steps", ctypes.c_int64),
        ("prefill_ms", ctypes.c_double), ("draft_ms", ctypes.c_double), ("verify_ms", ctypes.c_double),
        ("decode_ms", ctypes.c_double), ("total_ms", ctypes.c_double),
        ("stage_log", ctypes.POINTER(ctypes.c_int32)), ("stage_log_cap", ctypes.c_int32),
        ("gamma_log", ctypes.POINTER(ctypes.c_float)),
        ("n_guarded_noop_steps", ctypes.c_int64), ("noop_ms", ctypes.c_double),
    ]


class sd_adaptive(ctypes.Structure):
    _fields_ = [(n, ctypes.c_double) for n in ("gamma0", "alpha", "epsilon", "beta1", "beta2")]


class sd_sampling(ctypes.Structure):
    _fields_ = [("temperature", ctypes.c_float), ("top_p", ctypes.c_float), ("seed", ctypes.c_uint64)]


SD_SEARCH_MEASURED, SD_SEARCH_MODELED = 0, 1


class sd_search_params(ctypes.Structure):
    _fields_ = [
        ("n_init", ctypes.c_int32), ("iterations", ctypes.c_int32), ("n_candidates", ctypes.c_int32),
        ("length_scale", ctypes.c_double), ("noise", ctypes.c_double), ("xi", ctypes.c_double),
        ("seed", ctypes.c_uint64), ("objective", ctypes.c_int32), ("cost", ctypes.c_double * 5),
    ]


class sd_search_result(ctypes.Structure):
    _fields_ = [
        ("best_mask", ctypes.POINTER(ctypes.c_uint8)), ("best_value", ctypes.c_double),
        ("n_evaluated", ctypes.c_int32), ("masks", ctypes.POINTER(ctypes.c_uint8)),
        ("values", ctypes.POINTER(ctypes.c_double)), ("margins", ctypes.POINTER(ctypes.c_double)),
    ]


SEARCH_OBJECTIVE_FN = ctypes.CFUNCTYPE(ctypes.c_int, ctypes.POINTER(ctypes.c_uint8), ctypes.c_int32, ctypes.c_void_p,
                                       ctypes.POINTER(ctypes.c_double))

# Defaults of the skip-set search.
SEARCH_DEFAULTS = dict(n_init=8, iterations=32, n_candidates=64, length_scale=0.25, noise=1e-3, xi=0.01, seed=0)


# The paper's adaptive-exit settings (gamma0, epsilon, beta1, beta2; alpha
# for LLaMA-2-13B on CNN/DM).
PAPER_ADAPTIVE = dict(gamma0=0.6, alpha=0.9, epsilon=0.01, beta1=0.5, beta2=0.9)


_lib: Optional[ctypes.CDLL] = None


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libsd.so and declare every entry point's signature."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built: run `python -m paper_2309_08168_amd.build` first")
    lib = ctypes.CDLL(path)
    vp, i32, p = ctypes.c_void_p, ctypes.c_int32, ctypes.POINTER
    sig = {
        "sd_model_create": ([p(sd_config), p(sd_weights), vp, p(vp)], ctypes.c_int),
        "sd_model_destroy": ([vp], ctypes.c_int),
        "sd_kv_cache_bytes": ([p(sd_config), i32], ctypes.c_size_t),
        "sd_kv_cache_create": ([vp, i32, vp, p(vp)], ctypes.c_int),
        "sd_kv_cache_destroy": ([vp], ctypes.c_int),
        "sd_kv_cache_length": ([vp], i32),
        "sd_kv_cache_truncate": ([vp, i32], ctypes.c_int),
        "sd_kv_cache_set_length": ([vp, i32], ctypes.c_int),
        "sd_forward": ([vp, vp, i32, vp, vp, vp], ctypes.c_int),
        "sd_forward_static": ([vp, vp, i32, vp, vp, vp], ctypes.c_int),
        "sd_self_spec_generate": ([vp, vp, i32, i32, vp, i32, ctypes.c_float, vp, p(sd_stats)], ctypes.c_int),
        "sd_self_spec_generate_adaptive": ([vp, vp, i32, i32, vp, i32, p(sd_adaptive), vp, p(sd_stats)],
                                           ctypes.c_int),
        "sd_autoregressive_generate": ([vp, vp, i32, i32, vp, p(sd_stats)], ctypes.c_int),
        "sd_self_spec_sample": ([vp, vp, i32, i32, vp, i32, ctypes.c_float, vp, p(sd_sampling), vp, p(sd_stats)],
                                ctypes.c_int),
        "sd_autoregressive_sample": ([vp, vp, i32, i32, p(sd_sampling), vp, p(sd_stats)], ctypes.c_int),
        "sd_search_skip_set_fn": ([i32, p(sd_search_params), SEARCH_OBJECTIVE_FN, vp, p(sd_search_result)],
                                  ctypes.c_int),
        "sd_search_skip_set": ([vp, vp, i32, i32, i32, i32, ctypes.c_float, vp, p(sd_search_params),
                                p(sd_search_result)], ctypes.c_int),
        "sd_model_time_kernel": ([vp, i32, i32], ctypes.c_int),
        "sd_model_kernel_time": ([vp, p(ctypes.c_int64), p(ctypes.c_double), ctypes.c_char_p, i32,
                                  p(ctypes.c_int64), p(ctypes.c_int64)], ctypes.c_int),
        "sd_model_quantize_draft": ([vp, vp], ctypes.c_int),
        "sd_model_draft_fp8": ([vp, i32, i32, p(vp), p(vp)], ctypes.c_int),
        "sd_measure_read_bandwidth": ([vp, ctypes.c_size_t, i32, i32, i32, vp, vp, p(ctypes.c_double)], ctypes.c_int),
        "sd_last_error": ([], ctypes.c_char_p),
        "sd_version": ([], ctypes.c_char_p),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    _lib = lib
    return lib


def check(status: int):
    if status != SD_OK:
        raise SDError(status, load().sd_last_error().decode(errors="replace"))


def make_config(cfg) -> sd_config:
    """sd_config from a shape object with the fields of sd_synth.ModelConfig."""
    return sd_config(cfg.n_layers, cfg.d_model, cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.ffn_dim, cfg.vocab,
                     cfg.rms_eps, cfg.rope_base, SD_BF16 if cfg.dtype == "bf16" else SD_F32)


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


class DeviceWeights:
    """Weight tensors in device memory (torch allocations), keyed like sd_synth."""

    def __init__(self, cfg, host: Dict[str, np.ndarray], device="cuda"):
        import torch

        self.cfg = cfg
        self.tensors = {}
        for name, arr in host.items():
            a = np.ascontiguousarray(arr)
            t = torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a)
            self.tensors[name] = t.to(device, non_blocking=False)

    @classmethod
    def from_generator(cls, cfg, make, names, device="cuda"):
        """Upload tensors one by one from make(name) -> np.ndarray (host copies dropped)."""
        import torch

        self = cls.__new__(cls)
        self.cfg = cfg
        self.tensors = {}
        for name in names:
            a = np.ascontiguousarray(make(name))
            t = torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a)
            self.tensors[name] = t.to(device)
            del a, t
        return self

    def ptr(self, name: str) -> int:
        return self.tensors[name].data_ptr()


class Model:
    """An sd_model over DeviceWeights on a torch stream (default: current stream)."""

    def __init__(self, cfg, weights: DeviceWeights, stream=None):
        import torch

        lib = load()
        self.cfg = cfg
        self.weights = weights
        self.stream = stream if stream is not None else torch.cuda.current_stream()
        L = cfg.n_layers
        self._arrays = {
            key: (ctypes.c_void_p * L)(*[weights.ptr(f"layers.{l}.{key}") for l in range(L)])
            for key in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down")
        }
        w = sd_weights(weights.ptr("tok_emb"), weights.ptr("final_norm"), weights.ptr("lm_head"),
                       *[ctypes.cast(self._arrays[k], ctypes.POINTER(ctypes.c_void_p))
                         for k in ("attn_norm", "w_qkv", "w_o", "mlp_norm", "w_gate_up", "w_down")])
        self._cfg = make_config(cfg)
        h = ctypes.c_void_p()
        check(lib.sd_model_create(ctypes.byref(self._cfg), ctypes.byref(w), ctypes.c_void_p(self.stream.cuda_stream),
                                  ctypes.byref(h)))
        self._h = h

    def close(self):
        if getattr(self, "_h", None):
            load().sd_model_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # linear-layer classes of sd_model_time_kernel
    LAYERS = {"qkv": 0, "o": 1, "gate_up": 2, "down": 3, "head": 4}

    def time_kernel(self, layer: Optional[str], rows: int = 1):
        """Bracket launches of one layer class with HIP events (None: off)."""
        check(load().sd_model_time_kernel(self._h, -1 if layer is None else self.LAYERS[layer], rows))

    def kernel_time(self) -> dict:
        n_l, ms = ctypes.c_int64(), ctypes.c_double()
        n, k = ctypes.c_int64(), ctypes.c_int64()
        name = ctypes.create_string_buffer(256)
        check(load().sd_model_kernel_time(self._h, ctypes.byref(n_l), ctypes.byref(ms), name, 256, ctypes.byref(n),
                                          ctypes.byref(k)))
        return {"launches": n_l.value, "total_ms": ms.value, "kernel": name.value.decode(), "n": n.value,
                "k": k.value}

    def kv_cache_bytes(self, capacity: int) -> int:
        return int(load().sd_kv_cache_bytes(ctypes.byref(self._cfg), capacity))

    def cache(self, capacity: int, device_buf=None) -> "KVCache":
        return KVCache(self, capacity, device_buf)

    def forward(self, tokens, cache: "KVCache", skip=None, logits=None):
        """sd_forward; logits is an optional torch float32 cuda tensor [n, vocab]."""
        tok = np.ascontiguousarray(tokens, dtype=np.int32)
        sk = None if skip is None else np.ascontiguousarray(skip, dtype=np.uint8)
        lp = None if logits is None else ctypes.c_void_p(logits.data_ptr())
        check(load().sd_forward(self._h, _ptr(tok), tok.size, _ptr(sk), cache._h, lp))
        return logits

    def forward_static(self, tokens, cache: "KVCache", skip=None, logits=None):
        """sd_forward_static: sd_forward for up to 16 rows, its scratch in the
        library's static device array (no allocation)."""
        tok = np.ascontiguousarray(tokens, dtype=np.int32)
        sk = None if skip is None else np.ascontiguousarray(skip, dtype=np.uint8)
        lp = None if logits is None else ctypes.c_void_p(logits.data_ptr())
        check(load().sd_forward_static(self._h, _ptr(tok), tok.size, _ptr(sk), cache._h, lp))
        return logits

    def quantize_draft(self, skip):
        """sd_model_quantize_draft: FP8 copies of the weights of the sublayers
        skip keeps (None removes them)."""
        sk = None if skip is None else np.ascontiguousarray(skip, dtype=np.uint8)
        check(load().sd_model_quantize_draft(self._h, _ptr(sk)))

    def draft_fp8(self, layer: int, kind: int):
        """(bytes uint8 [N][K], exponents int32 [N]) of a quantized draft
        matrix copied to the host, or None; kind 0 QKV, 1 O, 2 gate/up, 3 down."""
        import torch

        q, e = ctypes.c_void_p(), ctypes.c_void_p()
        check(load().sd_model_draft_fp8(self._h, layer, kind, ctypes.byref(q), ctypes.byref(e)))
        if not q.value:
            return None
        c = self.cfg
        rows = [(c.n_heads + 2 * c.n_kv_heads) * c.head_dim, c.d_model, 2 * c.ffn_dim, c.d_model][kind]
        cols = [c.d_model, c.n_heads * c.head_dim, c.d_model, c.ffn_dim][kind]
        torch.cuda.synchronize()
        qb = np.empty((rows, cols), np.uint8)
        eb = np.empty(rows, np.int32)
        hip = ctypes.CDLL("libamdhip64.so")
        hip.hipMemcpy.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int]
        if hip.hipMemcpy(qb.ctypes.data, q, qb.nbytes, 2) or hip.hipMemcpy(eb.ctypes.data, e, eb.nbytes, 2):
            raise RuntimeError("hipMemcpy of the FP8 copy failed")
        return qb, eb

    def _sd_call(self, fn, prompt, max_new, skip, k_max, rule, log_cap):
        pr = np.ascontiguousarray(prompt, dtype=np.int32)
        sk = None if skip is None else np.ascontiguousarray(skip, dtype=np.uint8)
        out = np.zeros(max(max_new, 1), np.int32)
        cap = max(max_new, 1) if log_cap is None else log_cap
        log = np.zeros((cap, 2), np.int32)
        glog = np.zeros(cap, np.float32)
        st = sd_stats()
        st.stage_log = log.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
        st.gamma_log = glog.ctypes.data_as(ctypes.POINTER(ctypes.c_float))
        st.stage_log_cap = cap
        check(fn(self._h, _ptr(pr), pr.size, max_new, _ptr(sk), k_max, rule, _ptr(out), ctypes.byref(st)))
        return out[:max_new], _stats(st, log, glog)

    def generate_sd(self, prompt, max_new: int, skip, k_max: int, gamma: float, log_cap: Optional[int] = None):
        """sd_self_spec_generate (fixed threshold gamma)."""
        return self._sd_call(load().sd_self_spec_generate, prompt, max_new, skip, k_max, ctypes.c_float(gamma),
                             log_cap)

    def generate_sd_adaptive(self, prompt, max_new: int, skip, k_max: int, log_cap: Optional[int] = None,
                             **params):
        """sd_self_spec_generate_adaptive; params: gamma0, alpha, epsilon, beta1,
        beta2 (defaults: PAPER_ADAPTIVE)."""
        ad = sd_adaptive(**{**PAPER_ADAPTIVE, **params})
        return self._sd_call(load().sd_self_spec_generate_adaptive, prompt, max_new, skip, k_max,
                             ctypes.byref(ad), log_cap)

    def generate_ar(self, prompt, max_new: int):
        pr = np.ascontiguousarray(prompt, dtype=np.int32)
        out = np.zeros(max(max_new, 1), np.int32)
        st = sd_stats()
        check(load().sd_autoregressive_generate(self._h, _ptr(pr), pr.size, max_new, _ptr(out), ctypes.byref(st)))
        return out[:max_new], _stats(st, None)

    def generate_sd_sample(self, prompt, max_new: int, skip, k_max: int, temperature: float, top_p: float,
                           seed: int, gamma: Optional[float] = None, adaptive: Optional[dict] = None,
                           log_cap: Optional[int] = None):
        """sd_self_spec_sample: a fixed threshold gamma, or the adaptive rule
        when adaptive is a dict of its parameters (defaults: PAPER_ADAPTIVE)."""
        if gamma is None and adaptive is None:
            raise ValueError("gamma or adaptive is required")
        ad = None if adaptive is None else sd_adaptive(**{**PAPER_ADAPTIVE, **adaptive})
        sp = sd_sampling(temperature, top_p, seed)
        pr = np.ascontiguousarray(prompt, dtype=np.int32)
        sk = None if skip is None else np.ascontiguousarray(skip, dtype=np.uint8)
        out = np.zeros(max(max_new, 1), np.int32)
        cap = max(max_new, 1) if log_cap is None else log_cap
        log = np.zeros((cap, 2), np.int32)
        glog = np.zeros(cap, np.float32)
        st = sd_stats()
        st.stage_log = log.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
        st.gamma_log = glog.ctypes.data_as(ctypes.POINTER(ctypes.c_float))
        st.stage_log_cap = cap
        check(load().sd_self_spec_sample(self._h, _ptr(pr), pr.size, max_new, _ptr(sk), k_max,
                                         ctypes.c_float(0.0 if gamma is None else gamma),
                                         None if ad is None else ctypes.byref(ad), ctypes.byref(sp), _ptr(out),
                                         ctypes.byref(st)))
        return out[:max_new], _stats(st, log, glog)

    def search_skip_set(self, prompts, max_new: int, k_max: int, gamma: Optional[float] = None,
                        adaptive: Optional[dict] = None, objective: str = "measured", cost=None, **params) -> dict:
        """sd_search_skip_set over the rows of prompts (int array [n, t]):
        objective "measured" (GPU time per token) or "modeled" (cost, five
        floats); params override SEARCH_DEFAULTS."""
        if gamma is None and adaptive is None:
            raise ValueError("gamma or adaptive is required")
        ad = None if adaptive is None else sd_adaptive(**{**PAPER_ADAPTIVE, **adaptive})
        pr = np.ascontiguousarray(np.atleast_2d(prompts), dtype=np.int32)
        kind = {"measured": SD_SEARCH_MEASURED, "modeled": SD_SEARCH_MODELED}[objective]
        L = 2 * self.cfg.n_layers
        return _search_call(lambda sp, res: load().sd_search_skip_set(
            self._h, _ptr(pr), pr.shape[0], pr.shape[1], max_new, k_max, ctypes.c_float(0.0 if gamma is None else gamma),
            None if ad is None else ctypes.byref(ad), sp, res), L, kind, cost, params)

    def generate_ar_sample(self, prompt, max_new: int, temperature: float, top_p: float, seed: int):
        sp = sd_sampling(temperature, top_p, seed)
        pr = np.ascontiguousarray(prompt, dtype=np.int32)
        out = np.zeros(max(max_new, 1), np.int32)
        st = sd_stats()
        check(load().sd_autoregressive_sample(self._h, _ptr(pr), pr.size, max_new, ctypes.byref(sp), _ptr(out),
                                              ctypes.byref(st)))
        return out[:max_new], _stats(st, None)


def measure_read_bandwidth(buf, nbytes: int, wg_per_cu: int, iters: int, sink, stream=None, offset: int = 0,
                           loads_in_flight: int = 4) -> float:
    """sd_measure_read_bandwidth over nbytes of a torch device buffer from
    byte offset; returns the mean milliseconds of one read."""
    import torch

    st = stream if stream is not None else torch.cuda.current_stream()
    ms = ctypes.c_double()
    check(load().sd_measure_read_bandwidth(ctypes.c_void_p(buf.data_ptr() + offset), nbytes, wg_per_cu,
                                           loads_in_flight, iters,
                                           ctypes.c_void_p(sink.data_ptr()), ctypes.c_void_p(st.cuda_stream),
                                           ctypes.byref(ms)))
    return ms.value


def _search_call(call, n_dims: int, objective: int, cost, params: dict) -> dict:
    """Runs call(params, result) with result arrays sized for params."""
    prm = {**SEARCH_DEFAULTS, **params}
    sp = sd_search_params(prm["n_init"], prm["iterations"], prm["n_candidates"], prm["length_scale"], prm["noise"],
                          prm["xi"], prm["seed"], objective, (ctypes.c_double * 5)(*(cost or (0.0,) * 5)))
    n = max(prm["n_init"] + prm["iterations"], 1)
    best = np.zeros(max(n_dims, 1), np.uint8)
    masks = np.zeros((n, max(n_dims, 1)), np.uint8)
    values = np.zeros(n)
    margins = np.zeros(n)
    u8p, dp = ctypes.POINTER(ctypes.c_uint8), ctypes.POINTER(ctypes.c_double)
    res = sd_search_result(best.ctypes.data_as(u8p), 0.0, 0, masks.ctypes.data_as(u8p), values.ctypes.data_as(dp),
                           margins.ctypes.data_as(dp))
    check(call(ctypes.byref(sp), ctypes.byref(res)))
    k = res.n_evaluated
    return {"best_mask": best[:n_dims], "best_value": res.best_value, "masks": masks[:k, :n_dims],
            "values": values[:k], "margins": margins[:k]}


def search_skip_set_fn(objective, n_dims: int, **params) -> dict:
    """sd_search_skip_set_fn with a Python objective (a function of a uint8
    mask returning a float); params override SEARCH_DEFAULTS.  An exception
    in the objective stops the search and is raised again here."""
    err = []

    def trampoline(mask, n, user, value):
        try:
            value[0] = float(objective(np.ctypeslib.as_array(mask, (n,)).copy()))
            return SD_OK
        except Exception as e:  # noqa: BLE001 - carried across the C boundary
            err.append(e)
            return SD_ERR_INVALID_ARG

    fn = SEARCH_OBJECTIVE_FN(trampoline)
    try:
        return _search_call(lambda sp, res: load().sd_search_skip_set_fn(n_dims, sp, fn, None, res), n_dims, 0, None,
                            params)
    except SDError:
        if err:
            raise err[0]
        raise


def _stats(st: sd_stats, log, glog=None) -> dict:
    d = {k: getattr(st, k) for k, _ in sd_stats._fields_ if k not in ("stage_log", "stage_log_cap", "gamma_log")}
    if log is not None:
        d["stages"] = log[: min(st.n_stages, log.shape[0])].copy()
    if glog is not None:
        d["gammas"] = glog[: min(st.n_stages, glog.shape[0])].copy()
    return d


class KVCache:
    def __init__(self, model: Model, capacity: int, device_buf=None):
        self.model = model
        self.capacity = capacity
        self._buf = device_buf  # keep the caller's buffer alive
        h = ctypes.c_void_p()
        check(load().sd_kv_cache_create(model._h, capacity,
                                        None if device_buf is None else ctypes.c_void_p(device_buf.data_ptr()),
                                        ctypes.byref(h)))
        self._h = h

    def close(self):
        if getattr(self, "_h", None):
            load().sd_kv_cache_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def length(self) -> int:
        return int(load().sd_kv_cache_length(self._h))

    def truncate(self, n: int):
        check(load().sd_kv_cache_truncate(self._h, n))

    def set_length(self, n: int):
        check(load().sd_kv_cache_set_length(self._h, n))
