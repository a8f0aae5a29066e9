"""The oracle's pins are strong enough to catch plausible mistakes.

Each case plants one mistake in a copy of the oracle source, builds it on the
CPU, and checks that the pins used in test_oracle.py (the library-built
float64 model, losslessness, full acceptance with an empty skip set, the
stage closed forms) reject it.  The real oracle is never modified.
"""

import os

import numpy as np
import pytest

import oracle
import sd_synth as S
from tests import torch_ref

SRC = os.path.join(os.path.dirname(oracle.__file__), "sd_oracle.c")

MUTATIONS = {
    "rope_sign": ("v[i + half] = b * cs + a * sn;", "v[i + half] = b * cs - a * sn;"),
    "rope_pairing": ("double a = v[i], b = v[i + half];", "double a = v[2 * i], b = v[2 * i + 1];"),
    "gqa_head_map": ("int g = j / grp;", "int g = j % cf->n_kv_heads;"),
    "score_scale": ("double scale = 1.0 / sqrt((double)dh);", "double scale = 1.0 / (double)dh;"),
    "block_not_causal": ("attend(c, l, qkv + (int64_t)r * nqkv, start + r,",
                         "attend(c, l, qkv + (int64_t)r * nqkv, start + n - 1,"),
    "attn_residual": ("linear_layer(m, FP8_O, l, skip, m->w_o[l], d, (int64_t)H * dh, o, n, t);\n            for (int64_t i = 0; i < (int64_t)n * d; ++i)\n                h[i] += t[i];",
                      "linear_layer(m, FP8_O, l, skip, m->w_o[l], d, (int64_t)H * dh, o, n, t);\n            for (int64_t i = 0; i < (int64_t)n * d; ++i)\n                h[i] = t[i];"),
    "gate_up_swap": ("mm[(int64_t)r * F + f] = silu(gr[f]) * gr[F + f];", "mm[(int64_t)r * F + f] = silu(gr[F + f]) * gr[f];"),
    "silu_sign": ("return a / (1.0 + exp(-a));", "return a / (1.0 + exp(a));"),
    "norm_mean": ("double inv = 1.0 / sqrt(ss / (double)d + m->c.rms_eps);", "double inv = 1.0 / sqrt(ss + m->c.rms_eps);"),
    "accept_index": ("while (na < k && draft[na] == y[na])", "while (na < k && draft[na] == y[na + 1])"),
    "rollback_len": ("rc = orc_cache_truncate(c, lc + na + 1);", "rc = orc_cache_truncate(c, lc + na);"),
    "exit_after_token": ("if (p < gamma)\n                break;", "if (p >= gamma)\n                break;"),
    "kcap": ("if (kcap > max_new - emitted - 1)\n        kcap = max_new - emitted - 1;",
             "if (kcap > max_new - emitted - 2)\n        kcap = max_new - emitted - 2 > 0 ? max_new - emitted - 2 : 0;"),
    "draft_input": ("int32_t in = j == 0 ? last : draft[j - 1];", "int32_t in = last;"),
    "kv_not_rounded": ("if (m->c.wdtype != 1 || x == 0.0 || !isfinite(x))", "if (1)"),
    "kv_round_7bits": ("return ldexp(rint(ldexp(f, 8)), e - 8);", "return ldexp(rint(ldexp(f, 7)), e - 7);"),
    "adapt_sign": ("ar <= ad->alpha ? gamma_d + ad->epsilon : gamma_d - ad->epsilon",
                   "ar <= ad->alpha ? gamma_d - ad->epsilon : gamma_d + ad->epsilon"),
    "adapt_beta2": ("gamma_d = ad->beta2 * gamma_d + (1.0 - ad->beta2) * gamma_t;",
                    "gamma_d = (1.0 - ad->beta2) * gamma_d + ad->beta2 * gamma_t;"),
    "adapt_beta1_swap": ("ad->beta1 * ar + (1.0 - ad->beta1) * ar_e", "(1.0 - ad->beta1) * ar + ad->beta1 * ar_e"),
    "adapt_no_init": ("ar = n_updates == 0 ? ar_e : ad->beta1 * ar", "ar = n_updates < 0 ? ar_e : ad->beta1 * ar"),
    "adapt_rate_with_bonus": ("const double ar_e = (double)na / (double)k;",
                              "const double ar_e = (double)na / (double)(k + 1);"),
    # loader of externally filled caches ([L][2][KVH][len][dh])
    "cache_load_kv_swapped": ("double *dst = c->kv + kv_index(c, l, kvi, g, p);",
                              "double *dst = c->kv + kv_index(c, l, 1 - kvi, g, p);"),
    "cache_load_heads_first": ("for (int kvi = 0; kvi < 2; ++kvi)\n            for (int g = 0; g < cf->n_kv_heads; ++g)",
                               "for (int g = 0; g < cf->n_kv_heads; ++g)\n            for (int kvi = 0; kvi < 2; ++kvi)"),
    "cache_load_transposed": ("dst[e] = kv_dtype == 1 ? bf16_to_double(((const uint16_t *)kv)[src])",
                              "dst[e] = kv_dtype == 1 ? bf16_to_double(((const uint16_t *)kv)"
                              "[src - (size_t)p * cf->head_dim - (size_t)e + (size_t)e * (size_t)len + (size_t)p])"),
}


# Mistakes in the sampling variant, caught by the pins of test_oracle_sampling.py.
SAMPLING_MUTATIONS = {
    "philox_weyl": ("W1 = 0xBB67AE8584CAA73BULL", "W1 = 0xBB67AE8584CAA73DULL"),
    "philox_output_order": ("const uint64_t y1 = (uint64_t)p1;", "const uint64_t y1 = (uint64_t)p0;"),
    "warp_tie_order": ("return (x->id > y->id) - (x->id < y->id);", "return (x->id < y->id) - (x->id > y->id);"),
    "warp_temperature": ("pi[v] = exp(((double)(float)logits[v] - mx) / temperature);",
                         "pi[v] = exp(((double)(float)logits[v] - mx) * temperature);"),
    "warp_norm_all": ("        pi[v] /= zs;", "        pi[v] /= z;"),
    "accept_ratio_inverted": ("const double ratio = p[(size_t)na * V + d] / q[(size_t)na * V + d];",
                              "const double ratio = q[(size_t)na * V + d] / p[(size_t)na * V + d];"),
    "residual_swapped": ("res[v] = pn[v] > qn[v] ? pn[v] - qn[v] : 0.0;", "res[v] = qn[v] > pn[v] ? qn[v] - pn[v] : 0.0;"),
    "residual_from_p": ("y = tot > 0.0 ? draw(res, V, uf, &fm) : draw(pn, V, uf, &fm);", "y = draw(pn, V, uf, &fm);"),
    "final_uses_accept_uniform": ("orc_uniform(sp->seed, emitted + na, ORC_U_FINAL, stage)",
                                  "orc_uniform(sp->seed, emitted + na, ORC_U_ACCEPT, stage)"),
}


def _sampling_pins_hold(lib_path) -> bool:
    from tests import test_oracle_sampling as P

    try:
        for check in P.ALL_CHECKS:
            check(lib_path=lib_path)
        P.check_sd_matches_ar_distribution(lib_path=lib_path, n=8000, T=0.2, top_p=0.85, gamma=0.6, head_gain=1.6)
        return True
    except (oracle.OracleError, AssertionError, IndexError, ValueError):
        return False


def _pins_hold(lib_path) -> bool:
    """True when every pin passes for the oracle built at lib_path."""
    try:
        cfg = S.micro_config()
        w = S.make_weights(cfg, 0)
        m = oracle.Model(cfg, w, lib_path=lib_path)
        toks = S.prompt(cfg, 19, seed=3)
        got = m.score(toks)["logits"]
        ref = torch_ref.forward(cfg, S.weights_as_f64(cfg, w), toks)
        if not np.max(np.abs(got - ref)) <= 1e-10 * np.max(np.abs(ref)):  # NaN fails too
            return False
        cb = S.micro_config(n_layers=3, d_model=48, n_heads=2, n_kv_heads=1, head_dim=24, ffn_dim=80,
                            vocab=61, dtype="bf16", name="micro_bf16")
        wb = S.make_weights(cb, 0)
        got = oracle.Model(cb, wb, lib_path=lib_path).score(toks[:15] % cb.vocab)["logits"]
        ref = torch_ref.forward(cb, S.weights_as_f64(cb, wb), toks[:15] % cb.vocab)
        if not np.max(np.abs(got - ref)) <= 1e-10 * np.max(np.abs(ref)):
            return False
        tiny = S.MODELS["tiny"]
        mt = oracle.Model(tiny, S.make_weights(tiny, 0), lib_path=lib_path)
        pr = S.prompt(tiny, 16)
        ar, _ = mt.generate_ar(pr, 32)
        for mask, k, g in (("tiny", 4, 0.6), ("random3", 6, 0.0), ("none", 4, 0.0), ("tiny", 3, 0.0028)):
            sd = mt.generate_sd(pr, 32, S.skip_mask(tiny, mask, seed=11), k, g)
            if not np.array_equal(sd["tokens"], ar):
                return False
            st = sd["stages"]
            if int(np.sum(st[:, 1] + 1)) != 32 or np.any(st[:, 0] > k):
                return False
            if mask == "none" and g <= 0:
                if not np.array_equal(st[:, 0], st[:, 1]) or sd["n_stages"] != -(-32 // (k + 1)):
                    return False
            if g > 0:
                # drafts before the last of a stage were confident
                pm, i, emitted = sd["draft_pmax"], 0, 0
                for kk, nn in st:
                    if kk and (np.any(pm[i:i + kk - 1] < np.float32(g)) or
                               not (kk == min(k, 32 - emitted - 1) or pm[i + kk - 1] < np.float32(g))):
                        return False
                    i += kk
                    emitted += nn + 1
        # loading an externally filled cache
        from tests import test_oracle as O

        O.check_cache_load(lib_path)
        # adaptive draft exit (the pins of test_oracle_adaptive.py)
        from tests import test_oracle_adaptive as A

        for pin in (A.test_empty_skip_set_lowers_threshold_every_stage, A.test_target_at_one_raises_threshold_every_stage,
                    A.test_beta1_zero_steps_follow_each_stage, A.test_beta1_near_one_freezes_first_acceptance,
                    A.test_first_stage_initialises_the_average, A.test_exit_rule_uses_each_stages_threshold):
            pin(mt)
        return True
    except (oracle.OracleError, AssertionError):
        return False


def test_unmodified_oracle_passes(tmp_path):
    assert _pins_hold(oracle.LIB_PATH)
    assert _sampling_pins_hold(oracle.LIB_PATH)


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name, tmp_path):
    old, new = MUTATIONS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    mutated = tmp_path / "sd_oracle.c"
    mutated.write_text(src.replace(old, new))
    lib = oracle.build(src=str(mutated), out=str(tmp_path / f"liboracle_{name}.so"))
    assert not _pins_hold(lib), f"planted mistake {name} passed every pin"


@pytest.mark.parametrize("name", sorted(SAMPLING_MUTATIONS))
def test_planted_sampling_mistake_is_caught(name, tmp_path):
    old, new = SAMPLING_MUTATIONS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    mutated = tmp_path / "sd_oracle.c"
    mutated.write_text(src.replace(old, new))
    lib = oracle.build(src=str(mutated), out=str(tmp_path / f"liboracle_{name}.so"))
    assert not _sampling_pins_hold(lib), f"planted mistake {name} passed every sampling pin"


# Mistakes in the FP8 draft weights, caught by the pins of test_oracle_fp8.py.
FP8_MUTATIONS = {
    "fp8_ties_away": ("const double r = ldexp(rint(ldexp(a, -quantum)), quantum);",
                      "const double r = ldexp(floor(ldexp(a, -quantum) + 0.5), quantum);"),
    "fp8_scale_not_smallest": ("return e - 9 + (f > 0.875 ? 1 : 0);", "return e - 8 + (f > 0.875 ? 1 : 0);"),
    "fp8_subnormal_quantum": ("const int quantum = e - 1 < -6 ? -9 : e - 1 - 3;",
                              "const int quantum = e - 1 < -6 ? -10 : e - 1 - 3;"),
    "fp8_exponent_bias": ("ldexp(1.0 + (double)mt / 8.0, f - 7)", "ldexp(1.0 + (double)mt / 8.0, f - 8)"),
    "fp8_on_full_model": ("if (skip && m->fp8_q[kind] && m->fp8_q[kind][l])", "if (m->fp8_q[kind] && m->fp8_q[kind][l])"),
    "fp8_sublayer_swap": ("const int run = k < FP8_GATE_UP ? !skip[2 * l] : !skip[2 * l + 1];",
                          "const int run = k < FP8_GATE_UP ? !skip[2 * l + 1] : !skip[2 * l];"),
}


def _fp8_pins_hold(lib_path) -> bool:
    from tests import test_oracle_fp8 as P

    try:
        for check in P.ALL_CHECKS:
            check(lib_path=lib_path)
        return True
    except (oracle.OracleError, AssertionError, IndexError, ValueError):
        return False


def test_unmodified_oracle_passes_fp8_pins():
    assert _fp8_pins_hold(oracle.LIB_PATH)


@pytest.mark.parametrize("name", sorted(FP8_MUTATIONS))
def test_planted_fp8_mistake_is_caught(name, tmp_path):
    old, new = FP8_MUTATIONS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    mutated = tmp_path / "sd_oracle.c"
    mutated.write_text(src.replace(old, new))
    lib = oracle.build(src=str(mutated), out=str(tmp_path / f"liboracle_{name}.so"))
    assert not _fp8_pins_hold(lib), f"planted mistake {name} passed every FP8 pin"


# Mistakes in the skip-set search, caught by the pins of test_oracle_search.py.
SEARCH_SRC = os.path.join(os.path.dirname(oracle.__file__), "skip_search.py")
SEARCH_MUTATIONS = {
    "philox_key": ("philox4x64([a, purpose, c, 0], [seed, 1])", "philox4x64([a, purpose, c, 0], [seed, 0])"),
    "ei_sign": ("imp = best - mu - xi", "imp = mu - best - xi"),
    "ei_no_sigma": ("return imp * cdf + sigma * pdf", "return imp * cdf + pdf"),
    "kernel_not_scaled_by_L": ("np.exp(-hamming / (length_scale * A.shape[1]))", "np.exp(-hamming / length_scale)"),
    "posterior_var_sign": ("var[i] = 1.0 - k @", "var[i] = 1.0 + k @"),
    "no_noise": ("+ noise * np.eye(len(X))", ""),
    "standardise_sample_sd": ("np.sqrt(np.mean((y - y.mean()) ** 2))",
                              "np.sqrt(np.sum((y - y.mean()) ** 2) / max(len(y) - 1, 1))"),
    "worst_incumbent": ("incumbent = X[int(np.argmin(y))]", "incumbent = X[int(np.argmax(y))]"),
    "pick_least_ei": ("pick = int(np.argmax(ei))", "pick = int(np.argmin(ei))"),
    "best_is_max": ("best = float(ys.min())", "best = float(ys.max())"),
    "four_flips": ("flips = 1 + int(search_uniform(seed, t, P_NFLIP, c) * 3.0)",
                   "flips = 1 + int(search_uniform(seed, t, P_NFLIP, c) * 4.0)"),
    "density_range": ("p = 0.6 * search_uniform(seed, t, P_DENSITY, c)", "p = search_uniform(seed, t, P_DENSITY, c)"),
    "init_not_empty": ("p = 0.6 * i / n_init", "p = 0.6 * (i + 1) / (n_init + 1)"),
    "no_dedupe": ("if not any(np.array_equal(z, x) for x in X)]", "]"),
    "draft_mlp_cost_on_attention": ("att = int(np.sum(mask[0::2] == 0))", "att = int(np.sum(mask[1::2] == 0))"),
}


def _search_module(src: str):
    """The search oracle executed from src, as a module of the oracle package."""
    import types

    mod = types.ModuleType("oracle._mutated_skip_search")
    mod.__package__ = "oracle"
    exec(compile(src, SEARCH_SRC, "exec"), mod.__dict__)
    return mod


def _search_pins_hold(mod) -> bool:
    from tests import test_oracle_search as P

    try:
        for check in P.ALL_CHECKS:
            check(mod)
        return True
    except (AssertionError, IndexError, ValueError, np.linalg.LinAlgError):
        return False


def test_unmodified_search_oracle_passes():
    assert _search_pins_hold(_search_module(open(SEARCH_SRC).read()))


@pytest.mark.parametrize("name", sorted(SEARCH_MUTATIONS))
def test_planted_search_mistake_is_caught(name):
    old, new = SEARCH_MUTATIONS[name]
    src = open(SEARCH_SRC).read()
    assert src.count(old) == 1, f"mutation anchor for {name} not found exactly once"
    assert not _search_pins_hold(_search_module(src.replace(old, new))), f"planted mistake {name} passed every pin"
