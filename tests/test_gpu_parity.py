"""GPU parity: the HIP library (through its C ABI) against the CPU oracle on
the same seeded inputs.

- sd_forward logits: float32 models within 1e-4, bfloat16 within
  3e-2 * std(row), for 1..20 rows (single-row GEMV path, 16-row MFMA /
  VALU path, a ragged second chunk), with and without a skip mask, at
  several cache lengths, and through a cache rolled back by truncate.
- generation: autoregressive and self-speculative tokens equal the
  oracle's except after a reported near-tie; every GPU token is the
  oracle's choice (or within tau of it) given the GPU's own prefix; the
  stage trace (k_e, n_e) equals the oracle's while the tokens agree.
"""

import numpy as np
import pytest

import oracle
import sd_synth as S
from paper_2309_08168_amd import binding
from tests import gpu_util as U

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


# d_model 640: the MFMA-path input preparation covers one full 512-element
# slice and one partial slice per row
SLICES_BF16 = S.ModelConfig("slices_bf16", 2, 640, 5, 5, 128, 1280, 1000, "bf16")
MODELS = {"tiny": S.MODELS["tiny"], "mini_bf16": U.MINI_BF16, "micro_gqa": U.MICRO_GQA, "slices_bf16": SLICES_BF16}
_cache = {}


def _pair(name, seed=0):
    key = (name, seed)
    if key not in _cache:
        cfg = MODELS[name]
        w = S.make_weights(cfg, seed)
        _cache[key] = (cfg, w, oracle.Model(cfg, w), U.device_model(cfg, w))
    return _cache[key]


def _gpu_logits(dm, toks, cache, skip=None):
    out = torch.empty((len(toks), dm.cfg.vocab), dtype=torch.float32, device="cuda")
    dm.forward(toks, cache, skip=skip, logits=out)
    return out.cpu().numpy()


@pytest.mark.parametrize("name", list(MODELS))
@pytest.mark.parametrize("rows", [1, 2, 5, 16, 20])
def test_forward_logits(name, rows):
    cfg, w, om, dm = _pair(name)
    toks = S.prompt(cfg, 17 + rows, seed=rows)
    # prefix of 17 positions, then `rows` more
    oc = om.cache(64)
    om.forward(oc, toks[:17])
    ref = om.forward(oc, toks[17:])["logits"]
    gc = dm.cache(64)
    dm.forward(toks[:17], gc)
    got = _gpu_logits(dm, toks[17:], gc)
    assert gc.length == 17 + rows
    U.check_logits(cfg, got, ref, f"{name} rows={rows}")


@pytest.mark.parametrize("name", list(MODELS))
@pytest.mark.parametrize("rows", [1, 3, 13])
def test_forward_logits_with_skip(name, rows):
    cfg, w, om, dm = _pair(name)
    z = S.skip_mask(cfg, "random2", seed=3) if cfg.n_layers <= 2 else S.skip_mask(cfg, "tiny")
    toks = S.prompt(cfg, 9 + rows, seed=40 + rows)
    oc = om.cache(32)
    om.forward(oc, toks[:9])
    ref = om.forward(oc, toks[9:], skip=z)["logits"]
    gc = dm.cache(32)
    dm.forward(toks[:9], gc)
    got = _gpu_logits(dm, toks[9:], gc, skip=z)
    U.check_logits(cfg, got, ref, f"{name} skip rows={rows}")


@pytest.mark.parametrize("name", list(MODELS))
def test_forward_from_position_zero_and_rollback(name):
    cfg, w, om, dm = _pair(name)
    toks = S.prompt(cfg, 12, seed=7)
    ref = om.score(toks)["logits"]
    gc = dm.cache(16)
    got = _gpu_logits(dm, toks, gc)
    U.check_logits(cfg, got, ref, f"{name} from 0")
    # roll back 5 positions, write a different continuation, then the original
    gc.truncate(7)
    _gpu_logits(dm, (toks[7:] + 3) % cfg.vocab, gc)
    gc.truncate(7)
    got2 = _gpu_logits(dm, toks[7:], gc)
    U.check_logits(cfg, got2, ref[7:], f"{name} after rollback")


def test_forward_rows_are_independent_of_chunking():
    """One 12-row forward and twelve 1-row forwards give the same logits
    (within tolerance: different kernels)."""
    cfg, w, om, dm = _pair("mini_bf16")
    toks = S.prompt(cfg, 12, seed=9)
    a = _gpu_logits(dm, toks, dm.cache(16))
    c = dm.cache(16)
    b = np.concatenate([_gpu_logits(dm, toks[i:i + 1], c) for i in range(12)])
    ref = om.score(toks)["logits"]
    U.check_logits(cfg, a, ref, "block")
    U.check_logits(cfg, b, ref, "one by one")


GEN_CASES = [
    ("tiny", "tiny", 4, 0.6, 16, 32),
    ("tiny", "random3", 12, 0.0, 16, 32),
    ("tiny", "none", 4, 0.0, 16, 32),
    ("tiny", "tiny", 0, 0.6, 16, 9),
    ("tiny", "tiny", 3, 0.0028, 1, 20),
    ("tiny", "all", 2, 0.0, 5, 11),
    ("micro_gqa", "random2", 6, 0.0, 7, 24),
    ("mini_bf16", "random2", 12, 0.0, 24, 40),
    ("mini_bf16", "0,3", 4, 0.002, 24, 40),
]


@pytest.mark.parametrize("name,mask,k_max,gamma,t,max_new", GEN_CASES)
def test_generate_matches_oracle(name, mask, k_max, gamma, t, max_new):
    cfg, w, om, dm = _pair(name)
    pr = S.prompt(cfg, t, seed=t)
    z = S.skip_mask(cfg, mask, seed=11)
    ar_ref, ar_margin = om.generate_ar(pr, max_new)
    sd_ref = om.generate_sd(pr, max_new, z, k_max, gamma)
    std = om.score(np.concatenate([pr, ar_ref])[:-1])["logits"][t - 1:].std(axis=1)

    ar, ar_st = dm.generate_ar(pr, max_new)
    sd, sd_st = dm.generate_sd(pr, max_new, z, k_max, gamma)
    assert ar_st["n_emitted"] == max_new and sd_st["n_emitted"] == max_new

    n_ar = U.check_free_running(cfg, ar, ar_ref, ar_margin, std, f"{name} AR")
    n_sd = U.check_free_running(cfg, sd, sd_ref["tokens"], sd_ref["margin"], std, f"{name} SD")
    U.check_tokens_teacher_forced(cfg, om, pr, ar, f"{name} AR teacher-forced")
    U.check_tokens_teacher_forced(cfg, om, pr, sd, f"{name} SD teacher-forced")

    st = sd_st["stages"]
    assert int(np.sum(st[:, 1] + 1)) == max_new
    assert np.all((st[:, 1] <= st[:, 0]) & (st[:, 0] <= k_max))
    assert sd_st["n_drafted"] == st[:, 0].sum() and sd_st["n_accepted"] == st[:, 1].sum()
    # stage trace equals the oracle's over the stages whose tokens agree and
    # whose draft p_max is not within tolerance of gamma
    if n_sd == max_new and n_ar == max_new and sd_ref["min_gamma_gap"] > 1e-4:
        assert np.array_equal(st, sd_ref["stages"]), (st.tolist(), sd_ref["stages"].tolist())
    if mask == "none":
        assert np.array_equal(st[:, 0], st[:, 1])
    print(f"{name}: AR agrees for {n_ar}/{max_new}, SD for {n_sd}/{max_new}; stages {len(st)}, "
          f"acceptance {sd_st['n_accepted']}/{sd_st['n_drafted']}")


_planted = {}


def _planted_pair(name, mask, rho, gain):
    """A model whose masked sublayers are nearly redundant (long, confident drafts)."""
    key = (name, mask, rho, gain)
    if key not in _planted:
        cfg = MODELS[name]
        w = S.plant_redundancy(cfg, S.make_weights(cfg, 0), S.skip_mask(cfg, mask, seed=11), rho, gain)
        _planted[key] = (cfg, w, oracle.Model(cfg, w), U.device_model(cfg, w))
    return _planted[key]


ADAPT_CASES = [
    # model, mask, K_max, adaptive parameters, planted (rho, gain) or None, prompt, new tokens
    ("tiny", "tiny", 4, dict(gamma0=0.003, alpha=0.5), None, 16, 48),
    ("tiny", "none", 4, dict(), None, 16, 40),
    ("tiny", "tiny", 8, dict(gamma0=0.6, alpha=0.8), (0.05, 30.0), 16, 64),
    ("tiny", "tiny", 8, dict(gamma0=0.3, alpha=0.9, beta1=0.8), (0.05, 30.0), 16, 64),
    ("mini_bf16", "0,3", 12, dict(gamma0=0.002, alpha=0.3), None, 24, 40),
    ("mini_bf16", "0,3", 8, dict(gamma0=0.6, alpha=0.8), (0.02, 60.0), 24, 64),
]
# A draft's top-1 probability within this of the threshold may exit on the
# other side on the GPU: the logits differ by up to the parity tolerance,
# which moves p_max by ~1e-6 for float32 models and by a few 1e-3 for bf16.
GAMMA_TIE = {"f32": 1e-4, "bf16": 0.02}


@pytest.mark.parametrize("name,mask,k_max,params,planted,t,max_new", ADAPT_CASES)
def test_generate_adaptive_matches_oracle(name, mask, k_max, params, planted, t, max_new):
    """Adaptive draft exit (Sec. 3.4, Eqs. 2-4): tokens, stage trace and the
    threshold of every stage equal the oracle's."""
    cfg, w, om, dm = _pair(name) if planted is None else _planted_pair(name, mask, *planted)
    pr = S.prompt(cfg, t, seed=t)
    z = S.skip_mask(cfg, mask, seed=11)
    ref = om.generate_sd_adaptive(pr, max_new, z, k_max, **params)
    ar_ref, _ = om.generate_ar(pr, max_new)
    std = om.score(np.concatenate([pr, ar_ref])[:-1])["logits"][t - 1:].std(axis=1)
    sd, st = dm.generate_sd_adaptive(pr, max_new, z, k_max, **params)
    n_sd = U.check_free_running(cfg, sd, ref["tokens"], ref["margin"], std, f"{name} adaptive SD")
    U.check_tokens_teacher_forced(cfg, om, pr, sd, f"{name} adaptive SD teacher-forced")
    stg, g = st["stages"], st["gammas"]
    assert int(np.sum(stg[:, 1] + 1)) == max_new and np.all((stg[:, 1] <= stg[:, 0]) & (stg[:, 0] <= k_max))
    # the threshold moves by (1 - beta2) epsilon after every stage with drafts
    p = {**oracle.PAPER_ADAPTIVE, **params}
    step = (1 - p["beta2"]) * p["epsilon"]
    d = np.round(np.diff(g.astype(np.float64)) / step)
    assert np.all(np.abs(d[stg[:-1, 0] > 0]) == 1) and np.all(d[stg[:-1, 0] == 0] == 0)
    if n_sd == max_new and ref["min_gamma_gap"] > GAMMA_TIE[cfg.dtype]:
        assert np.array_equal(stg, ref["stages"]), (stg.tolist(), ref["stages"].tolist())
        assert np.array_equal(g, ref["gammas"])  # bit-exact: same float64 steps, same rounding
    print(f"{name}: adaptive SD agrees for {n_sd}/{max_new}; stages {len(stg)}, acceptance "
          f"{st['n_accepted']}/{st['n_drafted']}, gamma {g[0]:.4f} -> {g[-1]:.4f}")


def test_adaptive_rejects_bad_parameters():
    cfg, w, om, dm = _pair("tiny")
    with pytest.raises(binding.SDError):
        dm.generate_sd_adaptive(S.prompt(cfg, 4), 4, None, 2, alpha=float("nan"))


def test_generate_is_deterministic():
    cfg, w, om, dm = _pair("mini_bf16")
    pr = S.prompt(cfg, 24)
    z = S.skip_mask(cfg, "random2", seed=11)
    a, sa = dm.generate_sd(pr, 30, z, 5, 0.0)
    b, sb = dm.generate_sd(pr, 30, z, 5, 0.0)
    assert np.array_equal(a, b) and np.array_equal(sa["stages"], sb["stages"])


def test_generate_zero_and_one_token():
    cfg, w, om, dm = _pair("tiny")
    pr = S.prompt(cfg, 4)
    out, st = dm.generate_sd(pr, 0, None, 4, 0.6)
    assert out.size == 0 and st["n_emitted"] == 0
    out, st = dm.generate_sd(pr, 1, S.skip_mask(cfg, "tiny"), 4, 0.6)
    ref, _ = om.generate_ar(pr, 1)
    assert out.tolist() == ref.tolist() and st["n_stages"] == 1 and st["n_drafted"] == 0
