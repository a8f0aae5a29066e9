"""Pins of the oracle's sampling variant (appendix: self-speculative decoding
with random sampling, temperature and top-p, and the adaptive draft exit).

What fixes the expected values:
- Philox4x64-10: numpy's own implementation of the generator (a library
  routine); numpy advances the counter before its first block.
- The warped distribution: softmax closed forms, a hand-worked nucleus, the
  (probability, id) order on ties, and temperature as a logit scale.
- Autoregressive sampling draws from the warped distribution: a chi-square
  goodness-of-fit test against it.
- The defining property of speculative sampling: the tokens it emits have
  the distribution of autoregressive sampling from the full model, whatever
  the draft.  A chi-square test of the joint distribution of the first two
  tokens, on a small model whose draft differs enough from the full model
  that a third to two thirds of the drafts are rejected, against the exact
  joint distribution computed from the oracle's own forward and warp.
- Special cases with closed forms: K = 0 reproduces autoregressive sampling
  token for token (the counters coincide); an empty skip set accepts every
  draft (q = p); a nucleus of one token is greedy decoding; gamma above 1
  drafts one token per stage.

Each check is a function of the oracle build, so test_oracle_mutations.py
runs them against planted mistakes.
"""

import numpy as np
import pytest
from scipy import stats

import oracle
import sd_synth as S

# A small model whose draft (attention of layer 0 and MLP of layer 1
# skipped) disagrees with the full model about half the time: the skipped
# sublayers' output projections are scaled up 8x, so skipping them matters,
# and the lm-head gain spreads the logits over a few units at the sampling
# temperature (8 at T = 1, 1.6 at T = 0.2).
SMALL = S.micro_config(vocab=13, name="micro13")
SMALL_SKIP = np.array([1, 0, 0, 1], np.uint8)
SMALL_PROMPT = np.array([3, 11, 0, 7, 5], np.int32)


def small_model(lib_path=oracle.LIB_PATH, head_gain=8.0):
    w = S.plant_redundancy(SMALL, S.make_weights(SMALL, 2), SMALL_SKIP, 8.0, head_gain)
    return oracle.Model(SMALL, w, lib_path=lib_path)


def _chi2_pvalue(counts: np.ndarray, probs: np.ndarray, min_expected: float = 5.0) -> float:
    """Goodness of fit of counts to probs; cells of probability zero are left
    out (callers check they are empty), cells expected below min_expected
    are pooled."""
    live = probs > 0
    counts, probs = counts[live], probs[live]
    n = counts.sum()
    exp = probs * n
    big = exp >= min_expected
    obs = list(counts[big])
    ex = list(exp[big])
    if (~big).any():
        obs.append(counts[~big].sum())
        ex.append(exp[~big].sum())
    obs, ex = np.asarray(obs, float), np.asarray(ex, float)
    chi2 = float(((obs - ex) ** 2 / ex).sum())
    return float(stats.chi2.sf(chi2, len(obs) - 1))


def _next_dist(m, ctx, T, top_p):
    lg = m.score(np.asarray(ctx, np.int32))["logits"][-1]
    return oracle.warp(lg, T, top_p, lib_path=m._lib_path)[0]


def exact_joint2(m, prompt, T, top_p):
    """P(x1, x2) of autoregressive sampling after prompt."""
    V = m.cfg.vocab
    p1 = _next_dist(m, prompt, T, top_p)
    joint = np.zeros((V, V))
    for x1 in np.nonzero(p1 > 0)[0]:
        joint[x1] = p1[x1] * _next_dist(m, list(prompt) + [int(x1)], T, top_p)
    return joint


# ---------------------------------------------------------------------------
# checks (each a function of the oracle build)


def check_philox(lib_path=oracle.LIB_PATH):
    keys = [(0, 0), (0x0123456789ABCDEF, 0xFEDCBA9876543210), (2**64 - 1, 12345)]
    ctrs = [(1, 0, 0, 0), (6, 1, 7, 0), (2**63 + 5, 2**64 - 1, 3, 9), (123456789, 2, 0, 2**40)]
    for key in keys:
        for ctr in ctrs:
            prev = list(ctr)
            prev[0] -= 1  # numpy advances the counter before generating
            bg = np.random.Philox(key=np.array(key, dtype=np.uint64), counter=np.array(prev, dtype=np.uint64))
            want = bg.random_raw(4)
            got = oracle.philox4x64(ctr, key, lib_path=lib_path)
            assert np.array_equal(got, want), (key, ctr, got, want)


def check_uniforms(lib_path=oracle.LIB_PATH):
    """24-bit uniforms, U[0, 1) by a Kolmogorov-Smirnov test, distinct per
    purpose and stage."""
    u = np.array([oracle.uniform(7, i, oracle.U_DRAFT, 0, lib_path=lib_path) for i in range(4000)])
    assert np.all((u >= 0) & (u < 1)) and np.all(u * 2**24 == np.floor(u * 2**24))
    assert stats.kstest(u, "uniform").pvalue > 1e-3
    a = oracle.uniform(7, 5, oracle.U_DRAFT, 0, lib_path=lib_path)
    assert a != oracle.uniform(7, 5, oracle.U_ACCEPT, 0, lib_path=lib_path)
    assert a != oracle.uniform(7, 5, oracle.U_DRAFT, 1, lib_path=lib_path)
    assert a != oracle.uniform(8, 5, oracle.U_DRAFT, 0, lib_path=lib_path)


def check_warp(lib_path=oracle.LIB_PATH):
    def warp(lg, T, p):
        return oracle.warp(np.asarray(lg, float), T, p, lib_path=lib_path)

    # top_p = 1 is the softmax of logits / T
    rng = np.random.default_rng(4)
    lg = rng.normal(0, 2, 50).astype(np.float32).astype(np.float64)
    for T in (1.0, 0.5, 2.0):
        e = np.exp((lg - lg.max()) / T)
        pi, kept, cm = warp(lg, T, 1.0)
        assert kept == 50 and cm == np.inf and np.allclose(pi, e / e.sum(), rtol=1e-13, atol=0)
    # the nucleus of (0.5, 0.3, 0.15, 0.05): the shortest prefix reaching top_p, renormalised
    lg = np.log([0.5, 0.3, 0.15, 0.05])
    for top_p, want in ((0.45, [1, 0, 0, 0]), (0.75, [0.625, 0.375, 0, 0]), (0.85, [0.5 / 0.95, 0.3 / 0.95, 0.15 / 0.95, 0])):
        pi, kept, cm = warp(lg, 1.0, top_p)
        assert kept == np.count_nonzero(want) and np.allclose(pi, want, rtol=1e-6, atol=1e-12), (top_p, pi)
    assert abs(warp(lg, 1.0, 0.75)[2] - 0.05) < 1e-6  # masses 0.5 and 0.8 around 0.75
    # the order is by probability, not by id
    pi, kept, _ = warp(np.log([0.05, 0.3, 0.5, 0.15]), 1.0, 0.75)
    assert kept == 2 and np.allclose(pi, [0, 0.375, 0.625, 0], rtol=1e-6)
    # equal probabilities: lower ids first
    pi, kept, _ = warp(np.zeros(4), 1.0, 0.5)
    assert kept == 2 and np.allclose(pi, [0.5, 0.5, 0, 0])
    pi, kept, _ = warp(np.zeros(4), 1.0, 0.6)
    assert kept == 3 and np.allclose(pi, [1 / 3, 1 / 3, 1 / 3, 0])
    # temperature divides the logits (powers of two keep the float32 roundings exact)
    lg = rng.normal(0, 2, 40).astype(np.float32).astype(np.float64)
    for T in (0.25, 0.5, 4.0):
        a = warp(lg, T, 0.8)
        b = warp(lg / T, 1.0, 0.8)
        assert a[1] == b[1] and np.allclose(a[0], b[0], rtol=1e-12, atol=0)


def check_ar_sampling_distribution(lib_path=oracle.LIB_PATH, n=3000):
    m = small_model(lib_path)
    T, top_p = 1.0, 0.9
    p1 = _next_dist(m, SMALL_PROMPT, T, top_p)
    counts = np.zeros(SMALL.vocab)
    for seed in range(n):
        tok, _ = m.generate_ar_sample(SMALL_PROMPT, 1, T, top_p, seed)
        counts[tok[0]] += 1
    assert counts[p1 == 0].sum() == 0  # nothing outside the nucleus
    pv = _chi2_pvalue(counts, p1)
    assert pv > 1e-3, f"AR sampling does not fit its distribution (p = {pv:.3g})"


def check_sd_matches_ar_distribution(lib_path=oracle.LIB_PATH, n=12000, T=1.0, top_p=0.9, k_max=3, gamma=0.0,
                                     head_gain=8.0):
    m = small_model(lib_path, head_gain)
    joint = exact_joint2(m, SMALL_PROMPT, T, top_p)
    counts = np.zeros_like(joint)
    drafted = accepted = 0
    for seed in range(n):
        r = m.generate_sd_sample(SMALL_PROMPT, 2, SMALL_SKIP, k_max, T, top_p, seed, gamma=gamma)
        counts[r["tokens"][0], r["tokens"][1]] += 1
        drafted += r["n_drafted"]
        accepted += r["n_accepted"]
    rate = accepted / max(drafted, 1)
    assert 0.25 < rate < 0.75, f"acceptance {rate:.2f}: the test would not exercise both outcomes"
    assert counts[joint == 0].sum() == 0
    pv = _chi2_pvalue(counts.ravel(), joint.ravel())
    assert pv > 1e-3, f"speculative sampling does not match AR sampling (p = {pv:.3g}, acceptance {rate:.2f})"


def check_closed_forms(lib_path=oracle.LIB_PATH):
    tiny = S.MODELS["tiny"]
    mt = oracle.Model(tiny, S.make_weights(tiny, 0), lib_path=lib_path)
    pr = S.prompt(tiny, 16)
    z = S.skip_mask(tiny, "tiny")
    for seed in (1, 2):
        # K = 0: every stage is one full-model draw with the counters of AR sampling
        ar, _ = mt.generate_ar_sample(pr, 12, 0.8, 0.9, seed)
        sd = mt.generate_sd_sample(pr, 12, z, 0, 0.8, 0.9, seed, gamma=0.6)
        assert np.array_equal(sd["tokens"], ar) and np.all(sd["stages"] == 0)
        # an empty skip set: the draft is the full model, so every draft is accepted
        sd = mt.generate_sd_sample(pr, 12, None, 4, 0.8, 0.9, seed, gamma=0.0)
        assert sd["n_accepted"] == sd["n_drafted"] > 0
        # gamma above 1: the first draft of every stage already exits
        sd = mt.generate_sd_sample(pr, 12, z, 4, 0.8, 0.9, seed, gamma=1.5)
        budget = [min(4, 12 - e - 1) for e in np.cumsum([0] + list(sd["stages"][:-1, 1] + 1))]
        assert np.array_equal(sd["stages"][:, 0], np.minimum(budget, 1))
    # a nucleus of one token: sampling is greedy decoding, at any temperature
    greedy, _ = mt.generate_ar(pr, 16)
    for T in (0.3, 1.7):
        sd = mt.generate_sd_sample(pr, 16, z, 4, T, 1e-9, 3, gamma=0.6)
        assert np.array_equal(sd["tokens"], greedy)
        arr, _ = mt.generate_ar_sample(pr, 16, T, 1e-9, 3)
        assert np.array_equal(arr, greedy)


def check_stage_bookkeeping(lib_path=oracle.LIB_PATH):
    """Stage counts add up, drafts before a stage's last were confident, and
    the adaptive threshold starts at gamma0."""
    tiny = S.MODELS["tiny"]
    mt = oracle.Model(tiny, S.make_weights(tiny, 0), lib_path=lib_path)
    pr = S.prompt(tiny, 16)
    z = S.skip_mask(tiny, "tiny")
    for kw in (dict(gamma=0.02), dict(adaptive=dict(gamma0=0.02, alpha=0.5))):
        r = mt.generate_sd_sample(pr, 40, z, 5, 0.3, 0.95, 9, **kw)
        st, qm = r["stages"], r["draft_qmax"]
        assert int(np.sum(st[:, 1] + 1)) == 40 and np.all(st[:, 1] <= st[:, 0]) and np.all(st[:, 0] <= 5)
        i = emitted = 0
        for s_i, (kk, nn) in enumerate(st):
            g = r["gammas"][s_i]
            if kk:
                assert np.all(qm[i:i + kk - 1] >= g)
                assert kk == min(5, 40 - emitted - 1) or qm[i + kk - 1] < g
            i += kk
            emitted += nn + 1
        assert np.all(r["margin"] >= 0)
        if "adaptive" in kw:
            assert r["gammas"][0] == np.float32(0.02)


ALL_CHECKS = (check_philox, check_uniforms, check_warp, check_closed_forms, check_stage_bookkeeping,
              check_ar_sampling_distribution, check_sd_matches_ar_distribution)


# ---------------------------------------------------------------------------
# tests


def test_philox_matches_numpy():
    check_philox()


def test_uniforms():
    check_uniforms()


def test_warped_distribution():
    check_warp()


def test_closed_forms():
    check_closed_forms()


def test_stage_bookkeeping():
    check_stage_bookkeeping()


def test_ar_sampling_fits_its_distribution():
    check_ar_sampling_distribution()


def test_speculative_sampling_matches_ar_sampling():
    check_sd_matches_ar_distribution()


def test_speculative_sampling_matches_ar_sampling_low_temperature():
    """The paper's summarisation settings (temperature 0.2, top-p 0.85) with
    the static exit at 0.6."""
    check_sd_matches_ar_distribution(n=8000, T=0.2, top_p=0.85, gamma=0.6, head_gain=1.6)


def test_rejects_bad_parameters():
    m = small_model()
    for T, p in ((0.0, 0.9), (-1.0, 0.9), (1.0, 0.0), (1.0, 1.5), (float("nan"), 0.9)):
        with pytest.raises(oracle.OracleError):
            m.generate_sd_sample(SMALL_PROMPT, 4, SMALL_SKIP, 2, T, p, 0, gamma=0.5)
        with pytest.raises(oracle.OracleError):
            m.generate_ar_sample(SMALL_PROMPT, 4, T, p, 0)
