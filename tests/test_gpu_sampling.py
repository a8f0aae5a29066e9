"""GPU parity of the sampling variant (sd_self_spec_sample and
sd_autoregressive_sample) against the oracle.

- Same seed, same tokens: both sides draw the same Philox uniforms, so the
  GPU emits the oracle's tokens and stage trace, up to the first token one
  of whose decisions the oracle reports within delta of flipping (float32
  models, and a bf16 model whose measured logit error sets the bound).  delta =
  2 tol / T: a logit error of tol moves a warped probability by at most about
  2 tol / T relative, and so every CDF boundary, acceptance ratio and top-p
  cut by at most that in probability units.  The models have a planted
  lm-head gain, so the distributions are peaked like a trained model's and
  near-ties are rare; with flat random-weight distributions nearly every draw
  would sit within delta of a boundary.
- Distribution: on a small model whose draft is rejected about half the
  time, the GPU's first two tokens over many seeds fit the exact joint
  distribution of autoregressive sampling (chi-square), the defining property
  of speculative sampling.
- Closed forms on the GPU itself: K = 0 equals autoregressive sampling token
  for token, an empty skip set accepts every draft, a one-token nucleus is
  greedy decoding, the same seed repeats, bad parameters are rejected.
"""

import numpy as np
import pytest

import oracle
import sd_synth as S
from paper_2309_08168_amd import binding
from tests import gpu_util as U
from tests import test_oracle_sampling as P

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


_models = {}


def _pair(name, mask="tiny", rho=0.5, gain=16.0):
    key = (name, mask, rho, gain)
    if key not in _models:
        cfg = {"tiny": S.MODELS["tiny"], "micro_gqa": U.MICRO_GQA, "mini_bf16": U.MINI_BF16}[name]
        w = S.plant_redundancy(cfg, S.make_weights(cfg, 0), S.skip_mask(cfg, mask, seed=11), rho, gain)
        _models[key] = (cfg, w, oracle.Model(cfg, w), U.device_model(cfg, w))
    return _models[key]


def _f32(x):
    return float(np.float32(x))


def _first_flag(margin, delta):
    bad = np.nonzero(margin < delta)[0]
    return int(bad[0]) if bad.size else len(margin)


# (model, mask, K_max, gamma or None for adaptive, temperature, top_p, prompt, new tokens, seed)
CASES = [
    ("tiny", "tiny", 4, 0.6, 1.0, 0.9, 16, 40, 1),
    ("tiny", "tiny", 4, 0.3, 0.2, 0.85, 16, 40, 2),
    ("tiny", "tiny", 6, None, 0.6, 0.95, 16, 48, 3),
    ("tiny", "random3", 8, 0.0, 1.0, 1.0, 9, 40, 5),
    ("micro_gqa", "random2", 5, 0.2, 0.5, 0.9, 7, 32, 4),
]


@pytest.mark.parametrize("name,mask,k_max,gamma,T,top_p,t,max_new,seed", CASES)
def test_sample_matches_oracle(name, mask, k_max, gamma, T, top_p, t, max_new, seed):
    cfg, w, om, dm = _pair(name, mask)
    T, top_p = _f32(T), _f32(top_p)  # the library takes float32 parameters
    pr = S.prompt(cfg, t, seed=t)
    z = S.skip_mask(cfg, mask, seed=11)
    kw = dict(adaptive={}) if gamma is None else dict(gamma=gamma)
    ref = om.generate_sd_sample(pr, max_new, z, k_max, T, top_p, seed, **kw)
    ar_ref, ar_margin = om.generate_ar_sample(pr, max_new, T, top_p, seed)
    sd, st = dm.generate_sd_sample(pr, max_new, z, k_max, T, top_p, seed, **kw)
    ar, _ = dm.generate_ar_sample(pr, max_new, T, top_p, seed)
    delta = 2 * U.FP32_TOL / T

    n_sd = _first_flag(ref["margin"], delta)
    n_ar = _first_flag(ar_margin, delta)
    assert np.array_equal(sd[:n_sd], ref["tokens"][:n_sd]), (sd.tolist(), ref["tokens"].tolist())
    assert np.array_equal(ar[:n_ar], ar_ref[:n_ar]), (ar.tolist(), ar_ref.tolist())
    # the stage trace over the stages that end before the first flagged token
    # (and draft exits not within delta of the threshold)
    if ref["min_gamma_gap"] > delta:
        ends = np.cumsum(ref["stages"][:, 1] + 1)
        n_st = int(np.sum(ends <= n_sd))
        assert np.array_equal(st["stages"][:n_st], ref["stages"][:n_st])
        if gamma is None:
            assert np.array_equal(st["gammas"][:n_st], ref["gammas"][:n_st])
    s = st["stages"]
    assert int(np.sum(s[:, 1] + 1)) == max_new and np.all((s[:, 1] <= s[:, 0]) & (s[:, 0] <= k_max))
    assert np.all((sd >= 0) & (sd < cfg.vocab))
    print(f"{name} T={T} top_p={top_p}: SD equal for {n_sd}/{max_new}, AR for {n_ar}/{max_new}; "
          f"acceptance {st['n_accepted']}/{st['n_drafted']}")


# bfloat16 model (planted like the cases above): same seed, same tokens.  The
# bf16 tolerance (3e-2 std of a row) would flag nearly every draw of a
# peaked distribution, so the test first measures the GPU's logit error on
# this model over the oracle's own sampled sequence, through the decode-path
# kernels (1-, 2- and 5-row forwards, full model and draft mask), requires
# it within BF16_SAMPLE_TOL absolute, and takes delta = 2 BF16_SAMPLE_TOL / T.
BF16_SAMPLE_TOL = 1e-4
# Seeds chosen (on the CPU, with the oracle alone) so that the oracle's first
# decision within delta comes late, and the comparison covers most tokens.
BF16_CASES = [
    ("mini_bf16", "random2", 4, 0.6, 1.0, 0.9, 16, 40, 19),
    ("mini_bf16", "random2", 6, None, 0.6, 1.0, 16, 40, 29),
    ("mini_bf16", "random2", 5, 0.0, 0.5, 1.0, 12, 32, 9),
]


def _decode_path_error(cfg, om, dm, seq, start, z):
    """max |GPU - oracle| over the logits of rows start.. of seq, forwarded
    in chunks of 1, 2 and 5 rows, with the full model and with mask z."""
    worst = 0.0
    for skip in (None, z):
        oc, gc = om.cache(len(seq)), dm.cache(len(seq))
        om.forward(oc, seq[:start], want_logits=False)
        dm.forward(seq[:start], gc)
        i, sizes = start, [1, 2, 5]
        while i < len(seq):
            n = min(sizes[(i - start) % 3], len(seq) - i)
            ref = om.forward(oc, seq[i:i + n], skip=skip)["logits"]
            got = torch.empty((n, cfg.vocab), dtype=torch.float32, device="cuda")
            dm.forward(seq[i:i + n], gc, skip=skip, logits=got)
            worst = max(worst, float(np.abs(got.cpu().numpy().astype(np.float64) - ref).max()))
            i += n
    return worst


@pytest.mark.parametrize("name,mask,k_max,gamma,T,top_p,t,max_new,seed", BF16_CASES)
def test_sample_matches_oracle_bf16(name, mask, k_max, gamma, T, top_p, t, max_new, seed):
    cfg, w, om, dm = _pair(name, mask)
    T, top_p = _f32(T), _f32(top_p)
    pr = S.prompt(cfg, t, seed=t)
    z = S.skip_mask(cfg, mask, seed=11)
    kw = dict(adaptive={}) if gamma is None else dict(gamma=gamma)
    ref = om.generate_sd_sample(pr, max_new, z, k_max, T, top_p, seed, **kw)
    ar_ref, ar_margin = om.generate_ar_sample(pr, max_new, T, top_p, seed)
    seq = np.concatenate([pr, ref["tokens"]]).astype(np.int32)
    err = _decode_path_error(cfg, om, dm, seq, t - 1, z)
    # the bf16 parity bar holds, and this model's error is within the bound delta assumes
    assert err <= BF16_SAMPLE_TOL, f"GPU logit error {err:.3g} above {BF16_SAMPLE_TOL}"
    sd, st = dm.generate_sd_sample(pr, max_new, z, k_max, T, top_p, seed, **kw)
    ar, _ = dm.generate_ar_sample(pr, max_new, T, top_p, seed)
    delta = 2 * BF16_SAMPLE_TOL / T
    n_sd = _first_flag(ref["margin"], delta)
    n_ar = _first_flag(ar_margin, delta)
    assert np.array_equal(sd[:n_sd], ref["tokens"][:n_sd]), (sd.tolist(), ref["tokens"].tolist())
    assert np.array_equal(ar[:n_ar], ar_ref[:n_ar]), (ar.tolist(), ar_ref.tolist())
    if ref["min_gamma_gap"] > delta:
        ends = np.cumsum(ref["stages"][:, 1] + 1)
        n_st = int(np.sum(ends <= n_sd))
        assert np.array_equal(st["stages"][:n_st], ref["stages"][:n_st])
        if gamma is None:
            assert np.array_equal(st["gammas"][:n_st], ref["gammas"][:n_st])
    # the comparison must cover most of the run, else the case says little
    assert n_sd >= max_new // 2 and n_ar >= max_new // 2, (n_sd, n_ar)
    print(f"{name} bf16 T={T} top_p={top_p}: logit error {err:.2e}; SD equal for {n_sd}/{max_new}, "
          f"AR for {n_ar}/{max_new}; acceptance {st['n_accepted']}/{st['n_drafted']}")


def test_speculative_sampling_distribution_on_gpu():
    """The GPU's speculative sampling fits the exact AR joint distribution of
    the first two tokens (the small model of the oracle's pins)."""
    om = P.small_model()
    w = S.plant_redundancy(P.SMALL, S.make_weights(P.SMALL, 2), P.SMALL_SKIP, 8.0, 8.0)
    dm = U.device_model(P.SMALL, w)
    T, top_p = 1.0, _f32(0.9)
    joint = P.exact_joint2(om, P.SMALL_PROMPT, T, top_p)
    counts = np.zeros_like(joint)
    drafted = accepted = 0
    n = 4000
    for seed in range(n):
        tok, st = dm.generate_sd_sample(P.SMALL_PROMPT, 2, P.SMALL_SKIP, 3, T, top_p, 10_000 + seed, gamma=0.0)
        counts[tok[0], tok[1]] += 1
        drafted += st["n_drafted"]
        accepted += st["n_accepted"]
    rate = accepted / drafted
    assert 0.25 < rate < 0.75, rate
    assert counts[joint == 0].sum() == 0
    pv = P._chi2_pvalue(counts.ravel(), joint.ravel())
    print(f"GPU speculative sampling: acceptance {rate:.2f}, chi-square p = {pv:.3g} over {n} seeds")
    assert pv > 1e-3


@pytest.mark.parametrize("name", ["tiny", "mini_bf16"])
def test_closed_forms_on_gpu(name):
    cfg, w, om, dm = _pair(name, "tiny" if name == "tiny" else "0,3")
    pr = S.prompt(cfg, 12, seed=1)
    z = S.skip_mask(cfg, "tiny" if name == "tiny" else "0,3", seed=11)
    for seed in (7, 8):
        ar, _ = dm.generate_ar_sample(pr, 20, 0.8, 0.9, seed)
        sd0, st0 = dm.generate_sd_sample(pr, 20, z, 0, 0.8, 0.9, seed, gamma=0.6)
        assert np.array_equal(sd0, ar) and np.all(st0["stages"] == 0)
        sdn, stn = dm.generate_sd_sample(pr, 20, None, 4, 0.8, 0.9, seed, gamma=0.0)
        assert stn["n_accepted"] == stn["n_drafted"] > 0
        again, _ = dm.generate_sd_sample(pr, 20, z, 4, 0.8, 0.9, seed, gamma=0.3)
        once, _ = dm.generate_sd_sample(pr, 20, z, 4, 0.8, 0.9, seed, gamma=0.3)
        assert np.array_equal(again, once)
    other, _ = dm.generate_sd_sample(pr, 20, z, 4, 0.8, 0.9, 9, gamma=0.3)
    assert not np.array_equal(other, once)
    greedy, _ = dm.generate_ar(pr, 20)
    one, _ = dm.generate_sd_sample(pr, 20, z, 4, 0.5, 1e-9, 3, gamma=0.6)
    assert np.array_equal(one, greedy)


def test_sampling_rejects_bad_parameters():
    cfg, w, om, dm = _pair("tiny")
    pr = S.prompt(cfg, 4)
    for T, p in ((0.0, 0.9), (-1.0, 0.9), (float("inf"), 0.9), (1.0, 0.0), (1.0, 1.5), (float("nan"), 0.5)):
        with pytest.raises(binding.SDError):
            dm.generate_sd_sample(pr, 4, None, 2, T, p, 0, gamma=0.5)
        with pytest.raises(binding.SDError):
            dm.generate_ar_sample(pr, 4, T, p, 0)


def test_cut_through_tied_tokens():
    """Identical lm-head rows give every token the same logit: the warped
    distribution is uniform, the nucleus is the ceil(top_p V) lowest ids (a
    cut through one group of ties), the draft equals the full model (every
    draft accepted), and the draws are uniform over the nucleus."""
    cfg = U.MICRO_GQA
    w = S.make_weights(cfg, 3)
    w["lm_head"] = np.repeat(w["lm_head"][:1], cfg.vocab, axis=0).copy()
    dm = U.device_model(cfg, w)
    om = oracle.Model(cfg, w)
    pr = S.prompt(cfg, 5, seed=2)
    top_p = _f32(0.3)
    keep = int(np.ceil(top_p * cfg.vocab))
    ref = om.generate_sd_sample(pr, 30, S.skip_mask(cfg, "random2", seed=11), 4, 0.7, top_p, 5, gamma=0.0)
    counts = np.zeros(cfg.vocab)
    for seed in range(60):
        tok, st = dm.generate_sd_sample(pr, 30, S.skip_mask(cfg, "random2", seed=11), 4, 0.7, top_p, seed, gamma=0.0)
        assert st["n_accepted"] == st["n_drafted"]
        if seed == 5:
            assert np.array_equal(tok, ref["tokens"])
        np.add.at(counts, tok, 1)
    assert counts[keep:].sum() == 0 and np.all(counts[:keep] > 0)
    assert P._chi2_pvalue(counts[:keep], np.full(keep, 1.0 / keep)) > 1e-3
