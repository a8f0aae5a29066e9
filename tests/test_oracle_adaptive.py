"""Pins of the oracle's adaptive draft exit (Sec. 3.4, Eqs. 2-4).

The rule moves the threshold by exactly (1 - beta2) * epsilon per stage, up
when the smoothed acceptance AR is at most the target alpha and down
otherwise, so several special cases have closed forms that do not depend on
retyping the recurrence:
- an empty skip set accepts every draft (AR = 1): with alpha < 1 the threshold
  falls by (1 - beta2) epsilon at every stage, with alpha >= 1 it rises;
- beta1 = 0 makes AR the stage's own acceptance, so each step's direction is
  read off that stage's (k_e, n_e);
- beta1 near 1 freezes AR at the first stage's value (AR_1 = AR_e at e = 1),
  so every early step goes the same way;
and the decoding itself stays lossless.
"""

import numpy as np
import pytest

import oracle
import sd_synth as S

TINY = S.MODELS["tiny"]
STEP = (1 - 0.9) * 0.01  # (1 - beta2) * epsilon with the paper's settings


@pytest.fixture(scope="module")
def tiny():
    return oracle.Model(TINY, S.make_weights(TINY, 0))


def _steps(g):
    return np.round(np.diff(g.astype(np.float64)) / STEP).astype(int)


def test_empty_skip_set_lowers_threshold_every_stage(tiny):
    pr = S.prompt(TINY, 16)
    r = tiny.generate_sd_adaptive(pr, 40, S.skip_mask(TINY, "none"), 4, alpha=0.9)
    g = r["gammas"]
    assert np.all(r["stages"][:, 0] == r["stages"][:, 1])  # every draft accepted
    assert g[0] == np.float32(0.6)
    drafted = r["stages"][:-1, 0] > 0
    expect = 0.6 - STEP * np.cumsum(np.concatenate([[0], drafted.astype(int)]))
    assert np.allclose(g, expect.astype(np.float32), atol=1e-7)
    assert np.all(_steps(g)[drafted] == -1)


def test_target_at_one_raises_threshold_every_stage(tiny):
    pr = S.prompt(TINY, 16)
    r = tiny.generate_sd_adaptive(pr, 40, S.skip_mask(TINY, "tiny"), 4, alpha=1.0)
    drafted = r["stages"][:-1, 0] > 0
    st = _steps(r["gammas"])
    assert np.all(st[drafted] == 1) and np.all(st[~drafted] == 0)


def test_beta1_zero_steps_follow_each_stage(tiny):
    """AR = AR_e: stage e steps up exactly when n_e / k_e <= alpha."""
    pr = S.prompt(TINY, 16)
    for alpha in (0.0, 0.5, 0.99):
        r = tiny.generate_sd_adaptive(pr, 48, S.skip_mask(TINY, "tiny"), 4, alpha=alpha, beta1=0.0)
        k, n = r["stages"][:-1, 0], r["stages"][:-1, 1]
        st = _steps(r["gammas"])
        for e in range(len(st)):
            if k[e] == 0:
                assert st[e] == 0
            else:
                assert st[e] == (1 if n[e] <= alpha * k[e] else -1), (alpha, e)
        assert len(set(st.tolist())) > 1 or alpha in (0.0, 0.99)  # both directions occur at 0.5


def test_beta1_near_one_freezes_first_acceptance(tiny):
    """With beta1 = 0.99, AR stays within 0.01 per stage of AR_1 in {0, 1}."""
    pr = S.prompt(TINY, 16)
    r = tiny.generate_sd_adaptive(pr, 32, S.skip_mask(TINY, "tiny"), 1, alpha=0.5, beta1=0.99)
    k, n = r["stages"][:, 0], r["stages"][:, 1]
    first = np.nonzero(k > 0)[0][0]
    direction = 1 if n[first] == 0 else -1  # AR_1 = 0 -> up, AR_1 = 1 -> down
    st = _steps(r["gammas"])
    drafted = k[:-1] > 0
    assert np.all(st[drafted][:20] == direction)


def test_first_stage_initialises_the_average(tiny):
    """AR_1 = AR_e: with every draft accepted (AR_e = 1) and alpha = 0.5 the
    very first step is down, whatever beta1 is."""
    pr = S.prompt(TINY, 16)
    for beta1 in (0.5, 0.8, 0.99):
        r = tiny.generate_sd_adaptive(pr, 20, S.skip_mask(TINY, "none"), 3, alpha=0.5, beta1=beta1)
        assert _steps(r["gammas"])[0] == -1


@pytest.mark.parametrize("mask,k_max,alpha,gamma0", [("tiny", 4, 0.9, 0.6), ("random3", 6, 0.5, 0.0),
                                                     ("none", 4, 0.9, 0.6), ("tiny", 12, 0.8, 0.003)])
def test_adaptive_is_lossless(tiny, mask, k_max, alpha, gamma0):
    pr = S.prompt(TINY, 16)
    ar, _ = tiny.generate_ar(pr, 40)
    r = tiny.generate_sd_adaptive(pr, 40, S.skip_mask(TINY, mask, seed=11), k_max, alpha=alpha, gamma0=gamma0)
    assert np.array_equal(r["tokens"], ar)
    st = r["stages"]
    assert int(np.sum(st[:, 1] + 1)) == 40 and np.all(st[:, 1] <= st[:, 0]) and np.all(st[:, 0] <= k_max)


def test_exit_rule_uses_each_stages_threshold(tiny):
    pr = S.prompt(TINY, 16)
    n_new = 48
    r = tiny.generate_sd_adaptive(pr, n_new, S.skip_mask(TINY, "tiny"), 6, alpha=0.6, gamma0=0.003)
    pm, i, emitted = r["draft_pmax"], 0, 0
    for (k, n), g in zip(r["stages"], r["gammas"]):
        kcap = min(6, n_new - emitted - 1)
        if k:
            assert np.all(pm[i:i + k - 1] >= g)
            assert k == kcap or pm[i + k - 1] < g
        i += k
        emitted += n + 1
    assert i == pm.size


def test_adaptive_rejects_nan_parameters(tiny):
    with pytest.raises(oracle.OracleError):
        tiny.generate_sd_adaptive(S.prompt(TINY, 4), 4, None, 2, alpha=float("nan"))
