"""Pins of the oracle's skip-set search (Sec. 3.3, Eq. 1).

Each check takes the module under test, so the mutation tests can run the
same pins against copies with planted mistakes:

- uniforms: the search's Philox words equal numpy's Philox generator;
- surrogate: the posterior equals scikit-learn's Gaussian-process
  regressor with the Laplacian (L1) kernel, which on 0/1 vectors is the
  Hamming kernel; it interpolates at noise-free observations and reverts to
  the prior far from them;
- acquisition: expected improvement equals the integral that defines it,
  E[max(best - xi - f, 0)] under f ~ N(mu, sigma^2), taken by quadrature;
- candidates: local moves stay within 3 flips of the incumbent, random
  masks have the stated densities;
- search: on a 6-sublayer objective it finds the brute-force optimum, on a
  planted 24-sublayer objective it recovers the planted mask, it never
  evaluates a mask twice and it is deterministic in its seed.
"""

import math

import numpy as np
import pytest
from scipy import integrate, stats

from oracle import skip_search as O


def check_uniforms(mod=O):
    for seed in (0, 12345, 2**64 - 1):
        for ctr in ((1, 100, 0, 0), (7, 104, 96, 0), (2**40, 102, 3, 0)):
            prev = list(ctr)
            prev[0] -= 1  # numpy advances the counter before generating
            bg = np.random.Philox(key=np.array([seed, 1], np.uint64), counter=np.array(prev, np.uint64))
            want = int(bg.random_raw(4)[0]) // 2**40 / 2.0**24
            assert mod.search_uniform(seed, ctr[0], ctr[1], ctr[2]) == want, (seed, ctr)


def check_standardise(mod=O):
    y = np.array([3.0, 1.0, 4.0, 1.0, 5.0, 9.0])
    assert np.allclose(mod.standardise(y), (y - y.mean()) / np.std(y), rtol=0, atol=1e-15)
    assert np.array_equal(mod.standardise([2.5, 2.5, 2.5]), np.zeros(3))
    assert np.array_equal(mod.standardise([7.0]), np.zeros(1))


def _sklearn_posterior(X, ys, Z, length_scale, noise):
    from sklearn.gaussian_process import GaussianProcessRegressor
    from sklearn.gaussian_process.kernels import PairwiseKernel

    kern = PairwiseKernel(gamma=1.0 / (length_scale * X.shape[1]), metric="laplacian", gamma_bounds="fixed")
    gp = GaussianProcessRegressor(kernel=kern, alpha=noise, optimizer=None, normalize_y=False)
    gp.fit(X.astype(np.float64), ys)
    return gp.predict(Z.astype(np.float64), return_std=True)


def check_posterior(mod=O):
    rng = np.random.default_rng(5)
    for L, n, ls, noise in ((10, 7, 0.3, 1e-3), (24, 15, 0.25, 1e-2), (40, 30, 0.1, 1e-6)):
        X = (rng.random((n, L)) < 0.4).astype(np.uint8)
        ys = mod.standardise(rng.normal(size=n) * 3 + 1)
        Z = (rng.random((9, L)) < 0.4).astype(np.uint8)
        mu, sd = mod.posterior(X, ys, Z, ls, noise)
        mu_ref, sd_ref = _sklearn_posterior(X, ys, Z, ls, noise)
        assert np.allclose(mu, mu_ref, rtol=1e-9, atol=1e-12), (mu, mu_ref)
        assert np.allclose(sd, sd_ref, rtol=1e-7, atol=1e-9), (sd, sd_ref)
    # interpolation at noise-free observations, the prior far from them
    X = np.eye(6, dtype=np.uint8)
    ys = np.array([0.5, -1.0, 2.0, 0.0, 1.5, -0.25])
    mu, sd = mod.posterior(X, ys, X, 0.5, 1e-12)
    assert np.allclose(mu, ys, atol=1e-9) and np.all(sd < 1e-5)
    far = np.ones((1, 6), np.uint8)  # hamming 5 from every observation
    mu, sd = mod.posterior(X, ys, far, 0.01, 1e-12)
    assert abs(mu[0]) < 1e-12 and abs(sd[0] - 1.0) < 1e-12


def check_kernel(mod=O):
    a = np.array([1, 0, 1, 1, 0, 0, 1, 0], np.uint8)
    b = np.array([0, 0, 1, 0, 0, 1, 1, 1], np.uint8)
    k = mod.kernel(a, b, 0.5)[0, 0]
    # the product over coordinates of exp(-|a_j - b_j| / (0.5 L))
    assert math.isclose(k, math.prod(math.exp(-abs(int(x) - int(y)) / 4.0) for x, y in zip(a, b)), rel_tol=1e-15)
    assert mod.kernel(a, a, 0.5)[0, 0] == 1.0


def check_expected_improvement(mod=O):
    for mu, sigma, best, xi in ((0.0, 1.0, 0.0, 0.0), (0.3, 0.5, -0.2, 0.01), (-1.0, 0.2, 0.4, 0.05),
                                (2.0, 0.7, -1.5, 0.0), (0.1, 2.5, 0.1, 0.3)):
        want = integrate.quad(lambda f: (best - xi - f) * stats.norm.pdf(f, mu, sigma), -np.inf, best - xi,
                              epsabs=1e-13, epsrel=1e-12)[0]
        got = mod.expected_improvement(mu, sigma, best, xi)
        assert math.isclose(got, want, rel_tol=1e-9, abs_tol=1e-14), (mu, sigma, best, xi, got, want)
    assert mod.expected_improvement(-0.5, 0.0, 0.0, 0.1) == pytest.approx(0.4, abs=1e-15)
    assert mod.expected_improvement(0.5, 0.0, 0.0, 0.1) == 0.0


def check_candidates(mod=O):
    L, nc = 40, 64
    inc = (np.random.default_rng(1).random(L) < 0.3).astype(np.uint8)
    local_flips, dens = [], []
    for t in range(30):
        for c in range(nc):
            z = mod.candidate(9, t, c, nc, L, inc)
            assert z.shape == (L,) and set(np.unique(z)) <= {0, 1}
            if c < nc // 2:
                local_flips.append(int(np.sum(z != inc)))
            else:
                dens.append(z.mean())
    local_flips = np.array(local_flips)
    assert local_flips.max() <= 3 and np.all(np.isin(np.bincount(local_flips, minlength=4), np.arange(1, 10**6)))
    # random masks: density uniform on [0, 0.6) on average 0.3
    assert abs(np.mean(dens) - 0.3) < 0.02 and max(dens) < 0.75
    # initial design: densities 0.6 i / n, the first mask empty
    init = np.array([mod.initial_mask(3, i, 8, 400).mean() for i in range(8)])
    assert init[0] == 0.0 and np.all(np.abs(init - 0.6 * np.arange(8) / 8) < 0.06)


PLANTED24 = np.zeros(24, np.uint8)
PLANTED24[[1, 4, 6, 9, 13, 14, 17, 18, 20, 22]] = 1


def planted_objective(z, planted=PLANTED24, fac=0.8, K=8):
    """Modeled time per token of self-speculative decoding with K drafts per
    stage: a kept sublayer costs 1/L of a full step; each skipped sublayer
    outside the planted set multiplies the acceptance rate by fac."""
    z = np.asarray(z)
    L = len(planted)
    alpha = 0.97 * fac ** int(np.sum(z & (1 - planted))) * 0.995 ** int(np.sum(z & planted))
    draft = 0.02 + np.sum(z == 0) / L
    return (K * draft + 1.05) / ((1 - alpha ** (K + 1)) / (1 - alpha))


def check_search(mod=O):
    # brute force over all 64 masks of 6 sublayers
    planted6 = np.array([0, 1, 0, 0, 1, 0], np.uint8)
    every = np.array([[(m >> j) & 1 for j in range(6)] for m in range(64)], np.uint8)
    f6 = [planted_objective(z, planted6) for z in every]
    for seed, steps in ((0, 48), (3, 48), (5, 80)):
        r = mod.search(lambda z: planted_objective(z, planted6), 6, n_init=4, iterations=steps, n_candidates=32,
                       seed=seed)
        assert r["best_value"] == min(f6)
        assert np.array_equal(r["best_mask"], every[int(np.argmin(f6))])
        # past the 64 masks, steps evaluate nothing rather than a mask again
        later = [tuple(m) for m in r["masks"][4:]]
        assert len(set(later)) == len(later) and not set(later) & {tuple(m) for m in r["masks"][:4]}
    # the planted 24-sublayer mask, from every seed
    for seed in range(4):
        r = mod.search(planted_objective, 24, n_init=8, iterations=56, n_candidates=64, seed=seed)
        assert np.array_equal(r["best_mask"], PLANTED24), (seed, r["best_mask"])
        masks = [tuple(m) for m in r["masks"][8:]]
        assert len(set(masks)) == len(masks) and not set(masks) & {tuple(m) for m in r["masks"][:8]}
        assert np.all(np.isinf(r["margins"][:8])) and np.all(r["margins"][8:] > 0)
        assert np.allclose(r["values"], [planted_objective(m) for m in r["masks"]], rtol=0, atol=0)
    a = mod.search(planted_objective, 24, n_init=4, iterations=6, seed=11)
    b = mod.search(planted_objective, 24, n_init=4, iterations=6, seed=11)
    c = mod.search(planted_objective, 24, n_init=4, iterations=6, seed=12)
    assert np.array_equal(a["masks"], b["masks"]) and not np.array_equal(a["masks"], c["masks"])


def check_modeled_time(mod=O):
    # drafts accepted in full: K_max = 4, 20 tokens -> 4 stages of 4 drafts
    z = np.array([1, 0, 0, 0, 1, 1], np.uint8)  # kept: attention of layer 1, MLPs of layers 0 and 1
    cost = (0.5, 2.0, 3.0, 10.0, 0.25)
    draft = 0.5 + 1 * 2.0 + 2 * 3.0
    want = (16 * draft + 4 * 10.0 + 20 * 0.25) / 20
    assert math.isclose(mod.modeled_time([(16, 4)], z, cost, 20), want, rel_tol=1e-15)
    # autoregressive stages (no drafts): one verification per token
    assert math.isclose(mod.modeled_time([(0, 20), (0, 20)], z, cost, 20), 10.25, rel_tol=1e-15)


ALL_CHECKS = (check_uniforms, check_standardise, check_posterior, check_kernel, check_expected_improvement,
              check_candidates, check_search, check_modeled_time)


@pytest.mark.parametrize("check", ALL_CHECKS, ids=lambda f: f.__name__)
def test_search_pin(check):
    check()
