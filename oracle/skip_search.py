"""Skip-set search (Sec. 3.3, Eq. 1), plain numpy.

TEST INFRASTRUCTURE ONLY: the test suite and the benchmark's CPU baseline
may import this module; the product library never does.

z* = argmin_z f(z) over z in {0, 1}^L, L the number of sublayers, f(z) the
average time per emitted token of self-speculative decoding with the
sublayers of z bypassed in the draft.  The paper solves it with Bayesian
optimisation: a Gaussian-process surrogate of f and an acquisition that
trades exploration against exploitation pick the next z to evaluate, for a
fixed number of iterations.  It fixes nothing else; this module is one
definite reading of every other detail, step by step:

- z has one bit per sublayer, entry 2l the attention and 2l+1 the MLP of
  layer l (L = 2 n_layers, the count the paper gives for LLaMA-2-70B);
- initial design: n_init masks, mask i with each bit set with probability
  0.6 i / n_init, so mask 0 is empty (the full model as its own draft);
- surrogate: the observations are standardised (mean 0, population
  standard deviation 1; a deviation below 1e-12 counts as 1); a zero-mean GP
  with kernel k(a, b) = exp(-hamming(a, b) / (length_scale L)) and
  observation noise variance `noise` gives the posterior mean and standard
  deviation of the noise-free value;
- acquisition: expected improvement below the smallest standardised
  observation by a margin xi,
  EI = (best - mu - xi) Phi(u) + sigma phi(u), u = (best - mu - xi) / sigma
  (max(best - mu - xi, 0) when sigma = 0);
- each step scores n_candidates masks: the first n_candidates // 2 flip
  1 to 3 uniformly chosen bits of the incumbent (the best observation so
  far, first on ties), the rest set each bit with one probability drawn
  uniformly from [0, 0.6); masks evaluated before are dropped, the first
  maximiser of EI is evaluated next, and a step with no new candidate
  evaluates nothing;
- every random number is the top 24 bits of the first word of
  Philox4x64-10 with key (seed, 1) and counter (a, purpose, c, 0).

Parity of a search against this one is decision by decision: each step
also reports the margin between the chosen candidate's EI and the largest
EI strictly below it, and a decision whose margin is within rounding is
a near-tie that another implementation may take the other way.
"""

from __future__ import annotations

import math
from typing import Callable, List, Sequence

import numpy as np

from . import philox4x64

# Purposes of the search's uniforms (the second counter word).
P_INIT, P_NFLIP, P_FLIP, P_DENSITY, P_BIT = 100, 101, 102, 103, 104


def search_uniform(seed: int, a: int, purpose: int, c: int) -> float:
    w = philox4x64([a, purpose, c, 0], [seed, 1])
    return int(w[0]) // 2**40 / 2.0**24


def initial_mask(seed: int, i: int, n_init: int, L: int) -> np.ndarray:
    p = 0.6 * i / n_init
    return np.array([search_uniform(seed, i, P_INIT, j) < p for j in range(L)], np.uint8)


def candidate(seed: int, t: int, c: int, n_candidates: int, L: int, incumbent: np.ndarray) -> np.ndarray:
    if c < n_candidates // 2:
        z = incumbent.copy()
        flips = 1 + int(search_uniform(seed, t, P_NFLIP, c) * 3.0)
        for r in range(flips):
            j = int(search_uniform(seed, t, P_FLIP, c * 8 + r) * L)
            z[j] ^= 1
        return z
    p = 0.6 * search_uniform(seed, t, P_DENSITY, c)
    return np.array([search_uniform(seed, t, P_BIT, c * L + j) < p for j in range(L)], np.uint8)


def standardise(y: Sequence[float]) -> np.ndarray:
    y = np.asarray(y, np.float64)
    sd = float(np.sqrt(np.mean((y - y.mean()) ** 2)))
    return (y - y.mean()) / (sd if sd > 1e-12 else 1.0)


def kernel(A: np.ndarray, B: np.ndarray, length_scale: float) -> np.ndarray:
    """exp(-hamming / (length_scale L)) between the rows of A and of B."""
    A = np.atleast_2d(A).astype(np.int64)
    B = np.atleast_2d(B).astype(np.int64)
    hamming = np.abs(A[:, None, :] - B[None, :, :]).sum(-1)
    return np.exp(-hamming / (length_scale * A.shape[1]))


def posterior(X: np.ndarray, ys: np.ndarray, Z: np.ndarray, length_scale: float, noise: float):
    """GP posterior mean and standard deviation of the noise-free values at
    the rows of Z, given standardised observations ys at the rows of X.

    One row of Z at a time: two masks at the same distances from every
    observation then get the same values to the last bit, so such ties go
    to the first of them (batched products may round rows differently)."""
    K = kernel(X, X, length_scale) + noise * np.eye(len(X))
    alpha = np.linalg.solve(K, ys)
    mu = np.empty(len(Z))
    var = np.empty(len(Z))
    for i, z in enumerate(np.atleast_2d(Z)):
        k = kernel(z, X, length_scale)[0]
        mu[i] = k @ alpha
        var[i] = 1.0 - k @ np.linalg.solve(K, k)
    return mu, np.sqrt(np.maximum(var, 0.0))


def expected_improvement(mu: float, sigma: float, best: float, xi: float) -> float:
    imp = best - mu - xi
    if not sigma > 0.0:
        return max(imp, 0.0)
    u = imp / sigma
    cdf = 0.5 * math.erfc(-u / math.sqrt(2.0))
    pdf = math.exp(-0.5 * u * u) / math.sqrt(2.0 * math.pi)
    return imp * cdf + sigma * pdf


def search(objective: Callable[[np.ndarray], float], L: int, n_init: int = 8, iterations: int = 32,
           n_candidates: int = 64, length_scale: float = 0.25, noise: float = 1e-3, xi: float = 0.01,
           seed: int = 0) -> dict:
    """Bayesian optimisation of objective over {0, 1}^L.

    Returns the evaluated masks and values in order, the margin of each
    decision (inf for the initial design), and the best mask and value (the
    first minimum)."""
    X: List[np.ndarray] = []
    y: List[float] = []
    margins: List[float] = []
    for i in range(n_init):
        z = initial_mask(seed, i, n_init, L)
        X.append(z)
        y.append(float(objective(z)))
        margins.append(math.inf)
    for t in range(iterations):
        ys = standardise(y)
        incumbent = X[int(np.argmin(y))]
        cands = [candidate(seed, t, c, n_candidates, L, incumbent) for c in range(n_candidates)]
        fresh = [z for z in cands if not any(np.array_equal(z, x) for x in X)]
        if not fresh:
            continue
        mu, sigma = posterior(np.array(X), ys, np.array(fresh), length_scale, noise)
        best = float(ys.min())
        ei = np.array([expected_improvement(float(m), float(s), best, xi) for m, s in zip(mu, sigma)])
        pick = int(np.argmax(ei))
        below = ei[ei < ei[pick]]
        X.append(fresh[pick])
        y.append(float(objective(fresh[pick])))
        margins.append(float(ei[pick] - below.max()) if below.size else math.inf)
    b = int(np.argmin(y))
    return {"masks": np.array(X), "values": np.array(y), "margins": np.array(margins), "best_mask": X[b],
            "best_value": y[b]}


def modeled_time(counts, mask: np.ndarray, cost: Sequence[float], max_new: int) -> float:
    """Modeled time per emitted token of the decodes of several prompts,
    each (drafted tokens, stages): a draft step costs cost[0] plus cost[1]
    per attention and cost[2] per MLP sublayer it runs, a verification
    cost[3] plus cost[4] per row (drafts + 1)."""
    mask = np.asarray(mask)
    att = int(np.sum(mask[0::2] == 0))
    mlp = int(np.sum(mask[1::2] == 0))
    draft = cost[0] + cost[1] * att + cost[2] * mlp
    total = 0.0
    for drafted, stages in counts:
        total += drafted * draft + stages * cost[3] + cost[4] * (drafted + stages)
    return total / (len(counts) * max_new)
