"""The library's skip-set search (sd_search_skip_set_fn, host code) against
the oracle's search, decision by decision, on deterministic objectives.

Both draw the same Philox uniforms, so the initial masks and every
candidate list are identical bit for bit; the surrogates and acquisitions
agree to rounding.  A step's choice is therefore the oracle's unless the
oracle reports it within rounding of a tie (its margin below
TIE_MARGIN), after which the histories may part; no such step occurs in
these cases, so the whole trajectories must match.
"""

import math

import numpy as np
import pytest

from oracle import skip_search as O
from paper_2309_08168_amd import binding
from tests.test_oracle_search import PLANTED24, planted_objective

TIE_MARGIN = 1e-9


@pytest.fixture(scope="module", autouse=True)
def _lib():
    binding.load()


def _quadratic(L, seed):
    """A random quadratic pseudo-boolean function (not separable)."""
    rng = np.random.default_rng(seed)
    lin = rng.normal(size=L)
    quad = np.triu(rng.normal(size=(L, L)) * 0.3, 1)
    return lambda z: float(lin @ z + z @ quad @ z)


CASES = [
    # (name, L, objective, params)
    ("planted24", 24, planted_objective, dict(n_init=8, iterations=40, n_candidates=64, seed=1)),
    ("planted24_xi0", 24, planted_objective, dict(n_init=6, iterations=30, n_candidates=16, xi=0.0, seed=2)),
    ("quadratic40", 40, _quadratic(40, 3), dict(n_init=10, iterations=40, n_candidates=48, length_scale=0.4,
                                                noise=1e-2, seed=3)),
    ("quadratic80", 80, _quadratic(80, 4), dict(n_init=8, iterations=24, n_candidates=128, seed=4)),
    ("odd_candidates", 13, _quadratic(13, 5), dict(n_init=3, iterations=30, n_candidates=7, seed=5)),
    ("single_dim", 1, lambda z: float(z[0]), dict(n_init=1, iterations=5, n_candidates=3, seed=6)),
]


@pytest.mark.parametrize("name,L,f,params", CASES, ids=[c[0] for c in CASES])
def test_search_matches_oracle(name, L, f, params):
    prm = {**binding.SEARCH_DEFAULTS, **params}
    ref = O.search(f, L, **prm)
    got = binding.search_skip_set_fn(f, L, **params)
    first_tie = next((i for i, m in enumerate(ref["margins"]) if m < TIE_MARGIN), len(ref["margins"]))
    assert first_tie == len(ref["margins"]), f"oracle near-tie at evaluation {first_tie}"
    assert np.array_equal(got["masks"], ref["masks"])
    assert np.array_equal(got["values"], ref["values"])
    assert np.array_equal(got["best_mask"], ref["best_mask"]) and got["best_value"] == ref["best_value"]
    fin = np.isfinite(ref["margins"])
    assert np.array_equal(np.isfinite(got["margins"]), fin)
    assert np.allclose(got["margins"][fin], ref["margins"][fin], rtol=1e-6, atol=1e-12)
    print(f"{name}: {len(got['values'])} evaluations, best {got['best_value']:.6g}, "
          f"smallest margin {ref['margins'][fin].min() if fin.any() else math.inf:.3g}")


def test_search_recovers_planted_mask():
    got = binding.search_skip_set_fn(planted_objective, 24, n_init=8, iterations=56, n_candidates=64, seed=0)
    assert np.array_equal(got["best_mask"], PLANTED24)


def test_search_stops_evaluating_when_space_is_exhausted():
    # 3 sublayers: 8 masks, far fewer than the steps
    seen = []
    got = binding.search_skip_set_fn(lambda z: seen.append(z.copy()) or float(z.sum()), 3, n_init=2, iterations=40,
                                     n_candidates=16, seed=7)
    tail = [tuple(m) for m in got["masks"][2:]]
    assert len(got["values"]) == len(seen) <= 2 + 8 and len(set(tail)) == len(tail)
    assert got["best_value"] == 0.0


def test_search_rejects_bad_parameters():
    f = lambda z: 0.0  # noqa: E731
    for bad in (dict(n_init=0), dict(iterations=-1), dict(n_candidates=0), dict(length_scale=0.0),
                dict(noise=0.0), dict(xi=math.nan), dict(n_init=4000, iterations=100), dict(n_candidates=70000)):
        with pytest.raises(binding.SDError):
            binding.search_skip_set_fn(f, 8, **bad)
    for L in (0, 1025):
        with pytest.raises(binding.SDError):
            binding.search_skip_set_fn(f, L)


def test_objective_errors_stop_the_search():
    calls = []

    def failing(z):
        calls.append(1)
        if len(calls) == 3:
            raise KeyError("objective broke")
        return 1.0

    with pytest.raises(KeyError):
        binding.search_skip_set_fn(failing, 8, n_init=2, iterations=5)
    assert len(calls) == 3
    with pytest.raises(binding.SDError, match="non-finite"):
        binding.search_skip_set_fn(lambda z: math.inf, 8)
