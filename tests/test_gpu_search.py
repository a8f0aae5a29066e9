"""GPU: the skip-set search (sd_search_skip_set) with the library's own
self-speculative decoding as its objective.

- Modeled objective: a deterministic function of the decode's stage counts,
  so the search on the GPU must take the oracle's decisions, where the
  oracle's objective decodes with the oracle model.  The comparison runs up
  to the first evaluation at which a decode of the oracle had a token or a
  draft token within tau = 2 tol of a tie (the GPU may take the other token
  there, and the counts may differ) or the oracle's acquisition was within
  rounding of a tie; the cases are chosen so that the whole search compares.
- Measured objective: the GPU time per token; its values are not
  reproducible, so the checks are properties: every value positive and
  finite, distinct masks, the reported best the least value.
"""

import numpy as np
import pytest

import oracle
import sd_synth as S
from oracle import skip_search as O
from paper_2309_08168_amd import binding
from tests import gpu_util as U

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


TIE_MARGIN = 1e-9
TAU = 2 * U.FP32_TOL
# draft base, per attention, per MLP sublayer; verification base, per row
COST = (0.05, 0.1, 0.15, 1.0, 0.02)


def _planted(cfg, mask, rho=0.05, gain=16.0, seed=0):
    w = S.plant_redundancy(cfg, S.make_weights(cfg, seed), S.skip_mask(cfg, mask, seed=11), rho, gain)
    return w, oracle.Model(cfg, w), U.device_model(cfg, w)


# (model, planted mask, prompt seeds, prompt length, new tokens, K_max, gamma, search parameters,
#  whether the search recovers the planted mask)
CASES = [
    ("tiny", "tiny", (0, 1), 12, 24, 4, 0.0, dict(n_init=6, iterations=18, n_candidates=32, seed=1), False),
    ("tiny", "random3", (10, 11, 12), 10, 20, 6, 0.0, dict(n_init=4, iterations=14, n_candidates=16, xi=0.0, seed=2),
     True),
    ("micro_gqa", "random2", (0, 1), 7, 16, 5, 0.0, dict(n_init=3, iterations=12, n_candidates=8, seed=3), False),
]


@pytest.mark.parametrize("name,mask,seeds,t,max_new,k_max,gamma,params,recovers", CASES)
def test_modeled_search_matches_oracle(name, mask, seeds, t, max_new, k_max, gamma, params, recovers):
    cfg = {"tiny": S.MODELS["tiny"], "micro_gqa": U.MICRO_GQA}[name]
    w, om, dm = _planted(cfg, mask)
    prompts = np.stack([S.prompt(cfg, t, seed=s) for s in seeds])
    flagged = []

    def objective(z):
        counts, near = [], np.inf
        for pr in prompts:
            r = om.generate_sd(pr, max_new, z, k_max, gamma)
            near = min(near, r["min_draft_margin"], float(r["margin"].min()), r["min_gamma_gap"] if gamma else np.inf)
            counts.append((r["n_drafted"], r["n_stages"]))
        flagged.append(near < TAU)
        return O.modeled_time(counts, z, COST, max_new)

    ref = O.search(objective, 2 * cfg.n_layers, **{**binding.SEARCH_DEFAULTS, **params})
    got = dm.search_skip_set(prompts, max_new, k_max, gamma=gamma, objective="modeled", cost=COST, **params)
    n = len(ref["values"])
    stop = next((i for i in range(n) if flagged[i] or ref["margins"][i] < TIE_MARGIN), n)
    assert stop == n, f"{name}: oracle near-tie at evaluation {stop} of {n}"
    assert np.array_equal(got["masks"], ref["masks"])
    assert np.array_equal(got["values"], ref["values"])
    assert np.array_equal(got["best_mask"], ref["best_mask"]) and got["best_value"] == ref["best_value"]
    if recovers:
        assert np.array_equal(got["best_mask"], S.skip_mask(cfg, mask, seed=11))
    print(f"{name} planted {mask}: {n} evaluations, best {got['best_value']:.4f} at {got['best_mask'].tolist()}")


def test_measured_search_properties():
    cfg = S.MODELS["tiny"]
    w, om, dm = _planted(cfg, "tiny")
    prompts = np.stack([S.prompt(cfg, 12, seed=s) for s in range(2)])
    dm.generate_sd(prompts[0], 16, None, 4, 0.0)  # first-call set-up outside the search
    got = dm.search_skip_set(prompts, 24, 4, gamma=0.0, objective="measured", n_init=4, iterations=10,
                             n_candidates=16, noise=0.05, seed=4)
    v = got["values"]
    assert len(v) == 14 and np.all(np.isfinite(v)) and np.all(v > 0)
    assert got["best_value"] == v.min() and np.array_equal(got["best_mask"], got["masks"][int(np.argmin(v))])
    assert len({tuple(m) for m in got["masks"]}) == len(v)
    print(f"measured: {v.min():.4f}..{v.max():.4f} ms per token")


def test_adaptive_search_runs():
    cfg = U.MICRO_GQA
    w, om, dm = _planted(cfg, "random2")
    prompts = S.prompt(cfg, 7, seed=1)[None]
    got = dm.search_skip_set(prompts, 12, 4, adaptive={}, objective="modeled", cost=COST, n_init=2, iterations=4,
                             n_candidates=8)
    assert len(got["values"]) == 6 and np.all(np.isfinite(got["values"]))


def test_search_rejects_bad_arguments():
    cfg = U.MICRO_GQA
    w, om, dm = _planted(cfg, "random2")
    pr = S.prompt(cfg, 7)[None]
    with pytest.raises(binding.SDError):
        dm.search_skip_set(pr, 12, 4, gamma=0.0, objective="modeled", cost=(0, 0, float("inf"), 0, 0))
    with pytest.raises(binding.SDError):
        dm.search_skip_set(pr, 0, 4, gamma=0.0)
    with pytest.raises(binding.SDError):
        dm.search_skip_set(pr, 12, 16, gamma=0.0)  # K_max above 15: the decode rejects it
