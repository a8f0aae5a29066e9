"""Decode attention at long contexts and many query vectors per kv head.

One-layer bf16 models whose residual stream the attention output dominates
(H * head_dim = 2048 or 512 against d_model = 256), so the logits follow the
attention closely.  Contexts span several 128-key chunks with a ragged last
chunk, up to 33 chunks (more than the 16 partials the combine takes in one
group); a forward of 1..16 rows gives up to 8 * 16 = 128 query vectors per kv
head (8 tiles of 16 on the matrix-core path); head dims 128, 64 and 32; one
or two query vectors per kv head at head dim 128 (the VALU split kernel).

Tolerance: TIGHT_REL * std(oracle logits of the row), 30x tighter than the
bf16 model tolerance.  With one layer the GPU differs from the oracle only by
float32 rounding and by rare bf16 rounding flips of cached K/V;
test_tight_tolerance_sees_one_key (CPU) shows that hiding a single key from
the rows that should see it moves the logits by more than that.
"""

import numpy as np
import pytest

import oracle
import sd_synth as S
from tests import gpu_util as U
from tests import torch_ref

TIGHT_REL = 1e-3

CONFIGS = {
    "gqa8_dh128": S.ModelConfig("gqa8_dh128", 1, 256, 16, 2, 128, 256, 512, "bf16"),
    "gqa4_dh64": S.ModelConfig("gqa4_dh64", 1, 256, 8, 2, 64, 256, 512, "bf16"),
    "mha_dh32": S.ModelConfig("mha_dh32", 1, 256, 16, 16, 32, 256, 512, "bf16"),
    # one or two query vectors per kv head at head_dim 128 (the draft,
    # autoregressive and one-draft verification steps of the 7B/13B shapes)
    # take the VALU split kernel
    "mha_dh128": S.ModelConfig("mha_dh128", 1, 256, 16, 16, 128, 256, 512, "bf16"),
    "gqa2_dh128": S.ModelConfig("gqa2_dh128", 1, 256, 16, 8, 128, 256, 512, "bf16"),
}
CASES = [(name, pre, rows) for name in CONFIGS for pre, rows in [(300, 1), (300, 3), (300, 16), (700, 9)]]
# past 16 chunks of 128 keys the combine loops over its partials in groups
CASES += [("gqa8_dh128", 2100, 1), ("gqa4_dh64", 2100, 13), ("mha_dh32", 4100, 16)]
# the VALU kernel: one and two rows of multi-head attention, one row of
# grouped heads with two query heads per kv head; ragged last chunks, and
# more than 16 chunks
CASES += [("mha_dh128", 300, 2), ("mha_dh128", 700, 2), ("mha_dh128", 1283, 1), ("mha_dh128", 2300, 2),
          ("gqa2_dh128", 700, 1), ("gqa2_dh128", 2170, 1)]
_models = {}


def _pair(name):
    if name not in _models:
        cfg = CONFIGS[name]
        w = S.make_weights(cfg, 5)
        _models[name] = (cfg, w, oracle.Model(cfg, w), U.device_model(cfg, w))
    return _models[name]


def _tight(ref, got, what):
    tol = TIGHT_REL * ref.std(axis=-1)
    err = np.abs(got.astype(np.float64) - ref).max(axis=-1)
    ratio = float((err / tol).max())
    print(f"{what}: max|d|/tight tol {ratio:.3f}")
    assert np.all(err <= tol), f"{what}: max|d| {err.max():.3g} > {tol.min():.3g}"


@pytest.mark.gpu
@pytest.mark.parametrize("name,pre,rows", CASES)
def test_long_context_logits(name, pre, rows):
    torch = pytest.importorskip("torch")
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cfg, w, om, dm = _pair(name)
    toks = S.prompt(cfg, pre + rows, seed=pre + rows)
    oc = om.cache(pre + rows)
    om.forward(oc, toks[:pre], want_logits=False)
    ref = om.forward(oc, toks[pre:])["logits"]
    gc = dm.cache(pre + rows)
    for i in range(0, pre, 16):  # prefill in 16-row forwards, as the library's callers do
        dm.forward(toks[i:min(pre, i + 16)], gc)
    out = torch.empty((rows, cfg.vocab), dtype=torch.float32, device="cuda")
    dm.forward(toks[pre:], gc, logits=out)
    _tight(ref, out.cpu().numpy(), f"{name} ctx {pre}+{rows}")


def test_tight_tolerance_sees_one_key():
    """Hiding one key (position 150) from every row of a 16-row block after a
    300-token prefix moves the float64 logits of those rows by more than 3x
    the tight tolerance, for each configuration."""
    for name, cfg in CONFIGS.items():
        w64 = S.weights_as_f64(cfg, S.make_weights(cfg, 5))
        toks = S.prompt(cfg, 316, seed=316)
        full = torch_ref.forward(cfg, w64, toks)[300:]
        hidden = torch_ref.forward(cfg, w64, toks, hide_key=150)[300:]
        tol = TIGHT_REL * full.std(axis=-1)
        moved = np.abs(hidden - full).max(axis=-1) / tol
        assert moved.min() > 3.0, f"{name}: hiding a key moves logits by only {moved.min():.2f} tight tolerances"
