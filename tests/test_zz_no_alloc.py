"""The allocation-free forward (sd_forward_static) against sd_forward.

Two caches receive the same prefix through sd_forward; then each takes the
same forwards, one through sd_forward and the other through
sd_forward_static, and the logits must be identical (same kernels, same
order of every reduction), which is stricter than the oracle tolerance.
Two calls in a row, the second with fewer rows, on the matrix-core (13
rows), two-row and one-row paths of a bf16 model and the float32 VALU path
of the tiny model; a masked draft row; then the refusals (more than 16 rows,
a full cache).  The static scratch keeps the previous call's contents, so
the second, smaller call also checks that nothing stale leaks into it.
"""

import numpy as np
import pytest

import sd_synth as S
from tests import gpu_util as U

torch = pytest.importorskip("torch")

pytestmark = pytest.mark.gpu

CASES = {
    "mini_bf16": (U.MINI_BF16, 3, [13, 2, 1]),
    "tiny": (S.MODELS["tiny"], 0, [5, 1]),
}


def _logits(cfg, rows):
    return torch.full((rows, cfg.vocab), float("nan"), dtype=torch.float32, device="cuda")


@pytest.mark.parametrize("name", sorted(CASES))
def test_static_forward_equals_forward(name):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2309_08168_amd import binding

    cfg, seed, row_list = CASES[name]
    w = S.make_weights(cfg, seed)
    model = U.device_model(cfg, w)
    toks = S.prompt(cfg, 64, seed=17)
    pre = 20
    ca, cb = model.cache(64), model.cache(64)
    model.forward(toks[:pre], ca)
    model.forward(toks[:pre], cb)
    pos = pre
    for rows in row_list:
        ref = _logits(cfg, rows)
        got = _logits(cfg, rows)
        model.forward(toks[pos:pos + rows], ca, logits=ref)
        model.forward_static(toks[pos:pos + rows], cb, logits=got)
        assert ca.length == cb.length == pos + rows
        r, g = ref.cpu().numpy(), got.cpu().numpy()
        assert np.isfinite(r).all()
        assert np.array_equal(r, g), f"{name} {rows} rows: max |d| {np.abs(r - g).max()}"
        pos += rows
    # a draft row with the workload-style mask, after the rows above
    z = S.skip_mask(cfg, "random2" if cfg.n_layers == 2 else "tiny", 0)
    ref, got = _logits(cfg, 1), _logits(cfg, 1)
    model.forward(toks[pos:pos + 1], ca, skip=z, logits=ref)
    model.forward_static(toks[pos:pos + 1], cb, skip=z, logits=got)
    assert np.array_equal(ref.cpu().numpy(), got.cpu().numpy())
    # refusals leave the cache untouched
    n0 = cb.length
    with pytest.raises(binding.SDError) as e:
        model.forward_static(toks[:17], cb)
    assert e.value.status == binding.SD_ERR_INVALID_ARG and cb.length == n0
    full = model.cache(4)
    model.forward_static(toks[:3], full)
    with pytest.raises(binding.SDError) as e:
        model.forward_static(toks[:2], full)
    assert e.value.status == binding.SD_ERR_CAPACITY and full.length == 3
    model.close()
