"""GPU parity of the large-M forward (more than 16 rows on a bfloat16 model:
the prompt prefill, and long sd_forward calls) against the oracle.

- Logits of one long forward from position 0 and after a prefix, on models
  whose shapes leave ragged tails everywhere, and one whose narrow GEMMs
  split their reduction over work-groups: K of 136 and 200 (not a
  multiple of the 32-k stage), output widths of 160 and 400 (not a multiple
  of the 256-row tile), a vocabulary of 777 (odd leading dimension, scalar
  stores), grouped-query attention with head_dim 32, 64 and 128, and row
  counts across several 64- and 128-row tiles with a ragged last tile.
- A forward of 1100 rows runs as two chunks (1024 + 76).
- A masked forward (sublayers bypassed) equals the oracle's.
- Attention-dominated one-layer models at the tight tolerance of the
  attention tests (1e-3 std), prefilled in one forward.
- Decoding after a long prompt equals the oracle's tokens.
"""

import numpy as np
import pytest

import oracle
import sd_synth as S
from tests import gpu_util as U
from tests import test_gpu_attention as A

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


ODD_BF16 = S.ModelConfig("odd_bf16", 2, 136, 3, 1, 32, 200, 777, "bf16")
# wide enough that the residual-update GEMMs split their reduction (2 ways
# for the output projection, 4 for the down projection)
WIDE_BF16 = S.ModelConfig("wide_bf16", 1, 1024, 8, 8, 128, 2048, 512, "bf16")
# two layers whose output and down projections split their reduction (2
# and 4 ways): each split's partials are added into the residual stream by
# the norm that follows, whichever sublayer that is
WIDE2_BF16 = S.ModelConfig("wide2_bf16", 2, 1024, 8, 8, 128, 2048, 512, "bf16")
# a gate/up GEMM wide enough (14400 columns: 57 tiles of 256, the last one
# 64 wide) that forwards of 513 rows or more take the direct-to-LDS kernel
FFN_WIDE_BF16 = S.ModelConfig("ffn_wide_bf16", 1, 256, 4, 4, 64, 7200, 512, "bf16")
MODELS = {"mini_bf16": U.MINI_BF16, "odd_bf16": ODD_BF16, "gqa8_dh128": A.CONFIGS["gqa8_dh128"],
          "wide_bf16": WIDE_BF16}
# output and down projections of 10 column tiles of 256: at 1000 rows (4 row
# tiles) they split their reduction 4 ways on the 256 x 256 kernel (160
# work-groups)
D2560_BF16 = S.ModelConfig("d2560_bf16", 1, 2560, 20, 20, 128, 2048, 512, "bf16")
EXTRA = {"ffn_wide_bf16": FFN_WIDE_BF16, "wide2_bf16": WIDE2_BF16, "d2560_bf16": D2560_BF16}
_models = {}


def _pair(name, seed=0):
    if (name, seed) not in _models:
        cfg = MODELS[name] if name in MODELS else EXTRA[name]
        w = S.make_weights(cfg, seed)
        _models[(name, seed)] = (cfg, w, oracle.Model(cfg, w), U.device_model(cfg, w))
    return _models[(name, seed)]


def _logits(dm, toks, cache, skip=None):
    out = torch.empty((len(toks), dm.cfg.vocab), dtype=torch.float32, device="cuda")
    dm.forward(toks, cache, skip=skip, logits=out)
    return out.cpu().numpy()


@pytest.mark.parametrize("name", list(MODELS))
@pytest.mark.parametrize("rows", [17, 130, 300])
def test_long_forward_from_zero(name, rows):
    cfg, w, om, dm = _pair(name)
    toks = S.prompt(cfg, rows, seed=rows)
    ref = om.score(toks)["logits"]
    got = _logits(dm, toks, dm.cache(rows))
    r = U.check_logits(cfg, got, ref, f"{name} {rows} rows")
    print(f"{name} {rows} rows from 0: max |d| / tol {r:.3f}")


@pytest.mark.parametrize("rows", [600, 1000, 1024])
def test_forward_on_the_wide_gemm(rows):
    """gate/up of 3 or 4 x 57 tiles of 256 x 256 (a ragged last row tile at
    600 and 1000 rows, a 64-column last column tile): the direct-to-LDS GEMM."""
    cfg, w, om, dm = _pair("ffn_wide_bf16")
    toks = S.prompt(cfg, rows, seed=rows + 5)
    ref = om.score(toks)["logits"]
    got = _logits(dm, toks, dm.cache(rows))
    r = U.check_logits(cfg, got, ref, f"ffn_wide_bf16 {rows} rows")
    print(f"ffn_wide_bf16 {rows} rows from 0: max |d| / tol {r:.3f}")


@pytest.mark.parametrize("rows", [600, 1000])
def test_wide_gemm_forward_is_deterministic(rows):
    """Three forwards on the SwiGLU-fused gate/up GEMM (224- and 256-wide
    tiles) give bit-identical logits: no work-group writes its output where
    another still reads its input."""
    cfg, w, om, dm = _pair("ffn_wide_bf16")
    toks = S.prompt(cfg, rows, seed=rows + 13)
    first = _logits(dm, toks, dm.cache(rows))
    for _ in range(2):
        assert np.array_equal(_logits(dm, toks, dm.cache(rows)), first)


@pytest.mark.parametrize("name", ["mini_bf16", "odd_bf16"])
def test_long_forward_after_prefix(name):
    cfg, w, om, dm = _pair(name)
    toks = S.prompt(cfg, 90 + 75, seed=3)
    oc = om.cache(165)
    om.forward(oc, toks[:90], want_logits=False)
    ref = om.forward(oc, toks[90:])["logits"]
    gc = dm.cache(165)
    dm.forward(toks[:90], gc)
    got = _logits(dm, toks[90:], gc)
    assert gc.length == 165
    r = U.check_logits(cfg, got, ref, f"{name} 90 + 75 rows")
    print(f"{name} 75 rows after 90: max |d| / tol {r:.3f}")


def test_forward_of_two_chunks():
    cfg, w, om, dm = _pair("mini_bf16")
    toks = S.prompt(cfg, 1100, seed=11)
    ref = om.score(toks)["logits"]
    got = _logits(dm, toks, dm.cache(1100))
    r = U.check_logits(cfg, got, ref, "1100 rows")
    print(f"mini_bf16 1100 rows (two chunks): max |d| / tol {r:.3f}")


@pytest.mark.parametrize("mask", ["none", "1", "2", "3"])
def test_split_partials_fold_into_the_next_norm(mask):
    """Split output and down projections on a two-layer model: unmasked the
    partials go into the next MLP or attention norm and the final norm; with
    layer 0's MLP skipped (1) the output projection's go into layer 1's
    attention norm, with layer 1's attention skipped (2) the down
    projection's into layer 1's MLP norm, with layer 1's MLP skipped (3)
    into the final norm."""
    cfg, w, om, dm = _pair("wide2_bf16")
    z = S.skip_mask(cfg, mask, seed=0)
    toks = S.prompt(cfg, 300, seed=31)
    ref = om.forward(om.cache(300), toks, skip=z)["logits"]
    got = _logits(dm, toks, dm.cache(300), skip=z)
    r = U.check_logits(cfg, got, ref, f"wide2_bf16 mask {mask} 300 rows")
    print(f"wide2_bf16 mask {mask}: max |d| / tol {r:.3f}")


def test_split_reduction_on_the_wide_gemm():
    """The output and down projections of a d 2560 model over 1000 rows: 40
    tiles of 256 x 256, each reduction split 4 ways, the partials folded
    into the MLP norm and the final norm."""
    cfg, w, om, dm = _pair("d2560_bf16")
    toks = S.prompt(cfg, 1000, seed=41)
    ref = om.score(toks)["logits"]
    got = _logits(dm, toks, dm.cache(1000))
    r = U.check_logits(cfg, got, ref, "d2560_bf16 1000 rows")
    print(f"d2560_bf16 1000 rows: max |d| / tol {r:.3f}")


def test_generate_after_a_split_prefill():
    """The prompt prefill of a model with split residual updates and no
    logits: the last down projection's partials are added by a plain sum, and
    layer 1's keys and values depend on every fold before them."""
    cfg, w, om, dm = _pair("wide2_bf16")
    pr = S.prompt(cfg, 200, seed=23)
    z = S.skip_mask(cfg, "1", seed=0)
    ar_ref, ar_margin = om.generate_ar(pr, 16)
    sd_ref = om.generate_sd(pr, 16, z, 4, 0.0)
    ar, _ = dm.generate_ar(pr, 16)
    sd, _ = dm.generate_sd(pr, 16, z, 4, 0.0)
    std = om.score(np.concatenate([pr, ar_ref])[:-1])["logits"][len(pr) - 1:].std(axis=1)
    n_ar = U.check_free_running(cfg, ar, ar_ref, ar_margin, std, "wide2_bf16 AR after 200")
    n_sd = U.check_free_running(cfg, sd, sd_ref["tokens"], sd_ref["margin"], std, "wide2_bf16 SD after 200")
    U.check_tokens_teacher_forced(cfg, om, pr, sd, "wide2_bf16 SD after 200 teacher-forced")
    U.check_tokens_teacher_forced(cfg, om, pr, ar, "wide2_bf16 AR after 200 teacher-forced")
    print(f"wide2_bf16: AR equal for {n_ar}/16, SD for {n_sd}/16 after a 200-token prompt")


@pytest.mark.parametrize("name", ["mini_bf16", "odd_bf16"])
def test_long_masked_forward(name):
    cfg, w, om, dm = _pair(name)
    z = S.skip_mask(cfg, "random2", seed=3)
    toks = S.prompt(cfg, 20 + 40, seed=8)
    oc = om.cache(60)
    om.forward(oc, toks[:20], want_logits=False)
    ref = om.forward(oc, toks[20:], skip=z)["logits"]
    gc = dm.cache(60)
    dm.forward(toks[:20], gc)
    got = _logits(dm, toks[20:], gc, skip=z)
    U.check_logits(cfg, got, ref, f"{name} masked 40 rows")


@pytest.mark.parametrize("name", list(A.CONFIGS))
@pytest.mark.parametrize("pre,rows", [(300, 16), (700, 9)])
def test_attention_after_one_forward_prefill(name, pre, rows):
    """The attention tests' cases with the prefix written by one long forward."""
    cfg, w, om, dm = A._pair(name)
    toks = S.prompt(cfg, pre + rows, seed=pre + rows)
    oc = om.cache(pre + rows)
    om.forward(oc, toks[:pre], want_logits=False)
    ref_pre = om.forward(oc, toks[pre:])["logits"]
    gc = dm.cache(pre + rows)
    dm.forward(toks[:pre], gc)
    got = _logits(dm, toks[pre:], gc)
    A._tight(ref_pre, got, f"{name} one-forward prefill {pre}+{rows}")
    # and the long forward's own logits over the whole sequence
    ref_all = om.score(toks)["logits"]
    got_all = _logits(dm, toks, dm.cache(pre + rows))
    A._tight(ref_all, got_all, f"{name} {pre + rows} rows in one forward")


@pytest.mark.parametrize("name,mask,k_max,gamma", [("mini_bf16", "random2", 8, 0.0), ("odd_bf16", "0,3", 4, 0.002)])
def test_generate_after_long_prompt(name, mask, k_max, gamma):
    cfg, w, om, dm = _pair(name)
    pr = S.prompt(cfg, 200, seed=21)
    z = S.skip_mask(cfg, mask, seed=11)
    ar_ref, ar_margin = om.generate_ar(pr, 32)
    sd_ref = om.generate_sd(pr, 32, z, k_max, gamma)
    ar, _ = dm.generate_ar(pr, 32)
    sd, st = dm.generate_sd(pr, 32, z, k_max, gamma)
    std = om.score(np.concatenate([pr, ar_ref])[:-1])["logits"][len(pr) - 1:].std(axis=1)
    n_ar = U.check_free_running(cfg, ar, ar_ref, ar_margin, std, f"{name} AR after 200")
    n_sd = U.check_free_running(cfg, sd, sd_ref["tokens"], sd_ref["margin"], std, f"{name} SD after 200")
    assert st["prefill_ms"] > 0
    U.check_tokens_teacher_forced(cfg, om, pr, sd, f"{name} SD after 200 teacher-forced")
    print(f"{name}: AR equal for {n_ar}/32, SD for {n_sd}/32 after a 200-token prompt")
