"""GPU parity of the FP8 draft weights (sd_model_quantize_draft) against the
oracle (orc_set_draft_fp8).

- Quantization is integer-valued work: every byte and row exponent the
  library makes equals the oracle's, bit for bit, including rows with
  zeros, negative zeros, exact ties and extreme scales.
- Draft rows: one-row forwards with the skip mask read the FP8 copies; their
  logits match the oracle's FP8 draft within the bf16 tolerance, after a
  prefix the full (bf16) model wrote.  They differ from the bf16 draft by far
  more, so the test sees which weights were read.
- Generation: self-speculative decoding with the FP8 draft emits the
  oracle's tokens (which, verification being bf16, are greedy bf16
  decoding), and the same stage trace where the oracle reports no draft
  decision within tau.
- A two-layer model of the 13B widths (d 5120, 40 heads, FFN 13824,
  vocabulary 32000) checks the kernel shapes of the benchmark.
"""

import numpy as np
import pytest

import oracle
import sd_synth as S
from paper_2309_08168_amd import binding
from tests import gpu_util as U

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


KIND_NAMES = ["w_qkv", "w_o", "w_gate_up", "w_down"]


def _special_weights(cfg, seed):
    """Weights whose layer-0 output projection has rows of zeros, negative
    zeros, exact E4M3 ties and scales from 2^-30 to 2^10."""
    w = S.make_weights(cfg, seed)
    wo = S.bf16_bits_to_f32(w["layers.0.w_o"]).reshape(w["layers.0.w_o"].shape).copy()
    rng = np.random.default_rng(seed)
    wo[0] = 0.0
    wo[1, ::2] = -0.0
    wo[2, :] = 1.0
    wo[2, :6] = [448.0, 1.0625, 1.1875, 17.0, 2.0 ** -10, 3.0 * 2.0 ** -10]
    for r in range(3, 12):
        wo[r] *= np.float32(2.0) ** (10 * (r - 7))
    wo[12:20] = rng.standard_normal((8, wo.shape[1])).astype(np.float32)
    w = dict(w)
    w["layers.0.w_o"] = S.f32_to_bf16_bits(wo).reshape(wo.shape)
    w["layers.1.w_down"] = S.scale_tensor(w["layers.1.w_down"], 2.0 ** -24, "bf16")
    return w


_models = {}


def _pair(name):
    if name not in _models:
        if name == "special":
            cfg = U.MINI_BF16
            w = _special_weights(cfg, 3)
        elif name == "planted":
            cfg = U.MINI_BF16
            w = S.plant_redundancy(cfg, S.make_weights(cfg, 0), S.skip_mask(cfg, "random2", seed=11), 0.3, 12.0)
        else:
            cfg = S.ModelConfig("wide13_2l", 2, 5120, 40, 40, 128, 13824, 32000, "bf16")
            w = S.make_weights(cfg, 6)
        _models[name] = (cfg, w, oracle.Model(cfg, w), U.device_model(cfg, w))
    return _models[name]


@pytest.mark.parametrize("name,mask", [("special", "none"), ("planted", "random2")])
def test_quantized_bytes_match_oracle(name, mask):
    cfg, w, om, dm = _pair(name)
    z = S.skip_mask(cfg, mask, seed=11)
    dm.quantize_draft(z)
    n = 0
    for l in range(cfg.n_layers):
        for kind, kname in enumerate(KIND_NAMES):
            got = dm.draft_fp8(l, kind)
            if z[2 * l + (0 if kind < 2 else 1)]:
                assert got is None
                continue
            q, e = oracle.quantize_fp8_rows(w[f"layers.{l}.{kname}"])
            assert np.array_equal(got[1], e), (l, kname)
            assert np.array_equal(got[0], q), (l, kname, int(np.sum(got[0] != q)))
            n += 1
    assert n > 0
    dm.quantize_draft(None)
    assert dm.draft_fp8(0, 1) is None


def _draft_rows(cfg, om, dm, z, toks, pre, n, fp8):
    """Logits of n one-row draft forwards after a full-model prefix, GPU and oracle."""
    om.set_draft_fp8(z if fp8 else None)
    dm.quantize_draft(z if fp8 else None)
    oc, gc = om.cache(pre + n), dm.cache(pre + n)
    om.forward(oc, toks[:pre], want_logits=False)
    dm.forward(toks[:pre], gc)
    ref, got = [], []
    for i in range(pre, pre + n):
        ref.append(om.forward(oc, toks[i:i + 1], skip=z)["logits"][0])
        g = torch.empty((1, cfg.vocab), dtype=torch.float32, device="cuda")
        dm.forward(toks[i:i + 1], gc, skip=z, logits=g)
        got.append(g.cpu().numpy()[0])
    return np.array(got), np.array(ref)


@pytest.mark.parametrize("name,mask", [("planted", "random2"), ("special", "1")])
def test_fp8_draft_logits_match_oracle(name, mask):
    cfg, w, om, dm = _pair(name)
    z = S.skip_mask(cfg, mask, seed=11)
    toks = S.prompt(cfg, 24, seed=9)
    got, ref = _draft_rows(cfg, om, dm, z, toks, 16, 6, fp8=True)
    r = U.check_logits(cfg, got, ref, f"{name} FP8 draft rows")
    if name == "planted":
        # the bf16 draft is another model: far outside the tolerance of this
        # one (the special model's huge rows dominate its logit spread)
        _, ref_bf16 = _draft_rows(cfg, om, dm, z, toks, 16, 6, fp8=False)
        tol = U.row_tol(cfg, ref)
        assert np.max(np.abs(ref_bf16 - ref).max(axis=-1) / tol) > 3.0
    print(f"{name}: FP8 draft rows max |d|/tol {r:.3f}")


def test_fp8_draft_refuses_masked_multirow_forward():
    cfg, w, om, dm = _pair("planted")
    z = S.skip_mask(cfg, "random2", seed=11)
    dm.quantize_draft(z)
    c = dm.cache(8)
    with pytest.raises(binding.SDError) as e:
        dm.forward(S.prompt(cfg, 2, seed=1), c, skip=z)
    assert e.value.status == binding.SD_ERR_INVALID_ARG and c.length == 0
    dm.forward(S.prompt(cfg, 2, seed=1), c)  # the full model takes any row count
    dm.quantize_draft(None)


@pytest.mark.parametrize("k_max,gamma", [(4, 0.6), (8, 0.0), (6, 0.3)])
def test_fp8_draft_generate_matches_oracle(k_max, gamma):
    cfg, w, om, dm = _pair("planted")
    z = S.skip_mask(cfg, "random2", seed=11)
    om.set_draft_fp8(z)
    dm.quantize_draft(z)
    pr = S.prompt(cfg, 12, seed=13)
    n = 48
    ref = om.generate_sd(pr, n, z, k_max, gamma)
    ar, ar_margin = om.generate_ar(pr, n)
    sd, st = dm.generate_sd(pr, n, z, k_max, gamma)
    # verification is bf16: the oracle's FP8-draft output is its greedy output
    assert np.array_equal(ref["tokens"], ar)
    # near-ties of the emitted tokens from the oracle's own rows (tau = 2 tol per row)
    lg = om.score(np.concatenate([pr, ar])[:-1])["logits"][len(pr) - 1:]
    tau = 2 * U.row_tol(cfg, lg)
    flagged = np.nonzero(ar_margin < tau)[0]
    first = int(flagged[0]) if flagged.size else n
    assert np.array_equal(sd[:first], ar[:first]), (sd.tolist(), ar.tolist())
    stg = st["stages"]
    assert int(np.sum(stg[:, 1] + 1)) == n and np.all(stg[:, 1] <= stg[:, 0])
    # stage traces when no emitted token and no draft decision is near a tie
    # (draft rows: the largest full-row tau, doubled, bounds theirs)
    if first == n and ref["min_draft_margin"] > 2 * tau.max() and ref["min_gamma_gap"] > 2 * U.BF16_REL_TOL:
        assert np.array_equal(stg, ref["stages"])
    print(f"K={k_max} gamma={gamma}: tokens equal {first}/{n}; acceptance {st['n_accepted']}/{st['n_drafted']} "
          f"(oracle {ref['n_accepted']}/{ref['n_drafted']})")
    dm.quantize_draft(None)


@pytest.mark.big
def test_fp8_draft_at_13b_widths():
    cfg, w, om, dm = _pair("wide13")
    z = S.skip_mask(cfg, "3")  # the MLP of layer 1 skipped
    dm.quantize_draft(z)
    for l, kind in ((0, 0), (0, 2), (1, 1)):
        q, e = oracle.quantize_fp8_rows(w[f"layers.{l}.{KIND_NAMES[kind]}"])
        got = dm.draft_fp8(l, kind)
        assert np.array_equal(got[1], e) and np.array_equal(got[0], q)
    toks = S.prompt(cfg, 10, seed=2)
    got, ref = _draft_rows(cfg, om, dm, z, toks, 8, 2, fp8=True)
    r = U.check_logits(cfg, got, ref, "13B widths FP8 draft rows")
    print(f"13B widths: FP8 draft rows max |d|/tol {r:.3f}")
    dm.quantize_draft(None)
    _models.pop("wide13")
