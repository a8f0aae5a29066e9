"""Pins of the oracle's FP8 draft weights against what fixes them.

- Byte values: every OCP FP8 E4M3 byte decodes to PyTorch's own
  float8_e4m3fn value (NaN for the two NaN bytes).
- Quantizer: the bytes are PyTorch's round-to-nearest-even conversion of
  W * 2^-e, and e is the smallest exponent that keeps the row within 448
  (checked by brute force), on rows with zeros, negative zeros, ties and
  scales from tiny to large.
- Draft forward: with FP8 draft weights set, a forward with the skip mask
  equals a float64 library-built model (PyTorch SDPA) whose kept sublayers
  carry the dequantized weights; the full model still reads the bf16 weights.
- Losslessness: the verification keeps the bf16 weights, so self-speculative
  output with an FP8 draft still equals greedy autoregressive output.
"""

import numpy as np
import pytest

import oracle
import sd_synth as S
from tests import torch_ref

torch = pytest.importorskip("torch")

MICRO_BF16_GQA = S.micro_config(n_layers=2, d_model=64, n_heads=4, n_kv_heads=2, head_dim=16, ffn_dim=96,
                                vocab=97, dtype="bf16", name="micro_bf16_gqa")
KINDS = {"w_qkv": 0, "w_o": 0, "w_gate_up": 1, "w_down": 1}  # 0: attention sublayer, 1: MLP sublayer


def check_byte_values(lib_path=oracle.LIB_PATH):
    ref = torch.arange(256, dtype=torch.uint8).view(torch.float8_e4m3fn).to(torch.float64).numpy()
    got = np.array([oracle.fp8_value(b, lib_path) for b in range(256)])
    nan = np.isnan(ref)
    assert nan.sum() == 2 and np.array_equal(np.isnan(got), nan)
    assert np.array_equal(got[~nan], ref[~nan])


def _test_matrix(rng, n_rows=24, n_cols=40):
    """bf16 rows at many scales, with zeros, negative zeros and exact ties."""
    x = rng.standard_normal((n_rows, n_cols)).astype(np.float32)
    x *= np.float32(2.0) ** rng.integers(-30, 12, size=(n_rows, 1)).astype(np.float32)
    x[0] = 0.0
    x[1, ::3] = -0.0
    # exact halfway points between E4M3 neighbours after scaling: with the row
    # maximum 448 (e = 0), 1.0625 lies between 1.0 and 1.125, 17.0 between 16
    # and 18, and 2^-10 between 0 and 2^-9 (subnormal tie to even)
    x[2, :] = 1.0
    x[2, 0] = 448.0
    x[2, 1:6] = [1.0625, 1.1875, 17.0, 2.0 ** -10, 3.0 * 2.0 ** -10]
    return S.f32_to_bf16_bits(x).reshape(n_rows, n_cols)


def check_quantizer(lib_path=oracle.LIB_PATH):
    rng = np.random.default_rng(5)
    for _ in range(4):
        w = _test_matrix(rng)
        q, e = oracle.quantize_fp8_rows(w, lib_path)
        wf = S.bf16_bits_to_f32(w).reshape(w.shape).astype(np.float64)
        amax = np.abs(wf).max(axis=1)
        for n in range(w.shape[0]):
            if amax[n] == 0:
                assert e[n] == 0
                continue
            # the smallest exponent keeping the row within 448
            assert amax[n] * 2.0 ** -int(e[n]) <= 448.0 < amax[n] * 2.0 ** -(int(e[n]) - 1)
        scaled = torch.from_numpy(np.ldexp(wf, -e[:, None].astype(np.int64)).astype(np.float32))
        ref = scaled.to(torch.float8_e4m3fn).view(torch.uint8).numpy()
        assert np.array_equal(q, ref)
    # the hand-made ties of row 2 land on the even neighbours
    q, e = oracle.quantize_fp8_rows(_test_matrix(np.random.default_rng(0)), lib_path)
    vals = [oracle.fp8_value(b, lib_path) for b in q[2, :6]]
    assert e[2] == 0 and vals == [448.0, 1.0, 1.25, 16.0, 0.0, 2.0 ** -8]


def dequantized_weights(cfg, w, skip, lib_path=oracle.LIB_PATH):
    """float64 weights with every matrix of a kept sublayer replaced by its
    FP8 value * 2^e."""
    w64 = S.weights_as_f64(cfg, w)
    for l in range(cfg.n_layers):
        for name, sub in KINDS.items():
            if skip[2 * l + sub]:
                continue
            q, e = oracle.quantize_fp8_rows(w[f"layers.{l}.{name}"], lib_path)
            vals = np.array([oracle.fp8_value(b, lib_path) for b in range(256)])
            w64[f"layers.{l}.{name}"] = np.ldexp(vals[q], e[:, None].astype(np.int64))
    return w64


def check_draft_forward(lib_path=oracle.LIB_PATH):
    cfg = MICRO_BF16_GQA
    w = S.make_weights(cfg, 3)
    z = S.skip_mask(cfg, "1")  # MLP of layer 0 skipped: both attention sublayers and one MLP run
    toks = S.prompt(cfg, 11, seed=4)
    m = oracle.Model(cfg, w, lib_path=lib_path)
    m.set_draft_fp8(z)
    got = m.score(toks, skip=z)["logits"]
    ref = torch_ref.forward(cfg, dequantized_weights(cfg, w, z, lib_path), toks, skip=z, n_full=0)
    assert np.max(np.abs(got - ref)) <= 1e-10 * np.max(np.abs(ref))
    # the full model keeps the bf16 weights
    full = m.score(toks)["logits"]
    ref_full = torch_ref.forward(cfg, S.weights_as_f64(cfg, w), toks)
    assert np.max(np.abs(full - ref_full)) <= 1e-10 * np.max(np.abs(ref_full))
    # and the draft did change: FP8 is not the bf16 draft
    m.set_draft_fp8(None)
    bf16_draft = m.score(toks, skip=z)["logits"]
    assert np.max(np.abs(bf16_draft - got)) > 1e-4 * np.max(np.abs(got))


def check_lossless(lib_path=oracle.LIB_PATH):
    cfg = MICRO_BF16_GQA
    w = S.plant_redundancy(cfg, S.make_weights(cfg, 4), S.skip_mask(cfg, "2"), 0.2, 8.0)
    m = oracle.Model(cfg, w, lib_path=lib_path)
    pr = S.prompt(cfg, 6, seed=7)
    ar, _ = m.generate_ar(pr, 24)
    for mask, k, g in (("2", 4, 0.0), ("1,2", 6, 0.3), ("none", 3, 0.0)):
        z = S.skip_mask(cfg, mask)
        m.set_draft_fp8(z)
        sd = m.generate_sd(pr, 24, z, k, g)
        assert np.array_equal(sd["tokens"], ar)
        st = sd["stages"]
        assert int(np.sum(st[:, 1] + 1)) == 24
    m.set_draft_fp8(None)


ALL_CHECKS = [check_byte_values, check_quantizer, check_draft_forward, check_lossless]


@pytest.mark.parametrize("check", ALL_CHECKS, ids=lambda f: f.__name__)
def test_fp8_pins(check):
    check()


def test_set_draft_fp8_rejects_float32_models():
    cfg = S.MODELS["tiny"]
    m = oracle.Model(cfg, S.make_weights(cfg, 0))
    with pytest.raises(oracle.OracleError):
        m.set_draft_fp8(S.skip_mask(cfg, "tiny"))
