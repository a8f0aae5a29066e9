"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test names the property it pins.  A plausible mistake in the oracle
(a dropped residual, a wrong RoPE pairing or sign, a transposed q/k/v or
gate/up block, an off-by-one causal window, a wrong GQA head map, a wrong
acceptance count or rollback length) fails at least one of them.
"""

import numpy as np
import pytest

import oracle
import sd_synth as S
from tests import torch_ref

MICRO_GQA = S.micro_config()  # 2 layers, d 64, 4 q heads / 2 kv heads x 16, ffn 96, vocab 97
MICRO_BF16 = S.micro_config(n_layers=3, d_model=48, n_heads=2, n_kv_heads=1, head_dim=24, ffn_dim=80,
                            vocab=61, dtype="bf16", name="micro_bf16")


def _model(cfg, seed=0, weights=None):
    w = S.make_weights(cfg, seed) if weights is None else weights
    return oracle.Model(cfg, w), w


def _rel(a, b):
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


# --------------------------------------------------------------------------
# forward: library-built float64 model (F.rms_norm, SDPA, complex RoPE, silu)


@pytest.mark.parametrize("cfg", [MICRO_GQA, MICRO_BF16, S.MODELS["tiny"]], ids=lambda c: c.name)
def test_forward_matches_library_built_model(cfg):
    m, w = _model(cfg)
    toks = S.prompt(cfg, 19, seed=3)
    got = m.score(toks)["logits"]
    ref = torch_ref.forward(cfg, S.weights_as_f64(cfg, w), toks)
    assert _rel(got, ref) < 1e-10


@pytest.mark.parametrize("cfg", [MICRO_GQA, MICRO_BF16, S.MODELS["tiny"]], ids=lambda c: c.name)
def test_skipped_forward_matches_library_built_model(cfg):
    m, w = _model(cfg, seed=1)
    z = S.skip_mask(cfg, "random3", seed=5)
    toks = S.prompt(cfg, 13, seed=4)
    got = m.score(toks, skip=z)["logits"]
    ref = torch_ref.forward(cfg, S.weights_as_f64(cfg, w), toks, skip=z, n_full=0)
    assert _rel(got, ref) < 1e-10


def test_draft_rows_over_full_prefix_match_library_built_model():
    """Shared-cache reading: draft rows attend to K/V that the full model wrote."""
    cfg = MICRO_GQA
    m, w = _model(cfg, seed=2)
    z = S.skip_mask(cfg, "0,3")  # attention of layer 0, MLP of layer 1
    toks = S.prompt(cfg, 12, seed=6)
    c = m.cache(16)
    m.forward(c, toks[:9])
    got = np.concatenate([m.forward(c, toks[9:10], skip=z)["logits"], m.forward(c, toks[10:], skip=z)["logits"]])
    ref = torch_ref.forward(cfg, S.weights_as_f64(cfg, w), toks, skip=z, n_full=9)[9:]
    assert _rel(got, ref) < 1e-10


# --------------------------------------------------------------------------
# closed forms and textbook special cases


def _rmsnorm(x, g, eps):
    return g * x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)


def test_all_sublayers_skipped_is_bigram_table():
    """z = all ones: the draft is W_lm * RMSNorm(E[x]) and writes no KV."""
    cfg = S.MODELS["tiny"]
    m, w = _model(cfg)
    z = S.skip_mask(cfg, "all")
    toks = S.prompt(cfg, 7, seed=9)
    got = m.score(toks, skip=z)["logits"]
    ref = _rmsnorm(w["tok_emb"][toks].astype(np.float64), w["final_norm"].astype(np.float64), cfg.rms_eps) @ \
        w["lm_head"].astype(np.float64).T
    assert _rel(got, ref) < 1e-12


def test_position_zero_attention_returns_v0():
    """At position 0 the softmax has one key (weight 1) and RoPE is the identity."""
    cfg = MICRO_GQA
    m, w = _model(cfg, seed=3)
    W = S.weights_as_f64(cfg, w)
    tok = 17
    H, KVH, dh, d, Fd = cfg.n_heads, cfg.n_kv_heads, cfg.head_dim, cfg.d_model, cfg.ffn_dim
    h = W["tok_emb"][tok].copy()
    for l in range(cfg.n_layers):
        u = _rmsnorm(h, W[f"layers.{l}.attn_norm"], cfg.rms_eps)
        v = (W[f"layers.{l}.w_qkv"] @ u)[(H + KVH) * dh:].reshape(KVH, dh)
        o = np.repeat(v, H // KVH, axis=0).reshape(-1)
        h = h + W[f"layers.{l}.w_o"] @ o
        u = _rmsnorm(h, W[f"layers.{l}.mlp_norm"], cfg.rms_eps)
        gu = W[f"layers.{l}.w_gate_up"] @ u
        a = gu[:Fd]
        h = h + W[f"layers.{l}.w_down"] @ (a / (1 + np.exp(-a)) * gu[Fd:])
    ref = W["lm_head"] @ _rmsnorm(h, W["final_norm"], cfg.rms_eps)
    got = m.score([tok])["logits"][0]
    assert _rel(got, ref) < 1e-12
    assert d == h.size


def test_long_sequence_rope_positions_match_library_built_model():
    """RoPE angles at large positions (and the causal window) against the
    complex-multiplication form, through an incrementally filled cache."""
    cfg = S.micro_config(n_layers=1, d_model=32, n_heads=2, n_kv_heads=1, head_dim=16, ffn_dim=24, vocab=41)
    m, w = _model(cfg, seed=4)
    toks = S.prompt(cfg, 300, seed=5)
    c = m.cache(300)
    m.forward(c, toks[:290])
    got = m.forward(c, toks[290:])["logits"]
    ref = torch_ref.forward(cfg, S.weights_as_f64(cfg, w), toks)[290:]
    assert _rel(got, ref) < 1e-9


def test_rope_relative_position_in_library_model():
    """q(p).k(p') depends only on p - p': the checker model itself is shift
    invariant (positions offset by 1000 give the same logits)."""
    cfg = S.micro_config(n_layers=1, d_model=32, n_heads=2, n_kv_heads=2, head_dim=16, ffn_dim=8, vocab=5)
    w64 = S.weights_as_f64(cfg, S.make_weights(cfg, 4))
    seq = [1, 2, 1, 2, 1, 2]
    assert _rel(torch_ref.forward(cfg, w64, seq, start_pos=1000), torch_ref.forward(cfg, w64, seq)) < 1e-9


# --------------------------------------------------------------------------
# incremental KV decoding == from-scratch forward (brute force)


@pytest.mark.parametrize("cfg", [MICRO_GQA, MICRO_BF16, S.MODELS["tiny"]], ids=lambda c: c.name)
def test_incremental_equals_from_scratch(cfg):
    m, _ = _model(cfg, seed=6)
    toks = S.prompt(cfg, 21, seed=7)
    c = m.cache(32)
    chunks = [5, 1, 4, 1, 1, 9]
    rows, s = [], 0
    for n in chunks:
        rows.append(m.forward(c, toks[s:s + n])["logits"])
        s += n
    inc = np.concatenate(rows)
    for t in (1, 6, 13, 21):
        scratch = m.score(toks[:t])["logits"][-1]
        assert np.array_equal(inc[t - 1], scratch)


def test_truncate_then_rewrite_equals_fresh():
    cfg = MICRO_GQA
    m, _ = _model(cfg, seed=7)
    toks = S.prompt(cfg, 10, seed=8)
    other = (toks[6:] + 5) % cfg.vocab
    c = m.cache(12)
    m.forward(c, toks[:6])
    m.forward(c, other)          # rejected continuation
    c.truncate(6)
    got = m.forward(c, toks[6:])["logits"]
    ref = m.score(toks)["logits"][6:]
    assert np.array_equal(got, ref)


def test_ar_equals_argmax_of_teacher_forced_forward():
    """Algorithm 1: token i+1 is the argmax of the full-model logits after tokens 1..i."""
    cfg = S.MODELS["tiny"]
    m, _ = _model(cfg)
    pr = S.prompt(cfg, 16)
    out, margin = m.generate_ar(pr, 24)
    seq = np.concatenate([pr, out])
    r = m.score(seq[:-1])
    assert np.array_equal(r["argmax"][len(pr) - 1:], out)
    assert np.allclose(r["margin"][len(pr) - 1:], margin, rtol=0, atol=1e-12)
    lg = r["logits"][len(pr) - 1:]
    # lowest id among equal float32 maxima
    assert np.array_equal(np.argmax(lg.astype(np.float32), axis=1), out)


def test_cache_load_matches_written_cache():
    """Externally loaded K/V (layout [L][2][KVH][len][dh]) behaves like written K/V."""
    cfg = MICRO_GQA
    m, _ = _model(cfg, seed=8)
    kv = S.kv_fill(cfg, cfg.n_layers * 2 * cfg.n_kv_heads * 6 * cfg.head_dim, seed=1)
    c1 = m.cache(9)
    c1.load(kv, 6, cfg.dtype)
    a = m.forward(c1, [4, 5, 6])["logits"]
    c2 = m.cache(9)
    c2.load(kv, 6, cfg.dtype)
    b = np.concatenate([m.forward(c2, [4])["logits"], m.forward(c2, [5, 6])["logits"]])
    assert np.array_equal(a, b)
    # a different prefix must change the result
    c3 = m.cache(9)
    c3.load(kv * np.float32(0.5), 6, cfg.dtype)
    assert not np.allclose(m.forward(c3, [4, 5, 6])["logits"], a)


MICRO_BF16_GQA = S.micro_config(n_layers=2, d_model=64, n_heads=4, n_kv_heads=2, head_dim=16, ffn_dim=96,
                                vocab=97, dtype="bf16", name="micro_bf16_gqa")


def kv_layout(kv_pairs, length: int) -> np.ndarray:
    """K/V pairs of the library-built model ([T, KVH, dh] per layer) in the
    cache-load layout [L][2 (K, V)][KVH][length][dh]."""
    return np.stack([np.stack([k[:length].transpose(1, 0, 2), v[:length].transpose(1, 0, 2)]) for k, v in kv_pairs])


def check_cache_load(lib_path=oracle.LIB_PATH):
    """K/V written by the library-built float64 model for positions [0, P),
    loaded into an oracle cache, then an oracle forward of the remaining rows:
    its logits equal the library-built model's over the whole sequence.

    The loaded values come from a different implementation (torch SDPA
    model), so a layout mistake in the loader (K and V swapped, heads before
    K/V, positions and head_dim transposed, a dropped layer) changes what the
    rows attend to and fails.  Both a bf16 model (bf16 bits, the verify
    microbenchmark's case) and a float32 model (float32 values) are loaded."""
    for cfg, dt in ((MICRO_BF16_GQA, "bf16"), (MICRO_GQA, "f32")):
        w = S.make_weights(cfg, 9)
        toks = S.prompt(cfg, 14, seed=10)
        P = 9
        pairs = []
        ref = torch_ref.forward(cfg, S.weights_as_f64(cfg, w), toks, kv_out=pairs)
        assert len(pairs) == cfg.n_layers
        kv = kv_layout(pairs, P)
        if dt == "bf16":
            kvs = S.f32_to_bf16_bits(kv.astype(np.float32))
            assert np.array_equal(S.bf16_bits_to_f32(kvs), kv)  # exact: the model rounded them to bf16
        else:
            kvs = kv.astype(np.float32)
        m = oracle.Model(cfg, w, lib_path=lib_path)
        c = m.cache(16)
        c.load(kvs, P, dt)
        assert c.length == P
        got = m.forward(c, toks[P:])["logits"]
        # float32 model: the loaded values were rounded to float32, the oracle's own are exact
        tol = 1e-10 if dt == "bf16" else 1e-6
        assert _rel(got, ref[P:]) < tol, (cfg.name, _rel(got, ref[P:]))


def test_cache_load_matches_library_built_kv():
    check_cache_load()


# --------------------------------------------------------------------------
# decoding invariants (losslessness, acceptance, stage counts)

CASES = [
    ("tiny", "tiny", 4, 0.6), ("tiny", "random3", 12, 0.0), ("tiny", "random5", 3, 0.01),
    ("tiny", "all", 4, 0.0), ("tiny", "none", 5, 0.3), ("tiny", "tiny", 0, 0.6), ("tiny", "tiny", 1, 2.0),
]


@pytest.mark.parametrize("model,mask,k_max,gamma", CASES)
def test_self_spec_equals_autoregressive(model, mask, k_max, gamma):
    """Losslessness: greedy self-speculative output equals greedy AR output."""
    cfg = S.MODELS[model]
    m, _ = _model(cfg)
    pr = S.prompt(cfg, 16)
    z = S.skip_mask(cfg, mask, seed=11)
    ar, _ = m.generate_ar(pr, 32)
    sd = m.generate_sd(pr, 32, z, k_max, gamma)
    assert np.array_equal(sd["tokens"], ar)
    st = sd["stages"]
    assert int(np.sum(st[:, 1] + 1)) == 32
    assert np.all((0 <= st[:, 1]) & (st[:, 1] <= st[:, 0]) & (st[:, 0] <= k_max))
    assert sd["n_drafted"] == st[:, 0].sum() and sd["n_accepted"] == st[:, 1].sum()


@pytest.mark.parametrize("cfg", [MICRO_GQA, MICRO_BF16], ids=lambda c: c.name)
def test_self_spec_equals_autoregressive_micro(cfg):
    m, _ = _model(cfg, seed=12)
    for t, mask, k, g in ((1, "random2", 3, 0.0), (5, "0", 6, 0.05), (2, "all", 2, 0.0)):
        pr = S.prompt(cfg, t, seed=t)
        z = S.skip_mask(cfg, mask, seed=13)
        ar, _ = m.generate_ar(pr, 15)
        sd = m.generate_sd(pr, 15, z, k, g)
        assert np.array_equal(sd["tokens"], ar)


def test_empty_skip_accepts_every_draft():
    """z = 0 is the original model, so every draft is accepted."""
    cfg = S.MODELS["tiny"]
    m, _ = _model(cfg)
    pr = S.prompt(cfg, 16)
    for k, g in ((4, 0.6), (12, 0.0), (3, 0.002)):
        sd = m.generate_sd(pr, 32, S.skip_mask(cfg, "none"), k, g)
        assert np.array_equal(sd["stages"][:, 0], sd["stages"][:, 1])
        assert sd["n_accepted"] == sd["n_drafted"]


@pytest.mark.parametrize("k_max,max_new", [(4, 32), (12, 32), (1, 7), (3, 1)])
def test_stage_count_closed_forms(k_max, max_new):
    cfg = S.MODELS["tiny"]
    m, _ = _model(cfg)
    pr = S.prompt(cfg, 16)
    none = S.skip_mask(cfg, "none")
    # empty z and gamma <= 0: every stage drafts kcap and accepts all of them
    sd = m.generate_sd(pr, max_new, none, k_max, 0.0)
    assert sd["n_stages"] == -(-max_new // (k_max + 1))
    # gamma > 1: every stage with room for a draft exits after exactly one
    sd = m.generate_sd(pr, max_new, S.skip_mask(cfg, "tiny"), k_max, 1.5)
    kcap_pos = sd["stages"][:, 0]
    assert np.all(kcap_pos <= 1)
    emitted = np.concatenate([[0], np.cumsum(sd["stages"][:, 1] + 1)[:-1]])
    assert np.all(kcap_pos == np.minimum(1, max_new - emitted - 1))
    # K_max = 0: plain verification steps, one token each
    sd = m.generate_sd(pr, max_new, S.skip_mask(cfg, "tiny"), 0, 0.6)
    assert sd["n_stages"] == max_new and sd["n_drafted"] == 0


def test_draft_exit_keeps_low_confidence_token():
    """Sec. 3.4: drafting stops right after a token with p_max < gamma; that token is verified."""
    cfg = S.MODELS["tiny"]
    m, _ = _model(cfg)
    pr = S.prompt(cfg, 16)
    z = S.skip_mask(cfg, "tiny")
    gamma = 0.0029
    sd = m.generate_sd(pr, 32, z, 6, gamma)
    pm = sd["draft_pmax"]
    i = 0
    emitted = 0
    for k, n in sd["stages"]:
        kcap = min(6, 32 - emitted - 1)
        steps = pm[i:i + k]
        # every draft before the last one was confident; the last one either
        # hit the cap or fell below gamma
        assert np.all(steps[:-1] >= np.float32(gamma)) if k else True
        if k:
            assert k == kcap or steps[-1] < np.float32(gamma)
        i += k
        emitted += n + 1
    assert i == pm.size


def test_golden_tiny_fixture():
    """Regression fixture written by tests/golden/make_golden.py from the oracle."""
    import json
    import os

    path = os.path.join(os.path.dirname(__file__), "golden", "tiny_decode.json")
    g = json.load(open(path))
    cfg = S.MODELS["tiny"]
    m, _ = _model(cfg)
    wl = S.WORKLOADS["tiny"]
    pr = S.prompt(cfg, wl.prompt_len)
    assert pr.tolist() == g["prompt"]
    ar, _ = m.generate_ar(pr, wl.max_new)
    sd = m.generate_sd(pr, wl.max_new, S.skip_mask(cfg, wl.mask), wl.k_max, wl.gamma)
    assert ar.tolist() == g["ar_tokens"]
    assert sd["stages"].tolist() == g["sd_stages"]
