"""Error handling of the C ABI with a live model: invalid arguments are
rejected before anything is enqueued, and the model stays usable."""

import ctypes

import numpy as np
import pytest

import sd_synth as S
from paper_2309_08168_amd import binding
from tests import gpu_util as U

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def dm():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cfg = S.MODELS["tiny"]
    return U.device_model(cfg, S.make_weights(cfg, 0))


def _status(fn, *args):
    try:
        fn(*args)
    except binding.SDError as e:
        return e.status
    return binding.SD_OK


def test_invalid_arguments(dm):
    cfg = dm.cfg
    c = dm.cache(8)
    assert _status(dm.forward, [cfg.vocab], c) == binding.SD_ERR_INVALID_ARG
    assert _status(dm.forward, [-1], c) == binding.SD_ERR_INVALID_ARG
    assert _status(dm.forward, np.zeros(9, np.int32), c) == binding.SD_ERR_CAPACITY
    bad = np.zeros(2 * cfg.n_layers, np.uint8)
    bad[0] = 2
    assert _status(dm.forward, [1], c, bad) == binding.SD_ERR_INVALID_ARG
    assert c.length == 0
    pr = S.prompt(cfg, 4)
    assert _status(dm.generate_sd, pr, 4, None, 16, 0.5) == binding.SD_ERR_INVALID_ARG
    assert _status(dm.generate_sd, pr, 4, None, -1, 0.5) == binding.SD_ERR_INVALID_ARG
    assert _status(dm.generate_sd, pr, 4, None, 2, float("nan")) == binding.SD_ERR_INVALID_ARG
    assert _status(dm.generate_sd, [], 4, None, 2, 0.5) == binding.SD_ERR_INVALID_ARG
    assert _status(dm.generate_ar, pr, -1) == binding.SD_ERR_INVALID_ARG
    assert _status(c.truncate, 3) == binding.SD_ERR_INVALID_ARG
    assert _status(c.set_length, 9) == binding.SD_ERR_CAPACITY
    # still usable
    out, st = dm.generate_ar(pr, 3)
    assert st["n_emitted"] == 3


def test_caller_owned_cache_buffer(dm):
    cfg = dm.cfg
    nbytes = dm.kv_cache_bytes(20)
    buf = torch.zeros(nbytes // 4, dtype=torch.float32, device="cuda")
    c = dm.cache(20, device_buf=buf)
    toks = S.prompt(cfg, 6, seed=2)
    lg = torch.empty((6, cfg.vocab), dtype=torch.float32, device="cuda")
    dm.forward(toks, c, logits=lg)
    assert c.length == 6
    # the library wrote K/V of positions 0..5 into the caller's buffer
    kv = buf.view(cfg.n_layers, 2, cfg.n_kv_heads, 20, cfg.head_dim)
    assert torch.count_nonzero(kv[:, :, :, :6]).item() > 0
    assert torch.count_nonzero(kv[:, :, :, 6:]).item() == 0


def test_cache_outlives_model():
    """Destroying a model first detaches its caches; they can still be destroyed."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    cfg = S.MODELS["tiny"]
    m = U.device_model(cfg, S.make_weights(cfg, 0))
    c = m.cache(8)
    m.forward([1, 2], c)
    m2 = U.device_model(cfg, S.make_weights(cfg, 0))
    assert _status(m2.forward, [3], c) == binding.SD_ERR_INVALID_ARG  # another model's cache
    m.close()
    assert c.length == 2
    c.close()  # after its model: must not touch the freed model
    m2.close()


def test_kernel_timing_hook_samples_forwards(dm):
    """The measurement hook brackets the chosen class in one of every 16
    forwards of its regime: 32 autoregressive steps of the 4-layer model time
    the gate/up launches of steps 0 and 16 only, and timing changes no token."""
    cfg = dm.cfg
    prompt = S.prompt(cfg, 8)
    ref, _ = dm.generate_ar(prompt, 32)
    dm.time_kernel("gate_up", 1)
    out, _ = dm.generate_ar(prompt, 32)
    kt = dm.kernel_time()
    dm.time_kernel(None)
    assert np.array_equal(out, ref)
    assert kt["launches"] == 2 * cfg.n_layers
    assert kt["total_ms"] > 0.0
    assert kt["n"] == 2 * cfg.ffn_dim and kt["k"] == cfg.d_model
