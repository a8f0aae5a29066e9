"""Host logic of bench.py: byte accounting, the counter summaries, the
stale-counter guard and the one-GPU refusal.  No GPU is touched."""

import csv
import json
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import sd_synth as S  # noqa: E402

# Published parameter counts of the LLaMA-2 models whose shapes the workloads
# use (embedding and output matrices untied, no biases).
LLAMA2_PARAMS = {"7b": 6_738_415_616, "13b": 13_015_864_320, "70b": 68_976_648_192}


@pytest.mark.parametrize("name", ["7b", "13b", "70b"])
def test_shapes_match_published_parameter_counts(name):
    assert S.MODELS[name].param_count() == LLAMA2_PARAMS[name]


@pytest.mark.parametrize("name", ["7b", "13b", "70b"])
def test_full_step_reads_every_weight_but_the_embedding_table_once(name):
    """A full one-row step with no KV streams every parameter except the
    embedding table, of which it reads one row."""
    cfg = S.MODELS[name]
    es = 2
    want = (LLAMA2_PARAMS[name] - cfg.vocab * cfg.d_model + cfg.d_model) * es
    assert bench.step_bytes(cfg, None, 0, 0) == want


def test_step_bytes_kv_and_skips():
    cfg = S.MODELS["13b"]
    # 2 (K and V) x 40 kv heads x 128 x 2 bytes x 40 layers per cached position
    assert bench.step_bytes(cfg, None, 1, 0) - bench.step_bytes(cfg, None, 0, 0) == 819_200
    # one new position is written as well as read
    assert bench.step_bytes(cfg, None, 0, 1) - bench.step_bytes(cfg, None, 0, 0) == 819_200
    # skipping every sublayer leaves the head, the final norm and the embedding row
    skip = [1] * cfg.n_sublayers
    assert bench.step_bytes(cfg, skip, 4096, 1) == (cfg.vocab * cfg.d_model + 2 * cfg.d_model) * 2
    # skipping one MLP sublayer removes exactly its three matrices and its norm gain
    one = [0] * cfg.n_sublayers
    one[2 * 7 + 1] = 1
    drop = bench.step_bytes(cfg, None, 100, 1) - bench.step_bytes(cfg, one, 100, 1)
    assert drop == (3 * cfg.d_model * cfg.ffn_dim + cfg.d_model) * 2


@pytest.mark.parametrize("name", ["7b", "13b", "70b"])
def test_fp8_draft_step_bytes(name):
    """With FP8 draft copies a full-model weight set costs one byte per
    weight of the four sublayer matrices plus a 4-byte exponent per output
    row; the lm-head, the norms, the embedding row and the KV stay as they
    were."""
    cfg = S.MODELS[name]
    d, F, L = cfg.d_model, cfg.ffn_dim, cfg.n_layers
    qkv = (cfg.n_heads + 2 * cfg.n_kv_heads) * cfg.head_dim
    matrices = qkv * d + d * cfg.n_heads * cfg.head_dim + 3 * d * F
    exponent_rows = qkv + d + 2 * F + d
    for ctx, rows in ((0, 0), (1000, 1)):
        bf16 = bench.step_bytes(cfg, None, ctx, rows)
        fp8 = bench.step_bytes(cfg, None, ctx, rows, fp8=True)
        assert bf16 - fp8 == L * (matrices * 2 - matrices - 4 * exponent_rows)
    # a skipped sublayer costs nothing either way
    skip = [1] * cfg.n_sublayers
    assert bench.step_bytes(cfg, skip, 64, 1, fp8=True) == bench.step_bytes(cfg, skip, 64, 1)


def test_gate_up_bytes():
    # 13B, two rows: weights 27648 x 5120, gain 5120, two input rows of 5120
    # and two SwiGLU output rows of 13824
    assert bench.gate_up_bytes(27648, 5120, 2) == 27648 * 5120 * 2 + 5120 * 2 + 2 * 5120 * 4 + 2 * 13824 * 4
    assert bench.gate_up_bytes(27648, 5120, 2) - bench.gate_up_bytes(27648, 5120, 1) == (5120 + 13824) * 4


def _write_counter_csv(path, counter, rows):
    with open(path, "w", newline="") as f:
        w = csv.DictWriter(f, fieldnames=["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value",
                                          "Start_Timestamp", "End_Timestamp"])
        w.writeheader()
        for i, (name, value) in enumerate(rows):
            w.writerow({"Dispatch_Id": i, "Kernel_Name": name, "Counter_Name": counter, "Counter_Value": value,
                        "Start_Timestamp": 1000 * i, "End_Timestamp": 1000 * i + 500})


def _pmc_args(tmp_path, kernels, copy_bytes):
    class A:
        pass

    a = A()
    a.summarize_pmc = (str(tmp_path / "f.csv"), str(tmp_path / "w.csv"))
    a.kernels = ";".join(kernels)
    a.copy_bytes = copy_bytes
    a.command = "test"
    return a


def test_pmc_summary_calibrates_by_the_copy_and_takes_medians(tmp_path, monkeypatch):
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "traffic.json"))
    kern = "void sdk::k_linear_valu<unsigned short, 2, 8, 2, true, 64, 1>(sdk::LinearArgs)"
    copy = "__amd_rocclr_copyBuffer"
    gib = 1 << 30
    # the copy's FETCH_SIZE reads half its bytes (KiB), WRITE_SIZE all of them
    _write_counter_csv(tmp_path / "f.csv", "FETCH_SIZE",
                       [(copy, gib / 2 / 1024), (kern, 100.0), (kern, 140.0), (kern, 120.0), ("other", 7.0)])
    _write_counter_csv(tmp_path / "w.csv", "WRITE_SIZE",
                       [(copy, gib / 1024), (kern, 2.0), (kern, 2.0), (kern, 4.0), ("other", 1.0)])
    bench.run_summarize_pmc(_pmc_args(tmp_path, [kern], gib))
    out = json.load(open(tmp_path / "traffic.json"))
    assert out["copy_scale_fetch"] == pytest.approx(2.0)
    assert out["copy_scale_write"] == pytest.approx(1.0)
    e = out["kernels"][kern]
    assert e["fetch_bytes"] == pytest.approx(120.0 * 1024 * 2.0)
    assert e["write_bytes"] == pytest.approx(2.0 * 1024)
    assert e["bytes_per_launch"] == pytest.approx(e["fetch_bytes"] + e["write_bytes"])
    assert set(out["kernels"]) == {kern}
    assert out["source_hash"] == bench.source_hash()


def test_traffic_is_null_once_the_kernel_source_changes(tmp_path, monkeypatch):
    src = tmp_path / "kernels.hip"
    src.write_text("// version 1\n")
    monkeypatch.setattr(bench, "KERNEL_SOURCE", str(src))
    monkeypatch.setattr(bench, "TRAFFIC_FILE", str(tmp_path / "traffic.json"))
    json.dump({"source_hash": bench.source_hash(), "kernels": {"k": {"bytes_per_launch": 123.0}}},
              open(tmp_path / "traffic.json", "w"))
    assert bench.traffic_for("k") == 123.0
    assert bench.traffic_for("k", "13b") == 123.0
    # the counters were taken on the 13B shapes: another workload's launch of
    # the same kernel moves other bytes
    assert bench.traffic_for("k", "7b") is None
    assert bench.traffic_for("another kernel") is None
    src.write_text("// version 2\n")
    assert bench.traffic_for("k") is None
    os.remove(tmp_path / "traffic.json")
    assert bench.traffic_for("k") is None


def test_committed_traffic_matches_the_current_kernel_source():
    t = json.load(open(bench.TRAFFIC_FILE))
    assert t["source_hash"] == bench.source_hash(), "counters were taken on another version of the kernel source"
    (e,) = t["kernels"].values()
    # within 1% of the algorithmic bytes of the 13B two-row gate/up launch
    assert e["bytes_per_launch"] == pytest.approx(bench.gate_up_bytes(27648, 5120, 2), rel=0.01)


def test_forwards_group_dispatches_by_control_block_kernel():
    disp = [("k_set_ctl", {}, 1), ("k_embed", {}, 2), ("__amd_rocclr_copyBuffer", {}, 3), ("k_lin", {}, 4),
            ("k_set_ctl", {}, 5), ("at::native::fill", {}, 6), ("k_lin", {}, 7)]
    f = bench._forwards(disp)
    assert [[n for n, _, _ in fw] for fw in f] == [["k_embed", "k_lin"], ["k_lin"]]


def test_more_than_one_gpu_is_refused_before_touching_a_device():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_cpu_baseline_reports_decode_rates_and_the_host():
    """The oracle baseline separates prefill from decode and names the host."""
    wl = S.WORKLOADS["tiny"]
    cfg = S.MODELS["tiny"]
    w = S.make_weights(cfg, 0)
    r = bench.cpu_baseline(cfg, w, S.prompt(cfg, wl.prompt_len), wl, S.skip_mask(cfg, wl.mask))
    assert r["kind"] == "oracle" and r["unit"] == "tokens/s" and r["value"] > 0 and r["ar_value"] > 0
    assert r["prefill_rows"] == 7 and r["prefill_s"] >= 0
    assert r["cores"] >= 1 and r["nproc"] == os.cpu_count() and "cpu_model" in r
    assert 0 < r["attn_share_at_workload_ctx"] < 1
