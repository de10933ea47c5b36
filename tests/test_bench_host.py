"""Host logic of bench.py, without a GPU: the algorithmic work model that the
roofline divides by, the bound classification, the check that a committed
counter summary was taken on the current sources, and the single-GPU guard."""
import json
import os
import subprocess
import sys
from dataclasses import replace

import numpy as np

import bench
from paper_2608_22167_amd import workload as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_visible_keys_full_and_window():
    # a decode token at position L0 sees L0 + 1 keys, at most `window`
    assert bench._visible_sum(9, 1, 0) == 10
    assert bench._visible_sum(9, 1, 128) == 10
    assert bench._visible_sum(500, 1, 128) == 128
    # a 3-token chunk from position 0 sees 1 + 2 + 3 keys
    assert bench._visible_sum(0, 3, 0) == 6
    # past the window every token of a chunk sees exactly `window` keys
    assert bench._visible_sum(1000, 5, 128) == 5 * 128


def _decode_work(shape, idx, seq_lens):
    q = np.ones(len(seq_lens), np.int64)
    return bench.layer_work(shape, np.asarray(seq_lens, np.int64), q, np.asarray(idx))


def test_expert_weights_count_once_per_touched_expert():
    s = W.GPT_OSS_20B
    H, I = s.hidden, s.ffn_dim
    seqs = [100, 200, 300, 400]
    a, t_dec, t_pre = _decode_work(s, [[0, 1, 2, 3]] * 4, seqs)
    b, _, _ = _decode_work(s, [[0, 1, 2, 4]] * 3 + [[0, 1, 2, 3]], seqs)
    assert (t_dec, t_pre) == (4, 0)
    # one more expert touched: exactly one more expert's bf16 weights read
    assert b["expert_gu"][0] - a["expert_gu"][0] == 2 * I * H * 2
    assert b["expert_down"][0] - a["expert_down"][0] == H * I * 2
    # the same rows: the same products
    assert b["expert_gu"][1] == a["expert_gu"][1] == 2 * 16 * 2 * I * H


def test_mxfp4_experts_count_codes_and_scales():
    s = replace(W.GPT_OSS_20B, expert_fmt="mxfp4")
    H, I = s.hidden, s.ffn_dim
    a, _, _ = _decode_work(s, [[0, 1, 2, 3]], [50])
    b, _, _ = _decode_work(s, [[3, 2, 1, 0]], [50])
    c, _, _ = _decode_work(s, [[4, 5, 6, 7], [0, 1, 2, 3]], [50, 50])
    assert a == b  # the order of a token's selections does not matter
    # four more experts: their codes (half a byte a weight) and scales (a byte per 32)
    extra = c["expert_gu"][0] - a["expert_gu"][0]
    rows_extra = 4 * (H + I) * 2  # the second token's four rows in and out
    assert extra - rows_extra == 4 * (2 * I * H // 2 + 2 * I * H // 32)


def test_window_caps_attention_bytes():
    full, _, _ = _decode_work(W.GPT_OSS_20B, [[0, 1, 2, 3]], [10000])
    sw, _, _ = _decode_work(W.GPT_OSS_20B_SW, [[0, 1, 2, 3]], [10000])
    kv_per_key = W.GPT_OSS_20B.n_kv_heads * W.GPT_OSS_20B.head_dim * 2 * 2
    q_bytes = W.GPT_OSS_20B.n_q_heads * W.GPT_OSS_20B.head_dim * 2
    assert full["attn_split"][0] == 10001 * kv_per_key + q_bytes
    assert sw["attn_split"][0] == 128 * kv_per_key + q_bytes


def test_roofline_bound_follows_the_ridge():
    ridge = bench.MFMA_PEAK_TFLOPS["bf16"] * 1e12 / (bench.HBM_PEAK_GBS * 1e9)  # flop per byte
    low = bench.roofline_of(1e9, 1e9 * ridge / 2, 1e-3, "bf16")
    assert low["bound"] == "hbm" and low["unit"] == "GB/s"
    assert abs(low["achieved"] - 1000.0) < 0.1 and abs(low["frac"] - 1000.0 / bench.HBM_PEAK_GBS) < 1e-4
    high = bench.roofline_of(1e9, 1e9 * ridge * 2, 1e-3, "bf16")
    assert high["bound"] == "mfma" and high["unit"] == "TFLOP/s"
    assert abs(high["frac"] - high["achieved"] / bench.MFMA_PEAK_TFLOPS["bf16"]) < 1e-4
    # products with MXFP8 activations are priced at the fp8 rate
    s = replace(W.GPT_OSS_20B, expert_fmt="mxfp4_native")
    assert bench.peak_key("expert_gu", s) == "mxfp8" and bench.peak_key("qkv", s) == "bf16"


def test_counter_summary_used_only_on_matching_sources(tmp_path, monkeypatch):
    prof = tmp_path / "profiles"
    prof.mkdir()
    (prof / "expert_gu_demo_counters.md").write_text(
        "- hbm bytes per launch: 1.5e+09\n- sources sha256[:16]: 0123456789abcdef\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    monkeypatch.setattr(bench, "source_hash", lambda k: "0123456789abcdef")
    assert bench.traffic_from_profile("expert_gu", "demo") == 1.5e9
    monkeypatch.setattr(bench, "source_hash", lambda k: "fedcba9876543210")
    assert bench.traffic_from_profile("expert_gu", "demo") is None  # sources changed since
    assert bench.traffic_from_profile("expert_gu", "other") is None  # no summary


def test_source_hash_covers_the_kernel_sources():
    # GEMM kernels hash the GEMM sources, attention the attention sources
    assert bench.source_hash("expert_gu") == bench.source_hash("qkv")
    assert bench.source_hash("attn_split") == bench.source_hash("attn_prefill")
    assert bench.source_hash("expert_gu") != bench.source_hash("attn_split")
    assert bench.source_hash("lm_head") != bench.source_hash("expert_gu")


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert line["n_gpus"] == 2 and "one GPU" in line["error"]
