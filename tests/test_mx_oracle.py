"""Pins of the reference's MXFP8 activation rule (native MXFP4 experts),
CPU only: the E4M3 element values of the OCP MX v1.0 specification, exact
round trips, round-half-to-even and saturation, the shared-scale rule, the
format's error bound, and the MoE with MXFP8 activations against the dense
brute force that restates the rule with numpy."""
import os
from dataclasses import replace

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2608_22167_amd import workload as W
from tests import bruteforce as BF

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def test_e4m3_values_match_the_spec_table():
    for line in open(os.path.join(GOLDEN, "ocp_mx_fp8_e4m3.txt")):
        if line.startswith("#") or not line.strip():
            continue
        code, val = line.split()
        got = O.e4m3(int(code, 16))
        if val == "nan":
            assert np.isnan(got)
        else:
            assert got == float(val) and np.signbit(got) == val.startswith("-"), (code, got, val)


def test_e4m3_round_trip_and_monotone():
    vals = [O.e4m3(c) for c in range(0x7F)]
    assert all(a < b for a, b in zip(vals, vals[1:]))
    for c in list(range(0x7F)) + list(range(0x81, 0xFF)):
        assert O.e4m3_encode(O.e4m3(c)) == c, hex(c)


@pytest.mark.parametrize("x,code", [(1.0625, 0x38), (1.1875, 0x3A), (1000.0, 0x7E), (464.0, 0x7E), (440.0, 0x7E),
                                    (1.5 * 2.0 ** -9, 0x02), (0.5 * 2.0 ** -9, 0x00), (0.6 * 2.0 ** -9, 0x01),
                                    (-1.0625, 0xB8), (2.0 ** -6 - 2.0 ** -10, 0x08)])
def test_e4m3_rounding_ties_and_saturation(x, code):
    assert O.e4m3_encode(x) == code


def test_mxfp8_scale_rule_and_codes():
    row = np.zeros((1, 64))
    row[0, :4] = [1.0, -0.5, 0.25, 3.0]      # amax 3: floor(log2 3) - 8 = -7
    row[0, 32:34] = [1.9, 0.001]             # amax 1.9: e = -8, 1.9 * 256 = 486.4 saturates
    codes, scales = O.mxfp8_quant(row)
    assert scales.tolist() == [[120, 119]]
    assert O.e4m3(codes[0, 3]) * 2.0 ** -7 == 3.0 and O.e4m3(codes[0, 0]) * 2.0 ** -7 == 1.0
    assert codes[0, 32] == 0x7E
    zero, zs = O.mxfp8_quant(np.zeros((2, 32)))
    assert (zero == 0).all() and (zs == 0).all()


def test_mxfp8_error_bound_and_numpy_restatement():
    rng = np.random.default_rng(0)
    x = torch.from_numpy(rng.standard_normal((64, 256)) * np.exp2(rng.integers(-20, 20, (64, 1)))).to(
        torch.bfloat16).double().numpy()
    codes, scales = O.mxfp8_quant(x)
    deq = np.vectorize(O.e4m3)(codes) * np.exp2(np.repeat(scales.astype(np.float64) - 127, 32, axis=1))
    np.testing.assert_array_equal(deq, BF.mxfp8_round(x))
    # three mantissa bits: relative error at most 2^-4 where no saturation and no subnormal applies
    blk = np.abs(x).reshape(64, 8, 32).max(axis=2, keepdims=True)
    normal = (np.abs(x).reshape(64, 8, 32) >= blk * 2.0 ** -8).reshape(x.shape) & \
             (np.abs(x).reshape(64, 8, 32) < blk * 0.875).reshape(x.shape)
    rel = np.abs(deq - x)[normal] / np.abs(x)[normal]
    assert rel.max() <= 2.0 ** -4


def test_moe_with_mxfp8_activations_matches_bruteforce():
    shape = replace(W.GPT_OSS_20B, hidden=192, n_q_heads=8, n_kv_heads=2, head_dim=64, n_experts=8, top_k=3,
                    ffn_dim=128, expert_fmt="mxfp4_native")
    wl = W.custom(shape, [4], [1], 61)
    h = W.synth_normal(5, 7, (12, shape.hidden)).double().numpy()
    r = O.moe(shape, O.Weights(shape, wl.weights), h)
    Wn = BF.weights_np(wl.weights)
    Wn["w_gu"] = O.Weights(shape, wl.weights).arr["w_gu"].astype(np.float64)
    Wn["w_d"] = O.Weights(shape, wl.weights).arr["w_d"].astype(np.float64)
    hn = BF.rmsnorm(h, Wn["g2"], shape.rms_eps)
    for t in range(h.shape[0]):
        acc, sel, w, _ = BF.moe_token(hn[t], Wn, shape)
        np.testing.assert_allclose(r["out"][t], h[t] + acc, rtol=1e-10, atol=1e-11)
    # and it differs from the bf16-activation reading (the rounding is real)
    dense = O.moe(replace(shape, expert_fmt="mxfp4"), O.Weights(shape, wl.weights), h)
    assert np.abs(dense["out"] - r["out"]).max() > 1e-4
