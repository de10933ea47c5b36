"""Native MXFP4 experts on the GPU (MXFP4 weights x MXFP8 activations on the
scaled matrix cores) against the reference with its MXFP8 activation rule,
through the C ABI: the quantizer and the weights' slice-order copy bit for
bit, the MoE sub-block at a few to
thousands of rows per expert (ragged tiles and reduction tails), whole
layers, and the mixed prefill step at full size on sampled sequences."""
from dataclasses import replace

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2608_22167_amd import mcpu, workload as W
from tests import parity as PT
from tests.test_gpu_parity import compare_layer, reference, run_layer

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    torch.cuda.set_device(0)
    yield
    torch.cuda.empty_cache()


def test_mxfp8_quantize_bit_exact():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((300, 2880)) * np.exp2(rng.integers(-30, 30, (300, 1)))
    x[0, :32] = 0.0                                   # an all-zero block
    x[1, :32] = 1.9                                   # saturation at 448
    x[2, :32] = [1.0625, 1.1875] * 16                 # ties to even
    x[3, :32] = 2.0 ** -140                           # bf16 subnormals
    x[4, 32:64] = -np.arange(32) * 2.0 ** -12
    xb = torch.from_numpy(x).to(torch.bfloat16)
    codes, scales = mcpu.mxfp8_quantize(xb.cuda())
    torch.cuda.synchronize()
    rc, rs = O.mxfp8_quant(xb.double().numpy())
    np.testing.assert_array_equal(scales.cpu().numpy(), rs)
    np.testing.assert_array_equal(codes.cpu().numpy(), rc)


@pytest.mark.parametrize("groups,rows,cols", [(2, 32, 192), (1, 16, 2880), (3, 48, 64)])
def test_pack_mxfp4_layout_byte_exact(groups, rows, cols):
    """mcpu_pack_mxfp4 against the slice order the header states, rebuilt
    with numpy reshapes (192 columns: a last scale dword with two unused
    bytes, which hold 127)."""
    rng = np.random.default_rng(groups * 1000 + cols)
    codes = rng.integers(0, 256, (groups, rows, cols // 2), dtype=np.uint8)
    scales = rng.integers(2, 253, (groups, rows, cols // 32), dtype=np.uint8)
    out = mcpu.packed_mxfp4(torch.from_numpy(codes).cuda(), torch.from_numpy(scales).cuda())
    torch.cuda.synchronize()
    got = out.cpu().numpy()
    cb = (groups * rows * cols // 2 + 255) // 256 * 256
    want_c = codes.reshape(groups, rows, cols // 64, 32).transpose(0, 2, 1, 3).reshape(-1)
    np.testing.assert_array_equal(got[:want_c.size], want_c)
    kq = (cols // 32 + 3) // 4
    sp = np.full((groups, rows, kq * 4), 127, np.uint8)
    sp[:, :, :cols // 32] = scales
    want_s = sp.reshape(groups, rows, kq, 4).transpose(0, 2, 1, 3).reshape(-1)
    np.testing.assert_array_equal(got[cb:cb + want_s.size], want_s)
    assert got.size == cb + want_s.size


def _moe_check(s, T, seed, h_seed=4, sample=None):
    wl = W.custom(s, [4], [1], seed)
    dw = mcpu.DeviceWeights(s, wl.weights)
    h = W.synth_normal(9, h_seed, (T, s.hidden))
    out = torch.empty((T, s.hidden), device="cuda")
    idx = torch.empty((T, s.top_k), dtype=torch.int32, device="cuda")
    wt = torch.empty((T, s.top_k), device="cuda")
    ws = mcpu.workspace(mcpu.moe_forward_workspace_size(s, T))
    mcpu.moe_forward(s, dw, h.cuda(), out, idx, wt, None, ws)
    torch.cuda.synchronize()
    assert mcpu.mcpu_check_device_errors(ws) == 0
    rows = np.arange(T) if sample is None else np.unique(np.concatenate(
        [[0, T - 1], np.random.default_rng(seed).choice(T, sample, replace=False)]))
    weights = O.Weights(s, wl.weights)
    hh = h[torch.from_numpy(rows)]
    ref = O.moe(s, weights, hh)
    g_idx = idx.cpu().numpy()[rows]
    tie = PT.check_router(g_idx, ref["idx"], ref["logits"], s.top_k)
    if tie.any():
        f = ref["idx"].copy()
        f[tie] = g_idx[tie]
        ref = O.moe(s, weights, hh, force_idx=f)
    return PT.check("moe out (native MXFP4)", out.cpu().double().numpy()[rows], ref["out"], "bf16")


@pytest.mark.parametrize("T", [1, 40, 300, 3600])
def test_moe_native_small_shapes(T):
    """8 experts, top-2, hidden/ffn 576 (4.5 reduction stages of 128: a half
    stage at the end): from single rows to about 900 rows per expert."""
    s = replace(W.GPT_OSS_20B, hidden=576, n_q_heads=8, n_kv_heads=2, head_dim=64, n_experts=8, top_k=2,
                ffn_dim=576, expert_fmt="mxfp4_native")
    mx, rl = _moe_check(s, T, 1301 + T)
    print(f"  T={T}: max-abs {mx:.2e} rel-L2 {rl:.2e}")


@pytest.mark.parametrize("T", [256, 16384])
def test_moe_native_gpt_oss_shape_sampled(T):
    s = replace(W.GPT_OSS_20B, expert_fmt="mxfp4_native")
    mx, rl = _moe_check(s, T, 1311, sample=24)
    print(f"  T={T}: max-abs {mx:.2e} rel-L2 {rl:.2e}")


def test_native_layer_small():
    shape = replace(W.GPT_OSS_20B, hidden=256, n_q_heads=8, n_kv_heads=2, head_dim=64, n_experts=8, top_k=2,
                    ffn_dim=256, expert_fmt="mxfp4_native")
    wl = W.custom(shape, [0, 15, 16, 200, 1100], [1, 1, 40, 1, 17], 1321, sink_std=0.5)
    gpu, step = run_layer(wl)
    compare_layer(wl, gpu, step)


def test_native_mixed_step_full_size_sampled():
    """The mixed prefill step with native MXFP4 experts (the benchmark's
    compute-bound case): two decode sequences and the shortest chunk."""
    from tests.test_gpu_prefill import _run_layer_rows
    wl = W.mixed_prefill(expert_fmt="mxfp4_native")
    dec = np.nonzero(wl.q_lens == 1)[0]
    pre = np.nonzero(wl.q_lens > 1)[0]
    seqs = sorted({int(dec[np.argmax(wl.seq_lens[dec])]), int(dec[0]), int(pre[np.argmin(wl.q_lens[pre])])})
    sub, rows = W.restrict(wl, seqs)
    g, finite, wsum_ok = _run_layer_rows(wl, rows)
    assert finite and wsum_ok
    ref, _ = reference(sub, g)
    compare_layer(sub, g, None, ref)
