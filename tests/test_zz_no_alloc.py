"""decode_layer_noalloc (the static-scratch variant of decode_layer for
callers that cannot allocate) against decode_layer, through the C ABI.

Two calls in a row on the same GPU, the second with a smaller batch, each
compared with decode_layer on a caller workspace: the same kernels run on the
same inputs, so the outputs are bit-identical (stronger than the layer bar);
the call's device error word is handed back and cleared. A step needing more
scratch than the static array holds is rejected on the host.
"""
import ctypes

import numpy as np
import pytest
import torch

from paper_2608_22167_amd import mcpu, workload as W

pytestmark = pytest.mark.gpu


def _both(wl):
    s = wl.shape
    ref = mcpu.DeviceStep(wl)
    ref.run()
    T = wl.n_tokens
    x_out = torch.empty_like(ref.x_in)
    idx = torch.empty((T, s.top_k), dtype=torch.int32, device="cuda")
    w = torch.empty((T, s.top_k), device="cuda")
    err = torch.full((1,), -1, dtype=torch.int32, device="cuda")
    # the same pools and inputs as the reference step, re-appended at the same positions
    mcpu.decode_layer_noalloc(s, ref.weights, ref.pool, ref.page_table, ref.seq_lens, ref.cu_q, ref.host_seq_lens,
                              ref.host_cu_q, ref.x_in, x_out, idx, w, None, err)
    torch.cuda.synchronize()
    assert ref.device_errors() == 0
    assert int(err.item()) == 0
    return ref, x_out, idx, w


def test_noalloc_matches_decode_layer_twice_then_smaller():
    assert torch.cuda.is_available()
    torch.cuda.set_device(0)
    big = W.full_b64(seed=1201)
    small = W.custom(W.GPT_OSS_20B, [5, 130, 700, 16, 2049, 1], np.ones(6), 1202)
    for wl in (big, small):
        ref, x_out, idx, w = _both(wl)
        assert torch.equal(x_out, ref.x_out), wl.name
        assert torch.equal(idx, ref.topk_idx)
        assert torch.equal(w, ref.topk_w)
        d = (x_out - ref.x_out).abs().max().item()
        assert d <= 2e-2


def test_noalloc_reports_and_clears_device_errors():
    torch.cuda.set_device(0)
    wl = W.custom(W.GPT_OSS_20B, [40, 100], np.ones(2), 1203)
    wl.page_table[1, 0] = -1       # a missing page: the step sets the page bit
    step = mcpu.DeviceStep(wl)
    s = wl.shape
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    out = torch.empty_like(step.x_in)
    mcpu.decode_layer_noalloc(s, step.weights, step.pool, step.page_table, step.seq_lens, None, step.host_seq_lens,
                              None, step.x_in, out, None, None, None, err)
    torch.cuda.synchronize()
    assert int(err.item()) & mcpu.DEVERR_PAGE
    wl2 = W.custom(W.GPT_OSS_20B, [40, 100], np.ones(2), 1203)
    step2 = mcpu.DeviceStep(wl2)
    mcpu.decode_layer_noalloc(s, step2.weights, step2.pool, step2.page_table, step2.seq_lens, None,
                              step2.host_seq_lens, None, step2.x_in, out, None, None, None, err)
    torch.cuda.synchronize()
    assert int(err.item()) == 0     # the previous call's bits were cleared


def test_noalloc_rejects_steps_beyond_the_scratch():
    s = W.GPT_OSS_20B
    B = 600
    assert mcpu.decode_layer_workspace_size(s, B, B) > mcpu.NOALLOC_SCRATCH_BYTES
    L = mcpu.lib()
    cfg = mcpu.make_cfg(s)
    rc, pool = ctypes.c_void_p(), None
    h = ctypes.c_void_p()
    assert L.kv_pool_create(ctypes.byref(cfg), 64, 4096, 8192, ctypes.byref(h)) == 0
    hs = np.full(B, 10, np.int32)
    w = mcpu.LayerWeights()
    d = 1 << 32
    got = L.decode_layer_noalloc(ctypes.byref(cfg), ctypes.byref(w), h, B, d, 8, d, None, hs.ctypes.data, None, d,
                                 d + 4096, None, None, None, None, None)
    assert got == mcpu.MCPU_ENOMEM
    assert "scratch" in L.mcpu_last_error().decode()
    L.kv_pool_destroy(h)
