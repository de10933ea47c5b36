"""GPU path (libmcpu.so through the C ABI) against the CPU reference.

Sizes: small cases span several pages, several attention splits and ragged
page tails; the full-size workloads (64 sequences with 2k-16k contexts, 256
sliding-window sequences with log-normal contexts) are compared on sampled
sequences, which is exact because sequences are independent given their own
cache pages.
"""
import math
from dataclasses import replace

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2608_22167_amd import mcpu, workload as W
from tests import parity as PT

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    torch.cuda.set_device(0)
    yield


def _np(t):
    return t.detach().cpu().float().numpy().astype(np.float64)


def run_layer(wl):
    """decode_layer on the GPU; returns its outputs and the device step."""
    step = mcpu.DeviceStep(wl)
    s = wl.shape
    T = wl.n_tokens
    taps_t = dict(q=torch.empty((T, s.n_q_heads, s.head_dim), dtype=s.torch_dtype, device="cuda"),
                  o=torch.empty((T, s.attn_dim), dtype=s.torch_dtype, device="cuda"),
                  h1=torch.empty((T, s.hidden), dtype=torch.float32, device="cuda"))
    taps = mcpu.Taps(q=taps_t["q"].data_ptr(), o=taps_t["o"].data_ptr(), h1=taps_t["h1"].data_ptr())
    step.run(taps)
    torch.cuda.synchronize()
    assert step.device_errors() == 0
    out = dict(out=_np(step.x_out), idx=step.topk_idx.cpu().numpy(), w=_np(step.topk_w),
               q=_np(taps_t["q"]), o=_np(taps_t["o"]), h1=_np(taps_t["h1"]))
    return out, step


def reference(wl, gpu):
    """CPU reference; near-tie tokens re-run with the GPU's expert choice."""
    ref = O.decode_layer(wl)
    tie = PT.check_router(gpu["idx"], ref["idx"], ref["logits"], wl.shape.top_k)
    if tie.any():
        force = ref["idx"].copy()
        force[tie] = gpu["idx"][tie]
        ref = O.decode_layer(wl, force_idx=force)
    return ref, tie


def compare_layer(wl, gpu, step=None, ref=None):
    if ref is None:
        ref, _ = reference(wl, gpu)
    dt = wl.shape.dtype
    PT.check("q", gpu["q"], ref["q"], dt)
    PT.check("o", gpu["o"], ref["o"], dt)
    PT.check("h1", gpu["h1"], ref["h1"], dt)
    if wl.shape.expert_fmt == "mxfp4_native":
        # MXFP8 codes are a step function of the MoE input: a one-ulp bf16
        # difference of the normalised row (from h1's rounding) flips E4M3 codes
        # (12.5% steps), so the MoE increment is compared from the GPU's own h1
        # (teacher-forced, as in moe_forward); `out` below still checks the chain
        w = O.Weights(wl.shape, wl.weights)
        rm = O.moe(wl.shape, w, gpu["h1"])
        tie = PT.check_router(gpu["idx"], rm["idx"], rm["logits"], wl.shape.top_k)
        if tie.any():
            f = rm["idx"].copy()
            f[tie] = gpu["idx"][tie]
            rm = O.moe(wl.shape, w, gpu["h1"], force_idx=f)
        PT.check("moe (from the GPU's h1)", gpu["out"] - gpu["h1"], rm["moe"], dt)
    else:
        PT.check("moe", gpu["out"] - gpu["h1"], ref["out"] - ref["h1"], dt)
    PT.check("out", gpu["out"], ref["out"], dt)
    np.testing.assert_allclose(gpu["w"].sum(1), 1.0, rtol=1e-5)
    PT.check("topk_w", *PT.weights_by_expert(gpu["idx"], gpu["w"], ref["idx"], ref["w"]), dt)
    if step is not None:
        check_appended(wl, step, ref)
    return ref


def check_appended(wl, step, ref):
    """New keys/values in the device pools against the reference's. Both sides
    round the normalised row to bf16 and project it; they differ in the
    projection's summation order (fp32 vs float64) before rounding to the
    cache dtype, which moves an entry by at most one bf16 ulp. Where the two
    RMSNorms (fp32 vs float64) straddle a bf16 rounding boundary of one
    element of the normalised row, every k and v of that token also moves by
    |w| x ulp(xn) (about 1e-4, at most about 1.5e-3). So every entry is
    within max(1 bf16 ulp, 2e-3) of the reference's (one ulp from magnitude
    0.5 up); the share of entries beyond one ulp is printed. An fp32 cache is
    held to the fp32 bar."""
    s = wl.shape
    kp = step.k_pool.cpu().float().numpy()
    vp = step.v_pool.cpu().float().numpy()
    kr, vr = ref["k_pool"], ref["v_pool"]
    got_k, want_k, got_v, want_v = [], [], [], []
    for b in range(wl.batch):
        for i in range(int(wl.q_lens[b])):
            pos = int(wl.seq_lens[b]) + i
            page = wl.page_table[b, pos // 16]
            kl, vl = O.pool_to_logical(s, kp[page:page + 1], vp[page:page + 1])
            krl, vrl = O.pool_to_logical(s, kr[page:page + 1], vr[page:page + 1])
            slot = pos % 16
            got_k.append(kl[0, :, slot]); want_k.append(krl[0, :, slot])
            got_v.append(vl[0, :, slot]); want_v.append(vrl[0, :, slot])
    for name, got, want in (("k", got_k, want_k), ("v", got_v, want_v)):
        got, want = np.stack(got), np.stack(want)
        if s.dtype == "bf16":
            ulp = PT.bf16_ulp(np.maximum(np.abs(got), np.abs(want)))
            err = np.abs(got - want)
            bad = err > np.maximum(ulp, 2e-3)
            assert not bad.any(), f"appended {name}: {int(bad.sum())} entries beyond max(1 ulp, 2e-3), " \
                                  f"worst {err.max():.3e}"
            print(f"  appended {name}: {float((err > ulp).mean()):.2e} of entries beyond one bf16 ulp "
                  f"(max {float((err / ulp).max()):.2f} ulps)")
        else:
            PT.check(f"appended {name}", got, want, s.dtype)


# ---------------------------------------------------------------------------------- tiny fp32


def test_tiny_f32_layer():
    wl = W.tiny_f32(seed=1001)
    gpu, step = run_layer(wl)
    compare_layer(wl, gpu, step)


def test_tiny_f32_plain_swiglu_and_window():
    shape = replace(W.TINY, swiglu_alpha=1.0, swiglu_limit=math.inf, swiglu_beta=0.0, window=40)
    wl = W.custom(shape, [1, 40, 41, 100, 255], np.ones(5), 1011, sink_std=1.0)
    gpu, step = run_layer(wl)
    compare_layer(wl, gpu, step)


def test_tiny_f32_repeatable_bitwise():
    wl = W.tiny_f32(seed=1012, batch=8)
    a, _ = run_layer(wl)
    b, _ = run_layer(wl)
    for k in a:
        np.testing.assert_array_equal(a[k], b[k])


# ---------------------------------------------------------------------------------- bf16 layer


def _bf16_small(window=0, seed=1021, sink_std=0.02, bias=None, ctx=None):
    shape = replace(W.GPT_OSS_20B, window=window)
    ctx = [0, 1, 15, 16, 17, 127, 128, 129, 300, 1100] if ctx is None else ctx
    return W.custom(shape, ctx, np.ones(len(ctx)), seed, sink_std=sink_std, router_bias=bias)


def test_bf16_full_attention_layer():
    wl = _bf16_small()
    gpu, step = run_layer(wl)
    compare_layer(wl, gpu, step)


def test_bf16_sliding_window_layer():
    wl = _bf16_small(window=128, seed=1022, bias=W.zipf_router_bias(32, 1.1, 1022))
    gpu, step = run_layer(wl)
    compare_layer(wl, gpu, step)


@pytest.mark.parametrize("batch", [1, 17])
def test_bf16_layer_small_batches(batch):
    """One decode token (every expert GEMM group holds at most one row, the
    split projections one row of their 64-row tile) and 17 (one row past a
    16-row fragment)."""
    rng = np.random.default_rng(1024 + batch)
    ctx = [int(c) for c in rng.integers(1, 900, size=batch)]
    wl = _bf16_small(seed=1024 + batch, ctx=ctx)
    gpu, step = run_layer(wl)
    compare_layer(wl, gpu, step)


def test_bf16_sink_stress_layer():
    # Sinks of std 3 make some heads put nearly all weight on one key. With a
    # one-key context that head's output is the new token's bf16-stored value,
    # whose storage rounding alone (ulp 1/64 above 2) can exceed the 2e-2
    # max-abs bound, so this case starts at 16 cached keys; one-key contexts
    # are covered at the configured sink scale above.
    wl = _bf16_small(seed=1023, sink_std=3.0, ctx=[16, 17, 31, 127, 128, 129, 300, 1100])
    gpu, step = run_layer(wl)
    compare_layer(wl, gpu, step)


# ---------------------------------------------------------------------------------- attention only


def _attention_case(wl, q_scale=1.0, sinks=None, seed=5):
    s = wl.shape
    rng = np.random.default_rng(seed)
    q = torch.from_numpy((rng.standard_normal((wl.batch, s.n_q_heads, s.head_dim)) * q_scale)
                         .astype(np.float32)).to(s.torch_dtype)
    sk = wl.weights["sinks"] if sinks is None else torch.as_tensor(sinks, dtype=torch.float32)
    step = mcpu.DeviceStep(wl)
    o = torch.empty((wl.batch, s.attn_dim), dtype=s.torch_dtype, device="cuda")
    ws = mcpu.workspace(mcpu.paged_attention_workspace_size(s, wl.batch, wl.batch))
    mcpu.paged_attention(s, sk.cuda(), step.pool, step.page_table, step.seq_lens, None,
                         wl.seq_lens, None, q.cuda(), o, ws)
    torch.cuda.synchronize()
    assert mcpu.mcpu_check_device_errors(ws) == 0
    ref = O.attention(s, np.arange(wl.batch), wl.seq_lens, q, wl.k_pool, wl.v_pool, wl.page_table, sk)
    return _np(o), ref.reshape(wl.batch, -1), step, q, sk


@pytest.mark.parametrize("window", [0, 128])
def test_attention_sink_stress_and_overflow(window):
    wl = _bf16_small(window=window, seed=1031)
    ctx = wl.seq_lens.astype(np.float64) + 1
    rng = np.random.default_rng(3)
    # sinks taking 10-90% of the mass, and +/-30
    sinks = rng.uniform(-2.0, np.log(ctx.max()) + 3.0, size=wl.shape.n_q_heads).astype(np.float32)
    sinks[:4] = 30.0
    sinks[4:8] = -30.0
    got, ref, *_ = _attention_case(wl, sinks=sinks)
    PT.check("o(sink stress)", got, ref, "bf16")
    got, ref, *_ = _attention_case(wl, q_scale=50.0)
    PT.check("o(q x 50)", got, ref, "bf16")
    assert np.abs(got).max() > 0.1  # peaked softmax: not averaged away


def test_attention_page_permutation_bitwise():
    wl = _bf16_small(seed=1032)
    a, *_ = _attention_case(wl)
    perm = np.random.default_rng(11).permutation(wl.n_pages)
    kp, vp = torch.empty_like(wl.k_pool), torch.empty_like(wl.v_pool)
    kp[perm], vp[perm] = wl.k_pool, wl.v_pool
    wl.k_pool, wl.v_pool = kp, vp
    wl.page_table = np.where(wl.page_table >= 0, perm[np.maximum(wl.page_table, 0)], -1).astype(np.int32)
    b, *_ = _attention_case(wl)
    np.testing.assert_array_equal(a, b)


def test_attention_split_count_invariance_fp32():
    """The same query over the same pages, in batches whose total length makes
    the planner cut its 188 pages into 12, 6 and 2 splits (16, 37 and 184
    pages per split): the fp32 results agree within 1e-6 relative, and with
    the reference at the fp32 bar. Filler queries share one run of pages, so
    the batch is long without a large pool."""
    s = replace(W.TINY, window=0)
    ctx = 3000                                   # 188 pages
    n_pages = 200
    rng = np.random.default_rng(1035)
    shp = (n_pages, s.n_kv_heads, 16, s.head_dim)
    k_pool = torch.from_numpy(rng.standard_normal(shp).astype(np.float32))
    v_pool = torch.from_numpy(rng.standard_normal(shp).astype(np.float32))
    row = rng.permutation(n_pages)[:188].astype(np.int32)
    q0 = torch.from_numpy(rng.standard_normal((1, s.n_q_heads, s.head_dim)).astype(np.float32))
    sinks = torch.from_numpy(rng.uniform(-2, 6, s.n_q_heads).astype(np.float32))
    pool = mcpu.KVPool(s, k_pool.cuda(), v_pool.cuda())
    outs = []
    for n_fill in (0, 300, 1500):
        B = 1 + n_fill
        pt = np.tile(row, (B, 1))
        sl = np.full(B, ctx - 1, np.int32)       # each query at position ctx - 1 sees ctx keys
        q = torch.cat([q0, torch.from_numpy(rng.standard_normal((n_fill, s.n_q_heads, s.head_dim))
                                            .astype(np.float32))]) if n_fill else q0
        o = torch.empty((B, s.attn_dim), device="cuda")
        ws = mcpu.workspace(mcpu.paged_attention_workspace_size(s, B, B))
        mcpu.paged_attention(s, sinks.cuda(), pool, torch.from_numpy(pt).cuda(), torch.from_numpy(sl).cuda(),
                             None, sl, None, q.cuda(), o, ws)
        torch.cuda.synchronize()
        assert mcpu.mcpu_check_device_errors(ws) == 0
        outs.append(_np(o[:1]))
    for o in outs[1:]:
        assert PT.rel_l2(o, outs[0]) <= 1e-6, PT.rel_l2(o, outs[0])
    ref = O.attention(s, [0], [ctx - 1], q0, k_pool, v_pool, row[None, :], sinks).reshape(1, -1)
    for o in outs:
        PT.check("o(split count)", o, ref, "f32")


def test_attention_missing_page_sets_device_error():
    wl = _bf16_small(seed=1033)
    wl.page_table[9, 3] = -1
    s = wl.shape
    step = mcpu.DeviceStep(wl)
    q = torch.zeros((wl.batch, s.n_q_heads, s.head_dim), dtype=s.torch_dtype, device="cuda")
    o = torch.empty((wl.batch, s.attn_dim), dtype=s.torch_dtype, device="cuda")
    ws = mcpu.workspace(mcpu.paged_attention_workspace_size(s, wl.batch, wl.batch))
    mcpu.paged_attention(s, step.weights.t["sinks"], step.pool, step.page_table, step.seq_lens, None,
                         wl.seq_lens, None, q, o, ws)
    assert mcpu.mcpu_check_device_errors(ws) & mcpu.DEVERR_PAGE
    assert mcpu.mcpu_check_device_errors(ws) == 0   # read-and-clear


# ---------------------------------------------------------------------------------- append, MoE


def test_kv_pages_append_bit_exact():
    shape = W.GPT_OSS_20B
    wl = W.custom(shape, [3, 16, 31, 200], [1, 5, 1, 17], 1041, weights=False)
    step_pools = (wl.k_pool.cuda(), wl.v_pool.cuda())
    pool = mcpu.KVPool(shape, *step_pools)
    T = wl.n_tokens
    kn = W.synth_normal(7, 1, (T, 8, 64), dtype=torch.bfloat16)
    vn = W.synth_normal(7, 2, (T, 8, 64), dtype=torch.bfloat16)
    ws = mcpu.workspace(256)
    pt = torch.from_numpy(wl.page_table).cuda()
    mcpu.kv_pages_append(pool, pt, torch.from_numpy(wl.seq_lens).cuda(), torch.from_numpy(wl.cu_q).cuda(),
                         kn.cuda(), vn.cuda(), ws)
    torch.cuda.synchronize()
    assert mcpu.mcpu_check_device_errors(ws) == 0
    tok_seq = np.repeat(np.arange(wl.batch), wl.q_lens)
    tok_pos = np.concatenate([wl.seq_lens[b] + np.arange(wl.q_lens[b]) for b in range(wl.batch)])
    kr, vr = O.kv_append(shape, tok_seq, tok_pos, kn, vn, wl.k_pool, wl.v_pool, wl.page_table)
    np.testing.assert_array_equal(step_pools[0].cpu().float().numpy(), kr)
    np.testing.assert_array_equal(step_pools[1].cpu().float().numpy(), vr)


@pytest.mark.parametrize("kind", ["tiny_f32", "bf16", "tiny_f32_t1100", "bf16_t1030"])
def test_moe_forward_and_forced_selection(kind):
    """Routers: one token per 1024-thread workgroup up to 256 tokens (24 and 10
    tokens here; 8 experts put an expert's threads in two wavefronts), one per
    256-thread workgroup below 1024 (the 350- and 1000-token cases elsewhere),
    16 tokens per workgroup from 1024 on (1100 and 1030 tokens: a ragged last
    workgroup)."""
    if kind == "tiny_f32":
        wl = W.tiny_f32(seed=1051, batch=24)
    elif kind == "tiny_f32_t1100":
        wl = W.tiny_f32(seed=1053, batch=1100)
    elif kind == "bf16":
        wl = _bf16_small(seed=1052)
    else:
        shape = replace(W.GPT_OSS_20B, hidden=512, n_q_heads=8, n_kv_heads=2, ffn_dim=512)  # 32 experts, top 4
        wl = W.custom(shape, np.random.default_rng(1054).integers(0, 64, size=1030), np.ones(1030), 1054)
    s = wl.shape
    dw = mcpu.DeviceWeights(s, wl.weights)
    T = wl.n_tokens
    h = W.synth_normal(9, 3, (T, s.hidden))
    out = torch.empty((T, s.hidden), device="cuda")
    idx = torch.empty((T, s.top_k), dtype=torch.int32, device="cuda")
    wt = torch.empty((T, s.top_k), device="cuda")
    ws = mcpu.workspace(mcpu.moe_forward_workspace_size(s, T))
    mcpu.moe_forward(s, dw, h.cuda(), out, idx, wt, None, ws)
    torch.cuda.synchronize()
    ref = O.moe(s, O.Weights(s, wl.weights), h)
    tie = PT.check_router(idx.cpu().numpy(), ref["idx"], ref["logits"], s.top_k)
    if tie.any():
        f = ref["idx"].copy()
        f[tie] = idx.cpu().numpy()[tie]
        ref = O.moe(s, O.Weights(s, wl.weights), h, force_idx=f)
    PT.check("moe out", _np(out), ref["out"], s.dtype)
    # the same rows in, so the weights differ only by the logits' summation order
    gw, rw = PT.weights_by_expert(idx.cpu().numpy(), _np(wt), ref["idx"], ref["w"])
    np.testing.assert_allclose(gw, rw, atol=1e-5, rtol=0)
    # forced selection, including a repeated expert within one token
    force = np.random.default_rng(1).integers(0, s.n_experts, size=(T, s.top_k)).astype(np.int32)
    force[0, :] = force[0, 0]
    mcpu.moe_forward(s, dw, h.cuda(), out, idx, wt, torch.from_numpy(force).cuda(), ws)
    torch.cuda.synchronize()
    assert mcpu.mcpu_check_device_errors(ws) == 0
    ref = O.moe(s, O.Weights(s, wl.weights), h, force_idx=force)
    PT.check("moe out (forced)", _np(out), ref["out"], s.dtype)
    np.testing.assert_array_equal(idx.cpu().numpy(), force)


# ---------------------------------------------------------------------------------- full size, sampled


@pytest.mark.parametrize("which", ["full_b64", "sliding_b256"])
def test_full_size_every_sequence(which):
    """The 64-sequence full-attention and the 256-sequence sliding-window
    layers the benchmark times, every token against the reference (appended
    K/V included). Then, as a report and not a gate, the same GPU output
    against the reference that rounds only the cache entries (every
    activation kept in float64): how far the result depends on rounding the
    activations the layer stores."""
    wl = W.full_b64() if which == "full_b64" else W.sliding_b256()
    gpu, step = run_layer(wl)
    ref, tie = reference(wl, gpu)
    compare_layer(wl, gpu, step, ref)
    kv = O.decode_layer(wl, kv_only=True)
    k = wl.shape.top_k
    gap_ok = ~PT.near_tie_tokens(kv["logits"], k)
    flips = (np.sort(gpu["idx"], 1) != np.sort(kv["idx"], 1)).any(1)
    both = ~flips
    print(f"\n  {which}: vs the storage-rounding reference: out max-abs "
          f"{np.abs(gpu['out'] - ref['out']).max():.3e}, rel-L2 {PT.rel_l2(gpu['out'], ref['out']):.3e}, "
          f"near ties {int(tie.sum())}"
          f"\n  {which}: vs the cache-only-rounding reference: out max-abs "
          f"{np.abs(gpu['out'] - kv['out']).max():.3e}, rel-L2 {PT.rel_l2(gpu['out'], kv['out']):.3e} "
          f"(same sets: max-abs {np.abs(gpu['out'] - kv['out'])[both].max(initial=0):.3e}), "
          f"router set flips {int(flips.sum())} of {wl.n_tokens}, "
          f"{int((flips & gap_ok).sum())} of them at a reference gap above 1e-3")


# ---------------------------------------------------------------------------------- MXFP4 experts


def _mxfp4_shape(small=True):
    if small:
        return replace(W.GPT_OSS_20B, hidden=256, n_q_heads=8, n_kv_heads=2, head_dim=64, n_experts=8,
                       top_k=2, ffn_dim=256, expert_fmt="mxfp4")
    return replace(W.GPT_OSS_20B, expert_fmt="mxfp4")


@pytest.mark.parametrize("small", [True, False])
def test_mxfp4_experts_layer(small):
    shape = _mxfp4_shape(small)
    ctx = [0, 15, 16, 200, 1100] if small else [3, 129, 700, 2049]
    wl = W.custom(shape, ctx, np.ones(len(ctx)), 1061, sink_std=0.5)
    gpu, step = run_layer(wl)
    compare_layer(wl, gpu, step)


def test_mxfp4_bad_scale_sets_device_error():
    shape = _mxfp4_shape(True)
    wl = W.custom(shape, [10, 20], np.ones(2), 1062)
    wl.weights["w_gu_scales"] = wl.weights["w_gu_scales"].clone()
    wl.weights["w_gu_scales"][:, 0, 0] = 255  # NaN scale in every expert's first row
    dw = mcpu.DeviceWeights(shape, wl.weights)
    h = W.synth_normal(3, 4, (2, shape.hidden)).cuda()
    out = torch.empty_like(h)
    ws = mcpu.workspace(mcpu.moe_forward_workspace_size(shape, 2))
    mcpu.moe_forward(shape, dw, h, out, None, None, None, ws)
    assert mcpu.mcpu_check_device_errors(ws) & mcpu.DEVERR_MXFP4


# ---------------------------------------------------------------------------------- many rows per matrix


def _moe_shape(hidden, ffn, fmt):
    return replace(W.GPT_OSS_20B, hidden=hidden, n_q_heads=8, n_kv_heads=2, head_dim=64, n_experts=8, top_k=2,
                   ffn_dim=ffn, expert_fmt=fmt)


def _moe_forward_check(s, T, seed, h_seed):
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
    weights = O.Weights(s, wl.weights)
    ref = O.moe(s, weights, h)
    tie = PT.check_router(idx.cpu().numpy(), ref["idx"], ref["logits"], s.top_k)
    if tie.any():
        f = ref["idx"].copy()
        f[tie] = idx.cpu().numpy()[tie]
        ref = O.moe(s, weights, h, force_idx=f)
    PT.check("moe out", _np(out), ref["out"], "bf16")


@pytest.mark.parametrize("T", [16, 50])
def test_projections_packed_weights_bitwise_equal_row_major(T):
    """Decode steps of up to 64 tokens: the split projections read the
    streaming-order copies of w_qkv and w_o when they are given (QKV in its
    rotary block order, row by row from the copy), multiplying the same
    operands in the same order, so the layer's outputs equal those from the
    row-major weights bit for bit."""
    rng = np.random.default_rng(1091 + T)
    wl = W.custom(W.GPT_OSS_20B, rng.integers(1, 400, size=T), np.ones(T), 1091 + T)
    packed, step = run_layer(wl)
    assert "w_qkv_packed" in step.weights.t and "w_o_packed" in step.weights.t
    step.weights = mcpu.DeviceWeights(wl.shape, wl.weights, pack=False)
    assert "w_qkv_packed" not in step.weights.t
    step.run()
    torch.cuda.synchronize()
    assert step.device_errors() == 0
    np.testing.assert_array_equal(_np(step.x_out), packed["out"])
    np.testing.assert_array_equal(step.topk_idx.cpu().numpy(), packed["idx"])


@pytest.mark.parametrize("fmt", ["dense", "mxfp4"])
@pytest.mark.parametrize("hidden,ffn,T", [(512, 512, 1000), (1024, 1024, 3600)])
def test_moe_forward_many_rows(fmt, hidden, ffn, T):
    """Expert GEMMs with hundreds of rows per expert (64- and 128-row tiles,
    ragged last tiles in every group)."""
    _moe_forward_check(_moe_shape(hidden, ffn, fmt), T, 1071 + hidden, 4)


@pytest.mark.parametrize("fmt,T", [("dense", 40), ("mxfp4", 200), ("mxfp4", 350)])
def test_moe_forward_slab_rows(fmt, T):
    """Expert GEMMs on weight slabs: about 10 (bf16 weights, from the
    streaming-order copy; 64-row items) or 50 and 90 (MXFP4; 128-row items)
    rows per expert, so every group is one item with a ragged end; 576 = 4.5
    reduction chunks, so the last chunk is a half."""
    _moe_forward_check(_moe_shape(576, 576, fmt), T, 1075, 6)


def test_moe_forward_mxfp4_slab_hot_expert():
    """MXFP4 slabs with one expert far above the average: every one of 300
    tokens picks expert 0 (300 rows: two full 128-row items and a ragged
    third) and one of experts 1-7 (about 43 rows each, one item), 75 rows per
    expert on average."""
    s = _moe_shape(576, 576, "mxfp4")
    T = 300
    wl = W.custom(s, [4], [1], 1095)
    dw = mcpu.DeviceWeights(s, wl.weights)
    h = W.synth_normal(9, 10, (T, s.hidden))
    force = np.stack([np.zeros(T, dtype=np.int32), 1 + np.arange(T, dtype=np.int32) % 7], axis=1)
    out = torch.empty((T, s.hidden), device="cuda")
    ws = mcpu.workspace(mcpu.moe_forward_workspace_size(s, T))
    mcpu.moe_forward(s, dw, h.cuda(), out, None, None, torch.from_numpy(force).cuda(), ws)
    torch.cuda.synchronize()
    assert mcpu.mcpu_check_device_errors(ws) == 0
    ref = O.moe(s, O.Weights(s, wl.weights), h, force_idx=force)
    PT.check("moe out", _np(out), ref["out"], "bf16")


def test_dense_projections_ragged_rows_sampled():
    """300 decode tokens: the dense projections take 64-row tiles with a ragged
    last tile; compared on sampled sequences."""
    rng = np.random.default_rng(1081)
    ctx = rng.integers(1, 400, size=300)
    wl = W.custom(W.GPT_OSS_20B, ctx, np.ones(300), 1081)
    gpu, step = run_layer(wl)
    seqs = sorted({0, 63, 64, 255, 256, 299} | {int(b) for b in rng.choice(300, 4, replace=False)})
    sub, rows = W.restrict(wl, seqs)
    g = {k: v[rows] for k, v in gpu.items()}
    ref, _ = reference(sub, g)
    compare_layer(sub, g, None, ref)


def test_pack_weights_layout_bit_exact():
    """mcpu_pack_weights writes the documented streaming order, computed here on
    the host piece by piece, with zeros past the last column (192 columns = 1.5
    chunks of 128)."""
    rng = np.random.default_rng(1077)
    g, rows, cols = 3, 48, 192
    w = torch.from_numpy(rng.standard_normal((g, rows, cols)).astype(np.float32)).to(torch.bfloat16)
    packed = mcpu.packed_weights(w.cuda())
    torch.cuda.synchronize()
    got = packed.cpu().numpy().view(np.uint16).reshape(-1, 8)
    src = w.view(torch.int16).numpy().view(np.uint16)
    want = np.zeros_like(got)
    i = 0
    for e in range(g):
        for rb in range(rows // 16):
            for c in range(-(-cols // 128)):
                for t in range(4):
                    for lane in range(64):
                        col = 128 * c + 32 * t + 8 * (lane // 16)
                        if col < cols:
                            want[i] = src[e, 16 * rb + lane % 16, col:col + 8]
                        i += 1
    assert i == got.shape[0]
    np.testing.assert_array_equal(got, want)


@pytest.mark.parametrize("T", [40, 16384])
def test_moe_forward_packed_weights_bitwise_equal_row_major(T):
    """Short expert groups (40 tokens: weight slabs) and 256-row tiles (16384
    tokens: the direct-to-LDS GEMM) read the streaming-order copy when it is
    given; the products see the same operands in the same order, so the
    outputs are bit-identical to those from the row-major weights."""
    s = _moe_shape(576, 576, "dense")
    wl = W.custom(s, [4], [1], 1075)
    h = W.synth_normal(9, 6, (T, s.hidden)).cuda()
    outs = []
    for pack in (False, True):
        dw = mcpu.DeviceWeights(s, wl.weights, pack=pack)
        assert ("w_gu_packed" in dw.t) == pack
        out = torch.empty((T, s.hidden), device="cuda")
        ws = mcpu.workspace(mcpu.moe_forward_workspace_size(s, T))
        mcpu.moe_forward(s, dw, h, out, None, None, None, ws)
        torch.cuda.synchronize()
        assert mcpu.mcpu_check_device_errors(ws) == 0
        outs.append(out.cpu())
    assert torch.equal(outs[0], outs[1])


def test_split_projections_repeatable_sampled():
    """50 decode tokens: the dense projections split their reduction over
    workgroups, one ragged 64-row tile and a reduction ending in half a chunk
    (2880 = 22.5 x 128); a second run is bit-identical (partial tiles are
    summed in split order whatever order they arrive in), and sampled
    sequences match the oracle."""
    rng = np.random.default_rng(1083)
    ctx = rng.integers(1, 400, size=50)
    wl = W.custom(W.GPT_OSS_20B, ctx, np.ones(50), 1083)
    gpu, step = run_layer(wl)
    again, _ = run_layer(wl)
    for k in gpu:
        np.testing.assert_array_equal(gpu[k], again[k])
    seqs = sorted({0, 31, 48, 49} | {int(b) for b in rng.choice(50, 4, replace=False)})
    sub, rows = W.restrict(wl, seqs)
    g = {k: v[rows] for k, v in gpu.items()}
    ref, _ = reference(sub, g)
    compare_layer(sub, g, None, ref)


@pytest.mark.parametrize("fmt", ["dense", "mxfp4"])
def test_moe_forward_large_groups_sampled(fmt):
    """16384 tokens routed over the experts (thousands of rows each): the
    128 x 128-tile path with many tiles per group; tokens are independent given their routing, so a seeded sample of
    rows is compared (the grouping still covers every token)."""
    s = _moe_shape(1024, 1024, fmt)
    T = 16384
    wl = W.custom(s, [4], [1], 1091)
    dw = mcpu.DeviceWeights(s, wl.weights)
    h = W.synth_normal(9, 5, (T, s.hidden))
    out = torch.empty((T, s.hidden), device="cuda")
    idx = torch.empty((T, s.top_k), dtype=torch.int32, device="cuda")
    wt = torch.empty((T, s.top_k), device="cuda")
    ws = mcpu.workspace(mcpu.moe_forward_workspace_size(s, T))
    mcpu.moe_forward(s, dw, h.cuda(), out, idx, wt, None, ws)
    torch.cuda.synchronize()
    assert mcpu.mcpu_check_device_errors(ws) == 0
    rows = np.sort(np.random.default_rng(3).choice(T, 96, replace=False))
    rows[0], rows[-1] = 0, T - 1
    weights = O.Weights(s, wl.weights)
    ref = O.moe(s, weights, h[torch.from_numpy(rows)])
    g_idx = idx.cpu().numpy()[rows]
    tie = PT.check_router(g_idx, ref["idx"], ref["logits"], s.top_k)
    if tie.any():
        f = ref["idx"].copy()
        f[tie] = g_idx[tie]
        ref = O.moe(s, weights, h[torch.from_numpy(rows)], force_idx=f)
    PT.check("moe out", _np(out)[rows], ref["out"], "bf16")


def test_dense_projections_large_rows_sampled():
    """8200 decode tokens: the dense projections take 128 x 128 tiles with a
    ragged last tile; compared on sampled sequences."""
    rng = np.random.default_rng(1093)
    ctx = rng.integers(1, 64, size=8200)
    wl = W.custom(W.GPT_OSS_20B, ctx, np.ones(8200), 1093)
    step = mcpu.DeviceStep(wl)
    step.run()
    torch.cuda.synchronize()
    assert step.device_errors() == 0
    seqs = sorted({0, 255, 256, 8191, 8199} | {int(b) for b in rng.choice(8200, 4, replace=False)})
    sub, rows = W.restrict(wl, seqs)
    r = torch.from_numpy(np.asarray(rows, np.int64)).cuda()
    g = dict(out=_np(step.x_out.index_select(0, r)), idx=step.topk_idx.index_select(0, r).cpu().numpy())
    ref, _ = reference(sub, g)
    PT.check("out", g["out"], ref["out"], "bf16")
