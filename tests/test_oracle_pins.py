"""Pins of the CPU reference (oracle/) against things other than itself.

Each test ties one part of the reference to an independent fact: a dense
brute force with explicit masks (tests/bruteforce.py), a closed form, a
library routine in a special case, or an invariant. A plausible slip in the
reference (dropped sink, wrong window bound, swapped RoPE pair, wrong GQA
head mapping, gate/up swap, wrong nibble order, ...) fails at least one.
"""
import math

import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2608_22167_amd import workload as W
from tests import bruteforce as BF

RNG = np.random.default_rng(7)


def _tiny_attention_case(shape, ctx, seed, sink_std=0.02, window=None):
    if window is not None:
        from dataclasses import replace
        shape = replace(shape, window=window)
    wl = W.custom(shape, ctx, np.ones(len(ctx)), seed, sink_std=sink_std)
    return wl


# ------------------------------------------------------------------ bfloat16


def test_round_bf16_matches_torch_on_fp32_values():
    x = np.concatenate([RNG.standard_normal(20000) * 10.0 ** RNG.integers(-30, 30, 20000),
                        [1e-40, -3e-39, 3.3e38, 65504.0]]).astype(np.float32)
    ours = O.round_bf16(x.astype(np.float64))
    ref = torch.from_numpy(x).to(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(ours, ref)


def test_round_bf16_ties_to_even():
    # bfloat16 keeps 8 significant bits: the spacing just above 1 is 2^-7.
    assert O.lib().orc_round_bf16(1.0 + 2.0 ** -8) == 1.0                 # tie -> even (1.0)
    assert O.lib().orc_round_bf16(1.0 + 3 * 2.0 ** -8) == 1.0 + 2.0 ** -6  # tie -> even
    assert O.lib().orc_round_bf16(1.0 + 2.0 ** -8 + 2.0 ** -30) == 1.0 + 2.0 ** -7
    assert O.lib().orc_round_bf16(-(1.0 + 2.0 ** -8)) == -1.0


# ------------------------------------------------------------------ RMSNorm


def test_rmsnorm_matches_torch():
    x = RNG.standard_normal((5, 96))
    g = (1 + 0.1 * RNG.standard_normal(96)).astype(np.float32)
    ours = O.rmsnorm(x, g, 1e-5)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (96,), torch.from_numpy(g).double(), 1e-5)
    np.testing.assert_allclose(ours, ref.numpy(), rtol=1e-13, atol=1e-13)


def test_rmsnorm_scale_invariant_without_eps():
    x = RNG.standard_normal((3, 64))
    g = np.ones(64, np.float32)
    np.testing.assert_allclose(O.rmsnorm(37.5 * x, g, 0.0), O.rmsnorm(x, g, 0.0), rtol=1e-13)
    np.testing.assert_allclose((O.rmsnorm(x, g, 0.0) ** 2).mean(-1), 1.0, rtol=1e-13)


# ------------------------------------------------------------------ RoPE


def test_rope_rotates_the_half_split_pair():
    d = 8
    cos, sin = W.rope_table(50, d)
    v = np.zeros(d)
    v[1] = 1.0                       # unit vector in the first element of pair 1
    r = O.rope(v, 7, cos, sin)
    c, s = float(cos[7, 1]), float(sin[7, 1])
    expect = np.zeros(d)
    expect[1], expect[1 + d // 2] = c, s
    np.testing.assert_allclose(r, expect, atol=1e-15)


def test_rope_preserves_pair_norms_and_relative_position():
    d = 64
    cos, sin = W.rope_table(300, d)
    q, k = RNG.standard_normal(d), RNG.standard_normal(d)
    qr = O.rope(q, 123, cos, sin)
    np.testing.assert_allclose(qr[:32] ** 2 + qr[32:] ** 2, q[:32] ** 2 + q[32:] ** 2, rtol=1e-6)
    # q(m) . k(n) depends on m - n only (the table is cos/sin of pos * freq)
    a = O.rope(q, 200, cos, sin) @ O.rope(k, 150, cos, sin)
    b = O.rope(q, 60, cos, sin) @ O.rope(k, 10, cos, sin)
    assert abs(a - b) < 1e-5 * (abs(a) + 1)
    ident_c, ident_s = np.ones((10, d // 2), np.float32), np.zeros((10, d // 2), np.float32)
    np.testing.assert_array_equal(O.rope(q, 3, ident_c, ident_s), q)


# ------------------------------------------------------------------ SwiGLU


def test_swiglu_plain_form_is_silu_times_up():
    g, u = RNG.standard_normal(1000) * 4, RNG.standard_normal(1000) * 4
    ours = O.swiglu(g, u, 1.0, math.inf, 0.0)
    ref = torch.nn.functional.silu(torch.from_numpy(g)) * torch.from_numpy(u)
    np.testing.assert_allclose(ours, ref.numpy(), rtol=1e-12, atol=1e-14)


def test_swiglu_clamped_form_closed_values():
    a, L, b = 1.702, 7.0, 1.0
    sig = lambda z: 1 / (1 + math.exp(-z))
    # gate above the limit is capped; up below -L is clamped
    assert O.lib().orc_swiglu(10.0, 0.0, a, L, b) == pytest.approx(7.0 * sig(a * 7.0) * 1.0, rel=1e-15)
    assert O.lib().orc_swiglu(2.0, -10.0, a, L, b) == pytest.approx(2.0 * sig(a * 2.0) * (-6.0), rel=1e-15)
    assert O.lib().orc_swiglu(-3.0, 8.0, a, L, b) == pytest.approx(-3.0 * sig(-a * 3.0) * 8.0, rel=1e-15)


# ------------------------------------------------------------------ top-k


def test_topk_matches_stable_argsort_with_ties():
    for _ in range(200):
        lg = RNG.integers(-4, 5, size=32).astype(np.float64) * 0.5  # many exact ties
        ours = O.topk(lg, 4)
        ref = np.argsort(-lg.astype(np.float32), kind="stable")[:4]
        np.testing.assert_array_equal(ours, ref)


def test_topk_decides_in_fp32():
    lg = np.zeros(8)
    lg[3] = 1.0
    lg[5] = 1.0 + 1e-12    # equal after rounding to fp32 -> lower index first
    np.testing.assert_array_equal(O.topk(lg, 2), [3, 5])


# ------------------------------------------------------------------ page format


@pytest.mark.parametrize("d", [32, 64])
def test_page_format_roundtrip_and_matches_reshape_definition(d):
    from dataclasses import replace
    shape = replace(W.TINY, head_dim=d)
    k = RNG.standard_normal((5, 2, 16, d)).astype(np.float32)
    v = RNG.standard_normal((5, 2, 16, d)).astype(np.float32)
    kp, vp = O.pool_from_logical(shape, k, v)
    bkp, bvp = BF.pool_from_logical(k, v)
    np.testing.assert_array_equal(kp, bkp)
    np.testing.assert_array_equal(vp, bvp)
    k2, v2 = O.pool_to_logical(shape, kp, vp)
    np.testing.assert_array_equal(k2, k)
    np.testing.assert_array_equal(v2, v)
    # spot check the documented formula: K(slot 5, dim 13) of page 2, head 1
    flat = kp.reshape(5, 2, -1)
    assert flat[2, 1, ((13 // 8) * 16 + 5) * 8 + 13 % 8] == k[2, 1, 5, 13]
    flatv = vp.reshape(5, 2, -1)
    assert flatv[2, 1, (((13 // 16) * 4 + 5 // 4) * 16 + 13 % 16) * 4 + 5 % 4] == v[2, 1, 5, 13]


# ------------------------------------------------------------------ attention


def _attn_inputs(wl, q_scale=1.0, seed=3):
    s = wl.shape
    rng = np.random.default_rng(seed)
    T = wl.batch
    q = rng.standard_normal((T, s.n_q_heads, s.head_dim)) * q_scale
    tok_seq = np.arange(T, dtype=np.int32)
    tok_pos = (wl.seq_lens - 1).astype(np.int32)   # attend over the cached keys only
    return q, tok_seq, tok_pos


def _brute_attention(wl, q, tok_pos, sinks):
    s = wl.shape
    kl, vl = BF.pool_to_logical(wl.k_pool.float().numpy().astype(np.float64),
                                wl.v_pool.float().numpy().astype(np.float64))
    out = []
    for b in range(wl.batch):
        n = int(tok_pos[b]) + 1
        lo = max(0, n - 1 - s.window + 1) if s.window else 0
        K = np.zeros((n, s.n_kv_heads, s.head_dim))
        V = np.zeros_like(K)
        pos = np.arange(lo, n)
        pages = wl.page_table[b][pos // 16]
        K[pos], V[pos] = kl[pages, :, pos % 16, :], vl[pages, :, pos % 16, :]
        out.append(BF.attention_dense(q[b], K, V, n - 1, s.window, sinks, 1 / math.sqrt(s.head_dim)))
    return np.stack(out)


@pytest.mark.parametrize("window", [0, 128])
@pytest.mark.parametrize("sink_std", [0.02, 3.0])
def test_attention_matches_dense_bruteforce(window, sink_std):
    from dataclasses import replace
    shape = replace(W.TINY, window=window)
    wl = W.custom(shape, [1, 15, 16, 17, 127, 129, 200, 301], np.ones(8), 11, sink_std=sink_std)
    q, ts, tp = _attn_inputs(wl)
    ours = O.attention(shape, ts, tp, q, wl.k_pool, wl.v_pool, wl.page_table, wl.weights["sinks"])
    ref = _brute_attention(wl, q, tp, wl.weights["sinks"].double().numpy())
    np.testing.assert_allclose(ours, ref, rtol=1e-12, atol=1e-13)


def test_attention_without_sink_is_sdpa():
    wl = W.custom(W.TINY, [40, 77, 150], np.ones(3), 12)
    q, ts, tp = _attn_inputs(wl)
    ours = O.attention(W.TINY, ts, tp, q, wl.k_pool, wl.v_pool, wl.page_table, None)
    kl, vl = BF.pool_to_logical(wl.k_pool.numpy(), wl.v_pool.numpy())
    for b in range(3):
        n = int(tp[b]) + 1
        K, V = BF.dense_seq(kl, vl, wl.page_table[b], n)
        Kt = torch.from_numpy(K.astype(np.float64)).permute(1, 0, 2).repeat_interleave(4, 0)
        Vt = torch.from_numpy(V.astype(np.float64)).permute(1, 0, 2).repeat_interleave(4, 0)
        qt = torch.from_numpy(q[b]).unsqueeze(1)
        ref = torch.nn.functional.scaled_dot_product_attention(qt, Kt, Vt).squeeze(1)
        np.testing.assert_allclose(ours[b], ref.numpy(), rtol=1e-10, atol=1e-12)


def test_attention_sink_closed_forms():
    # K = 0 and V = 1: every visible key has logit 0, so o = c / (c + e^s) exactly
    wl = W.custom(W.TINY, [30, 64, 100], np.ones(3), 13, sink_std=1.5)
    wl.k_pool.zero_()
    wl.v_pool.fill_(1.0)
    q, ts, tp = _attn_inputs(wl)
    o = O.attention(W.TINY, ts, tp, q, wl.k_pool, wl.v_pool, wl.page_table, wl.weights["sinks"])
    s = wl.weights["sinks"].double().numpy()
    for b in range(3):
        c = int(tp[b]) + 1
        np.testing.assert_allclose(o[b], (c / (c + np.exp(s)))[:, None] * np.ones((1, 32)), rtol=1e-13)
    # V = 1 with random K: o = 1 - sink share, i.e. the softmax-with-sink row sum
    wl2 = W.custom(W.TINY, [30, 64, 100], np.ones(3), 14, sink_std=2.0)
    wl2.v_pool.fill_(1.0)
    q, ts, tp = _attn_inputs(wl2)
    o2 = O.attention(W.TINY, ts, tp, q, wl2.k_pool, wl2.v_pool, wl2.page_table, wl2.weights["sinks"])
    o3 = O.attention(W.TINY, ts, tp, q, wl2.k_pool, wl2.v_pool, wl2.page_table, None)
    np.testing.assert_allclose(o3, 1.0, rtol=1e-13)
    assert (o2 < 1).all() and (o2 > 0).all()
    # large sink: the sink takes (nearly) all the mass
    wl2.weights["sinks"].fill_(30.0)
    o4 = O.attention(W.TINY, ts, tp, q, wl2.k_pool, wl2.v_pool, wl2.page_table, wl2.weights["sinks"])
    assert np.abs(o4).max() < 101 * math.exp(-30 + 10)


def test_attention_large_logits_stay_finite():
    wl = W.custom(W.TINY, [90, 200], np.ones(2), 15)
    q, ts, tp = _attn_inputs(wl, q_scale=50.0)
    ours = O.attention(W.TINY, ts, tp, q, wl.k_pool, wl.v_pool, wl.page_table, wl.weights["sinks"])
    assert np.isfinite(ours).all()
    ref = _brute_attention(wl, q, tp, wl.weights["sinks"].double().numpy())
    np.testing.assert_allclose(ours, ref, rtol=1e-10, atol=1e-12)


def test_attention_page_permutation_is_bitwise_invariant():
    wl = W.custom(W.TINY, [70, 33, 180], np.ones(3), 16)
    q, ts, tp = _attn_inputs(wl)
    a = O.attention(W.TINY, ts, tp, q, wl.k_pool, wl.v_pool, wl.page_table, wl.weights["sinks"])
    perm = np.random.default_rng(1).permutation(wl.n_pages)
    kp, vp = torch.empty_like(wl.k_pool), torch.empty_like(wl.v_pool)
    kp[perm], vp[perm] = wl.k_pool, wl.v_pool
    pt = np.where(wl.page_table >= 0, perm[np.maximum(wl.page_table, 0)], -1).astype(np.int32)
    b = O.attention(W.TINY, ts, tp, q, kp, vp, pt, wl.weights["sinks"])
    np.testing.assert_array_equal(a, b)


def test_attention_window_beyond_context_equals_full():
    from dataclasses import replace
    wl = W.custom(W.TINY, [10, 47, 60], np.ones(3), 17)
    q, ts, tp = _attn_inputs(wl)
    a = O.attention(W.TINY, ts, tp, q, wl.k_pool, wl.v_pool, wl.page_table, wl.weights["sinks"])
    b = O.attention(replace(W.TINY, window=61), ts, tp, q, wl.k_pool, wl.v_pool, wl.page_table,
                    wl.weights["sinks"])
    np.testing.assert_array_equal(a, b)
    c = O.attention(replace(W.TINY, window=20), ts, tp, q, wl.k_pool, wl.v_pool, wl.page_table,
                    wl.weights["sinks"])
    assert not np.allclose(a[2], c[2])


def test_attention_gqa_head_mapping():
    # only KV head 1 carries values: query heads 4..7 (group 1) see them, 0..3 do not
    wl = W.custom(W.TINY, [50], np.ones(1), 18)
    kl, vl = BF.pool_to_logical(wl.k_pool.numpy(), wl.v_pool.numpy())
    vl[:, 0] = 0.0
    _, vp = BF.pool_from_logical(kl, vl)
    q, ts, tp = _attn_inputs(wl)
    o = O.attention(W.TINY, ts, tp, q, wl.k_pool, vp, wl.page_table, None)
    assert np.abs(o[0, :4]).max() == 0.0 and np.abs(o[0, 4:]).min() > 0.0


# ------------------------------------------------------------------ KV append


def test_kv_append_positions_and_rounding():
    from dataclasses import replace
    shape = replace(W.GPT_OSS_20B, hidden=128, n_q_heads=8, n_kv_heads=2, head_dim=64)
    wl = W.custom(shape, [15, 16, 40], np.ones(3), 19, weights=False)
    rng = np.random.default_rng(0)
    kn = rng.standard_normal((3, 2, 64))
    vn = rng.standard_normal((3, 2, 64))
    kp, vp = O.kv_append(shape, [0, 1, 2], wl.seq_lens, kn, vn, wl.k_pool, wl.v_pool, wl.page_table)
    kl, vl = BF.pool_to_logical(kp, vp)
    for b in range(3):
        p = int(wl.seq_lens[b])
        page = wl.page_table[b][p // 16]
        np.testing.assert_array_equal(kl[page, :, p % 16, :], BF.bf16(kn[b]))
        np.testing.assert_array_equal(vl[page, :, p % 16, :], BF.bf16(vn[b]))
    # nothing else changed
    changed = (kp != wl.k_pool.float().numpy()).reshape(wl.n_pages, -1).any(1)
    assert changed.sum() <= 3


# ------------------------------------------------------------------ MoE


def _moe_shape():
    return W.TINY


def test_moe_matches_naive_loop():
    wl = W.tiny_f32(seed=21, batch=6)
    Wt = O.Weights(wl.shape, wl.weights)
    h = np.random.default_rng(1).standard_normal((6, wl.shape.hidden))
    r = O.moe(wl.shape, Wt, h)
    Wn = BF.weights_np(wl.weights)
    hn = BF.rmsnorm(h, Wn["g2"], wl.shape.rms_eps)
    for t in range(6):
        acc, sel, w, lg = BF.moe_token(hn[t], Wn, wl.shape)
        np.testing.assert_array_equal(r["idx"][t], sel)
        np.testing.assert_allclose(r["w"][t], w, rtol=1e-12)
        np.testing.assert_allclose(r["out"][t], h[t] + acc, rtol=1e-11, atol=1e-12)
        np.testing.assert_allclose(r["logits"][t], lg, rtol=1e-11, atol=1e-13)
    np.testing.assert_allclose(r["w"].sum(1), 1.0, rtol=1e-14)


def test_moe_identical_experts_is_dense_ffn():
    wl = W.tiny_f32(seed=22, batch=5)
    Wd = dict(wl.weights)
    for k in ("w_gu", "b_gu", "w_d", "b_d"):
        Wd[k] = Wd[k][:1].expand_as(Wd[k]).contiguous()
    Wt = O.Weights(wl.shape, Wd)
    h = np.random.default_rng(2).standard_normal((5, wl.shape.hidden))
    r = O.moe(wl.shape, Wt, h)
    s = wl.shape
    hn = BF.stored(BF.rmsnorm(h, Wd["g2"].double().numpy(), s.rms_eps), s.dtype)
    gu = hn @ Wd["w_gu"][0].double().numpy().T + Wd["b_gu"][0].double().numpy()
    a = BF.stored(BF.swiglu(gu[:, 0::2], gu[:, 1::2], s.swiglu_alpha, s.swiglu_limit, s.swiglu_beta), s.dtype)
    y = a @ Wd["w_d"][0].double().numpy().T + Wd["b_d"][0].double().numpy()
    np.testing.assert_allclose(r["out"], h + y, rtol=1e-11, atol=1e-12)


def test_moe_top1_is_the_argmax_expert_ffn():
    from dataclasses import replace
    s = replace(W.TINY, top_k=1)
    wl = W.custom(s, [20, 30], np.ones(2), 23)
    Wt = O.Weights(s, wl.weights)
    h = np.random.default_rng(3).standard_normal((2, s.hidden))
    r = O.moe(s, Wt, h)
    Wn = BF.weights_np(wl.weights)
    for t in range(2):
        hn = BF.rmsnorm(h[t:t + 1], Wn["g2"], s.rms_eps)[0]
        e = int(np.argmax(Wn["w_r"] @ hn + Wn["b_r"]))
        assert r["idx"][t, 0] == e and r["w"][t, 0] == 1.0
        gu = Wn["w_gu"][e] @ BF.stored(hn, s.dtype) + Wn["b_gu"][e]
        y = Wn["w_d"][e] @ BF.stored(BF.swiglu(gu[0::2], gu[1::2], s.swiglu_alpha, s.swiglu_limit,
                                               s.swiglu_beta), s.dtype) + Wn["b_d"][e]
        np.testing.assert_allclose(r["out"][t], h[t] + y, rtol=1e-11, atol=1e-12)


def test_moe_expert_permutation_invariance():
    wl = W.tiny_f32(seed=24, batch=4)
    h = np.random.default_rng(4).standard_normal((4, wl.shape.hidden))
    r = O.moe(wl.shape, O.Weights(wl.shape, wl.weights), h)
    perm = np.random.default_rng(5).permutation(wl.shape.n_experts)   # new id -> old id
    Wp = dict(wl.weights)
    for k in ("w_gu", "b_gu", "w_d", "b_d", "w_r", "b_r"):
        Wp[k] = wl.weights[k][torch.from_numpy(perm)].contiguous()
    rp = O.moe(wl.shape, O.Weights(wl.shape, Wp), h)
    np.testing.assert_allclose(rp["out"], r["out"], rtol=1e-12, atol=1e-13)
    np.testing.assert_array_equal(np.sort(perm[rp["idx"]], 1), np.sort(r["idx"], 1))


def test_moe_force_idx_overrides_selection():
    wl = W.tiny_f32(seed=25, batch=3)
    Wt = O.Weights(wl.shape, wl.weights)
    h = np.random.default_rng(6).standard_normal((3, wl.shape.hidden))
    force = np.array([[0, 1], [7, 3], [5, 2]], dtype=np.int32)
    r = O.moe(wl.shape, Wt, h, force_idx=force)
    Wn = BF.weights_np(wl.weights)
    hn = BF.rmsnorm(h, Wn["g2"], wl.shape.rms_eps)
    for t in range(3):
        acc, _, _, _ = BF.moe_token(hn[t], Wn, wl.shape, force=force[t])
        np.testing.assert_allclose(r["out"][t], h[t] + acc, rtol=1e-11, atol=1e-12)


# ------------------------------------------------------------------ whole layer


@pytest.mark.parametrize("kind", ["tiny_f32", "bf16_small", "bf16_window"])
def test_decode_layer_matches_dense_bruteforce(kind):
    from dataclasses import replace
    if kind == "tiny_f32":
        wl = W.tiny_f32(seed=31)
    else:
        shape = replace(W.GPT_OSS_20B, hidden=192, n_q_heads=8, n_kv_heads=2, head_dim=64,
                        n_experts=8, top_k=3, ffn_dim=96, window=128 if kind == "bf16_window" else 0)
        wl = W.custom(shape, [3, 16, 130, 257], np.ones(4), 32, sink_std=1.0)
    r = O.decode_layer(wl)
    ref = BF.decode_layer(wl)
    np.testing.assert_allclose(r["q"], ref["q"], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(r["o"], ref["o"], rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(r["h1"], ref["h1"], rtol=1e-10, atol=1e-12)
    np.testing.assert_array_equal(r["idx"], ref["idx"])
    np.testing.assert_allclose(r["out"], ref["out"], rtol=1e-10, atol=1e-11)


@pytest.mark.parametrize("kind", ["bf16_small", "bf16_window"])
def test_decode_layer_cache_only_rounding_matches_dense_bruteforce(kind):
    """The reporting mode that rounds only the cache entries (no stored
    activations) against the dense brute force with the same rule; it must
    differ from the default mode (the rounding points are real)."""
    from dataclasses import replace
    shape = replace(W.GPT_OSS_20B, hidden=192, n_q_heads=8, n_kv_heads=2, head_dim=64,
                    n_experts=8, top_k=3, ffn_dim=96, window=128 if kind == "bf16_window" else 0)
    wl = W.custom(shape, [3, 16, 130, 257], [1, 3, 1, 2], 33, sink_std=1.0)
    r = O.decode_layer(wl, kv_only=True)
    ref = BF.decode_layer(wl, kv_only=True)
    np.testing.assert_allclose(r["q"], ref["q"], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(r["o"], ref["o"], rtol=1e-10, atol=1e-12)
    np.testing.assert_array_equal(r["idx"], ref["idx"])
    np.testing.assert_allclose(r["out"], ref["out"], rtol=1e-10, atol=1e-11)
    assert np.abs(r["out"] - O.decode_layer(wl)["out"]).max() > 1e-6


def test_decode_layer_row_subset_equals_full_step():
    """Evaluating a subset of rows (every token still appended) returns exactly
    the full step's values at those rows, including a forced selection."""
    from dataclasses import replace
    shape = replace(W.TINY, window=0)
    wl = W.custom(shape, [33, 0, 60, 7], [5, 20, 1, 3], 44)
    full = O.decode_layer(wl)
    rows = np.array([0, 4, 6, 24, 27])
    sub = O.decode_layer(wl, rows=rows)
    for k in ("out", "q", "o", "h1", "idx", "w", "logits", "moe"):
        np.testing.assert_array_equal(sub[k], full[k][rows], err_msg=k)
    np.testing.assert_array_equal(sub["k_pool"], full["k_pool"])
    force = np.tile(np.arange(shape.top_k, dtype=np.int32), (wl.n_tokens, 1))
    fsub = O.decode_layer(wl, rows=rows, force_idx=force)
    np.testing.assert_array_equal(fsub["out"], O.decode_layer(wl, force_idx=force)["out"][rows])


def test_decode_layer_chunk_equals_sequential_decode():
    from dataclasses import replace
    shape = replace(W.TINY, window=0)
    n = 5
    wl = W.custom(shape, [33, 60], [n, 1], 41)
    chunk = O.decode_layer(wl)
    # the same tokens one at a time, each step starting from the previous pools
    kp, vp = wl.k_pool, wl.v_pool
    x = wl.x_in
    outs = []
    for i in range(n):
        seq = W.custom(shape, [33 + i], [1], 41, weights=False, kv=False)
        seq.weights, seq.k_pool, seq.v_pool = wl.weights, kp, vp
        seq.page_table = wl.page_table[:1]
        seq.n_pages = wl.n_pages
        seq.x_in = x[i:i + 1]
        r = O.decode_layer(seq)
        kp, vp = torch.from_numpy(r["k_pool"]), torch.from_numpy(r["v_pool"])
        outs.append(r["out"][0])
    np.testing.assert_allclose(chunk["out"][:n], np.stack(outs), rtol=1e-12, atol=1e-13)


def test_decode_layer_page_permutation_bitwise():
    wl = W.tiny_f32(seed=42)
    a = O.decode_layer(wl)
    perm = np.random.default_rng(9).permutation(wl.n_pages)
    kp, vp = torch.empty_like(wl.k_pool), torch.empty_like(wl.v_pool)
    kp[perm], vp[perm] = wl.k_pool, wl.v_pool
    wl.k_pool, wl.v_pool = kp, vp
    wl.page_table = np.where(wl.page_table >= 0, perm[np.maximum(wl.page_table, 0)], -1).astype(np.int32)
    b = O.decode_layer(wl)
    np.testing.assert_array_equal(a["out"], b["out"])


def test_decode_layer_rejects_missing_page():
    wl = W.tiny_f32(seed=43)
    wl.page_table[1, 0] = -1
    with pytest.raises(ValueError):
        O.decode_layer(wl)


# ------------------------------------------------------------------ MXFP4


def _golden_e2m1():
    import os
    path = os.path.join(os.path.dirname(__file__), "golden", "ocp_mx_fp4_e2m1.txt")
    vals = {}
    for line in open(path):
        line = line.split("#")[0].strip()
        if line:
            code, val = line.split()
            vals[int(code, 2)] = float(val)
    return vals


def test_e2m1_table_matches_ocp_spec():
    gold = _golden_e2m1()
    assert len(gold) == 16
    for code, val in gold.items():
        assert O.e2m1(code) == val


def test_mxfp4_dequant_scales_and_nibble_order():
    rows, cols = 3, 64
    rng = np.random.default_rng(0)
    codes = rng.integers(0, 256, size=(rows, cols // 2), dtype=np.uint8)
    scales = np.array([[127, 100], [0, 200], [130, 127]], dtype=np.uint8)
    out = O.mxfp4_dequant(codes, scales, rows, cols)
    gold = _golden_e2m1()
    for r in range(rows):
        for j in range(cols):
            byte = int(codes[r, j // 2])
            code = byte & 0xF if j % 2 == 0 else byte >> 4
            assert out[r, j] == np.float32(gold[code] * 2.0 ** (int(scales[r, j // 32]) - 127))
    with pytest.raises(ValueError):
        O.mxfp4_dequant(codes, np.full((rows, 2), 255, np.uint8), rows, cols)
