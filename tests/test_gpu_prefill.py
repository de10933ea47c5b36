"""Chunked prefill (tool observations appended as multi-token chunks) on the
GPU against the CPU reference: whole layers with mixed decode and prefill
sequences, the attention call alone under sink stress and page permutation,
and the full-size mixed step (192 decode sequences plus 64 chunks of
256-4096 tokens) on sampled sequences.

Sequences adding 16 or more tokens take the prefill kernel (blocks of 32
tokens for 8 query heads per KV head, 64 for 4); shorter additions take the
split-K decode path, so the cases below cover both sides of that boundary,
ragged last blocks, empty contexts and windows shorter than the chunk.
"""
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


def test_prefill_tiny_f32_layer():
    shape = W.TINY  # 4 query heads per KV head: 64-token blocks
    wl = W.custom(shape, [0, 10, 100, 250, 3], [20, 70, 1, 130, 15], 1101, sink_std=1.0)
    gpu, step = run_layer(wl)
    compare_layer(wl, gpu, step)


@pytest.mark.parametrize("hq,hkv", [(16, 1), (4, 2)])
def test_prefill_head_groupings_without_prefill_kernel(hq, hkv):
    """16 and 2 query heads per KV head have no prefill-kernel instance: their
    chunks go to split-K attention, with the same results."""
    shape = replace(W.TINY, n_q_heads=hq, n_kv_heads=hkv)
    wl = W.custom(shape, [0, 10, 100, 3], [20, 70, 1, 33], 1105 + hq, sink_std=1.0)
    gpu, step = run_layer(wl)
    compare_layer(wl, gpu, step)


@pytest.mark.parametrize("window", [0, 128])
def test_prefill_bf16_layer(window):
    shape = replace(W.GPT_OSS_20B, window=window)
    wl = W.custom(shape, [0, 3, 200, 1500, 40], [40, 17, 1, 300, 15], 1102 + window, sink_std=0.5)
    gpu, step = run_layer(wl)
    compare_layer(wl, gpu, step)


def _attention(wl, sinks, pool_k, pool_v, page_table, q_scale=1.0):
    s = wl.shape
    T = wl.n_tokens
    q = W.synth_normal(wl.seed, 901, (T, s.n_q_heads, s.head_dim), std=q_scale, dtype=s.torch_dtype)
    pool = mcpu.KVPool(s, pool_k.cuda(), pool_v.cuda())
    o = torch.empty((T, s.n_q_heads * s.head_dim), dtype=s.torch_dtype, device="cuda")
    ws = mcpu.workspace(mcpu.paged_attention_workspace_size(s, wl.batch, T))
    mcpu.paged_attention(s, sinks.cuda(), pool, torch.from_numpy(page_table).cuda(),
                         torch.from_numpy(wl.seq_lens).cuda(), torch.from_numpy(wl.cu_q).cuda(),
                         wl.seq_lens, wl.cu_q, q.cuda(), o, ws)
    torch.cuda.synchronize()
    assert mcpu.mcpu_check_device_errors(ws) == 0
    return q, o.cpu()


@pytest.mark.parametrize("window", [0, 128])
def test_prefill_attention_sink_stress_and_page_permutation(window):
    """Sinks far above and far below the scores, and the same step with the
    pool's pages renumbered: identical bits."""
    shape = replace(W.GPT_OSS_20B, window=window)
    wl = W.custom(shape, [0, 700, 31, 16], [64, 100, 33, 1], 1111 + window, weights=False)
    sinks = torch.from_numpy(np.tile([12.0, -12.0, 0.0, 3.0], shape.n_q_heads // 4).astype(np.float32))
    q, o = _attention(wl, sinks, wl.k_pool, wl.v_pool, wl.page_table)
    tok_seq = np.repeat(np.arange(wl.batch), wl.q_lens)
    tok_pos = np.concatenate([wl.seq_lens[b] + np.arange(wl.q_lens[b]) for b in range(wl.batch)])
    ref = O.attention(shape, tok_seq, tok_pos, q, wl.k_pool, wl.v_pool, wl.page_table, sinks)
    PT.check("prefill attention", o.float().numpy().reshape(ref.shape), ref, shape.dtype)
    perm = np.random.default_rng(7).permutation(wl.n_pages).astype(np.int32)
    inv = np.argsort(perm).astype(np.int32)
    k2 = torch.empty_like(wl.k_pool)
    v2 = torch.empty_like(wl.v_pool)
    k2[torch.from_numpy(inv).long()] = wl.k_pool
    v2[torch.from_numpy(inv).long()] = wl.v_pool
    pt2 = np.where(wl.page_table >= 0, inv[np.maximum(wl.page_table, 0)], -1).astype(np.int32)
    _, o2 = _attention(wl, sinks, k2, v2, pt2)
    assert torch.equal(o.view(torch.int16), o2.view(torch.int16))


@pytest.mark.parametrize("window", [0, 128])
def test_prefill_attention_large_scores_and_extreme_sinks(window):
    """Queries scaled x 50 (scores up to about 200, so the lazy rescale of the
    running maximum is taken on most steps) with sinks of +30 and -30: the
    max-subtracted softmax stays finite and matches the reference."""
    shape = replace(W.GPT_OSS_20B, window=window)
    wl = W.custom(shape, [0, 900, 47, 16], [96, 130, 40, 1], 1113 + window, weights=False)
    sinks = torch.from_numpy(np.tile([30.0, -30.0, 0.5, 4.0], shape.n_q_heads // 4).astype(np.float32))
    q, o = _attention(wl, sinks, wl.k_pool, wl.v_pool, wl.page_table, q_scale=50.0)
    tok_seq = np.repeat(np.arange(wl.batch), wl.q_lens)
    tok_pos = np.concatenate([wl.seq_lens[b] + np.arange(wl.q_lens[b]) for b in range(wl.batch)])
    ref = O.attention(shape, tok_seq, tok_pos, q, wl.k_pool, wl.v_pool, wl.page_table, sinks)
    got = o.float().numpy().reshape(ref.shape)
    assert np.isfinite(got).all()
    PT.check("prefill attention (q x 50, sinks +-30)", got, ref, shape.dtype)
    assert np.abs(got[:, 1::4]).max() > 0.1   # the -30 sink heads: peaked, not averaged away


def _run_layer_rows(wl, rows):
    """decode_layer on the whole step; only the given token rows come back."""
    step = mcpu.DeviceStep(wl)
    s = wl.shape
    T = wl.n_tokens
    taps_t = dict(q=torch.empty((T, s.n_q_heads, s.head_dim), dtype=s.torch_dtype, device="cuda"),
                  o=torch.empty((T, s.attn_dim), dtype=s.torch_dtype, device="cuda"),
                  h1=torch.empty((T, s.hidden), dtype=torch.float32, device="cuda"))
    step.run(mcpu.Taps(q=taps_t["q"].data_ptr(), o=taps_t["o"].data_ptr(), h1=taps_t["h1"].data_ptr()))
    torch.cuda.synchronize()
    assert step.device_errors() == 0
    r = torch.from_numpy(np.asarray(rows, np.int64)).cuda()
    pick = lambda t: t.index_select(0, r).float().cpu().numpy().astype(np.float64)
    out = dict(out=pick(step.x_out), idx=step.topk_idx.index_select(0, r).cpu().numpy(), w=pick(step.topk_w),
               q=pick(taps_t["q"]), o=pick(taps_t["o"]), h1=pick(taps_t["h1"]))
    finite = bool(torch.isfinite(step.x_out).all())
    wsum = step.topk_w.sum(1)
    wsum_ok = bool(((wsum - 1).abs() <= 1e-5).all())
    return out, finite, wsum_ok


def test_mixed_step_full_size_sampled():
    """The 192 + 64 sequence mixed step at full size (151k tokens), compared on
    two decode sequences and the prefill sequence with the shortest chunk."""
    wl = W.mixed_prefill()
    dec = np.nonzero(wl.q_lens == 1)[0]
    pre = np.nonzero(wl.q_lens > 1)[0]
    seqs = sorted({int(dec[np.argmax(wl.seq_lens[dec])]), int(dec[0]), int(pre[np.argmin(wl.q_lens[pre])])})
    sub, rows = W.restrict(wl, seqs)
    g, finite, wsum_ok = _run_layer_rows(wl, rows)
    assert finite and wsum_ok
    ref, _ = reference(sub, g)
    compare_layer(sub, g, None, ref)


def test_mixed_step_full_size_longest_chunk_sampled():
    """The full-size mixed step on the prefill sequence with the longest
    context among those adding at least 2048 tokens: every chunk token is
    appended by the reference, and a seeded subset of its rows (first, last
    and eight others) goes through attention, the output projection and the
    MoE, so the chunk's ring of pages is compared at full depth."""
    wl = W.mixed_prefill()
    pre = np.nonzero(wl.q_lens >= 2048)[0]
    b = int(pre[np.argmax(wl.seq_lens[pre])])
    sub, rows = W.restrict(wl, [b])
    n = int(wl.q_lens[b])
    rng = np.random.default_rng(1114)
    local = np.unique(np.concatenate([[0, n - 1], rng.choice(n, 8, replace=False)])).astype(np.int32)
    g, finite, wsum_ok = _run_layer_rows(wl, np.asarray(rows)[local])
    assert finite and wsum_ok
    print(f"  sequence {b}: {int(wl.seq_lens[b])} cached + {n} new tokens, rows {local.tolist()}")
    ref = O.decode_layer(sub, rows=local)
    tie = PT.check_router(g["idx"], ref["idx"], ref["logits"], sub.shape.top_k)
    if tie.any():
        force = np.zeros((sub.n_tokens, sub.shape.top_k), np.int32)
        force[local] = ref["idx"]
        force[local[tie]] = g["idx"][tie]
        ref = O.decode_layer(sub, rows=local, force_idx=force)
    compare_layer(sub, g, None, ref)
