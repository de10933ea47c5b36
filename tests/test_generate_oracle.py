"""Pins of the trajectory reference (oracle/generate.py), CPU only: one
causal prefill of a whole trajectory gives every position the same residual
row as feeding the trajectory one token at a time through every layer with
the caches carried along (and the same as feeding it in uneven chunks)."""
import numpy as np
import torch

from oracle import generate as OG
from oracle import oracle as O
from paper_2608_22167_amd import workload as W
from paper_2608_22167_amd.generate import GenSpec

SMALL = W.replace(W.GPT_OSS_20B, hidden=128, n_q_heads=4, n_kv_heads=2, head_dim=32, n_experts=4, top_k=2,
                  ffn_dim=128)


def _setup(window=16, n_layers=3, vocab=512):
    spec = GenSpec(n_layers=n_layers, base=SMALL, vocab=vocab, window=window, max_ctx=256)
    ss = spec.stack_spec()
    lw = [W.stack_weights_host(ss, i) for i in range(n_layers)]
    emb = W.lm_weights_host(spec.seed, SMALL.hidden, vocab)["embed"]
    return spec, ss, lw, emb


def _chunked(ss, lw, emb, tokens, chunks):
    """The trajectory fed chunk by chunk (sizes `chunks`), caches carried."""
    N = len(tokens)
    n_pages = (N + 15) // 16
    pt = np.arange(n_pages, dtype=np.int32)[None, :]
    pools = []
    for i in range(ss.n_layers):
        s = ss.shape(i)
        shp = (n_pages, s.n_kv_heads, 16, s.head_dim)
        pools.append([torch.zeros(shp, dtype=torch.bfloat16), torch.zeros(shp, dtype=torch.bfloat16)])
    rows, start = [], 0
    for q in chunks:
        x = emb[torch.from_numpy(np.asarray(tokens[start:start + q]))].double()
        for i in range(ss.n_layers):
            wl = W.Workload(name="chunk", shape=ss.shape(i), seed=ss.seed, seq_lens=np.array([start], np.int32),
                            q_lens=np.array([q], np.int32), page_table=pt, n_pages=n_pages, weights=lw[i])
            wl.k_pool, wl.v_pool = pools[i]
            wl.x_in = x
            r = O.decode_layer(wl)
            pools[i] = [torch.from_numpy(r["k_pool"]), torch.from_numpy(r["v_pool"])]
            x = torch.from_numpy(r["out"])
        rows.append(x.numpy())
        start += q
    return np.concatenate(rows)


def test_whole_trajectory_prefill_equals_token_by_token():
    spec, ss, lw, emb = _setup()
    tokens = np.random.default_rng(1).integers(0, spec.vocab, 37)
    whole = OG.trajectory_rows(ss, lw, emb, tokens)
    one = _chunked(ss, lw, emb, tokens, [1] * len(tokens))
    np.testing.assert_allclose(whole, one, rtol=1e-10, atol=1e-10)


def test_whole_trajectory_prefill_equals_uneven_chunks():
    spec, ss, lw, emb = _setup(window=20)
    tokens = np.random.default_rng(2).integers(0, spec.vocab, 50)
    whole = OG.trajectory_rows(ss, lw, emb, tokens)
    np.testing.assert_allclose(whole, _chunked(ss, lw, emb, tokens, [7, 1, 1, 25, 16]), rtol=1e-10, atol=1e-10)


def test_window_layers_see_only_their_window():
    """Changing a token more than a window before position p changes row p
    only through the full-attention layers: with every layer windowed (one
    layer, even index), row p is unchanged."""
    spec, ss, lw, emb = _setup(window=16, n_layers=1)
    tokens = np.random.default_rng(3).integers(0, spec.vocab, 40)
    a = OG.trajectory_rows(ss, lw, emb, tokens)
    t2 = tokens.copy()
    t2[2] = (t2[2] + 1) % spec.vocab
    b = OG.trajectory_rows(ss, lw, emb, t2)
    np.testing.assert_array_equal(a[19:], b[19:])     # positions 19.. see keys 4..: token 2 is outside
    assert np.abs(a[2:18] - b[2:18]).max() > 0
