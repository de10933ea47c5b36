"""CPU reference of whole trajectories through the decoder stack. TEST
INFRASTRUCTURE ONLY.

A trajectory's tokens are embedded and run through every layer as one causal
prefill chunk on an empty cache (the single-layer reference with seq_lens 0
and the whole trajectory as the chunk), which by causality gives every
position the residual row that incremental generation reaches one token or
one chunk at a time. The vocabulary head (orc_lm_head) then gives the token a
row samples, or the log-probability of a given next token.
"""
from __future__ import annotations

import numpy as np
import torch

from oracle import oracle as O

PAGE = 16


def trajectory_rows(ss, layer_weights, embed, tokens):
    """Final residual rows [N, H] (float64) of trajectory `tokens` through the
    stack `ss` (a StackSpec), with host layer weights layer_weights[i] (dicts
    as stack_weights_host returns) and the bf16 embedding table."""
    from paper_2608_22167_amd import workload as W
    tokens = np.asarray(tokens, np.int64)
    N = len(tokens)
    x = embed[torch.from_numpy(tokens)].double()
    n_pages = (N + PAGE - 1) // PAGE
    pt = np.arange(n_pages, dtype=np.int32)[None, :]
    for i in range(ss.n_layers):
        s = ss.shape(i)
        wl = W.Workload(name="trajectory", shape=s, seed=ss.seed, seq_lens=np.zeros(1, np.int32),
                        q_lens=np.array([N], np.int32), page_table=pt, n_pages=n_pages, weights=layer_weights[i])
        shp = (n_pages, s.n_kv_heads, PAGE, s.head_dim)
        wl.k_pool = torch.zeros(shp, dtype=torch.bfloat16)
        wl.v_pool = torch.zeros(shp, dtype=torch.bfloat16)
        wl.x_in = x
        x = torch.from_numpy(O.decode_layer(wl)["out"])
    return x.numpy()
