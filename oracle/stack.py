"""CPU reference of the layer stack on sampled sequences. TEST INFRASTRUCTURE ONLY.

Each sampled sequence is independent of the others given its own cache pages,
so the reference restricts the step to the sample: it regenerates on the host
exactly the pages those sequences read (the generator is counter based) and
evaluates the per-layer reference layer by layer. Each layer is evaluated
twice: once to learn the routing (which does not depend on the expert
weights), then, after drawing and dequantising only the experts that routing
uses, with that selection forced.

Three ways to chain the layers:
  free running      the reference's own output feeds the next layer; wherever
                    its k-th and (k+1)-th fp32 router logits lie within 1e-3,
                    the GPU's selection (if given) is used, since both are then
                    correct; elsewhere the selections must agree exactly;
  teacher forced    every layer takes the GPU's own input to that layer
                    (`inputs`), so each layer is checked at the single-layer
                    bar however deep it sits;
  following the GPU the reference adopts the GPU's selection at every layer
                    (`follow_gpu`), which isolates the numerical drift of a
                    deep chain once teacher forcing has shown every selection
                    correct.
"""
from __future__ import annotations

import numpy as np
import torch

from oracle import oracle as O

TIE_GAP = 1e-3


def _near_ties(logits, k):
    lf = np.sort(np.asarray(logits, np.float32), axis=1)[:, ::-1]
    return (lf[:, k - 1] - lf[:, k]).astype(np.float64) <= TIE_GAP


def reference_stack(spec, seqs, n_layers=None, gpu_idx=None, inputs=None, follow_gpu=False):
    """seqs: sampled sequence ids; gpu_idx: [L][B][k] selections of the GPU run;
    inputs: per-layer input rows [n, H] of the sampled sequences (teacher forcing).
    Returns (final residual [n, H] float64, per-layer dicts with the layer's
    output `out`, selection `idx`, near-tie mask `ties` and `mismatch`, the rows
    whose GPU selection differs from the reference's outside a near tie)."""
    from paper_2608_22167_amd import workload as W
    seqs = np.asarray(sorted(int(s) for s in seqs))
    L = spec.n_layers if n_layers is None else n_layers
    if follow_gpu and gpu_idx is None:
        raise ValueError("follow_gpu needs the GPU's selections")
    x = W.stack_x_in(spec)[torch.from_numpy(seqs)].double().numpy()
    info = []
    s0 = spec.shape(0)
    E, I, H = s0.n_experts, s0.ffn_dim, s0.hidden
    # dense fp32 expert arrays reused by every layer: the routing pass never
    # reads them, the second pass reads only the experts re-drawn for the layer
    w_gu = np.zeros((E, 2 * I, H), np.float32)
    w_d = np.zeros((E, H, I), np.float32)
    for layer in range(L):
        if inputs is not None:
            x = np.asarray(inputs[layer], np.float64)
        s = spec.shape(layer)
        pt = spec.page_table(layer)[seqs]
        used = np.unique(pt[pt >= 0])
        remap = -np.ones(spec.n_pages(layer), np.int64)
        remap[used] = np.arange(len(used))
        Wd = W.stack_weights_host(spec, layer, experts=[])
        Wd["w_gu"], Wd["w_d"] = w_gu, w_d
        sub = W.Workload(name="stack_sample", shape=s, seed=spec.seed, seq_lens=spec.seq_lens[seqs],
                         q_lens=np.ones(len(seqs), np.int32),
                         page_table=np.where(pt >= 0, remap[np.maximum(pt, 0)], -1).astype(np.int32),
                         n_pages=len(used), weights=Wd)
        sub.k_pool = W.stack_pages_host(spec, layer, "k", used)
        sub.v_pool = W.stack_pages_host(spec, layer, "v", used)
        sub.x_in = torch.from_numpy(x)
        weights = O.Weights(s, Wd)
        g = None if gpu_idx is None else np.asarray(gpu_idx[layer])[seqs]
        if follow_gpu:
            sel, ties, mismatch = g.copy(), np.zeros(len(seqs), bool), np.zeros(len(seqs), bool)
        else:
            # routing pass (expert weights are still zero)
            ra = O.decode_layer(sub, weights)
            sel = ra["idx"].copy()
            ties = _near_ties(ra["logits"], s.top_k)
            mismatch = np.zeros(len(seqs), bool)
            if g is not None:
                mismatch = (~ties) & (np.sort(g, 1) != np.sort(sel, 1)).any(1)
                sel[ties] = g[ties]
        # draw and dequantise only the experts the sample uses
        for e in np.unique(sel):
            e = int(e)
            for key, arr, rows, cols in (("w_gu", w_gu, 2 * I, H), ("w_d", w_d, H, I)):
                codes = W.synth_bytes(spec.seed, spec.tid(layer, key + "_codes"), (rows, cols // 2),
                                      offset=e * rows * (cols // 2))
                raw = W.synth_bytes(spec.seed, spec.tid(layer, key + "_scales"), (rows, cols // 32),
                                    offset=e * rows * (cols // 32))
                O.mxfp4_dequant(codes, 117 + raw % 3, rows, cols, out=arr[e])
        rb = O.decode_layer(sub, weights, force_idx=sel)
        x = rb["out"]
        info.append(dict(out=x, idx=sel, ties=ties, mismatch=mismatch))
    return x, info
