"""CPU reference of the layer stack on sampled sequences. TEST INFRASTRUCTURE ONLY.

Each sampled sequence is independent of the others given its own cache pages,
so the reference restricts the step to the sample: it regenerates on the host
exactly the pages those sequences read (the generator is counter based) and
chains the per-layer reference from the step's input through every layer,
each layer's output feeding the next. Each layer is evaluated twice: once to
learn the routing (which does not depend on the expert weights), then, after
drawing and dequantising only the experts that routing uses, with that
selection forced.

Routing is an argmax, so wherever two experts' logits are closer than the
two computations can be apart, either choice is correct. Given the GPU run's
selections, and optionally its logits, a row whose GPU set differs from the
reference's is accepted when every swapped pair of experts lies within the
row's gap of each other under the reference's logits; the gap is 1e-3, or
twice the row's largest logit difference between the two runs when that is
larger (each side may be off by that much). An accepted row continues with
the GPU's set, one of the correct results; any other difference is a
mismatch.
"""
from __future__ import annotations

import numpy as np
import torch

from oracle import oracle as O

TIE_GAP = 1e-3  # the single-layer bar: the k-th and (k+1)-th fp32 logits within 1e-3


def _swap_ok(ref_logits, ref_sel, gpu_sel, gap):
    """True where each expert the GPU took instead of one of the reference's is
    within gap of it under the reference's logits."""
    ok = np.ones(len(ref_sel), bool)
    for r in range(len(ref_sel)):
        a, b = set(int(e) for e in ref_sel[r]), set(int(e) for e in gpu_sel[r])
        for e_ref in a - b:
            for e_gpu in b - a:
                if ref_logits[r, e_ref] - ref_logits[r, e_gpu] > gap[r]:
                    ok[r] = False
    return ok


def reference_stack(spec, seqs, n_layers=None, gpu_idx=None, gpu_logits=None):
    """seqs: sampled sequence ids; gpu_idx: [L][B][k] selections of the GPU run;
    gpu_logits: [L][B][E] its router logits. Returns (final residual [n, H]
    float64, per-layer dicts with the layer's output `out`, selection `idx`,
    accepted differing rows `adopted`, the rows' logit gaps `gap`, the largest
    logit difference `logit_err` and `mismatch`, the rows whose GPU selection
    is not a correct one)."""
    from paper_2608_22167_amd import workload as W
    seqs = np.asarray(sorted(int(s) for s in seqs))
    L = spec.n_layers if n_layers is None else n_layers
    x = W.stack_x_in(spec)[torch.from_numpy(seqs)].double().numpy()
    info = []
    s0 = spec.shape(0)
    E, I, H = s0.n_experts, s0.ffn_dim, s0.hidden
    # dense fp32 expert arrays reused by every layer: the routing pass never
    # reads them, the second pass reads only the experts re-drawn for the layer
    w_gu = np.zeros((E, 2 * I, H), np.float32)
    w_d = np.zeros((E, H, I), np.float32)
    for layer in range(L):
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
        # routing pass (expert weights are still zero)
        ra = O.decode_layer(sub, weights)
        sel = ra["idx"].copy()
        n = len(seqs)
        mismatch, adopted = np.zeros(n, bool), np.zeros(n, bool)
        gap, logit_err = np.full(n, TIE_GAP), np.zeros(n)
        if gpu_idx is not None:
            g = np.asarray(gpu_idx[layer])[seqs]
            if gpu_logits is not None:
                logit_err = np.abs(np.asarray(gpu_logits[layer], np.float64)[seqs] - ra["logits"]).max(1)
                gap = np.maximum(gap, 2.0 * logit_err)
            differ = (np.sort(g, 1) != np.sort(sel, 1)).any(1)
            ok = _swap_ok(ra["logits"], sel, g, gap)
            adopted = differ & ok
            mismatch = differ & ~ok
            sel[adopted] = g[adopted]
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
        info.append(dict(out=x, idx=sel, adopted=adopted, gap=gap, logit_err=logit_err, mismatch=mismatch))
    return x, info
