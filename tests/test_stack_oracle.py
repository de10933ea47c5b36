"""Pins of the stack reference (oracle/stack.py), CPU only.

The stack reference restricts each layer to a sample of sequences,
regenerates only the pages and experts the sample reads, and learns the
routing in a first pass before drawing the chosen experts. None of that may
change the result: the plain definition of a stack is the single-layer
reference applied layer after layer to the whole batch with every expert
drawn. The tests below compare the two on a small stack, and pin the rule
that accepts a differing expert selection on crafted logits.
"""
from dataclasses import replace

import numpy as np
import pytest
import torch

from oracle import oracle as O
from oracle import stack as OS
from paper_2608_22167_amd import workload as W

SMALL = replace(W.GPT_OSS_20B, hidden=256, n_q_heads=8, n_kv_heads=2, head_dim=64, n_experts=8, top_k=2,
                ffn_dim=256)


# ------------------------------------------------------------------------------- swap rule


def test_swap_ok_accepts_same_sets_in_any_order():
    lg = np.array([[0.5, 0.1, 0.9, -0.2]])
    assert OS.swap_ok(lg, [[2, 0]], [[0, 2]]).all()


def test_swap_ok_within_and_beyond_the_gap():
    # reference top-2 = {0, 1}; expert 2 sits 5e-4 below expert 1, expert 3 sits 2e-3 below
    lg = np.array([[1.0, 0.5, 0.4995, 0.498]] * 3)
    ref = np.array([[0, 1]] * 3)
    gpu = np.array([[0, 2], [0, 3], [2, 3]])
    np.testing.assert_array_equal(OS.swap_ok(lg, ref, gpu, 1e-3), [True, False, False])
    # the same swaps under a wider per-row gap
    np.testing.assert_array_equal(OS.swap_ok(lg, ref, gpu, [1e-3, 3e-3, 3e-3]), [True, True, False])


def test_swap_ok_rejects_displacing_a_far_higher_expert():
    # GPU drops expert 0 (logit 1.0) for expert 2 (0.4995): 0.5005 apart, far beyond the gap,
    # although expert 2 is within the gap of the reference's other pick. A sign slip (the
    # adopted expert's logit minus the displaced one's) or an absolute value of the wrong
    # pair would accept it.
    lg = np.array([[1.0, 0.5, 0.4995, -1.0]])
    assert not OS.swap_ok(lg, [[0, 1]], [[2, 1]], 1e-3).any()
    # displacing expert 1 instead is within the gap
    assert OS.swap_ok(lg, [[0, 1]], [[0, 2]], 1e-3).all()


def test_swap_ok_rejects_a_repeated_expert():
    lg = np.array([[1.0, 1.0, 0.0, 0.0]])
    assert not OS.swap_ok(lg, [[0, 1]], [[0, 0]], 1.0).any()


# ------------------------------------------------------------------------------- restricted stack


def _small_stack(n_layers=3):
    return W.stack24(seed=1501, batch=6, median=40, cap=200, n_layers=n_layers, slack=1.25, base=SMALL)


def _plain_chain(spec, n_layers, force=None):
    """The definition: every layer's full batch through the single-layer
    reference, all experts drawn, all pages regenerated, chained."""
    x = W.stack_x_in(spec).double()
    outs, idxs = [], []
    for layer in range(n_layers):
        s = spec.shape(layer)
        pt = spec.page_table(layer)
        wl = W.Workload(name="plain", shape=s, seed=spec.seed, seq_lens=spec.seq_lens,
                        q_lens=np.ones(spec.batch, np.int32), page_table=pt, n_pages=spec.n_pages(layer),
                        weights=W.stack_weights_host(spec, layer))
        pages = np.arange(spec.n_pages(layer))
        wl.k_pool = W.stack_pages_host(spec, layer, "k", pages)
        wl.v_pool = W.stack_pages_host(spec, layer, "v", pages)
        wl.x_in = x
        r = O.decode_layer(wl, force_idx=None if force is None else force[layer])
        x = torch.from_numpy(r["out"])
        outs.append(r["out"])
        idxs.append(r["idx"])
    return outs, np.stack(idxs)


def test_restricted_chain_equals_plain_layer_chain():
    spec = _small_stack()
    outs, idx = _plain_chain(spec, 3)
    seqs = np.array([0, 2, 5])
    ref, info = OS.reference_stack(spec, seqs, n_layers=3)
    for layer in range(3):
        np.testing.assert_array_equal(info[layer]["out"], outs[layer][seqs])
        np.testing.assert_array_equal(np.sort(info[layer]["idx"], 1), np.sort(idx[layer][seqs], 1))
        assert not info[layer]["adopted"].any()
    np.testing.assert_array_equal(ref, outs[-1][seqs])


def test_teacher_forced_layer_equals_plain_layer():
    """reference_layer from a given input equals the plain layer on that input."""
    spec = _small_stack()
    outs, idx = _plain_chain(spec, 2)
    seqs = np.array([1, 3, 4])
    ra, rb = OS.reference_layer(spec, 1, seqs, outs[0][seqs])
    np.testing.assert_array_equal(rb["out"], outs[1][seqs])
    np.testing.assert_array_equal(np.sort(ra["idx"], 1), np.sort(idx[1][seqs], 1))


def test_chain_adopts_a_differing_gpu_selection():
    """A GPU set that differs is followed (and its logit gap reported); the
    chain then equals the plain chain forced to that set."""
    spec = _small_stack(2)
    _, idx = _plain_chain(spec, 2)
    gpu = idx.copy()
    b = 2
    ref_set = set(idx[0, b].tolist())
    gpu[0, b, 1] = next(e for e in range(SMALL.n_experts) if e not in ref_set)
    seqs = np.array([0, b])
    ref, info = OS.reference_stack(spec, seqs, n_layers=2, gpu_idx=gpu)
    np.testing.assert_array_equal(info[0]["adopted"], [False, True])
    assert info[0]["gap"][1] != 0.0 and info[0]["gap"][0] == 0.0
    forced, _ = _plain_chain(spec, 2, force=[gpu[0], None])
    np.testing.assert_array_equal(info[0]["out"], forced[0][seqs])


@pytest.mark.parametrize("seed", [1502])
def test_small_stack_routes_are_exact_topk(seed):
    """The restricted routing pass selects the top-k of its own logits."""
    spec = W.stack24(seed=seed, batch=4, median=30, cap=100, n_layers=1, slack=1.25, base=SMALL)
    seqs = np.arange(4)
    x = W.stack_x_in(spec).double().numpy()
    ra, _ = OS.reference_layer(spec, 0, seqs, x)
    for r in range(4):
        order = np.argsort(-ra["logits"][r], kind="stable")[:SMALL.top_k]
        assert sorted(order.tolist()) == sorted(ra["idx"][r].tolist())
