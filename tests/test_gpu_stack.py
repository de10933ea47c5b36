"""The decoder-layer stack (alternating sliding-window and full attention,
MXFP4 experts) on the GPU against the CPU reference, and the device twin of
the seeded input generator against the host generator.

The stack is generated in HBM by the device generator; the reference
regenerates on the host only what its sampled sequences read. Each layer is
compared at the single-layer bar from the residual rows the GPU fed into it
(teacher-forced); the reference's own free-running chain is reported as the
drift over depth.
"""
import numpy as np
import pytest
import torch

from oracle import stack as OS
from paper_2608_22167_amd import mcpu, workload as W
from tests import parity as PT

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    torch.cuda.set_device(0)
    yield
    torch.cuda.empty_cache()


# ------------------------------------------------------------------------------------- generators


@pytest.mark.parametrize("n,offset", [(1, 0), (7, 3), (4099, 0), (100003, 12345)])
def test_device_generator_bf16_bitwise(n, offset):
    dev = W.fill_normal_device(torch.empty(n, dtype=torch.bfloat16, device="cuda"), 77, 5, std=0.02,
                               mean=1.0, offset=offset)
    host = W.synth_normal(77, 5, (n,), std=0.02, mean=1.0, dtype=torch.bfloat16, offset=offset)
    assert torch.equal(dev.cpu().view(torch.int16), host.view(torch.int16))


@pytest.mark.parametrize("n,offset", [(9, 0), (65537, 7), (1 << 20, (1 << 32) - (1 << 20))])
def test_device_generator_fast_bf16_bitwise(n, offset):
    dev = W.fill_fast_normal_device(torch.empty(n, dtype=torch.bfloat16, device="cuda"), 78, 20,
                                    offset=offset)
    host = W.synth_fast_normal(78, 20, n, offset=offset)
    assert torch.equal(dev.cpu().view(torch.int16), host.view(torch.int16))


@pytest.mark.parametrize("n,offset", [(3, 0), (70001, 99)])
def test_device_generator_bytes_bitwise(n, offset):
    dev = W.fill_bytes_device(torch.empty(n, dtype=torch.uint8, device="cuda"), 79, 30, offset=offset)
    host = W.synth_bytes(79, 30, (n,), offset=offset)
    assert torch.equal(dev.cpu(), host)


# ------------------------------------------------------------------------------------------ stack


def _sample(spec, extra, seed):
    """The longest and shortest sequences plus `extra` seeded others."""
    lens = spec.seq_lens
    rng = np.random.default_rng(seed)
    pick = {int(np.argmax(lens)), int(np.argmin(lens))}
    pick |= {int(i) for i in rng.choice(spec.batch, size=extra, replace=False)}
    return sorted(pick)


def _run(spec, n_layers, seqs):
    st = mcpu.DeviceStack(spec, n_layers=n_layers)
    rows = torch.tensor(seqs, device="cuda")
    H = spec.shape_full.hidden
    logits = torch.empty((n_layers, spec.batch, spec.shape_full.n_experts), dtype=torch.float32, device="cuda")
    inputs = torch.empty((n_layers, len(seqs), H), dtype=torch.float32, device="cuda")
    outputs = torch.empty((n_layers, len(seqs), H), dtype=torch.float32, device="cuda")
    out = st.run(logits=logits, rows=rows, inputs=inputs)
    torch.cuda.synchronize()
    assert st.device_errors() == 0
    # layer i's output is layer i+1's input; the last layer's is the step's output
    outputs[:-1] = inputs[1:]
    outputs[-1] = out.index_select(0, rows)
    got = dict(inputs=inputs.double().cpu().numpy(), outputs=outputs.double().cpu().numpy(),
               idx=st.topk_idx.cpu().numpy(), logits=logits.cpu().numpy())
    again = st.run()
    torch.cuda.synchronize()
    assert torch.equal(out, again), "stack step is not repeatable"
    del st, out, again
    torch.cuda.empty_cache()
    return got


def _gpu_topk_consistent(idx, logits, rows):
    """The GPU's selections are the top-k of its own fp32 logits (ties to the lower id)."""
    k = idx.shape[-1]
    for layer in range(idx.shape[0]):
        for r in rows:
            order = np.argsort(-logits[layer, r].astype(np.float32), kind="stable")[:k]
            assert sorted(order.tolist()) == sorted(idx[layer, r].tolist()), (layer, r)


def _compare(spec, n_layers, seqs):
    """Teacher-forced: every layer, started from the rows the GPU fed into it,
    meets the single-layer bar (max-abs 2e-2, rel-L2 1e-2 on the layer's
    output; expert sets exact unless every swapped expert is within the 1e-3
    logit gap under the reference's logits, in which case the reference is
    evaluated with the GPU's set). The free-running reference chain is then
    reported as the drift over depth and bounded by depth x the bar."""
    got = _run(spec, n_layers, seqs)
    _gpu_topk_consistent(got["idx"], got["logits"], seqs)
    seqs = np.asarray(seqs)
    experts = OS._Experts(spec)
    errs = []
    for layer in range(n_layers):
        g_idx = got["idx"][layer][seqs]
        state = {}

        def choose(ra, g_idx=g_idx, state=state):
            sel = ra["idx"].copy()
            differ = (np.sort(g_idx, 1) != np.sort(sel, 1)).any(1)
            ok = OS.swap_ok(ra["logits"], sel, g_idx, OS.TIE_GAP)
            assert ok.all(), f"layer {layer}: router sets differ beyond the tie gap at sampled rows " \
                             f"{seqs[~ok]}: GPU {g_idx[~ok]} vs reference {sel[~ok]}"
            sel[differ] = g_idx[differ]
            state["swapped"] = int(differ.sum())
            return sel

        ra, rb = OS.reference_layer(spec, layer, seqs, got["inputs"][layer], choose, experts)
        lerr = np.abs(got["logits"][layer][seqs].astype(np.float64) - ra["logits"]).max()
        mx, rl = PT.check(f"stack layer {layer}", got["outputs"][layer], rb["out"], "bf16")
        # the layer's own increment (both sides start from the same rows): rel-L2 against its norm
        x0 = got["inputs"][layer]
        PT.check(f"stack layer {layer} increment", got["outputs"][layer] - x0, rb["out"] - x0, "bf16")
        errs.append((layer, mx, rl, lerr, state["swapped"]))
        print(f"  layer {layer:2d}: max-abs {mx:.2e} rel-L2 {rl:.2e} logit err {lerr:.2e} "
              f"near-tie swaps {state['swapped']}", flush=True)
    # drift of the free-running chain (reported; bounded by depth x the bar)
    ref, info = OS.reference_stack(spec, seqs, n_layers=n_layers, gpu_idx=got["idx"])
    adopted = sum(int(d["adopted"].sum()) for d in info)
    mx = np.abs(got["outputs"][-1] - ref).max()
    print(f"  free-running chain after {n_layers} layers: max-abs {mx:.2e}, rel-L2 "
          f"{PT.rel_l2(got['outputs'][-1], ref):.2e}, GPU sets adopted {adopted}")
    PT.check(f"stack{n_layers} drift", got["outputs"][-1], ref, "bf16", scale=n_layers)


def test_stack_depth4_small_batch():
    spec = W.stack24(seed=1006, batch=16, median=1024, cap=8192, n_layers=4)
    _compare(spec, 4, _sample(spec, 4, 11))


@pytest.mark.timeout(900)
def test_stack24_full_size_sampled():
    """The 24-layer, 512-sequence stack the benchmark times, on sampled sequences."""
    spec = W.stack24()
    _compare(spec, spec.n_layers, _sample(spec, 1, 12))
