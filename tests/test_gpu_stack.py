"""The decoder-layer stack (alternating sliding-window and full attention,
MXFP4 experts) on the GPU against the CPU reference, and the device twin of
the seeded input generator against the host generator.

The stack is generated in HBM by the device generator; the reference
regenerates on the host only what its sampled sequences read and chains its
own layers from the step's input. A stack is compared at L times the
single-layer tolerance: each layer adds its own rounding error, and the
residual connection passes the errors of earlier layers on with a gain close
to one.
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
    logits = torch.empty((n_layers, spec.batch, spec.shape_full.n_experts), dtype=torch.float32, device="cuda")
    out = st.run(logits=logits)
    torch.cuda.synchronize()
    assert st.device_errors() == 0
    got = out.index_select(0, rows).double().cpu().numpy()
    idx = st.topk_idx.cpu().numpy()
    lg = logits.cpu().numpy()
    again = st.run()
    torch.cuda.synchronize()
    assert torch.equal(out, again), "stack step is not repeatable"
    del st, out, again
    torch.cuda.empty_cache()
    return got, idx, lg


def _gpu_topk_consistent(idx, logits, rows):
    """The GPU's selections are the top-k of its own fp32 logits (ties to the lower id)."""
    k = idx.shape[-1]
    for layer in range(idx.shape[0]):
        for r in rows:
            order = np.argsort(-logits[layer, r].astype(np.float32), kind="stable")[:k]
            assert sorted(order.tolist()) == sorted(idx[layer, r].tolist()), (layer, r)


def _compare(spec, n_layers, seqs):
    got, idx, lg = _run(spec, n_layers, seqs)
    _gpu_topk_consistent(idx, lg, seqs)
    ref, info = OS.reference_stack(spec, seqs, n_layers=n_layers, gpu_idx=idx, gpu_logits=lg)
    for layer, d in enumerate(info):
        assert not d["mismatch"].any(), \
            f"layer {layer}: router sets differ at sampled rows {np.nonzero(d['mismatch'])[0]} " \
            f"(logit differences {d['logit_err']})"
        # the logits themselves stay within the depth-scaled bar
        assert d["logit_err"].max() <= 2e-2 * (layer + 1), (layer, d["logit_err"])
    return PT.check(f"stack{n_layers}", got, ref, "bf16", scale=n_layers)


def test_stack_depth4_small_batch():
    spec = W.stack24(seed=1006, batch=16, median=1024, cap=8192, n_layers=4)
    _compare(spec, 4, _sample(spec, 4, 11))


@pytest.mark.timeout(900)
def test_stack24_full_size_sampled():
    """The 24-layer, 512-sequence stack the benchmark times, on sampled sequences."""
    spec = W.stack24()
    _compare(spec, spec.n_layers, _sample(spec, 1, 12))
