"""The decoder-layer stack (alternating sliding-window and full attention,
MXFP4 experts) on the GPU against the CPU reference, and the device twin of
the seeded input generator against the host generator.

The stack is generated in HBM by the device generator; the reference
regenerates on the host only what its sampled sequences read. A stack is
compared at L times the single-layer tolerance: each layer adds its own
rounding error, and the residual connection passes the errors of earlier
layers on with a gain close to one.
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
    out, caps = st.run(capture_rows=rows)
    torch.cuda.synchronize()
    assert st.device_errors() == 0
    xs = [c.double().cpu().numpy() for c in caps]
    idx = st.topk_idx.cpu().numpy()
    again = st.run()
    torch.cuda.synchronize()
    assert torch.equal(out, again), "stack step is not repeatable"
    del st, out, again, caps
    torch.cuda.empty_cache()
    return xs, idx


def _no_mismatch(info):
    for layer, d in enumerate(info):
        assert not d["mismatch"].any(), \
            f"layer {layer}: router sets differ at sampled rows {np.nonzero(d['mismatch'])[0]}"


def test_stack_depth4_small_batch():
    """Free-running chain: the reference's own output feeds its next layer."""
    spec = W.stack24(seed=1006, batch=16, median=1024, cap=8192, n_layers=4)
    seqs = _sample(spec, 4, 11)
    xs, idx = _run(spec, 4, seqs)
    ref, info = OS.reference_stack(spec, seqs, n_layers=4, gpu_idx=idx)
    _no_mismatch(info)
    PT.check("stack4", xs[-1], ref, "bf16", scale=4)


@pytest.mark.timeout(900)
def test_stack24_full_size_sampled():
    """The 24-layer, 512-sequence stack the benchmark times, on sampled sequences.

    Teacher forced: every layer, given the GPU's own input to it, matches the
    reference at the single-layer bar, routing included. Then the reference
    chain that follows the GPU's (thereby validated) routing bounds the
    accumulated drift of the whole stack at 24 times that bar."""
    spec = W.stack24()
    seqs = _sample(spec, 1, 12)
    xs, idx = _run(spec, spec.n_layers, seqs)
    _, info = OS.reference_stack(spec, seqs, gpu_idx=idx, inputs=xs[:-1])
    _no_mismatch(info)
    for layer, d in enumerate(info):
        PT.check(f"layer {layer}", xs[layer + 1], d["out"], "bf16")
    ref, _ = OS.reference_stack(spec, seqs, gpu_idx=idx, follow_gpu=True)
    PT.check("stack24", xs[-1], ref, "bf16", scale=spec.n_layers)
