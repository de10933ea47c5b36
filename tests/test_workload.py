"""The seeded input generator follows its stated definition, bit for bit."""
import numpy as np
import torch

from paper_2608_22167_amd import workload as W

M64 = (1 << 64) - 1


def _mix(z):
    z = ((z ^ (z >> 30)) * 0xBF58476D1CE4E5B9) & M64
    z = ((z ^ (z >> 27)) * 0x94D049BB133111EB) & M64
    return z ^ (z >> 31)


def _draw(seed, tid, i, std, mean):
    key = _mix(_mix(seed) ^ tid)
    h = _mix((key + (i + 1) * 0x9E3779B97F4A7C15) & M64)
    s = sum((h >> (8 * b)) & 0xFF for b in range(8))
    c = np.float32(std / W.IH_STD)
    return np.float32(np.float32(s - 1020) * c) + np.float32(mean)


def test_generator_definition_fp32_and_offsets():
    x = W.synth_normal(1234, 9, (4096,), std=0.02, mean=1.0)
    for i in (0, 1, 77, 4095):
        assert x[i].item() == float(_draw(1234, 9, i, 0.02, 1.0))
    y = W.synth_normal(1234, 9, (96,), std=0.02, mean=1.0, offset=4000)
    assert torch.equal(y, x[4000:4096])


def test_generator_bf16_is_rounded_fp32():
    a = W.synth_normal(5, 3, (10000,), dtype=torch.float32)
    b = W.synth_normal(5, 3, (10000,), dtype=torch.bfloat16)
    assert torch.equal(a.to(torch.bfloat16), b)
    assert abs(a.mean().item()) < 0.03 and abs(a.std().item() - 1) < 0.03


def test_page_tables_are_sparse_permutations():
    wl = W.custom(W.TINY, [17, 100, 3], [1, 1, 40], 3, weights=False)
    used = wl.page_table[wl.page_table >= 0]
    assert len(np.unique(used)) == len(used) and used.max() < wl.n_pages
    for b in range(3):
        need = (int(wl.seq_lens[b]) + int(wl.q_lens[b]) + 15) // 16
        assert (wl.page_table[b, :need] >= 0).all() and (wl.page_table[b, need:] == -1).all()
