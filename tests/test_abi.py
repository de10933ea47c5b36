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
    assert L.kv_pages_free(h, 1, np.array([9], np.int32).ctypes.data) == mcpu.MCPU_EINVAL
    assert "not allocated" in L.mcpu_last_error().decode()
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


def test_packed_mxfp4_size_and_argument_checks():
    """mcpu_packed_mxfp4_bytes: the codes (rounded up to 256 bytes), then one
    scale dword per row and 128 columns; mcpu_pack_mxfp4 rejects bad
    arguments on the host (dummy addresses: every case returns before a
    launch)."""
    L = mcpu.lib()
    assert L.mcpu_packed_mxfp4_bytes(32, 5760, 2880) == 32 * 5760 * 1440 + 32 * 23 * 5760 * 4
    assert L.mcpu_packed_mxfp4_bytes(1, 16, 64) == 512 + 16 * 4     # 512 code bytes, already whole
    assert L.mcpu_packed_mxfp4_bytes(1, 16, 192) == 1536 + 2 * 16 * 4
    for bad in [(0, 16, 64), (1, 8, 64), (1, 16, 96), (1, 16, 0), (-1, 16, 64)]:
        assert L.mcpu_packed_mxfp4_bytes(*bad) == 0, bad
    a, s, b = 1 << 20, 1 << 24, 1 << 30
    assert L.mcpu_pack_mxfp4(a, s, b, 1, 16, 96, None) == mcpu.MCPU_EINVAL
    assert L.mcpu_pack_mxfp4(None, s, b, 1, 16, 64, None) == mcpu.MCPU_EINVAL
    assert L.mcpu_pack_mxfp4(a, s, b + 16, 1, 16, 64, None) == mcpu.MCPU_EINVAL      # dst not 256-aligned
    assert L.mcpu_pack_mxfp4(a + 8, s, b, 1, 16, 64, None) == mcpu.MCPU_EINVAL       # codes misaligned
    assert L.mcpu_pack_mxfp4(a, s, a + 256, 1, 16, 64, None) == mcpu.MCPU_EINVAL     # overlaps the codes
    assert L.mcpu_pack_mxfp4(a, b + 256, b, 1, 16, 64, None) == mcpu.MCPU_EINVAL     # overlaps the scales


def test_native_experts_need_their_slice_order_copies():
    """A native-MXFP4 layer without w_gu_packed / w_d_packed is rejected
    before any launch."""
    import dataclasses
    shape = dataclasses.replace(W.GPT_OSS_20B, expert_fmt="mxfp4_native")
    L = mcpu.lib()
    cfg = mcpu.make_cfg(shape)
    w = _dummy_weights(mxfp4=True)
    rc = L.moe_forward(ctypes.byref(cfg), ctypes.byref(w), 4, _DUMMY, _DUMMY, None, None, None, _DUMMY + (1 << 24),
                       1 << 30, None)
    assert rc == mcpu.MCPU_EINVAL
    assert b"w_gu_packed" in L.mcpu_last_error()


# dummy device addresses: never dereferenced, every call below returns on the host
_DUMMY = 1 << 32


def _dummy_weights(mxfp4=False, drop=None):
    names = [n for n, _ in mcpu.LayerWeights._fields_ if n != "rope_max_pos"]
    kw = {n: _DUMMY + 4096 * i for i, n in enumerate(names)}
    kw["w_gu_packed"] = kw["w_d_packed"] = kw["w_qkv_packed"] = kw["w_o_packed"] = None
    if not mxfp4:
        kw["s_gu"] = kw["s_d"] = None
    if drop:
        kw[drop] = None
    return mcpu.LayerWeights(rope_max_pos=4096, **kw)


def _decode_call(shape, w, ws_bytes, x_in=_DUMMY + (1 << 24), page_table=_DUMMY + (2 << 24), pool=None):
    L = mcpu.lib()
    cfg = mcpu.make_cfg(shape)
    if pool is None:
        rc, pool = _fake_pool(shape, 64)
        assert rc == 0
    hs = np.array([5, 17, 40], np.int32)
    rc = L.decode_layer(ctypes.byref(cfg), ctypes.byref(w), pool, 3, page_table, 8, _DUMMY + (3 << 24), None,
                        hs.ctypes.data, None, x_in, _DUMMY + (4 << 24), None, None, None,
                        _DUMMY + (5 << 24), ws_bytes, None)
    return rc


def test_decode_layer_rejects_null_pointers_and_small_workspace():
    """Host-detected errors return before any launch (mcpu.h): NULL weight and
    buffer pointers give MCPU_EINVAL, a workspace below
    decode_layer_workspace_size gives MCPU_ENOMEM, each with a message."""
    L = mcpu.lib()
    s = W.TINY
    need = mcpu.decode_layer_workspace_size(s, 3, 3)
    for name in ("g1", "w_qkv", "w_o", "rope_cos", "g2", "w_r", "w_gu", "b_d"):
        assert _decode_call(s, _dummy_weights(drop=name), need) == mcpu.MCPU_EINVAL, name
        assert "NULL" in L.mcpu_last_error().decode()
    assert _decode_call(s, _dummy_weights(), need, x_in=None) == mcpu.MCPU_EINVAL
    assert _decode_call(s, _dummy_weights(), need, page_table=None) == mcpu.MCPU_EINVAL
    # MXFP4 experts without their scale arrays
    mx = replace(W.GPT_OSS_20B, expert_fmt="mxfp4")
    w = _dummy_weights(mxfp4=True, drop="s_gu")
    assert _decode_call(mx, w, mcpu.decode_layer_workspace_size(mx, 3, 3)) == mcpu.MCPU_EINVAL
    assert "scale" in L.mcpu_last_error().decode()
    # streaming-order projection copies on a layer that is not bf16
    w = _dummy_weights()
    w.w_qkv_packed = _DUMMY + (6 << 24)
    assert s.dtype != "bf16" and _decode_call(s, w, need) == mcpu.MCPU_EINVAL
    assert "packed projection" in L.mcpu_last_error().decode()
    # workspace one byte short
    assert _decode_call(s, _dummy_weights(), need - 1) == mcpu.MCPU_ENOMEM
    assert "workspace" in L.mcpu_last_error().decode()
    # the pool of another layer shape
    rc, other = _fake_pool(replace(W.TINY, head_dim=64), 64)
    assert rc == 0
    assert _decode_call(s, _dummy_weights(), need, pool=other) == mcpu.MCPU_EINVAL


def test_moe_forward_rejects_null_pointers_and_small_workspace():
    L = mcpu.lib()
    s = W.TINY
    cfg = mcpu.make_cfg(s)
    need = mcpu.moe_forward_workspace_size(s, 10)

    def call(w, h=_DUMMY + (1 << 24), out=_DUMMY + (2 << 24), ws=_DUMMY + (3 << 24), nbytes=need, n=10):
        return L.moe_forward(ctypes.byref(cfg), ctypes.byref(w), n, h, out, None, None, None, ws, nbytes, None)

    for name in ("g2", "w_r", "b_r", "w_gu", "b_gu", "w_d", "b_d"):
        assert call(_dummy_weights(drop=name)) == mcpu.MCPU_EINVAL, name
    assert call(_dummy_weights(), h=None) == mcpu.MCPU_EINVAL
    assert call(_dummy_weights(), out=None) == mcpu.MCPU_EINVAL
    assert call(_dummy_weights(), ws=None) == mcpu.MCPU_EINVAL
    assert call(_dummy_weights(), nbytes=need - 256) == mcpu.MCPU_ENOMEM
    assert call(_dummy_weights(), n=-1) == mcpu.MCPU_EINVAL
    assert call(_dummy_weights(), h=None, n=0) == mcpu.MCPU_OK   # nothing to do, nothing launched


def test_paged_attention_rejects_mismatched_cu_q_and_small_workspace():
    L = mcpu.lib()
    s = W.TINY
    cfg = mcpu.make_cfg(s)
    rc, pool = _fake_pool(s, 64)
    assert rc == 0
    hs = np.array([5, 17], np.int32)
    hc = np.array([0, 1, 2], np.int32)
    need = mcpu.paged_attention_workspace_size(s, 2, 2)
    d = _DUMMY
    # cu_q given without its host copy
    assert L.paged_attention(ctypes.byref(cfg), None, pool, 2, d, 8, d, d, hs.ctypes.data, None, d, d, d, need,
                             None) == mcpu.MCPU_EINVAL
    assert L.paged_attention(ctypes.byref(cfg), None, pool, 2, d, 8, d, d, hs.ctypes.data, hc.ctypes.data, d, d,
                             d, need - 1, None) == mcpu.MCPU_ENOMEM
    # a position beyond the page table's width
    far = np.array([5, 8 * 16], np.int32)
    assert L.paged_attention(ctypes.byref(cfg), None, pool, 2, d, 8, d, None, far.ctypes.data, None, d, d, d,
                             need, None) == mcpu.MCPU_EINVAL
    assert "beyond page table" in L.mcpu_last_error().decode()
