"""Python binding of the C ABI in include/mcpu.h (argument marshalling only).

Every function keeps the C name and forwards device pointers of torch
tensors plus the current HIP stream; all arithmetic runs in libmcpu.so's
gfx950 kernels. There is no fallback: if the library is missing or a call
fails, an exception is raised.
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmcpu.so")

MCPU_OK, MCPU_EINVAL, MCPU_ENOMEM, MCPU_EHIP, MCPU_EUNSUPPORTED, MCPU_EDEVICE = 0, -1, -2, -3, -4, -5
MCPU_F32, MCPU_BF16 = 0, 1
MCPU_EXPERT_DENSE, MCPU_EXPERT_MXFP4, MCPU_EXPERT_MXFP4_NATIVE = 0, 1, 2
_EXPERT_FMT = {"dense": MCPU_EXPERT_DENSE, "mxfp4": MCPU_EXPERT_MXFP4, "mxfp4_native": MCPU_EXPERT_MXFP4_NATIVE}
DEVERR_PAGE, DEVERR_ROPE, DEVERR_EXPERT, DEVERR_PLAN, DEVERR_MXFP4 = 1, 2, 4, 8, 16

EXPORTED = ("mcpu_last_error", "kv_pool_create", "kv_pool_destroy", "kv_pool_free_pages",
            "kv_pages_alloc", "kv_pages_free", "kv_pages_append", "paged_attention_workspace_size",
            "paged_attention", "moe_forward_workspace_size", "moe_forward",
            "decode_layer_workspace_size", "decode_layer", "mcpu_check_device_errors",
            "mcpu_timing_start", "mcpu_timing_read", "mcpu_packed_weights_bytes", "mcpu_pack_weights",
            "lm_head_workspace_size", "lm_head_sample", "embed_tokens", "decode_layer_noalloc",
            "mcpu_mxfp8_quantize", "mcpu_packed_mxfp4_bytes", "mcpu_pack_mxfp4")
NOALLOC_SCRATCH_BYTES = 128 << 20  # the static scratch of decode_layer_noalloc, per GPU

KERNELS = ("attn_plan", "rmsnorm", "qkv", "attn_split", "attn_combine", "oproj", "router", "permute",
           "expert_gu", "expert_down", "moe_combine", "kv_append", "attn_prefill", "lm_head")
DEVERR_TOKEN = 32


class McpuError(RuntimeError):
    def __init__(self, code, msg):
        super().__init__(f"mcpu status {code}: {msg}")
        self.code = code


class LayerCfg(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "hidden", "n_q_heads", "n_kv_heads", "head_dim", "n_experts", "top_k", "ffn_dim",
        "page_size", "window", "dtype", "expert_fmt")] + [
        (n, ctypes.c_float) for n in ("rms_eps", "swiglu_alpha", "swiglu_limit", "swiglu_beta")]


class LayerWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "g1", "w_qkv", "b_qkv", "w_o", "b_o", "g2", "w_r", "b_r", "w_gu", "b_gu", "w_d", "b_d",
        "s_gu", "s_d", "sinks", "rope_cos", "rope_sin")] + [("rope_max_pos", ctypes.c_int32)] + [
        (n, ctypes.c_void_p) for n in ("w_gu_packed", "w_d_packed", "w_qkv_packed", "w_o_packed")]


class LmHead(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("vocab", ctypes.c_int32), ("rms_eps", ctypes.c_float),
                ("g_final", ctypes.c_void_p), ("w_lm", ctypes.c_void_p), ("w_lm_packed", ctypes.c_void_p)]


class Taps(ctypes.Structure):
    _fields_ = [("q", ctypes.c_void_p), ("o", ctypes.c_void_p), ("h1", ctypes.c_void_p),
                ("logits", ctypes.c_void_p)]


_LIB = None


def lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run __graft_entry__.build() first")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_size_t
        i32p = ctypes.POINTER(ctypes.c_int32)
        L.mcpu_last_error.restype = ctypes.c_char_p
        L.kv_pool_create.argtypes = [vp, i32, vp, vp, ctypes.POINTER(vp)]
        L.kv_pool_destroy.argtypes = [vp]
        L.kv_pool_free_pages.argtypes = [vp]
        L.kv_pool_free_pages.restype = i32
        L.kv_pages_alloc.argtypes = [vp, i32, vp]
        L.kv_pages_free.argtypes = [vp, i32, vp]
        L.kv_pages_append.argtypes = [vp, i32, vp, i32, vp, vp, i32, vp, vp, vp, sz, vp]
        L.paged_attention_workspace_size.argtypes = [vp, i32, i32]
        L.paged_attention_workspace_size.restype = sz
        L.paged_attention.argtypes = [vp, vp, vp, i32, vp, i32, vp, vp, vp, vp, vp, vp, vp, sz, vp]
        L.moe_forward_workspace_size.argtypes = [vp, i32]
        L.moe_forward_workspace_size.restype = sz
        L.moe_forward.argtypes = [vp, vp, i32, vp, vp, vp, vp, vp, vp, sz, vp]
        L.decode_layer_workspace_size.argtypes = [vp, i32, i32]
        L.decode_layer_workspace_size.restype = sz
        L.decode_layer.argtypes = [vp, vp, vp, i32, vp, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                   vp, sz, vp]
        L.decode_layer_noalloc.argtypes = [vp, vp, vp, i32, vp, i32, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.mcpu_check_device_errors.argtypes = [vp, vp, i32p]
        L.mcpu_packed_weights_bytes.argtypes = [i32, i32, i32]
        L.mcpu_packed_weights_bytes.restype = sz
        L.mcpu_pack_weights.argtypes = [i32, vp, vp, i32, i32, i32, vp]
        L.lm_head_workspace_size.argtypes = [i32, i32, i32]
        L.lm_head_workspace_size.restype = sz
        L.lm_head_sample.argtypes = [vp, i32, vp, vp, ctypes.c_float, ctypes.c_uint64, vp, vp, vp, vp, vp, vp,
                                     vp, vp, sz, vp]
        L.embed_tokens.argtypes = [vp, i32, i32, i32, vp, vp, vp, sz, vp]
        L.mcpu_mxfp8_quantize.argtypes = [vp, ctypes.c_int64, i32, vp, vp, vp]
        L.mcpu_packed_mxfp4_bytes.argtypes = [i32, i32, i32]
        L.mcpu_packed_mxfp4_bytes.restype = sz
        L.mcpu_pack_mxfp4.argtypes = [vp, vp, vp, i32, i32, i32, vp]
        L.mcpu_timing_start.argtypes = [i32, i32]
        L.mcpu_timing_read.argtypes = [i32, vp, i32, i32p]
        _LIB = L
    return _LIB


def _check(rc):
    if rc != MCPU_OK:
        raise McpuError(rc, lib().mcpu_last_error().decode())


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    if isinstance(t, np.ndarray):
        assert t.flags["C_CONTIGUOUS"]
        return t.ctypes.data
    assert t.is_contiguous()
    return t.data_ptr()


def _stream(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return ctypes.c_void_p(s.cuda_stream)


def _host_i32(a) -> Optional[np.ndarray]:
    if a is None:
        return None
    if isinstance(a, torch.Tensor):
        a = a.cpu().numpy()
    return np.ascontiguousarray(a, dtype=np.int32)


# ---------------------------------------------------------------------------
# config / weights
# ---------------------------------------------------------------------------


def make_cfg(shape) -> LayerCfg:
    return LayerCfg(hidden=shape.hidden, n_q_heads=shape.n_q_heads, n_kv_heads=shape.n_kv_heads,
                    head_dim=shape.head_dim, n_experts=shape.n_experts, top_k=shape.top_k,
                    ffn_dim=shape.ffn_dim, page_size=shape.page_size, window=shape.window,
                    dtype=MCPU_F32 if shape.dtype == "f32" else MCPU_BF16,
                    expert_fmt=_EXPERT_FMT[shape.expert_fmt],
                    rms_eps=shape.rms_eps, swiglu_alpha=shape.swiglu_alpha,
                    swiglu_limit=shape.swiglu_limit, swiglu_beta=shape.swiglu_beta)


def packed_weights(w: torch.Tensor, stream=None) -> torch.Tensor:
    """Streaming-order copy of bf16 weights [groups, rows, cols] (mcpu_pack_weights)."""
    assert w.dtype == torch.bfloat16 and w.dim() == 3 and w.is_cuda and w.is_contiguous()
    g, rows, cols = (int(d) for d in w.shape)
    n = lib().mcpu_packed_weights_bytes(g, rows, cols)
    if n == 0:
        raise McpuError(MCPU_EINVAL, f"weights {tuple(w.shape)} cannot be packed (rows % 16, cols % 64)")
    out = torch.empty(n, dtype=torch.uint8, device=w.device)
    _check(lib().mcpu_pack_weights(MCPU_BF16, _ptr(w), _ptr(out), g, rows, cols, _stream(stream)))
    return out


def packed_mxfp4(codes: torch.Tensor, scales: torch.Tensor, stream=None) -> torch.Tensor:
    """Slice-order copy of MXFP4 weights (mcpu_pack_mxfp4): codes uint8
    [groups, rows, cols/2], scales uint8 [groups, rows, cols/32]."""
    assert codes.dtype == torch.uint8 and scales.dtype == torch.uint8 and codes.dim() == 3 and codes.is_cuda
    assert codes.is_contiguous() and scales.is_contiguous()
    g, rows, half = (int(d) for d in codes.shape)
    n = lib().mcpu_packed_mxfp4_bytes(g, rows, 2 * half)
    if n == 0:
        raise McpuError(MCPU_EINVAL, f"MXFP4 weights {tuple(codes.shape)} cannot be packed (rows % 16, cols % 64)")
    out = torch.empty(n, dtype=torch.uint8, device=codes.device)
    _check(lib().mcpu_pack_mxfp4(_ptr(codes), _ptr(scales), _ptr(out), g, rows, 2 * half, _stream(stream)))
    return out


class DeviceWeights:
    """Layer parameters copied to the GPU, with the mcpu_layer_weights struct.
    With pack=True, bf16 dense experts and the bf16 projections also get their
    streaming-order copies; native MXFP4 experts always get their slice-order
    copies."""

    def __init__(self, shape, W, device="cuda", pack=True):
        self.t = {k: v.to(device).contiguous() for k, v in W.items()}
        t = self.t
        mx = shape.expert_fmt != "dense"
        if pack and not mx and shape.dtype == "bf16" and shape.hidden % 64 == 0 and shape.ffn_dim % 64 == 0:
            t["w_gu_packed"] = packed_weights(t["w_gu"])
            t["w_d_packed"] = packed_weights(t["w_d"])
        if pack and shape.dtype == "bf16" and shape.hidden % 64 == 0 and shape.attn_dim % 64 == 0 and "w_qkv" in t:
            t["w_qkv_packed"] = packed_weights(t["w_qkv"].view(1, *t["w_qkv"].shape))
            t["w_o_packed"] = packed_weights(t["w_o"].view(1, *t["w_o"].shape))
        if shape.expert_fmt == "mxfp4_native" and "w_gu_packed" not in t:
            t["w_gu_packed"] = packed_mxfp4(t["w_gu_codes"], t["w_gu_scales"])
            t["w_d_packed"] = packed_mxfp4(t["w_d_codes"], t["w_d_scales"])
        p = lambda k: _ptr(t[k]) if k in t else None
        self.struct = LayerWeights(
            g1=p("g1"), w_qkv=p("w_qkv"), b_qkv=p("b_qkv"), w_o=p("w_o"), b_o=p("b_o"), g2=p("g2"),
            w_r=p("w_r"), b_r=p("b_r"),
            w_gu=p("w_gu_codes") if mx else p("w_gu"), b_gu=p("b_gu"),
            w_d=p("w_d_codes") if mx else p("w_d"), b_d=p("b_d"),
            s_gu=p("w_gu_scales") if mx else None, s_d=p("w_d_scales") if mx else None,
            sinks=p("sinks"), rope_cos=p("rope_cos"), rope_sin=p("rope_sin"),
            rope_max_pos=int(t["rope_cos"].shape[0]) if "rope_cos" in t else 0,
            w_gu_packed=p("w_gu_packed"), w_d_packed=p("w_d_packed"), w_qkv_packed=p("w_qkv_packed"),
            w_o_packed=p("w_o_packed"))


# ---------------------------------------------------------------------------
# page pool
# ---------------------------------------------------------------------------


class KVPool:
    """mcpu_kv_pool over caller-owned device K/V pools (kept alive here)."""

    def __init__(self, shape, k_pool: torch.Tensor, v_pool: torch.Tensor):
        self.shape = shape
        self.cfg = make_cfg(shape)
        self.k, self.v = k_pool, v_pool
        self.n_pages = int(k_pool.shape[0])
        h = ctypes.c_void_p()
        _check(lib().kv_pool_create(ctypes.byref(self.cfg), self.n_pages, _ptr(k_pool), _ptr(v_pool),
                                    ctypes.byref(h)))
        self.handle = h

    def free_pages(self) -> int:
        return lib().kv_pool_free_pages(self.handle)

    def close(self):
        if self.handle:
            lib().kv_pool_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def kv_pool_create(shape, k_pool, v_pool) -> KVPool:
    return KVPool(shape, k_pool, v_pool)


def kv_pages_alloc(pool: KVPool, n: int) -> np.ndarray:
    out = np.empty(max(n, 1), dtype=np.int32)
    _check(lib().kv_pages_alloc(pool.handle, n, _ptr(out)))
    return out[:n]


def kv_pages_free(pool: KVPool, ids) -> None:
    ids = _host_i32(ids)
    _check(lib().kv_pages_free(pool.handle, len(ids), _ptr(ids) if len(ids) else None))


def kv_pages_append(pool: KVPool, page_table, seq_lens, cu_q, k_new, v_new, workspace, stream=None):
    batch = int(seq_lens.shape[0])
    n_tokens = int(k_new.shape[0])
    _check(lib().kv_pages_append(pool.handle, batch, _ptr(page_table), int(page_table.shape[1]),
                                 _ptr(seq_lens), _ptr(cu_q), n_tokens, _ptr(k_new), _ptr(v_new),
                                 _ptr(workspace), workspace.numel() * workspace.element_size(),
                                 _stream(stream)))


def workspace(nbytes: int, device="cuda") -> torch.Tensor:
    """Zero-filled, 256-byte aligned device workspace."""
    return torch.zeros(max(nbytes, 256), dtype=torch.uint8, device=device)


def paged_attention_workspace_size(shape, max_batch, max_tokens) -> int:
    cfg = make_cfg(shape)
    return lib().paged_attention_workspace_size(ctypes.byref(cfg), max_batch, max_tokens)


def paged_attention(shape, sinks, pool: KVPool, page_table, seq_lens, cu_q, host_seq_lens, host_cu_q,
                    q, o, workspace, stream=None):
    cfg = make_cfg(shape)
    hs, hc = _host_i32(host_seq_lens), _host_i32(host_cu_q)
    _check(lib().paged_attention(ctypes.byref(cfg), _ptr(sinks), pool.handle, int(seq_lens.shape[0]),
                                 _ptr(page_table), int(page_table.shape[1]), _ptr(seq_lens), _ptr(cu_q),
                                 _ptr(hs), _ptr(hc), _ptr(q), _ptr(o), _ptr(workspace),
                                 workspace.numel(), _stream(stream)))


def moe_forward_workspace_size(shape, max_tokens) -> int:
    cfg = make_cfg(shape)
    return lib().moe_forward_workspace_size(ctypes.byref(cfg), max_tokens)


def moe_forward(shape, weights: DeviceWeights, h, out, topk_idx=None, topk_w=None, force_idx=None,
                workspace=None, stream=None):
    cfg = make_cfg(shape)
    _check(lib().moe_forward(ctypes.byref(cfg), ctypes.byref(weights.struct), int(h.shape[0]), _ptr(h),
                             _ptr(out), _ptr(topk_idx), _ptr(topk_w), _ptr(force_idx),
                             _ptr(workspace), workspace.numel(), _stream(stream)))


def decode_layer_workspace_size(shape, max_batch, max_tokens) -> int:
    cfg = make_cfg(shape)
    return lib().decode_layer_workspace_size(ctypes.byref(cfg), max_batch, max_tokens)


def decode_layer(shape, weights: DeviceWeights, pool: KVPool, page_table, seq_lens, cu_q, host_seq_lens,
                 host_cu_q, x_in, x_out, topk_idx=None, topk_w=None, taps: Optional[Taps] = None,
                 workspace=None, stream=None):
    cfg = make_cfg(shape)
    hs, hc = _host_i32(host_seq_lens), _host_i32(host_cu_q)
    _check(lib().decode_layer(ctypes.byref(cfg), ctypes.byref(weights.struct), pool.handle,
                              int(seq_lens.shape[0]), _ptr(page_table), int(page_table.shape[1]),
                              _ptr(seq_lens), _ptr(cu_q), _ptr(hs), _ptr(hc), _ptr(x_in), _ptr(x_out),
                              _ptr(topk_idx), _ptr(topk_w),
                              ctypes.byref(taps) if taps is not None else None,
                              _ptr(workspace), workspace.numel(), _stream(stream)))


def decode_layer_noalloc(shape, weights: DeviceWeights, pool: KVPool, page_table, seq_lens, cu_q, host_seq_lens,
                         host_cu_q, x_in, x_out, topk_idx=None, topk_w=None, taps: Optional[Taps] = None,
                         device_errors=None, stream=None):
    """decode_layer on the library's static scratch (no workspace argument)."""
    cfg = make_cfg(shape)
    hs, hc = _host_i32(host_seq_lens), _host_i32(host_cu_q)
    _check(lib().decode_layer_noalloc(ctypes.byref(cfg), ctypes.byref(weights.struct), pool.handle,
                                      int(seq_lens.shape[0]), _ptr(page_table), int(page_table.shape[1]),
                                      _ptr(seq_lens), _ptr(cu_q), _ptr(hs), _ptr(hc), _ptr(x_in), _ptr(x_out),
                                      _ptr(topk_idx), _ptr(topk_w), ctypes.byref(taps) if taps is not None else None,
                                      _ptr(device_errors), _stream(stream)))


def mcpu_check_device_errors(workspace, stream=None) -> int:
    bits = ctypes.c_int32(0)
    rc = lib().mcpu_check_device_errors(_ptr(workspace), _stream(stream), ctypes.byref(bits))
    if rc not in (MCPU_OK, MCPU_EDEVICE):
        _check(rc)
    return bits.value


def mcpu_timing_start(kernel: str, n: int) -> None:
    _check(lib().mcpu_timing_start(KERNELS.index(kernel), n))


def mcpu_timing_read(kernel: str, n: int) -> np.ndarray:
    ms = np.zeros(max(n, 1), dtype=np.float32)
    rec = ctypes.c_int32(0)
    _check(lib().mcpu_timing_read(KERNELS.index(kernel), _ptr(ms), n, ctypes.byref(rec)))
    return ms[:rec.value].astype(np.float64)


# ---------------------------------------------------------------------------
# generation ends: embedding, vocabulary head, sampling
# ---------------------------------------------------------------------------


class DeviceLmHead:
    """Final RMSNorm gain and unembedding [V, H] bf16 on the GPU, with the
    mcpu_lm_head struct; pack=True adds the streaming-order copy that
    few-row batches read."""

    def __init__(self, g_final, w_lm, rms_eps=1e-5, device="cuda", pack=True):
        self.g = g_final.to(device=device, dtype=torch.float32).contiguous()
        self.w = w_lm.to(device=device, dtype=torch.bfloat16).contiguous()
        V, H = (int(d) for d in self.w.shape)
        self.hidden, self.vocab = H, V
        self.packed = packed_weights(self.w.view(1, V, H)) if pack and H % 64 == 0 else None
        self.struct = LmHead(hidden=H, vocab=V, rms_eps=rms_eps, g_final=_ptr(self.g), w_lm=_ptr(self.w),
                             w_lm_packed=_ptr(self.packed))


def lm_head_workspace_size(hidden, vocab, max_tokens) -> int:
    return lib().lm_head_workspace_size(hidden, vocab, max_tokens)


def lm_head_sample(head: DeviceLmHead, x, temperature, seed=0, seq_ids=None, positions=None, targets=None,
                   tokens=None, logprob=None, target_logprob=None, lse=None, workspace=None, stream=None,
                   x_rows=None):
    """lm_head_sample on rows x [T, H] fp32 (or on rows x[x_rows]); outputs
    are device tensors (nullable)."""
    T = int(x.shape[0] if x_rows is None else x_rows.shape[0])
    _check(lib().lm_head_sample(ctypes.byref(head.struct), T, _ptr(x), _ptr(x_rows), float(temperature), int(seed),
                                _ptr(seq_ids), _ptr(positions), _ptr(targets), _ptr(tokens), _ptr(logprob),
                                _ptr(target_logprob), _ptr(lse), _ptr(workspace),
                                workspace.numel() * workspace.element_size(), _stream(stream)))


def mxfp8_quantize(x, stream=None):
    """bf16 rows [R, C] on the GPU -> (codes uint8 [R, C], scales uint8 [R, C/32])."""
    assert x.dtype == torch.bfloat16 and x.is_contiguous()
    R, C = (int(d) for d in x.shape)
    codes = torch.empty((R, C), dtype=torch.uint8, device=x.device)
    scales = torch.empty((R, C // 32), dtype=torch.uint8, device=x.device)
    _check(lib().mcpu_mxfp8_quantize(_ptr(x), R, C, _ptr(codes), _ptr(scales), _stream(stream)))
    return codes, scales


def embed_tokens(table, tokens, x_out, workspace, stream=None):
    V, H = (int(d) for d in table.shape)
    _check(lib().embed_tokens(_ptr(table), V, H, int(tokens.shape[0]), _ptr(tokens), _ptr(x_out), _ptr(workspace),
                              workspace.numel() * workspace.element_size(), _stream(stream)))


# ---------------------------------------------------------------------------
# a workload resident on the GPU
# ---------------------------------------------------------------------------


class DeviceStep:
    """Uploads a workload (weights, pools, tables, inputs) and runs decode_layer on it."""

    def __init__(self, wl, device="cuda"):
        s = wl.shape
        self.wl = wl
        self.shape = s
        self.weights = DeviceWeights(s, wl.weights, device)
        self.k_pool = wl.k_pool.to(device)
        self.v_pool = wl.v_pool.to(device)
        self.pool = KVPool(s, self.k_pool, self.v_pool)
        self.page_table = torch.from_numpy(np.ascontiguousarray(wl.page_table)).to(device)
        self.seq_lens = torch.from_numpy(np.ascontiguousarray(wl.seq_lens)).to(device)
        self.host_seq_lens = np.ascontiguousarray(wl.seq_lens, dtype=np.int32)
        if wl.is_decode:
            self.cu_q, self.host_cu_q = None, None
        else:
            self.host_cu_q = np.ascontiguousarray(wl.cu_q, dtype=np.int32)
            self.cu_q = torch.from_numpy(self.host_cu_q).to(device)
        T = wl.n_tokens
        self.x_in = wl.x_in.to(device)
        self.x_out = torch.empty_like(self.x_in)
        self.topk_idx = torch.empty((T, s.top_k), dtype=torch.int32, device=device)
        self.topk_w = torch.empty((T, s.top_k), dtype=torch.float32, device=device)
        self.ws = workspace(decode_layer_workspace_size(s, wl.batch, T), device)

    def run(self, taps: Optional[Taps] = None, stream=None):
        decode_layer(self.shape, self.weights, self.pool, self.page_table, self.seq_lens, self.cu_q,
                     self.host_seq_lens, self.host_cu_q, self.x_in, self.x_out, self.topk_idx,
                     self.topk_w, taps, self.ws, stream)

    def device_errors(self) -> int:
        return mcpu_check_device_errors(self.ws)


class DeviceStack:
    """A stack of decoder layers resident on the GPU (per-layer weights and KV
    pools, one page table per attention kind), stepped by calling decode_layer
    once per layer. The residual stream ping-pongs between two buffers so the
    step's input x_in is left intact and the step can be re-run."""

    def __init__(self, spec, device="cuda", n_layers=None):
        from paper_2608_22167_amd import workload as W
        self.spec = spec
        self.n_layers = spec.n_layers if n_layers is None else n_layers
        self.weights, self.k, self.v, self.pools = [], [], [], []
        for i in range(self.n_layers):
            s = spec.shape(i)
            self.weights.append(DeviceWeights(s, W.stack_weights_device(spec, i, device), device))
            self.k.append(W.stack_pool_device(spec, i, "k", device))
            self.v.append(W.stack_pool_device(spec, i, "v", device))
            self.pools.append(KVPool(s, self.k[i], self.v[i]))
        self.pt_full = torch.from_numpy(np.ascontiguousarray(spec.page_table_full)).to(device)
        self.pt_sw = torch.from_numpy(np.ascontiguousarray(spec.page_table_sw)).to(device)
        self.seq_lens = torch.from_numpy(np.ascontiguousarray(spec.seq_lens)).to(device)
        self.host_seq_lens = np.ascontiguousarray(spec.seq_lens, dtype=np.int32)
        B, H, K = spec.batch, spec.shape_full.hidden, spec.shape_full.top_k
        self.x_in = W.stack_x_in(spec).to(device)
        self.buf = [torch.empty_like(self.x_in), torch.empty_like(self.x_in)]
        self.topk_idx = torch.empty((self.n_layers, B, K), dtype=torch.int32, device=device)
        ws = max(decode_layer_workspace_size(spec.shape(i), B, B) for i in range(min(2, self.n_layers)))
        self.ws = workspace(ws, device)

    def run(self, stream=None, logits: Optional[torch.Tensor] = None, rows: Optional[torch.Tensor] = None,
            inputs: Optional[torch.Tensor] = None) -> torch.Tensor:
        """One step through every layer; returns the final residual stream.
        logits, if given ([n_layers, B, E] fp32), receives each layer's router
        logits; inputs, if given ([n_layers, len(rows), H] fp32), receives the
        residual-stream rows `rows` (device int64) that enter each layer."""
        x = self.x_in
        for i in range(self.n_layers):
            y = self.buf[i % 2]
            pt = self.pt_sw if self.spec.is_sw(i) else self.pt_full
            if inputs is not None:
                torch.index_select(x, 0, rows, out=inputs[i])
            taps = None if logits is None else Taps(logits=logits[i].data_ptr())
            decode_layer(self.spec.shape(i), self.weights[i], self.pools[i], pt, self.seq_lens, None,
                         self.host_seq_lens, None, x, y, self.topk_idx[i], None, taps, self.ws, stream)
            x = y
        return x

    def device_errors(self) -> int:
        return mcpu_check_device_errors(self.ws)
