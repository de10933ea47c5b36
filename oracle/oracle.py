"""ctypes wrapper of the CPU reference (mcpu_oracle.c). TEST INFRASTRUCTURE ONLY.

Only tests, the smoke check and the benchmark's CPU-baseline leg import this
module. It takes host arrays (numpy or CPU torch tensors), converts them to
the fp32 / fp64 arrays the C code reads, and returns numpy results.
"""
from __future__ import annotations

import ctypes
import os
from typing import Dict, Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB = None

c_i32p = ctypes.POINTER(ctypes.c_int32)


class OrcCfg(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int32) for n in (
        "hidden", "n_q_heads", "n_kv_heads", "head_dim", "n_experts", "top_k", "ffn_dim",
        "page_size", "window", "kv_bf16", "kv_only", "act_mx")] + [
        (n, ctypes.c_double) for n in ("rms_eps", "swiglu_alpha", "swiglu_limit", "swiglu_beta")]


class OrcWeights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in (
        "g1", "w_qkv", "b_qkv", "w_o", "b_o", "g2", "w_r", "b_r", "w_gu", "b_gu", "w_d", "b_d",
        "sinks", "rope_cos", "rope_sin")] + [("rope_max_pos", ctypes.c_int32)]


def lib():
    global _LIB
    if _LIB is None:
        path = os.path.join(_HERE, "libmcpu_oracle.so")
        if not os.path.exists(path):
            from oracle.build import build
            build()
        _LIB = ctypes.CDLL(path)
        L = _LIB
        vp, i32, i64, f64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_double
        L.orc_round_bf16.restype = f64
        L.orc_round_bf16.argtypes = [f64]
        L.orc_round_bf16_array.argtypes = [i64, vp, vp]
        L.orc_rmsnorm.argtypes = [i64, i32, vp, vp, f64, vp]
        L.orc_rope.argtypes = [i32, i32, vp, vp, vp]
        L.orc_swiglu.restype = f64
        L.orc_swiglu.argtypes = [f64, f64, f64, f64, f64]
        L.orc_swiglu_array.argtypes = [i64, vp, vp, f64, f64, f64, vp]
        L.orc_topk.argtypes = [i32, i32, vp, vp]
        L.orc_kv_append.argtypes = [vp, i32, vp, vp, vp, vp, vp, vp, vp, i32, i32]
        L.orc_attention.argtypes = [vp, i32, vp, vp, vp, vp, vp, vp, i32, i32, vp, vp]
        L.orc_moe.argtypes = [vp, vp, i32, vp, vp, vp, vp, vp, vp, vp]
        L.orc_decode_layer.argtypes = [vp, vp, i32, vp, i32, i32, vp, vp, vp, vp, vp, vp,
                                       vp, vp, vp, vp, vp, vp, vp, vp]
        L.orc_decode_layer_rows.argtypes = [vp, vp, i32, vp, i32, i32, vp, vp, vp, vp, vp, i32, vp,
                                            vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.orc_e2m1.restype = f64
        L.orc_e2m1.argtypes = [i32]
        L.orc_mxfp4_dequant.argtypes = [i64, i32, vp, vp, vp]
        L.orc_philox4x32_10.argtypes = [vp, vp, vp]
        L.orc_sample_uniform.restype = f64
        L.orc_sample_uniform.argtypes = [ctypes.c_uint64, i32, i32, i32]
        L.orc_gumbel.restype = f64
        L.orc_gumbel.argtypes = [f64]
        L.orc_lm_head.argtypes = [i32, i32, i32, vp, vp, f64, vp, f64, ctypes.c_uint64, vp, vp, vp, vp, vp, vp,
                                  vp, vp, vp]
        L.orc_e4m3.restype = f64
        L.orc_e4m3.argtypes = [i32]
        L.orc_e4m3_encode.argtypes = [f64]
        L.orc_mxfp8_quant.argtypes = [i64, i32, vp, vp, vp]
        L.orc_pool_to_logical.argtypes = [vp, i32, vp, vp, vp, vp]
        L.orc_pool_from_logical.argtypes = [vp, i32, vp, vp, vp, vp]
    return _LIB


# ---------------------------------------------------------------------------
# array helpers
# ---------------------------------------------------------------------------


def _np(a, dtype) -> np.ndarray:
    """Host copy as a C-contiguous numpy array of dtype (bf16 torch tensors go via fp32)."""
    try:
        import torch
        if isinstance(a, torch.Tensor):
            a = a.detach().cpu()
            if a.dtype == torch.bfloat16:
                a = a.float()
            a = a.numpy()
    except ImportError:  # pragma: no cover
        pass
    return np.ascontiguousarray(np.asarray(a), dtype=dtype)


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


def make_cfg(shape, kv_only=False) -> OrcCfg:
    return OrcCfg(hidden=shape.hidden, n_q_heads=shape.n_q_heads, n_kv_heads=shape.n_kv_heads,
                  head_dim=shape.head_dim, n_experts=shape.n_experts, top_k=shape.top_k,
                  ffn_dim=shape.ffn_dim, page_size=shape.page_size, window=shape.window,
                  kv_bf16=1 if shape.dtype == "bf16" else 0, kv_only=1 if kv_only else 0,
                  act_mx=1 if getattr(shape, "expert_fmt", "") == "mxfp4_native" else 0,
                  rms_eps=shape.rms_eps,
                  swiglu_alpha=shape.swiglu_alpha, swiglu_limit=shape.swiglu_limit,
                  swiglu_beta=shape.swiglu_beta)


class Weights:
    """fp32 host copies of a layer's parameters (MXFP4 experts are decoded first)."""

    def __init__(self, shape, W: Dict):
        self.shape = shape
        f = lambda k: _np(W[k], np.float32)
        self.arr = {k: f(k) for k in ("g1", "w_qkv", "b_qkv", "w_o", "b_o", "g2", "w_r", "b_r",
                                      "b_gu", "b_d", "sinks", "rope_cos", "rope_sin")}
        if "w_gu" in W:
            self.arr["w_gu"] = f("w_gu")
            self.arr["w_d"] = f("w_d")
        else:
            E, I, H = shape.n_experts, shape.ffn_dim, shape.hidden
            self.arr["w_gu"] = mxfp4_dequant(W["w_gu_codes"], W["w_gu_scales"], 2 * I, H).reshape(E, 2 * I, H)
            self.arr["w_d"] = mxfp4_dequant(W["w_d_codes"], W["w_d_scales"], H, I).reshape(E, H, I)
        a = self.arr
        self.struct = OrcWeights(**{k: a[k].ctypes.data for k in a},
                                 rope_max_pos=a["rope_cos"].shape[0])


# ---------------------------------------------------------------------------
# entry points
# ---------------------------------------------------------------------------


def round_bf16(x) -> np.ndarray:
    x = _np(x, np.float64)
    out = np.empty_like(x)
    lib().orc_round_bf16_array(x.size, _p(x), _p(out))
    return out


def rmsnorm(x, g, eps) -> np.ndarray:
    x = _np(x, np.float64)
    g = _np(g, np.float32)
    out = np.empty_like(x)
    lib().orc_rmsnorm(x.shape[0], x.shape[1], _p(x), _p(g), eps, _p(out))
    return out


def rope(v, pos: int, cos, sin) -> np.ndarray:
    v = _np(v, np.float64).copy()
    cos, sin = _np(cos, np.float32), _np(sin, np.float32)
    lib().orc_rope(v.shape[-1], pos, _p(cos), _p(sin), _p(v))
    return v


def swiglu(gate, up, alpha, limit, beta) -> np.ndarray:
    g, u = _np(gate, np.float64), _np(up, np.float64)
    out = np.empty_like(g)
    lib().orc_swiglu_array(g.size, _p(g), _p(u), alpha, limit, beta, _p(out))
    return out


def topk(logits, k: int) -> np.ndarray:
    lg = _np(logits, np.float64)
    out = np.empty(k, dtype=np.int32)
    lib().orc_topk(lg.shape[-1], k, _p(lg), _p(out))
    return out


def e2m1(code: int) -> float:
    return lib().orc_e2m1(code)


def mxfp4_dequant(codes, scales, rows_per_mat: int, cols: int, out=None) -> np.ndarray:
    """out, if given, is a C-contiguous float32 array of rows * cols elements."""
    c = _np(codes, np.uint8)
    s = _np(scales, np.uint8)
    rows = c.size // (cols // 2)
    if out is None:
        out = np.empty((rows, cols), dtype=np.float32)
    elif out.dtype != np.float32 or out.size != rows * cols or not out.flags.c_contiguous:
        raise ValueError("mxfp4_dequant: out must be contiguous float32 of rows * cols elements")
    rc = lib().orc_mxfp4_dequant(rows, cols, _p(c), _p(s), _p(out))
    if rc:
        raise ValueError("invalid MXFP4 input")
    return out


def pool_to_logical(shape, k_pool, v_pool):
    """Page-format pools -> logical [n_pages, Hkv, 16, d] arrays."""
    kp, vp = _np(k_pool, np.float32), _np(v_pool, np.float32)
    n_pages = kp.shape[0]
    ko, vo = np.empty_like(kp), np.empty_like(vp)
    cfg = make_cfg(shape)
    lib().orc_pool_to_logical(ctypes.byref(cfg), n_pages, _p(kp), _p(vp), _p(ko), _p(vo))
    return ko, vo


def pool_from_logical(shape, k_log, v_log):
    kl, vl = _np(k_log, np.float32), _np(v_log, np.float32)
    ko, vo = np.empty_like(kl), np.empty_like(vl)
    cfg = make_cfg(shape)
    lib().orc_pool_from_logical(ctypes.byref(cfg), kl.shape[0], _p(kl), _p(vl), _p(ko), _p(vo))
    return ko, vo


def kv_append(shape, tok_seq, tok_pos, k_new, v_new, k_pool, v_pool, page_table):
    """Returns updated fp32 copies of the pools."""
    cfg = make_cfg(shape)
    ts, tp = _np(tok_seq, np.int32), _np(tok_pos, np.int32)
    kn, vn = _np(k_new, np.float64), _np(v_new, np.float64)
    kp, vpl = _np(k_pool, np.float32).copy(), _np(v_pool, np.float32).copy()
    pt = _np(page_table, np.int32)
    rc = lib().orc_kv_append(ctypes.byref(cfg), ts.size, _p(ts), _p(tp), _p(kn), _p(vn), _p(kp),
                             _p(vpl), _p(pt), pt.shape[1], kp.shape[0])
    if rc:
        raise ValueError("kv_append: page missing for a position")
    return kp, vpl


def attention(shape, tok_seq, tok_pos, q, k_pool, v_pool, page_table, sinks=None) -> np.ndarray:
    """o [T, Hq, d] for queries q [T, Hq, d] against the paged cache."""
    cfg = make_cfg(shape)
    ts, tp = _np(tok_seq, np.int32), _np(tok_pos, np.int32)
    qq = _np(q, np.float64)
    kp, vpl = _np(k_pool, np.float32), _np(v_pool, np.float32)
    pt = _np(page_table, np.int32)
    sk = None if sinks is None else _np(sinks, np.float32)
    o = np.empty_like(qq)
    rc = lib().orc_attention(ctypes.byref(cfg), ts.size, _p(ts), _p(tp), _p(qq), _p(kp), _p(vpl),
                             _p(pt), pt.shape[1], kp.shape[0], _p(sk), _p(o))
    if rc:
        raise ValueError("attention: page missing for a visible key")
    return o


def moe(shape, weights: Weights, h, force_idx=None) -> Dict[str, np.ndarray]:
    cfg = make_cfg(shape)
    hh = _np(h, np.float64)
    T = hh.shape[0]
    out = np.empty_like(hh)
    moe_out = np.empty_like(hh)
    idx = np.empty((T, shape.top_k), dtype=np.int32)
    w = np.empty((T, shape.top_k), dtype=np.float64)
    lg = np.empty((T, shape.n_experts), dtype=np.float64)
    fi = None if force_idx is None else _np(force_idx, np.int32)
    rc = lib().orc_moe(ctypes.byref(cfg), ctypes.byref(weights.struct), T, _p(hh), _p(out), _p(idx),
                       _p(w), _p(lg), _p(moe_out), _p(fi))
    if rc:
        raise ValueError("moe: invalid configuration")
    return dict(out=out, idx=idx, w=w, logits=lg, moe=moe_out)


def decode_layer(wl, weights: Optional[Weights] = None, force_idx=None, k_pool=None,
                 v_pool=None, rows=None, kv_only=False) -> Dict[str, np.ndarray]:
    """One decoder-layer step of workload wl. Returns every intermediate the
    tests compare: q (after rotation), o, h1, moe, out, idx, w, logits and the
    pools after the append. rows (optional, ascending token rows): every new
    token is appended, but only these rows are evaluated and returned (in
    that order). kv_only: round only the cache entries (see mcpu_oracle.c)."""
    s = wl.shape
    cfg = make_cfg(s, kv_only)
    if weights is None:
        weights = Weights(s, wl.weights)
    kp = _np(wl.k_pool if k_pool is None else k_pool, np.float32).copy()
    vpl = _np(wl.v_pool if v_pool is None else v_pool, np.float32).copy()
    pt = _np(wl.page_table, np.int32)
    sl = _np(wl.seq_lens, np.int32)
    cu = None if wl.is_decode else _np(wl.cu_q, np.int32)
    x = _np(wl.x_in, np.float64)
    T, H = x.shape
    sel = None if rows is None else _np(rows, np.int32)
    if sel is not None:
        T = len(sel)
    r = dict(out=np.empty((T, H)), q=np.empty((T, s.n_q_heads, s.head_dim)),
             o=np.empty((T, s.n_q_heads * s.head_dim)), h1=np.empty((T, H)),
             idx=np.empty((T, s.top_k), dtype=np.int32), w=np.empty((T, s.top_k)),
             logits=np.empty((T, s.n_experts)), moe=np.empty((T, H)))
    fi = None if force_idx is None else _np(force_idx, np.int32)
    outs = (_p(r["out"]), _p(r["q"]), _p(r["o"]), _p(r["h1"]), _p(r["idx"]), _p(r["w"]), _p(r["logits"]),
            _p(r["moe"]), _p(fi))
    if sel is None:
        rc = lib().orc_decode_layer(ctypes.byref(cfg), ctypes.byref(weights.struct), wl.batch, _p(pt),
                                    pt.shape[1], kp.shape[0], _p(sl), _p(cu), _p(kp), _p(vpl), _p(x), *outs)
    else:
        rc = lib().orc_decode_layer_rows(ctypes.byref(cfg), ctypes.byref(weights.struct), wl.batch, _p(pt),
                                         pt.shape[1], kp.shape[0], _p(sl), _p(cu), _p(kp), _p(vpl), _p(x),
                                         len(sel), _p(sel), *outs)
    if rc:
        raise ValueError("decode_layer: invalid input (missing page or position beyond RoPE table)")
    r["k_pool"], r["v_pool"] = kp, vpl
    return r


# ---------------------------------------------------------------------------
# generation ends: vocabulary head and sampling
# ---------------------------------------------------------------------------


def philox4x32_10(ctr, key) -> np.ndarray:
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.empty(4, dtype=np.uint32)
    lib().orc_philox4x32_10(_p(c), _p(k), _p(out))
    return out


def sample_uniform(seed: int, seq: int, pos: int, v: int) -> float:
    return lib().orc_sample_uniform(seed, seq, pos, v)


def gumbel(u: float) -> float:
    return lib().orc_gumbel(u)


def lm_head(x, g_final, w_lm, eps, temperature, seed=0, seq_ids=None, positions=None, targets=None,
            want_logits=False) -> Dict[str, np.ndarray]:
    """Vocabulary head and next-token choice for rows x [T, H] (see
    orc_lm_head). Returns tokens, logprob, lse, target_logprob (if targets),
    and logits / pert [T, V] if want_logits."""
    xx = _np(x, np.float64)
    T, H = xx.shape
    g = _np(g_final, np.float32)
    w = _np(w_lm, np.float32)
    V = w.shape[0]
    si = None if seq_ids is None else _np(seq_ids, np.int32)
    ps = None if positions is None else _np(positions, np.int32)
    tg = None if targets is None else _np(targets, np.int32)
    r = dict(tokens=np.empty(T, np.int32), logprob=np.empty(T), lse=np.empty(T))
    if tg is not None:
        r["target_logprob"] = np.empty(T)
    if want_logits:
        r["logits"] = np.empty((T, V))
        r["pert"] = np.empty((T, V))
    rc = lib().orc_lm_head(T, H, V, _p(xx), _p(g), eps, _p(w), float(temperature), int(seed), _p(si), _p(ps),
                           _p(tg), _p(r["tokens"]), _p(r["logprob"]), _p(r["lse"]), _p(r.get("target_logprob")),
                           _p(r.get("logits")), _p(r.get("pert")))
    if rc:
        raise ValueError("lm_head: sampling needs seq_ids and positions")
    return r


def e4m3(code: int) -> float:
    return lib().orc_e4m3(code)


def e4m3_encode(x: float) -> int:
    return lib().orc_e4m3_encode(float(x))


def mxfp8_quant(x):
    """Rows x [R, C] (C a multiple of 32) -> (codes uint8 [R, C], scales uint8 [R, C/32])."""
    xx = _np(x, np.float64)
    R, C = xx.shape
    codes = np.empty((R, C), np.uint8)
    scales = np.empty((R, C // 32), np.uint8)
    if lib().orc_mxfp8_quant(R, C, _p(xx), _p(codes), _p(scales)):
        raise ValueError("mxfp8_quant: columns must be a multiple of 32")
    return codes, scales
