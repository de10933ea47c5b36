"""Seeded synthetic workloads for the decode step (inputs only).

The paper trains gpt-oss-20b and says the Run stage of its rollout pipeline is
GPU bound and dominated by generation (Sec. 3.2; Sec. 4.2 measures rollout
throughput in tokens/s). It publishes no trajectories or weights we can use,
so every tensor here is drawn from a seeded generator with the shapes of a
gpt-oss-20b decoder layer (model card cited in Sec. 4) and context lengths
modelled on the response lengths of Sec. 4.1.

This module draws random numbers and lays out page tables. It holds none of
the layer's arithmetic: the GPU path and the CPU reference both consume what
it returns. Large tensors come from the counter-based generator in
``csrc/synth.c`` (Irwin-Hall(8) variates, variance 1, reproducible bit for bit
on any IEEE-754 machine); small integer arrays from ``numpy.random``.
"""
from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass, field, replace
from typing import Dict, Optional

import numpy as np
import torch

PAGE = 16

# --------------------------------------------------------------------------
# shapes
# --------------------------------------------------------------------------


@dataclass(frozen=True)
class LayerShape:
    hidden: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    n_experts: int
    top_k: int
    ffn_dim: int
    window: int = 0            # 0 = full attention, else keys [p-window+1, p]
    dtype: str = "bf16"        # "f32" or "bf16": matrices, KV cache, GEMM operands
    expert_fmt: str = "dense"  # "dense" (same dtype), "mxfp4", or "mxfp4_native" (MXFP8 activations)
    page_size: int = PAGE
    rms_eps: float = 1e-5
    swiglu_alpha: float = 1.702
    swiglu_limit: float = 7.0
    swiglu_beta: float = 1.0

    def __post_init__(self):
        if self.dtype not in ("f32", "bf16") or self.expert_fmt not in ("dense", "mxfp4", "mxfp4_native"):
            raise ValueError(f"dtype {self.dtype!r} / expert_fmt {self.expert_fmt!r}")

    @property
    def qkv_dim(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def attn_dim(self) -> int:
        return self.n_q_heads * self.head_dim

    @property
    def torch_dtype(self):
        return torch.float32 if self.dtype == "f32" else torch.bfloat16


TINY = LayerShape(hidden=256, n_q_heads=8, n_kv_heads=2, head_dim=32, n_experts=8,
                  top_k=2, ffn_dim=256, dtype="f32")
GPT_OSS_20B = LayerShape(hidden=2880, n_q_heads=64, n_kv_heads=8, head_dim=64,
                         n_experts=32, top_k=4, ffn_dim=2880, dtype="bf16")
GPT_OSS_20B_SW = replace(GPT_OSS_20B, window=128)

# --------------------------------------------------------------------------
# counter-based generator (csrc/synth.c)
# --------------------------------------------------------------------------

_HERE = os.path.dirname(os.path.abspath(__file__))
_SYNTH = None


def _synth():
    global _SYNTH
    if _SYNTH is None:
        path = os.path.join(_HERE, "libmcpu_synth.so")
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(path)
        u64, i64, f32, vp = ctypes.c_uint64, ctypes.c_int64, ctypes.c_float, ctypes.c_void_p
        lib.synth_fill_f32.argtypes = [u64, u64, u64, i64, f32, f32, vp]
        lib.synth_fill_bf16.argtypes = [u64, u64, u64, i64, f32, f32, vp]
        lib.synth_fill_u8.argtypes = [u64, u64, u64, i64, vp]
        lib.synth_fill_fast_bf16.argtypes = [u64, u64, ctypes.c_uint32, i64, f32, f32, vp]
        _SYNTH = lib
    return _SYNTH


IH_STD = math.sqrt(8 * (256 * 256 - 1) / 12.0)  # std of a sum of eight uniform bytes


def synth_normal(seed: int, tid: int, shape, std: float = 1.0, mean: float = 0.0,
                 dtype=torch.float32, offset: int = 0) -> torch.Tensor:
    """Seeded N(mean, std^2)-like tensor (Irwin-Hall(8)); fp32 or bf16."""
    n = int(np.prod(shape)) if len(shape) else 1
    c = float(np.float32(std / IH_STD))
    if dtype == torch.float32:
        out = torch.empty(n, dtype=torch.float32)
        _synth().synth_fill_f32(seed, tid, offset, n, c, float(np.float32(mean)), out.data_ptr())
    elif dtype == torch.bfloat16:
        out = torch.empty(n, dtype=torch.bfloat16)
        _synth().synth_fill_bf16(seed, tid, offset, n, c, float(np.float32(mean)), out.data_ptr())
    else:
        raise ValueError(dtype)
    return out.view(*shape)


IH4_STD = math.sqrt(4 * (256 * 256 - 1) / 12.0)  # std of a sum of four uniform bytes


def synth_fast_normal(seed: int, tid: int, n: int, std: float = 1.0, offset: int = 0) -> torch.Tensor:
    """Bulk Irwin-Hall(4) bf16 values for KV pools (indices below 2^32)."""
    out = torch.empty(n, dtype=torch.bfloat16)
    _synth().synth_fill_fast_bf16(seed, tid, offset, n, float(np.float32(std / IH4_STD)), 0.0, out.data_ptr())
    return out


# --- device twin (csrc/synth_fill.hip): the same values, generated in HBM ----------

_SYNTH_DEV = None


def _synth_dev():
    global _SYNTH_DEV
    if _SYNTH_DEV is None:
        path = os.path.join(_HERE, "libmcpu_synth_dev.so")
        if not os.path.exists(path):
            raise RuntimeError(f"{path} is not built; run __graft_entry__.build()")
        lib = ctypes.CDLL(path)
        u64, i64, f32, vp = ctypes.c_uint64, ctypes.c_int64, ctypes.c_float, ctypes.c_void_p
        lib.synth_fill_device_bf16.argtypes = [u64, u64, u64, i64, f32, f32, vp, vp]
        lib.synth_fill_device_fast_bf16.argtypes = [u64, u64, ctypes.c_uint32, i64, f32, f32, vp, vp]
        lib.synth_fill_device_u8.argtypes = [u64, u64, u64, i64, vp, vp]
        _SYNTH_DEV = lib
    return _SYNTH_DEV


def _stream_ptr():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def fill_normal_device(out: torch.Tensor, seed: int, tid: int, std: float = 1.0, mean: float = 0.0,
                       offset: int = 0) -> torch.Tensor:
    """Device twin of synth_normal (bf16 only)."""
    assert out.dtype == torch.bfloat16 and out.is_contiguous()
    c = float(np.float32(std / IH_STD))
    rc = _synth_dev().synth_fill_device_bf16(seed, tid, offset, out.numel(), c, float(np.float32(mean)),
                                             out.data_ptr(), _stream_ptr())
    if rc:
        raise RuntimeError(f"device fill failed ({rc})")
    return out


def fill_fast_normal_device(out: torch.Tensor, seed: int, tid: int, std: float = 1.0, offset: int = 0):
    """Device twin of synth_fast_normal."""
    assert out.dtype == torch.bfloat16 and out.is_contiguous() and offset + out.numel() <= 2 ** 32
    rc = _synth_dev().synth_fill_device_fast_bf16(seed, tid, offset, out.numel(), float(np.float32(std / IH4_STD)),
                                                  0.0, out.data_ptr(), _stream_ptr())
    if rc:
        raise RuntimeError(f"device fill failed ({rc})")
    return out


def fill_bytes_device(out: torch.Tensor, seed: int, tid: int, offset: int = 0) -> torch.Tensor:
    assert out.dtype == torch.uint8 and out.is_contiguous()
    rc = _synth_dev().synth_fill_device_u8(seed, tid, offset, out.numel(), out.data_ptr(), _stream_ptr())
    if rc:
        raise RuntimeError(f"device fill failed ({rc})")
    return out


def synth_bytes(seed: int, tid: int, shape, offset: int = 0) -> torch.Tensor:
    n = int(np.prod(shape))
    out = torch.empty(n, dtype=torch.uint8)
    _synth().synth_fill_u8(seed, tid, offset, n, out.data_ptr())
    return out.view(*shape)


# tensor ids of the generator streams (per layer: + 100 * layer)
TID = dict(g1=1, w_qkv=2, b_qkv=3, w_o=4, b_o=5, g2=6, w_r=7, b_r=8, w_gu=9, b_gu=10,
           w_d=11, b_d=12, sinks=13, k_pool=20, v_pool=21, x_in=22,
           w_gu_codes=30, w_gu_scales=31, w_d_codes=32, w_d_scales=33)

# --------------------------------------------------------------------------
# the generation ends: token embedding, final RMSNorm gain, unembedding
# (gpt-oss vocabulary of 201088 ids); the embedding rows are N(0, 1) like the
# residual stream the layer workloads start from
# --------------------------------------------------------------------------

GPT_OSS_VOCAB = 201088
LM_TID = dict(g_final=90, w_lm=91, embed=92)


def lm_weights_host(seed: int, hidden: int, vocab: int, embed: bool = True) -> Dict[str, torch.Tensor]:
    W = dict(g_final=synth_normal(seed, LM_TID["g_final"], (hidden,), std=0.02, mean=1.0),
             w_lm=synth_normal(seed, LM_TID["w_lm"], (vocab, hidden), std=0.02, dtype=torch.bfloat16))
    if embed:
        W["embed"] = synth_normal(seed, LM_TID["embed"], (vocab, hidden), dtype=torch.bfloat16)
    return W


def lm_weights_device(seed: int, hidden: int, vocab: int, device="cuda") -> Dict[str, torch.Tensor]:
    """The same tensors generated in HBM (the host regenerates any rows it needs)."""
    W = dict(g_final=synth_normal(seed, LM_TID["g_final"], (hidden,), std=0.02, mean=1.0).to(device))
    W["w_lm"] = fill_normal_device(torch.empty((vocab, hidden), dtype=torch.bfloat16, device=device), seed,
                                   LM_TID["w_lm"], std=0.02)
    W["embed"] = fill_normal_device(torch.empty((vocab, hidden), dtype=torch.bfloat16, device=device), seed,
                                    LM_TID["embed"])
    return W


# --------------------------------------------------------------------------
# workload
# --------------------------------------------------------------------------


@dataclass
class Workload:
    name: str
    shape: LayerShape
    seed: int
    seq_lens: np.ndarray          # int32 [B]: tokens cached before the step
    q_lens: np.ndarray            # int32 [B]: new tokens per sequence (1 = decode)
    page_table: np.ndarray        # int32 [B, max_pages]: physical page or -1
    n_pages: int                  # pool size in pages
    weights: Dict[str, torch.Tensor] = field(default_factory=dict)
    k_pool: Optional[torch.Tensor] = None   # [n_pages, Hkv, 16, d] (page format in mcpu.h)
    v_pool: Optional[torch.Tensor] = None
    x_in: Optional[torch.Tensor] = None     # fp32 [T, hidden]
    notes: str = ""

    @property
    def batch(self) -> int:
        return int(self.seq_lens.shape[0])

    @property
    def n_tokens(self) -> int:
        return int(self.q_lens.sum())

    @property
    def cu_q(self) -> np.ndarray:
        return np.concatenate([[0], np.cumsum(self.q_lens)]).astype(np.int32)

    @property
    def is_decode(self) -> bool:
        return bool(np.all(self.q_lens == 1))

    @property
    def max_pages(self) -> int:
        return int(self.page_table.shape[1])

    def visible_keys(self) -> int:
        """Number of (query, key) pairs per KV head, i.e. keys each query attends to."""
        tot = 0
        W = self.shape.window
        for b in range(self.batch):
            for i in range(int(self.q_lens[b])):
                p = int(self.seq_lens[b]) + i
                lo = max(0, p - W + 1) if W else 0
                tot += p - lo + 1
        return tot


def rope_table(max_pos: int, head_dim: int, theta: float = 150000.0):
    """cos/sin tables [max_pos, head_dim/2] (fp32) for the pair (j, j + d/2).

    A model parameter like the weights: both sides read the same table, so its
    exact frequencies cannot affect parity.
    """
    half = head_dim // 2
    inv = theta ** (-np.arange(half, dtype=np.float64) * 2.0 / head_dim)
    ang = np.arange(max_pos, dtype=np.float64)[:, None] * inv[None, :]
    return (torch.from_numpy(np.cos(ang).astype(np.float32)),
            torch.from_numpy(np.sin(ang).astype(np.float32)))


def _pages(seq_lens, q_lens, window, rng, slack=1.25):
    """Random sparse page placement; pages wholly left of the window are -1."""
    B = len(seq_lens)
    need_hi = [(int(s) + int(q) + PAGE - 1) // PAGE for s, q in zip(seq_lens, q_lens)]
    need_lo = []
    for s in seq_lens:
        lo = max(0, int(s) - window + 1) if window else 0
        need_lo.append(lo // PAGE)
    max_pages = max(need_hi)
    n_needed = sum(h - l for h, l in zip(need_hi, need_lo))
    n_pages = max(n_needed + 1, int(math.ceil(slack * n_needed)))
    perm = rng.permutation(n_pages)[:n_needed].astype(np.int32)
    pt = np.full((B, max_pages), -1, dtype=np.int32)
    k = 0
    for b in range(B):
        cnt = need_hi[b] - need_lo[b]
        pt[b, need_lo[b]:need_hi[b]] = perm[k:k + cnt]
        k += cnt
    return pt, n_pages


def make_workload(name: str, shape: LayerShape, seq_lens, q_lens, seed: int,
                  router_bias: Optional[np.ndarray] = None, weights: bool = True,
                  kv: bool = True, sink_std: float = 0.02, layer: int = 0,
                  notes: str = "") -> Workload:
    """Draw every input of one decoder-layer step.

    Weights N(0, 0.02) (gains 1 + N(0, 0.02)), cached K/V and x_in N(0, 1).
    """
    seq_lens = np.asarray(seq_lens, dtype=np.int32)
    q_lens = np.asarray(q_lens, dtype=np.int32)
    rng = np.random.default_rng(seed)
    pt, n_pages = _pages(seq_lens, q_lens, shape.window, rng)
    wl = Workload(name=name, shape=shape, seed=seed, seq_lens=seq_lens, q_lens=q_lens,
                  page_table=pt, n_pages=n_pages, notes=notes)
    s = shape
    dt = s.torch_dtype
    base = 100 * layer
    T = int(q_lens.sum())
    if weights:
        W = {}
        nrm = lambda key, shp, std=0.02, mean=0.0, d=torch.float32: synth_normal(
            seed, base + TID[key], shp, std=std, mean=mean, dtype=d)
        W["g1"] = nrm("g1", (s.hidden,), mean=1.0)
        W["w_qkv"] = nrm("w_qkv", (s.qkv_dim, s.hidden), d=dt)
        W["b_qkv"] = nrm("b_qkv", (s.qkv_dim,))
        W["w_o"] = nrm("w_o", (s.hidden, s.attn_dim), d=dt)
        W["b_o"] = nrm("b_o", (s.hidden,))
        W["g2"] = nrm("g2", (s.hidden,), mean=1.0)
        W["w_r"] = nrm("w_r", (s.n_experts, s.hidden), d=dt)
        if router_bias is None:
            W["b_r"] = nrm("b_r", (s.n_experts,))
        else:
            W["b_r"] = torch.from_numpy(np.asarray(router_bias, dtype=np.float32))
        if s.expert_fmt == "dense":
            W["w_gu"] = nrm("w_gu", (s.n_experts, 2 * s.ffn_dim, s.hidden), d=dt)
            W["w_d"] = nrm("w_d", (s.n_experts, s.hidden, s.ffn_dim), d=dt)
        else:
            W.update(mxfp4_random(seed, base, s))
        W["b_gu"] = nrm("b_gu", (s.n_experts, 2 * s.ffn_dim))
        W["b_d"] = nrm("b_d", (s.n_experts, s.hidden))
        W["sinks"] = nrm("sinks", (s.n_q_heads,), std=sink_std)
        max_pos = int((seq_lens + q_lens).max()) + 1
        W["rope_cos"], W["rope_sin"] = rope_table(max_pos, s.head_dim)
        wl.weights = W
    if kv:
        shp = (n_pages, s.n_kv_heads, PAGE, s.head_dim)
        wl.k_pool = synth_normal(seed, base + TID["k_pool"], shp, dtype=dt)
        wl.v_pool = synth_normal(seed, base + TID["v_pool"], shp, dtype=dt)
    wl.x_in = synth_normal(seed, base + TID["x_in"], (T, s.hidden))
    return wl


def mxfp4_random(seed: int, base: int, s: LayerShape) -> Dict[str, torch.Tensor]:
    """Random MXFP4 expert weights: uniform e2m1 codes, e8m0 scales in {117,118,119}.

    Codes: [E, rows, cols/2] bytes, low nibble = even column. Scales: [E, rows, cols/32].
    """
    E, I, H = s.n_experts, s.ffn_dim, s.hidden
    out = {}
    for key, rows, cols in (("w_gu", 2 * I, H), ("w_d", H, I)):
        out[key + "_codes"] = synth_bytes(seed, base + TID[key + "_codes"], (E, rows, cols // 2))
        raw = synth_bytes(seed, base + TID[key + "_scales"], (E, rows, cols // 32))
        out[key + "_scales"] = (117 + (raw % 3)).to(torch.uint8)
    return out


def zipf_router_bias(n_experts: int, s: float, seed: int) -> np.ndarray:
    """Router bias b[e] = log p_{pi(e)} with p_r proportional to r^-s, pi a seeded permutation."""
    r = np.arange(1, n_experts + 1, dtype=np.float64)
    p = r ** (-s)
    p /= p.sum()
    perm = np.random.default_rng(seed + 7).permutation(n_experts)
    return np.log(p[perm]).astype(np.float32)


def lognormal_lengths(rng, n, median, sigma, cap, lo=1):
    x = np.exp(rng.normal(math.log(median), sigma, size=n))
    return np.clip(np.round(x), lo, cap).astype(np.int32)


# --------------------------------------------------------------------------
# the named configurations (seed 1000 + index)
# --------------------------------------------------------------------------


def tiny_f32(seed=1001, batch=4, **kw) -> Workload:
    """Tiny fp32 layer: hidden 256, 8/2 heads, d 32, 8 experts top-2, I 256;
    full attention with sinks; contexts U{64..256}; B = 4."""
    rng = np.random.default_rng(seed + 1)
    ctx = rng.integers(64, 257, size=batch)
    return make_workload("tiny_f32_b%d" % batch, kw.pop("shape", TINY), ctx, np.ones(batch), seed, **kw)


def full_b64(seed=1002, batch=64, ctx_lo=2048, ctx_hi=16384, **kw) -> Workload:
    """gpt-oss-20b-shaped full-attention layer, bf16, B = 64, contexts U{2048..16384}."""
    rng = np.random.default_rng(seed + 1)
    ctx = rng.integers(ctx_lo, ctx_hi + 1, size=batch)
    return make_workload("full_attn_bf16_b%d_ctx%d-%d" % (batch, ctx_lo, ctx_hi),
                         kw.pop("shape", GPT_OSS_20B), ctx, np.ones(batch), seed, **kw)


def sliding_b256(seed=1003, batch=256, median=4096, cap=32768, **kw) -> Workload:
    """Sliding-window (128) layer, bf16, B = 256, contexts log-normal (median 4096,
    sigma 1, cap 32768); router bias Zipf(s = 1.1) over a seeded expert permutation."""
    rng = np.random.default_rng(seed + 1)
    ctx = lognormal_lengths(rng, batch, median, 1.0, cap)
    bias = zipf_router_bias(GPT_OSS_20B.n_experts, 1.1, seed)
    return make_workload("sliding128_bf16_b%d_lognormal%d" % (batch, median),
                         kw.pop("shape", GPT_OSS_20B_SW), ctx, np.ones(batch), seed,
                         router_bias=bias, **kw)


def mixed_prefill(seed=1004, n_dec=192, n_pre=64, ctx_lo=1024, ctx_hi=24576,
                  chunk_lo=256, chunk_hi=4096, expert_fmt="dense", **kw) -> Workload:
    """Mixed step: n_dec decode sequences + n_pre sequences appending tool-observation
    chunks of U{256..4096} tokens; contexts U{1024..24576}; full attention, bf16
    (experts bf16, or MXFP4 with expert_fmt)."""
    rng = np.random.default_rng(seed + 1)
    B = n_dec + n_pre
    ctx = rng.integers(ctx_lo, ctx_hi + 1, size=B)
    q = np.ones(B, dtype=np.int32)
    q[n_dec:] = rng.integers(chunk_lo, chunk_hi + 1, size=n_pre)
    shape = replace(kw.pop("shape", GPT_OSS_20B), expert_fmt=expert_fmt)
    tag = {"dense": "bf16", "mxfp4": "mxfp4", "mxfp4_native": "mxfp4x8"}[expert_fmt]
    return make_workload("mixed_%s_%ddec_%dpre" % (tag, n_dec, n_pre), shape, ctx, q, seed, **kw)


def restrict(wl: Workload, seqs):
    """The same step restricted to sequences `seqs`, with a compact page pool
    holding only their pages (same values). Returns (workload, token rows)."""
    seqs = np.asarray(seqs)
    pt = wl.page_table[seqs]
    used = np.unique(pt[pt >= 0])
    remap = -np.ones(wl.n_pages, np.int64)
    remap[used] = np.arange(len(used))
    sub = Workload(name=wl.name + "_subset", shape=wl.shape, seed=wl.seed, seq_lens=wl.seq_lens[seqs],
                   q_lens=wl.q_lens[seqs],
                   page_table=np.where(pt >= 0, remap[np.maximum(pt, 0)], -1).astype(np.int32),
                   n_pages=len(used), weights=wl.weights)
    idx = torch.from_numpy(used)
    sub.k_pool, sub.v_pool = wl.k_pool[idx], wl.v_pool[idx]
    cu = wl.cu_q
    rows = np.concatenate([np.arange(cu[b], cu[b + 1]) for b in seqs])
    sub.x_in = wl.x_in[torch.from_numpy(rows)]
    return sub, rows


def custom(shape: LayerShape, ctx, q, seed, name="custom", **kw) -> Workload:
    return make_workload(name, shape, ctx, q, seed, **kw)


# --------------------------------------------------------------------------
# the 24-layer stack: alternating sliding-window (even layers) and full (odd)
# attention, MXFP4 experts, 512 sequences, log-normal contexts (median 8192,
# sigma 1, cap 65536). Large tensors are generated in HBM by the device twin
# of the generator; the host regenerates exactly the slices it needs.
# --------------------------------------------------------------------------


@dataclass
class StackSpec:
    name: str
    seed: int
    n_layers: int
    shape_full: LayerShape
    shape_sw: LayerShape
    seq_lens: np.ndarray
    page_table_full: np.ndarray
    n_pages_full: int
    page_table_sw: np.ndarray
    n_pages_sw: int
    rope_max_pos: int

    @property
    def batch(self) -> int:
        return int(self.seq_lens.shape[0])

    def is_sw(self, layer: int) -> bool:
        return layer % 2 == 0

    def shape(self, layer: int) -> LayerShape:
        return self.shape_sw if self.is_sw(layer) else self.shape_full

    def page_table(self, layer: int) -> np.ndarray:
        return self.page_table_sw if self.is_sw(layer) else self.page_table_full

    def n_pages(self, layer: int) -> int:
        return self.n_pages_sw if self.is_sw(layer) else self.n_pages_full

    def tid(self, layer: int, key: str) -> int:
        return 100 * (layer + 1) + TID[key]

    def kv_bytes_read(self) -> int:
        """K/V bytes the step's attention reads over all layers (2 KiB per visible key per layer)."""
        s = self.shape_full
        per_key = s.n_kv_heads * s.head_dim * 2 * 2
        full = int((self.seq_lens.astype(np.int64) + 1).sum())
        sw = int(np.minimum(self.seq_lens.astype(np.int64) + 1, self.shape_sw.window).sum())
        n_full = sum(0 if self.is_sw(i) else 1 for i in range(self.n_layers))
        return per_key * (n_full * full + (self.n_layers - n_full) * sw)


def stack24(seed=1005, batch=512, median=8192, cap=65536, n_layers=24, slack=1.05,
            base: LayerShape = None) -> StackSpec:
    """24-layer gpt-oss-20b-shaped stack, bf16 attention and router, MXFP4
    experts (base: another bf16 layer shape for small test stacks)."""
    rng = np.random.default_rng(seed + 1)
    ctx = lognormal_lengths(rng, batch, median, 1.0, cap)
    q = np.ones(batch, dtype=np.int32)
    full = replace(GPT_OSS_20B if base is None else base, expert_fmt="mxfp4", window=0)
    sw = replace(full, window=128)
    pt_f, np_f = _pages(ctx, q, 0, np.random.default_rng(seed + 2), slack)
    pt_s, np_s = _pages(ctx, q, 128, np.random.default_rng(seed + 3), slack)
    return StackSpec(name="stack%d_mxfp4_b%d_lognormal%d" % (n_layers, batch, median), seed=seed,
                     n_layers=n_layers, shape_full=full, shape_sw=sw, seq_lens=ctx,
                     page_table_full=pt_f, n_pages_full=np_f, page_table_sw=pt_s, n_pages_sw=np_s,
                     rope_max_pos=int(ctx.max()) + 2)


def stack_small_weights(spec: StackSpec, layer: int) -> Dict[str, torch.Tensor]:
    """Gains, biases, sinks and the RoPE table of one layer (host, fp32)."""
    s = spec.shape(layer)
    nrm = lambda key, shp, std=0.02, mean=0.0: synth_normal(spec.seed, spec.tid(layer, key), shp, std=std, mean=mean)
    W = dict(g1=nrm("g1", (s.hidden,), mean=1.0), b_qkv=nrm("b_qkv", (s.qkv_dim,)), b_o=nrm("b_o", (s.hidden,)),
             g2=nrm("g2", (s.hidden,), mean=1.0), b_r=nrm("b_r", (s.n_experts,)),
             b_gu=nrm("b_gu", (s.n_experts, 2 * s.ffn_dim)), b_d=nrm("b_d", (s.n_experts, s.hidden)),
             sinks=nrm("sinks", (s.n_q_heads,)))
    W["rope_cos"], W["rope_sin"] = rope_table(spec.rope_max_pos, s.head_dim)
    return W


def _mx_dims(s: LayerShape):
    E, I, H = s.n_experts, s.ffn_dim, s.hidden
    return {"w_gu": (E, 2 * I, H), "w_d": (E, H, I)}


def stack_weights_host(spec: StackSpec, layer: int, experts=None) -> Dict[str, torch.Tensor]:
    """All of a layer's parameters on the host. MXFP4 experts not in `experts`
    (when given) are left zero-filled, so only the experts a sample uses are drawn."""
    s = spec.shape(layer)
    W = stack_small_weights(spec, layer)
    nb = lambda key, shp: synth_normal(spec.seed, spec.tid(layer, key), shp, std=0.02, dtype=torch.bfloat16)
    W["w_qkv"] = nb("w_qkv", (s.qkv_dim, s.hidden))
    W["w_o"] = nb("w_o", (s.hidden, s.attn_dim))
    W["w_r"] = nb("w_r", (s.n_experts, s.hidden))
    if experts is not None and len(experts) == 0:
        return W  # no expert tensors wanted
    for key, (E, rows, cols) in _mx_dims(s).items():
        codes = torch.zeros((E, rows, cols // 2), dtype=torch.uint8)
        scales = torch.zeros((E, rows, cols // 32), dtype=torch.uint8)
        for e in (range(E) if experts is None else experts):
            codes[e] = synth_bytes(spec.seed, spec.tid(layer, key + "_codes"), (rows, cols // 2),
                                   offset=e * rows * (cols // 2))
            raw = synth_bytes(spec.seed, spec.tid(layer, key + "_scales"), (rows, cols // 32),
                              offset=e * rows * (cols // 32))
            scales[e] = 117 + raw % 3
        W[key + "_codes"], W[key + "_scales"] = codes, scales
    return W


def stack_weights_device(spec: StackSpec, layer: int, device="cuda") -> Dict[str, torch.Tensor]:
    """The same parameters generated in HBM (the large tensors never touch the host)."""
    s = spec.shape(layer)
    W = {k: v.to(device) for k, v in stack_small_weights(spec, layer).items()}
    for key, shp in (("w_qkv", (s.qkv_dim, s.hidden)), ("w_o", (s.hidden, s.attn_dim)),
                     ("w_r", (s.n_experts, s.hidden))):
        W[key] = fill_normal_device(torch.empty(shp, dtype=torch.bfloat16, device=device), spec.seed,
                                    spec.tid(layer, key), std=0.02)
    for key, (E, rows, cols) in _mx_dims(s).items():
        W[key + "_codes"] = fill_bytes_device(torch.empty((E, rows, cols // 2), dtype=torch.uint8, device=device),
                                              spec.seed, spec.tid(layer, key + "_codes"))
        raw = fill_bytes_device(torch.empty((E, rows, cols // 32), dtype=torch.uint8, device=device), spec.seed,
                                spec.tid(layer, key + "_scales"))
        W[key + "_scales"] = (117 + raw % 3).to(torch.uint8)
    return W


def stack_pool_device(spec: StackSpec, layer: int, which: str, device="cuda") -> torch.Tensor:
    """K or V pool of one layer, [n_pages, Hkv, 16, d] bf16, bulk generator, N(0, 1)."""
    s = spec.shape(layer)
    pool = torch.empty((spec.n_pages(layer), s.n_kv_heads, PAGE, s.head_dim), dtype=torch.bfloat16, device=device)
    return fill_fast_normal_device(pool.view(-1), spec.seed, spec.tid(layer, which + "_pool")).view(pool.shape)


def stack_pages_host(spec: StackSpec, layer: int, which: str, pages) -> torch.Tensor:
    """The listed pages of a layer's K or V pool, regenerated on the host."""
    s = spec.shape(layer)
    per = s.n_kv_heads * PAGE * s.head_dim
    out = torch.empty((len(pages), s.n_kv_heads, PAGE, s.head_dim), dtype=torch.bfloat16)
    for i, p in enumerate(pages):
        out[i] = synth_fast_normal(spec.seed, spec.tid(layer, which + "_pool"), per, offset=int(p) * per).view(
            s.n_kv_heads, PAGE, s.head_dim)
    return out


def stack_x_in(spec: StackSpec) -> torch.Tensor:
    return synth_normal(spec.seed, TID["x_in"], (spec.batch, spec.shape_full.hidden))
