"""Dense float64 brute force of the decoder-layer step, for pinning the oracle.

Written independently of oracle/: it never calls it, works on dense
per-sequence arrays with explicit mask matrices instead of the paged loops,
and implements the page format with numpy reshapes instead of index loops.
"""
import numpy as np
import torch

PAGE = 16


# --- page format (as documented in include/mcpu.h) via reshapes -----------------


def pool_from_logical(k_log: np.ndarray, v_log: np.ndarray):
    """logical [n_pages, Hkv, 16, d] -> page-format arrays of the same shape."""
    n, G, P, d = k_log.shape
    k = k_log.reshape(n, G, P, d // 8, 8).transpose(0, 1, 3, 2, 4).reshape(n, G, P, d)
    v = v_log.reshape(n, G, 4, 4, d // 16, 16).transpose(0, 1, 4, 2, 5, 3).reshape(n, G, P, d)
    return np.ascontiguousarray(k), np.ascontiguousarray(v)


def pool_to_logical(k_pool: np.ndarray, v_pool: np.ndarray):
    n, G, P, d = k_pool.shape
    k = k_pool.reshape(n, G, d // 8, P, 8).transpose(0, 1, 3, 2, 4).reshape(n, G, P, d)
    v = v_pool.reshape(n, G, d // 16, 4, 16, 4).transpose(0, 1, 3, 5, 2, 4).reshape(n, G, P, d)
    return np.ascontiguousarray(k), np.ascontiguousarray(v)


def dense_seq(k_log, v_log, page_table_row, n_tokens):
    """Gather one sequence's first n_tokens keys/values: [n_tokens, Hkv, d]."""
    pos = np.arange(n_tokens)
    pages = page_table_row[pos // PAGE]
    assert (pages >= 0).all()
    return k_log[pages, :, pos % PAGE, :], v_log[pages, :, pos % PAGE, :]


def bf16(x):
    """Round float64 straight to bfloat16 (8 significant bits, nearest-even)."""
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)
    q = np.maximum(e - 8, -133)
    return np.where(x == 0, x, np.ldexp(np.rint(np.ldexp(x, -q)), q))


# --- attention -------------------------------------------------------------------


def attention_dense(q, K, V, p, window, sink, scale):
    """q [Hq, d]; K, V [n, Hkv, d] for positions 0..n-1; query at position p.

    Explicit mask row over all n positions, sink as an extra logit column whose
    value vector is zero.
    """
    Hq, d = q.shape
    n, Hkv, _ = K.shape
    grp = Hq // Hkv
    j = np.arange(n)
    lo = max(0, p - window + 1) if window else 0
    mask = (j >= lo) & (j <= p)
    out = np.zeros((Hq, d))
    for h in range(Hq):
        g = h // grp
        z = (K[:, g, :] @ q[h]) * scale
        z = np.where(mask, z, -np.inf)
        cols = np.concatenate([z, [sink[h] if sink is not None else -np.inf]])
        m = cols.max()
        e = np.exp(cols - m)
        vals = np.concatenate([V[:, g, :], np.zeros((1, d))], axis=0)
        out[h] = (e[:, None] * vals).sum(0) / e.sum()
    return out


# --- layer ------------------------------------------------------------------------


def rmsnorm(x, g, eps):
    return x / np.sqrt((x * x).mean(-1, keepdims=True) + eps) * g


def rope(v, pos, cos, sin):
    h = v.shape[-1] // 2
    c, s = cos[pos].astype(np.float64), sin[pos].astype(np.float64)
    a, b = v[..., :h], v[..., h:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


def swiglu(gate, up, alpha, limit, beta):
    gate = np.minimum(gate, limit)
    up = np.clip(up, -limit, limit)
    return gate * (1.0 / (1.0 + np.exp(-alpha * gate))) * (up + beta)


def stored(x, dtype):
    """A value as a layer of this dtype stores it (bfloat16 or binary32)."""
    x = np.asarray(x, np.float64)
    return bf16(x) if dtype == "bf16" else x.astype(np.float32).astype(np.float64)


def moe_token(hn, W, shape, force=None, kv_only=False):
    """The router reads hn itself; the experts read its stored copy and store
    their SwiGLU activations (kv_only: neither is rounded). Native MXFP4
    experts read both stored rows as MXFP8."""
    f = lambda k: np.asarray(W[k], dtype=np.float64)
    act = (lambda x, dt: np.asarray(x, np.float64)) if kv_only else stored
    mx = (lambda x: mxfp8_round(x)) if shape.expert_fmt == "mxfp4_native" else (lambda x: x)
    logits = f("w_r") @ hn + f("b_r")
    hs = mx(act(hn, shape.dtype))
    lf = logits.astype(np.float32)
    order = np.argsort(-lf, kind="stable")
    sel = order[: shape.top_k] if force is None else np.asarray(force)
    w = np.exp(logits[sel] - logits[sel].max())
    w /= w.sum()
    acc = np.zeros(shape.hidden)
    for e, we in zip(sel, w):
        gu = f("w_gu")[e] @ hs + f("b_gu")[e]
        a = mx(act(swiglu(gu[0::2], gu[1::2], shape.swiglu_alpha, shape.swiglu_limit, shape.swiglu_beta),
                   shape.dtype))
        acc += we * (f("w_d")[e] @ a + f("b_d")[e])
    return acc, sel, w, logits


def weights_np(W):
    out = {}
    for k, v in W.items():
        out[k] = v.float().numpy().astype(np.float64) if isinstance(v, torch.Tensor) else np.asarray(v, np.float64)
    return out


def decode_layer(wl, kv_only=False):
    """Whole step, dense. Returns dict(out, o, h1, idx, w, q). kv_only: only
    the cache entries are rounded to the layer dtype, no activation."""
    s = wl.shape
    act = (lambda x, dt: np.asarray(x, np.float64)) if kv_only else stored
    W = weights_np(wl.weights)
    x = wl.x_in.double().numpy()
    T = x.shape[0]
    kl, vl = pool_to_logical(wl.k_pool.float().numpy().astype(np.float64),
                             wl.v_pool.float().numpy().astype(np.float64))
    d, Hq, Hkv = s.head_dim, s.n_q_heads, s.n_kv_heads
    xn = act(rmsnorm(x, W["g1"], s.rms_eps), s.dtype)
    qkv = xn @ W["w_qkv"].T + W["b_qkv"]
    A = Hq * d
    cu = wl.cu_q
    q_all = np.zeros((T, Hq, d))
    o_all = np.zeros((T, A))
    for b in range(wl.batch):
        r0, r1 = cu[b], cu[b + 1]
        L0 = int(wl.seq_lens[b])
        n = L0 + (r1 - r0)
        Kd = np.zeros((n, Hkv, d))
        Vd = np.zeros((n, Hkv, d))
        lo_needed = max(0, L0 - s.window + 1) if s.window else 0
        pos = np.arange(lo_needed, L0)
        if len(pos):
            pages = wl.page_table[b][pos // PAGE]
            Kd[pos] = kl[pages, :, pos % PAGE, :]
            Vd[pos] = vl[pages, :, pos % PAGE, :]
        for i, r in enumerate(range(r0, r1)):
            p = L0 + i
            row = qkv[r]
            q = act(rope(row[:A].reshape(Hq, d), p, W["rope_cos"], W["rope_sin"]), s.dtype)
            k = stored(rope(row[A:A + Hkv * d].reshape(Hkv, d), p, W["rope_cos"], W["rope_sin"]), s.dtype)
            v = stored(row[A + Hkv * d:].reshape(Hkv, d), s.dtype)
            Kd[p], Vd[p] = k, v
            q_all[r] = q
        for i, r in enumerate(range(r0, r1)):
            p = L0 + i
            o_all[r] = act(attention_dense(q_all[r], Kd, Vd, p, s.window, W["sinks"],
                                           1.0 / np.sqrt(d)).reshape(-1), s.dtype)
    h1 = x + o_all @ W["w_o"].T + W["b_o"]
    hn = rmsnorm(h1, W["g2"], s.rms_eps)
    out = np.zeros_like(h1)
    idx = np.zeros((T, s.top_k), dtype=np.int64)
    ws = np.zeros((T, s.top_k))
    for t in range(T):
        acc, sel, w, _ = moe_token(hn[t], W, s, kv_only=kv_only)
        out[t] = h1[t] + acc
        idx[t], ws[t] = sel, w
    return dict(out=out, o=o_all, h1=h1, idx=idx, w=ws, q=q_all)


# MXFP8 (OCP MX v1.0) restated with numpy: the E4M3 grid spacing at |v| is
# 2^(max(floor(log2 |v|), -6) - 3); round half to even on that grid (numpy's
# rint), saturate at 448; scale 2^(floor(log2 amax) - 8) per 32 elements.
def e4m3_round(y):
    y = np.asarray(y, np.float64)
    a = np.abs(y)
    with np.errstate(divide="ignore"):
        ex = np.floor(np.log2(np.where(a > 0, a, 1.0)))
    step = np.exp2(np.maximum(ex, -6.0) - 3.0)
    r = np.rint(a / step) * step
    return np.sign(y) * np.minimum(r, 448.0)


def mxfp8_round(x):
    """Rows x [..., C] (C % 32 == 0) replaced by their MXFP8 values."""
    x = np.asarray(x, np.float64)
    b = x.reshape(-1, 32)
    amax = np.abs(b).max(axis=1, keepdims=True)
    with np.errstate(divide="ignore"):
        e = np.where(amax > 0, np.floor(np.log2(np.where(amax > 0, amax, 1.0))) - 8.0, -127.0)
    e = np.clip(e, -127.0, 127.0)
    return (e4m3_round(b / np.exp2(e)) * np.exp2(e)).reshape(x.shape)
