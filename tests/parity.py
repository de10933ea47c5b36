"""Comparison helpers for GPU-vs-reference parity tests.

Tolerances: bf16 layers max-abs 2e-2 and relative-L2 1e-2; fp32 layers 1e-4
for both. Router selections must match exactly wherever the reference's k-th
and (k+1)-th logits (in fp32) differ by more than 1e-3; tokens inside that gap
are re-run on the reference with the GPU's selection.
"""
import numpy as np

TOL = {"bf16": (2e-2, 1e-2), "f32": (1e-4, 1e-4)}
TIE_GAP = 1e-3


def rel_l2(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.linalg.norm(a - b) / max(np.linalg.norm(b), 1e-300))


def check(name, got, ref, dtype, scale=1.0):
    atol, rtol = TOL[dtype]
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    assert got.shape == ref.shape, (name, got.shape, ref.shape)
    assert np.isfinite(got).all(), f"{name}: non-finite values"
    err = np.abs(got - ref)
    mx = float(err.max()) if got.size else 0.0
    rl = rel_l2(got, ref)
    where = np.unravel_index(int(err.argmax()), err.shape) if got.size else ()
    msg = (f"{name}: max-abs {mx:.3e} (tol {atol * scale:.1e}) at {tuple(int(i) for i in where)} "
           f"(ref {float(ref[where]) if got.size else 0.0:.4g}), rel-L2 {rl:.3e} (tol {rtol * scale:.1e})")
    assert mx <= atol * scale and rl <= rtol * scale, msg
    return mx, rl


def near_tie_tokens(logits, k):
    """Tokens whose k-th and (k+1)-th largest fp32 logits are within TIE_GAP."""
    lf = np.sort(np.asarray(logits, np.float32), axis=1)[:, ::-1]
    if lf.shape[1] <= k:
        return np.zeros(lf.shape[0], bool)
    return (lf[:, k - 1] - lf[:, k]).astype(np.float64) <= TIE_GAP


def check_router(gpu_idx, ref_idx, ref_logits, k):
    """Exact set equality outside near ties; returns the near-tie mask."""
    tie = near_tie_tokens(ref_logits, k)
    g = np.sort(np.asarray(gpu_idx), 1)
    r = np.sort(np.asarray(ref_idx), 1)
    bad = (~tie) & (g != r).any(1)
    assert not bad.any(), f"router sets differ at tokens {np.nonzero(bad)[0][:10]}"
    return tie


def bf16_ulp(x):
    """Spacing of bfloat16 numbers at |x| (normal range; 2^-133 below it)."""
    a = np.abs(np.asarray(x, np.float64))
    e = np.floor(np.log2(np.maximum(a, 2.0 ** -126)))
    return np.exp2(e - 7)


def weights_by_expert(gpu_idx, gpu_w, ref_idx, ref_w):
    """Top-k weights of both sides in ascending expert order per token (the
    sets must already agree), for element-wise comparison."""
    gi, ri = np.asarray(gpu_idx), np.asarray(ref_idx)
    go, ro = np.argsort(gi, 1, kind="stable"), np.argsort(ri, 1, kind="stable")
    gs, rs = np.take_along_axis(gi, go, 1), np.take_along_axis(ri, ro, 1)
    assert (gs == rs).all(), "expert sets differ"
    return (np.take_along_axis(np.asarray(gpu_w, np.float64), go, 1),
            np.take_along_axis(np.asarray(ref_w, np.float64), ro, 1))
