"""Pins of the reference's generation ends (oracle: orc_lm_head and its
sampling draws), CPU only.

The sampling rule is pinned to what fixes it independently of the code: the
Philox4x32-10 known-answer vectors, the Gumbel distribution's closed-form
moments, the law of the sampled tokens (softmax of the logits over the
temperature, by a chi-square test), library routines for the projection and
the log-sum-exp, and the independence of a row's draw from the batch.
"""
import math
import os

import numpy as np
import pytest
import torch
from scipy import special, stats

from oracle import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _kat():
    rows = []
    for line in open(os.path.join(GOLDEN, "philox4x32_10_kat.txt")):
        if line.startswith("#") or not line.strip():
            continue
        w = [int(x, 16) for x in line.split()]
        rows.append((w[:4], w[4:6], w[6:10]))
    return rows


@pytest.mark.parametrize("case", range(3))
def test_philox_known_answers(case):
    ctr, key, want = _kat()[case]
    np.testing.assert_array_equal(O.philox4x32_10(ctr, key), np.array(want, np.uint32))


def test_uniforms_strictly_inside_and_uniform():
    u = np.array([O.sample_uniform(7, s, p, v) for s in range(4) for p in range(50) for v in range(100)])
    assert (u > 0).all() and (u < 1).all()
    # Kolmogorov-Smirnov against U(0, 1)
    assert stats.kstest(u, "uniform").pvalue > 1e-4
    # the 23-bit grid: u * 2^23 - 1/2 is an integer
    k = u * 2.0 ** 23 - 0.5
    np.testing.assert_array_equal(k, np.round(k))


def test_gumbel_moments():
    """Mean = Euler-Mascheroni constant, variance = pi^2 / 6."""
    rng = np.random.default_rng(0)
    u = rng.uniform(size=200000)
    g = np.array([O.gumbel(x) for x in u])
    se = math.sqrt(math.pi ** 2 / 6 / len(g))
    assert abs(g.mean() - np.euler_gamma) < 5 * se
    assert abs(g.var() - math.pi ** 2 / 6) < 0.03
    assert O.gumbel(math.exp(-1.0)) == pytest.approx(0.0, abs=1e-15)


def _head(V=8, H=64, seed=3, scale=1.0):
    rng = np.random.default_rng(seed)
    w = (rng.standard_normal((V, H)) * 0.2 * scale).astype(np.float32)
    g = (1 + 0.02 * rng.standard_normal(H)).astype(np.float32)
    x = rng.standard_normal((1, H))
    return x, g, w


@pytest.mark.parametrize("temperature", [0.7, 1.6])
def test_sampled_tokens_follow_softmax_over_temperature(temperature):
    x, g, w = _head()
    T = 30000
    xs = np.repeat(x, T, axis=0)
    pos = np.arange(T, dtype=np.int32)
    r = O.lm_head(xs, g, w, 1e-5, temperature, seed=11, seq_ids=np.full(T, 5, np.int32), positions=pos,
                  want_logits=True)
    lg = r["logits"][0]
    p = special.softmax(lg / temperature)
    obs = np.bincount(r["tokens"], minlength=len(p))
    chi2 = ((obs - T * p) ** 2 / (T * p)).sum()
    assert stats.chi2.sf(chi2, len(p) - 1) > 1e-4, (obs, T * p)
    # the other temperature's law is rejected: the rule divides by the temperature
    other = special.softmax(lg * temperature)
    chi2o = ((obs - T * other) ** 2 / (T * other)).sum()
    assert stats.chi2.sf(chi2o, len(p) - 1) < 1e-6


def test_logits_logsumexp_and_logprobs_match_library_routines():
    rng = np.random.default_rng(4)
    T, H, V = 6, 128, 1000
    x = rng.standard_normal((T, H)) * 3
    g = (1 + 0.02 * rng.standard_normal(H)).astype(np.float32)
    w = torch.from_numpy(rng.standard_normal((V, H)) * 0.02).to(torch.bfloat16).float().numpy()
    tgt = rng.integers(0, V, T).astype(np.int32)
    tau = float(np.float32(0.7))
    r = O.lm_head(x, g, w, 1e-5, tau, seed=9, seq_ids=np.arange(T, dtype=np.int32),
                  positions=np.full(T, 17, np.int32), targets=tgt, want_logits=True)
    xn = torch.nn.functional.rms_norm(torch.from_numpy(x), (H,), torch.from_numpy(g).double(), eps=1e-5)
    xn = xn.to(torch.bfloat16).double().numpy()
    np.testing.assert_allclose(r["logits"], xn @ w.T.astype(np.float64), rtol=1e-12, atol=1e-12)
    s = r["logits"] / tau
    np.testing.assert_allclose(r["lse"], special.logsumexp(s, axis=1), rtol=1e-13)
    ls = special.log_softmax(s, axis=1)
    np.testing.assert_allclose(r["logprob"], ls[np.arange(T), r["tokens"]], rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(r["target_logprob"], ls[np.arange(T), tgt], rtol=1e-12, atol=1e-12)
    # the chosen token maximises the fp32-rounded perturbed score, lowest id first
    for t in range(T):
        pf = r["pert"][t].astype(np.float32)
        assert r["tokens"][t] == int(np.argmax(pf))
        # and the perturbation is the row's own Gumbel draw
        v = int(rng.integers(0, V))
        gv = O.gumbel(O.sample_uniform(9, t, 17, v))
        assert r["pert"][t, v] == pytest.approx(s[t, v] + gv, rel=0, abs=1e-12)


def test_greedy_is_argmax_of_logits():
    x, g, w = _head(V=64, H=64, seed=5)
    xs = np.concatenate([x, -x, 2 * x])
    r = O.lm_head(xs, g, w, 1e-5, 0.0, want_logits=True)
    np.testing.assert_array_equal(r["tokens"], np.argmax(r["logits"].astype(np.float32), axis=1))
    np.testing.assert_allclose(r["logprob"], special.log_softmax(r["logits"], axis=1).max(axis=1), rtol=1e-12)


def test_draw_depends_on_sequence_and_position_not_on_row():
    x, g, w = _head(V=256, H=64, seed=6)
    T = 12
    xs = np.repeat(x, T, axis=0) + 0.0
    seq = np.arange(T, dtype=np.int32) % 3
    pos = (np.arange(T, dtype=np.int32) * 7) % 5
    a = O.lm_head(xs, g, w, 1e-5, 0.7, seed=21, seq_ids=seq, positions=pos)
    perm = np.random.default_rng(1).permutation(T)
    b = O.lm_head(xs[perm], g, w, 1e-5, 0.7, seed=21, seq_ids=seq[perm], positions=pos[perm])
    np.testing.assert_array_equal(b["tokens"], a["tokens"][perm])
    np.testing.assert_array_equal(b["logprob"], a["logprob"][perm])
    # rows with the same (sequence, position) draw the same token; another seed draws differently
    c = O.lm_head(xs, g, w, 1e-5, 0.7, seed=22, seq_ids=seq, positions=pos)
    assert (c["tokens"] != a["tokens"]).any()
