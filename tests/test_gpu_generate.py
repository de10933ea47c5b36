"""The generation ends on the GPU (token embedding, vocabulary head with
temperature sampling and log-probabilities) against the reference, through
the C ABI.

Token choices are exact wherever the reference's two best perturbed scores
(s + g, in units of logits over the temperature) are more than DELTA apart;
inside that gap either token is a correct draw, and the GPU's must then score
within DELTA of the best. DELTA covers the logits' fp32 accumulation (about
1e-5) and a flipped bf16 rounding of one normalised element (|w| x ulp, up to
about 3e-4), divided by the temperature. Log-probabilities and the log-sum-exp
are held to 2e-3 absolute.
"""
import numpy as np
import pytest
import torch

from oracle import oracle as O
from paper_2608_22167_amd import mcpu, workload as W

pytestmark = pytest.mark.gpu

DELTA = 2e-3
LP_TOL = 2e-3
TAU = float(np.float32(0.7))


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    torch.cuda.set_device(0)
    yield
    torch.cuda.empty_cache()


def _run_head(head, x, temperature, seed, seq, pos, targets=None):
    T = x.shape[0]
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a, np.int32)).cuda()
    tok = torch.empty(T, dtype=torch.int32, device="cuda")
    lp, lse, tlp = (torch.empty(T, device="cuda") for _ in range(3))
    ws = mcpu.workspace(mcpu.lm_head_workspace_size(head.hidden, head.vocab, T))
    mcpu.lm_head_sample(head, x.cuda().contiguous(), temperature, seed, dev(seq), dev(pos),
                        None if targets is None else dev(targets), tok, lp, tlp if targets is not None else None,
                        lse, ws)
    torch.cuda.synchronize()
    assert mcpu.mcpu_check_device_errors(ws) == 0
    out = dict(tokens=tok.cpu().numpy(), logprob=lp.cpu().numpy().astype(np.float64),
               lse=lse.cpu().numpy().astype(np.float64))
    if targets is not None:
        out["target_logprob"] = tlp.cpu().numpy().astype(np.float64)
    return out


def _check(gpu, ref, rows=None):
    """gpu: outputs for all rows; ref: reference outputs for `rows` (default all)."""
    rows = np.arange(len(ref["tokens"])) if rows is None else np.asarray(rows)
    near = 0
    for i, r in enumerate(rows):
        p = ref["pert"][i]
        best = int(ref["tokens"][i])
        g = int(gpu["tokens"][r])
        if g != best:
            second = np.partition(p, -2)[-2]
            assert p[best] - second <= DELTA and p[best] - p[g] <= DELTA, \
                f"row {r}: GPU token {g} (score {p[g]:.6f}) vs reference {best} ({p[best]:.6f})"
            near += 1
        else:
            assert abs(gpu["logprob"][r] - ref["logprob"][i]) <= LP_TOL, (r, gpu["logprob"][r], ref["logprob"][i])
    np.testing.assert_allclose(gpu["lse"][rows], ref["lse"], atol=LP_TOL, rtol=0)
    if "target_logprob" in gpu:
        np.testing.assert_allclose(gpu["target_logprob"][rows], ref["target_logprob"], atol=LP_TOL, rtol=0)
    return near


def _small_head(hidden, vocab, seed):
    Wt = W.lm_weights_host(seed, hidden, vocab, embed=False)
    return Wt, mcpu.DeviceLmHead(Wt["g_final"], Wt["w_lm"])


@pytest.mark.parametrize("T,vocab", [(1, 4096), (37, 4096), (300, 4096), (600, 65536)])
@pytest.mark.parametrize("temperature", [TAU, 0.0])
def test_lm_head_sample_small(T, vocab, temperature):
    """Few rows (weight slabs), 300 rows (64 x 64 tiles, records through LDS)
    and 600 rows over a 65536-id vocabulary (128 x 128 tiles, records folded
    from the product registers, a partial last row tile); sampling and greedy."""
    H = 256
    Wt, head = _small_head(H, vocab, 2001)
    rng = np.random.default_rng(T + vocab)
    x = torch.from_numpy(rng.standard_normal((T, H)).astype(np.float32) * 2)
    seq = rng.integers(0, 1000, T)
    pos = rng.integers(0, 70000, T)
    tgt = rng.integers(0, vocab, T)
    gpu = _run_head(head, x, temperature, 77, seq, pos, tgt)
    rows = np.arange(T) if T <= 64 else np.sort(rng.choice(T, 24, replace=False))
    ref = O.lm_head(x[rows], Wt["g_final"], Wt["w_lm"], 1e-5, temperature, seed=77, seq_ids=seq[rows],
                    positions=pos[rows], targets=tgt[rows], want_logits=True)
    near = _check(gpu, ref, rows)
    print(f"  T={T} V={vocab} temperature={temperature}: {near} near-tie rows")


@pytest.mark.parametrize("T", [64, 256, 512])
def test_lm_head_sample_full_vocabulary_sampled(T):
    """gpt-oss-20b shapes: hidden 2880, 201088 ids (1.16 GB of bf16 weights),
    64 rows (streaming-order weight slabs), 256 rows (the benchmarked head) and
    512 rows (128 x 128 tiles, records folded from the product registers);
    compared on seeded rows."""
    H, V = 2880, W.GPT_OSS_VOCAB
    Wd = W.lm_weights_device(2002, H, V)
    head = mcpu.DeviceLmHead(Wd["g_final"], Wd["w_lm"])
    rng = np.random.default_rng(T)
    x = W.synth_normal(2002, 93, (T, H))
    seq = rng.integers(0, 4096, T)
    pos = rng.integers(0, 65536, T)
    tgt = rng.integers(0, V, T)
    gpu = _run_head(head, x, TAU, 5, seq, pos, tgt)
    rows = np.unique(np.concatenate([[0, T - 1], rng.choice(T, 3, replace=False)]))
    w_host = W.synth_normal(2002, W.LM_TID["w_lm"], (V, H), std=0.02, dtype=torch.bfloat16)
    ref = O.lm_head(x[torch.from_numpy(rows)], Wd["g_final"].cpu(), w_host, 1e-5, TAU, seed=5, seq_ids=seq[rows],
                    positions=pos[rows], targets=tgt[rows], want_logits=True)
    near = _check(gpu, ref, rows)
    print(f"  T={T}: rows {rows.tolist()}, {near} near-tie rows, tokens {gpu['tokens'][rows].tolist()}")
    assert torch.equal(Wd["w_lm"].cpu().view(torch.int16), w_host.view(torch.int16))


def test_lm_head_draw_is_independent_of_the_batch():
    """A row's token depends on (seed, sequence, position) only: permuting the
    rows permutes the results bit for bit, and the same rows inside a larger
    batch (another GEMM tiling) draw the same tokens outside near ties."""
    H, V, T = 256, 4096, 40
    Wt, head = _small_head(H, V, 2003)
    rng = np.random.default_rng(3)
    x = torch.from_numpy(rng.standard_normal((T, H)).astype(np.float32))
    seq, pos = rng.integers(0, 50, T), rng.integers(0, 500, T)
    a = _run_head(head, x, TAU, 9, seq, pos)
    perm = rng.permutation(T)
    b = _run_head(head, x[torch.from_numpy(perm)], TAU, 9, seq[perm], pos[perm])
    np.testing.assert_array_equal(b["tokens"], a["tokens"][perm])
    np.testing.assert_array_equal(b["logprob"], a["logprob"][perm])
    big_x = torch.cat([x, torch.from_numpy(rng.standard_normal((300, H)).astype(np.float32))])
    big = _run_head(head, big_x, TAU, 9, np.concatenate([seq, rng.integers(0, 50, 300)]),
                    np.concatenate([pos, rng.integers(0, 500, 300)]))
    ref = O.lm_head(x, Wt["g_final"], Wt["w_lm"], 1e-5, TAU, seed=9, seq_ids=seq, positions=pos, want_logits=True)
    _check({k: v[:T] for k, v in big.items()}, ref)


def test_embed_tokens_bit_exact_and_bad_id():
    V, H, T = 1000, 2880, 33
    table = W.synth_normal(2004, 92, (V, H), dtype=torch.bfloat16).cuda()
    rng = np.random.default_rng(4)
    ids = rng.integers(0, V, T).astype(np.int32)
    x = torch.empty((T, H), device="cuda")
    ws = mcpu.workspace(256)
    mcpu.embed_tokens(table, torch.from_numpy(ids).cuda(), x, ws)
    torch.cuda.synchronize()
    assert mcpu.mcpu_check_device_errors(ws) == 0
    assert torch.equal(x.cpu(), table.cpu()[torch.from_numpy(ids).long()].float())
    ids[5] = V
    mcpu.embed_tokens(table, torch.from_numpy(ids).cuda(), x, ws)
    assert mcpu.mcpu_check_device_errors(ws) & mcpu.DEVERR_TOKEN
    assert float(x[5].abs().max()) == 0.0


# ------------------------------------------------------------------------------ the generator


def _generator_case():
    from paper_2608_22167_amd.generate import GenSpec, Generator
    base = W.replace(W.GPT_OSS_20B, hidden=256, n_q_heads=8, n_kv_heads=2, head_dim=64, n_experts=8, top_k=2,
                     ffn_dim=256)
    spec = GenSpec(n_layers=4, base=base, vocab=4096, window=128, pages_full=512, pages_sw=128, max_ctx=4096)
    return spec, Generator(spec, max_tokens_per_step=512)


def test_generator_turns_against_reference_trajectories():
    """Continuous batching over multi-turn trajectories: five sequences join
    at different steps, generate 6-token turns, wait, take tool observations
    of 5-60 tokens, and leave after three turns. Every sampled token and its
    log-probability is checked against the reference trajectory (its whole
    history as one causal prefill, then the head with the same draws); window
    pages stay bounded while sequences grow, and every page comes back."""
    from oracle import generate as OG
    spec, gen = _generator_case()
    free0 = gen.free_pages()
    rng = np.random.default_rng(7)
    prompts = {sid: rng.integers(0, spec.vocab, n).tolist() for sid, n in zip(range(5), [3, 40, 17, 1, 100])}
    join = {0: 0, 1: 0, 2: 3, 3: 5, 4: 9}
    turns = {sid: 0 for sid in prompts}
    made = {sid: 0 for sid in prompts}
    samples = {sid: [] for sid in prompts}      # (position, token, logprob)
    waiting, finished, histories = {}, set(), {}
    max_sw = 0
    step = 0
    while len(finished) < len(prompts):
        for sid, at in join.items():
            if at == step:
                gen.add(sid, prompts[sid])
        for sid in list(waiting):
            waiting[sid] -= 1
            if waiting[sid] == 0:
                del waiting[sid]
                gen.resume(sid, rng.integers(0, spec.vocab, int(rng.integers(5, 60))).tolist())
        out = gen.step()
        for sid, (tok, lp) in out.items():
            s = gen.seqs[sid]
            samples[sid].append((s.length, tok, lp))
            made[sid] += 1
            if made[sid] % 6 == 0:           # the turn ends in a tool call
                turns[sid] += 1
                gen.hold(sid)
                if turns[sid] == 3:
                    histories[sid] = list(s.history) + [tok]
                    gen.release(sid)
                    finished.add(sid)
                else:
                    waiting[sid] = 2
        max_sw = max([max_sw] + [len(s.pages_sw) for s in gen.seqs.values()])
        step += 1
        assert step < 400
    assert gen.check_errors() == 0
    assert gen.free_pages() == free0, "pages leaked"
    assert max_sw <= 128 // 16 + 2, max_sw
    ss = spec.stack_spec()
    lw = [W.stack_weights_host(ss, i) for i in range(spec.n_layers)]
    lm = W.lm_weights_host(spec.seed, ss.shape_full.hidden, spec.vocab)
    near = 0
    for sid, hist in histories.items():
        rows = OG.trajectory_rows(ss, lw, lm["embed"], hist[:-1])
        pos = np.array([p for p, _, _ in samples[sid]])
        ref = O.lm_head(rows[pos - 1], lm["g_final"], lm["w_lm"], ss.shape_full.rms_eps, spec.temperature,
                        seed=spec.seed, seq_ids=np.full(len(pos), sid, np.int32), positions=pos, want_logits=True)
        got = dict(tokens=np.array([t for _, t, _ in samples[sid]]), logprob=np.array([l for _, _, l in samples[sid]]),
                   lse=ref["lse"])
        # the history holds the GPU's tokens: each one must be the reference's draw
        np.testing.assert_array_equal(np.array(hist)[pos], got["tokens"])
        near += _check(got, ref)
    print(f"  {step} steps, {sum(len(v) for v in samples.values())} sampled tokens, {near} near ties, "
          f"at most {max_sw} window pages per sequence")
    # the log-probability pass over the finished trajectories
    trajs = [histories[sid] for sid in sorted(histories)]
    scores = gen.score(trajs)
    assert gen.free_pages() == free0
    for sid, tr, sc in zip(sorted(histories), trajs, scores):
        rows = OG.trajectory_rows(ss, lw, lm["embed"], tr[:-1])
        n = len(tr) - 1
        ref = O.lm_head(rows, lm["g_final"], lm["w_lm"], ss.shape_full.rms_eps, spec.temperature,
                        seq_ids=np.zeros(n, np.int32), positions=np.zeros(n, np.int32),
                        targets=np.array(tr[1:], np.int32))
        np.testing.assert_allclose(sc, ref["target_logprob"], atol=LP_TOL, rtol=0)
        # a sampled token's log-probability is the same number from both passes
        for p, tok, lp in samples[sid]:
            assert abs(sc[p - 1] - lp) <= LP_TOL
