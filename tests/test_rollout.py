"""The rollout pipeline's scheduling (paper_2608_22167_amd/rollout.py) on
the CPU, with a stand-in generator whose tokens depend only on (sequence,
position) and whose steps take time like a GPU's: stage order, the per-stage
and in-flight limits, complete and identical trajectories under any
concurrency, and the coupled-versus-decoupled throughput gap."""
import time

import numpy as np
import pytest

from paper_2608_22167_amd import rollout as R


class StandInGenerator:
    """Generator's scheduling surface (add, step, hold, resume, release,
    seqs, held) without a model: a step costs a fixed time plus a little per
    token, and the token sampled at position p of sequence s is a hash of
    (s, p)."""

    def __init__(self, step_s=0.004, per_token_s=2e-6):
        self.seqs, self.held = {}, {}
        self.step_s, self.per_token_s = step_s, per_token_s
        self.steps = 0
        self.max_batch = 0

    def add(self, sid, tokens):
        s = self.seqs.setdefault(sid, dict(length=0, pending=[]))
        s["pending"].extend(tokens)

    def hold(self, sid):
        self.held[sid] = self.seqs[sid]["pending"][:]
        self.seqs[sid]["pending"].clear()

    def resume(self, sid, obs):
        self.add(sid, self.held.pop(sid, []) + list(obs))

    def release(self, sid):
        self.seqs.pop(sid)
        self.held.pop(sid, None)

    @staticmethod
    def token(sid, pos):
        return (sid * 1000003 + pos * 7919) % 4096

    def step(self):
        ready = [(sid, s) for sid, s in self.seqs.items() if s["pending"]]
        if not ready:
            return {}
        n_tok = sum(len(s["pending"]) for _, s in ready)
        time.sleep(self.step_s + self.per_token_s * n_tok)
        out = {}
        for sid, s in ready:
            s["length"] += len(s["pending"])
            s["pending"] = [self.token(sid, s["length"])]
            out[sid] = (s["pending"][0], -1.0)
        self.steps += 1
        self.max_batch = max(self.max_batch, len(ready))
        return out


def _run(cfg, gen=None):
    gen = gen or StandInGenerator()
    eng = R.Engine(gen)
    try:
        res = R.run_pipeline(cfg, eng)
    finally:
        eng.close()
    return res, gen


def _expected_tokens(cfg, tid):
    plan = R.trajectory_plan(cfg, tid)
    toks = []
    inp = plan["prompt"]
    for turn in range(cfg.turns):
        toks.extend(inp)
        for _ in range(cfg.tokens_per_turn):
            toks.append(StandInGenerator.token(tid, len(toks)))
        if turn < cfg.turns - 1:
            inp = plan["obs"][turn]
    return toks


FAST = dict(acquire_s=(0.01, 0.03), tool_s=(0.02, 0.08), eval_s=(0.0, 0.01), prompt_tokens=(4, 20),
            obs_tokens=(2, 10), tokens_per_turn=4, turns=3)


def test_pipeline_limits_order_and_trajectories():
    cfg = R.RolloutConfig(n_trajectories=30, acquire_workers=3, run_workers=6, eval_workers=2, in_flight=8, **FAST)
    res, gen = _run(cfg)
    recs = res["records"]
    assert len(recs) == 30
    assert res["max_live"] <= 8 and res["max_running"] <= 6 and res["max_acquiring"] <= 3
    assert res["max_running"] == 6          # the run pool fills up
    for tid, r in recs.items():
        t = r.t
        assert t["queued"] <= t["acq0"] <= t["acq1"] <= t["run0"] <= t["run1"] <= t["eval0"] <= t["eval1"]
        assert len(r.sampled) == cfg.turns * cfg.tokens_per_turn
        assert r.tokens == _expected_tokens(cfg, tid)
        for pos, tok, _ in r.sampled:
            assert r.tokens[pos] == tok
    assert gen.seqs == {} and gen.held == {}   # every sequence released
    assert gen.max_batch > 1                   # continuous batching: steps serve several sequences


def test_trajectories_do_not_depend_on_concurrency():
    a, _ = _run(R.RolloutConfig(n_trajectories=12, acquire_workers=2, run_workers=2, in_flight=4, **FAST))
    b, _ = _run(R.RolloutConfig(n_trajectories=12, acquire_workers=4, run_workers=12, in_flight=12, **FAST))
    for tid in range(12):
        assert a["records"][tid].tokens == b["records"][tid].tokens


def test_decoupled_run_pool_raises_throughput():
    """Tool stalls dominate the episode: with run workers equal to acquire
    workers the engine idles; doubling and quadrupling the run pool at the
    same in-flight capacity raises generated tokens per second."""
    base = dict(n_trajectories=48, acquire_workers=4, in_flight=16, eval_workers=4, turns=4, tokens_per_turn=4,
                acquire_s=(0.02, 0.04), tool_s=(0.15, 0.25), eval_s=(0.0, 0.01), prompt_tokens=(4, 8),
                obs_tokens=(2, 4))
    rates = {}
    for rw in (4, 8, 16):
        res, _ = _run(R.RolloutConfig(run_workers=rw, **base))
        rates[rw] = res["tokens_per_s"]
    assert rates[8] > 1.3 * rates[4] and rates[16] > rates[8], rates
