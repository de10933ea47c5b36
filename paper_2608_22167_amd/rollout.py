"""The rollout pipeline on one GPU: Acquire -> Run -> Eval with per-stage
worker pools, driving the continuous-batching generator.

The paper's rollout-orchestration layer runs each trajectory through three
overlapping stages (Sec. 3.2): acquire an environment, run the episode (turns
of generation on the GPU, each ended by a tool call that stalls in the
environment), and evaluate it. The stages are bound by different resources,
so each gets its own worker pool; the run stage gets more workers than the
acquire stage (at least twice as many by default), while the number of live
environments (the in-flight capacity) is held fixed. With run workers equal
to acquire workers (the coupled setting) the GPU idles whenever the shared
limit is spent on trajectories still acquiring or waiting on a tool; with
more run workers (decoupled) already-acquired trajectories keep generating
(Sec. 4.2; the sweep holds acquire at 24 workers and in-flight capacity at
120 and varies run workers over 24-120, rollout experiment details).

Here environments and tools are synthetic: acquiring, each tool call and the
evaluation are timed stalls (seeded, per trajectory and turn), and tool
observations are seeded token chunks, so a trajectory's content depends only
on its id; the pipeline decides only when things happen. Generation is real:
a single engine thread owns the GPU and advances every sequence that has
input in one continuous-batching step (`Generator.step`). A run worker owns
one episode: it submits the turn's input, waits for the engine to produce the
turn's tokens, then stalls on the tool while the engine serves others.
"""
from __future__ import annotations

import queue
import threading
import time
from concurrent.futures import Future, ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np


@dataclass
class RolloutConfig:
    n_trajectories: int = 48
    acquire_workers: int = 24
    run_workers: int = 48          # the decoupled default: twice the acquire pool
    eval_workers: int = 8
    in_flight: int = 120           # live environments (acquired, not yet released)
    turns: int = 3
    tokens_per_turn: int = 16      # generated tokens per turn (the turn ends in a tool call)
    prompt_tokens: tuple = (32, 96)   # uniform range of the first input
    obs_tokens: tuple = (8, 64)       # uniform range of each tool observation
    acquire_s: tuple = (0.05, 0.15)   # uniform stall ranges (seconds)
    tool_s: tuple = (0.05, 0.3)
    eval_s: tuple = (0.01, 0.03)
    vocab: int = 4096
    seed: int = 4001


def _rng(cfg: RolloutConfig, tid: int, what: int):
    return np.random.default_rng([cfg.seed, tid, what])


def trajectory_plan(cfg: RolloutConfig, tid: int) -> dict:
    """Everything a trajectory's environment contributes, drawn from its id:
    the stall lengths, the prompt and the tool observations."""
    r = _rng(cfg, tid, 0)
    prompt = r.integers(0, cfg.vocab, int(r.integers(cfg.prompt_tokens[0], cfg.prompt_tokens[1] + 1))).tolist()
    obs = [r.integers(0, cfg.vocab, int(r.integers(cfg.obs_tokens[0], cfg.obs_tokens[1] + 1))).tolist()
           for _ in range(cfg.turns - 1)]
    return dict(acquire=float(r.uniform(*cfg.acquire_s)), tools=[float(r.uniform(*cfg.tool_s))
                                                                  for _ in range(cfg.turns - 1)],
                eval=float(r.uniform(*cfg.eval_s)), prompt=prompt, obs=obs)


class Engine:
    """The GPU side: one thread owns the generator and steps every sequence
    with pending input; `generate` (from any thread) feeds a sequence its
    input and returns a future of the next n sampled tokens (with their
    log-probabilities). A sampled token that ends a request is held back and
    fed before the sequence's next input, so turns join seamlessly."""

    def __init__(self, gen):
        self.gen = gen
        self.inbox: "queue.Queue" = queue.Queue()
        self.want: Dict[int, list] = {}
        self.busy_s = 0.0
        self.steps = 0
        self.tokens = 0
        self.batch_hist: List[int] = []
        self._stop = False
        self._error: Optional[BaseException] = None
        self.thread = threading.Thread(target=self._loop, name="engine", daemon=True)
        self.thread.start()

    def generate(self, sid: int, tokens: List[int], n: int) -> Future:
        f: Future = Future()
        self.inbox.put(("gen", sid, list(tokens), n, f))
        return f

    def release(self, sid: int) -> Future:
        f: Future = Future()
        self.inbox.put(("release", sid, None, 0, f))
        return f

    def close(self):
        self._stop = True
        self.inbox.put(("stop", 0, None, 0, None))
        self.thread.join()
        if self._error:
            raise self._error

    def _take(self, msg):
        kind, sid, tokens, n, f = msg
        if kind == "gen":
            if sid in self.gen.held:
                self.gen.resume(sid, tokens)
            else:
                self.gen.add(sid, tokens)
            self.want[sid] = [n, [], f]
        elif kind == "release":
            self.gen.release(sid)
            f.set_result(None)

    def _loop(self):
        try:
            while not self._stop:
                block = not self.want
                try:
                    msg = self.inbox.get(block=block, timeout=0.5 if block else None)
                    if msg[0] == "stop":
                        break
                    self._take(msg)
                    while True:
                        msg = self.inbox.get_nowait()
                        if msg[0] == "stop":
                            self._stop = True
                            break
                        self._take(msg)
                except queue.Empty:
                    pass
                if not self.want:
                    continue
                t0 = time.perf_counter()
                out = self.gen.step()
                self.busy_s += time.perf_counter() - t0
                self.steps += 1
                self.batch_hist.append(len(out))
                for sid, (tok, lp) in out.items():
                    w = self.want.get(sid)
                    if w is None:
                        continue
                    w[1].append((tok, lp))
                    self.tokens += 1
                    if len(w[1]) == w[0]:
                        self.gen.hold(sid)
                        del self.want[sid]
                        w[2].set_result(w[1])
        except BaseException as e:  # surfaces in close()
            self._error = e
            for w in self.want.values():
                w[2].set_exception(e)


@dataclass
class TrajectoryRecord:
    tid: int
    tokens: List[int] = field(default_factory=list)      # the whole trajectory as fed
    sampled: List[tuple] = field(default_factory=list)   # (position, token, logprob)
    t: Dict[str, float] = field(default_factory=dict)    # stage timestamps


def run_pipeline(cfg: RolloutConfig, engine: Engine) -> dict:
    """Runs cfg.n_trajectories trajectories through the three stages and
    returns the records and throughput statistics."""
    live = threading.BoundedSemaphore(cfg.in_flight)
    acquire = ThreadPoolExecutor(cfg.acquire_workers, thread_name_prefix="acquire")
    run = ThreadPoolExecutor(cfg.run_workers, thread_name_prefix="run")
    evaluate = ThreadPoolExecutor(cfg.eval_workers, thread_name_prefix="eval")
    lock = threading.Lock()
    counters = dict(live=0, max_live=0, running=0, max_running=0, acquiring=0, max_acquiring=0)
    records: Dict[int, TrajectoryRecord] = {}
    done = threading.Event()
    n_done = [0]
    errors: List[BaseException] = []
    t_start = time.perf_counter()

    def bump(key, d):
        with lock:
            counters[key] += d
            counters["max_" + key] = max(counters["max_" + key], counters[key])

    def stage_eval(rec: TrajectoryRecord, plan: dict):
        try:
            rec.t["eval0"] = time.perf_counter()
            time.sleep(plan["eval"])
            rec.t["eval1"] = time.perf_counter()
        finally:
            bump("live", -1)
            live.release()
            with lock:
                n_done[0] += 1
                if n_done[0] == cfg.n_trajectories:
                    done.set()

    def stage_run(rec: TrajectoryRecord, plan: dict):
        try:
            bump("running", 1)
            rec.t["run0"] = time.perf_counter()
            inp = plan["prompt"]
            for turn in range(cfg.turns):
                rec.tokens.extend(inp)
                got = engine.generate(rec.tid, inp, cfg.tokens_per_turn).result()
                for tok, lp in got:
                    rec.sampled.append((len(rec.tokens), tok, lp))
                    rec.tokens.append(tok)
                if turn < cfg.turns - 1:
                    time.sleep(plan["tools"][turn])     # the tool call stalls in the environment
                    inp = plan["obs"][turn]
            engine.release(rec.tid).result()
            rec.t["run1"] = time.perf_counter()
            bump("running", -1)
            evaluate.submit(stage_eval, rec, plan)
        except BaseException as e:
            errors.append(e)
            done.set()

    def stage_acquire(rec: TrajectoryRecord, plan: dict):
        try:
            bump("acquiring", 1)
            rec.t["acq0"] = time.perf_counter()
            time.sleep(plan["acquire"])
            rec.t["acq1"] = time.perf_counter()
            bump("acquiring", -1)
            run.submit(stage_run, rec, plan)
        except BaseException as e:
            errors.append(e)
            done.set()

    def feeder():
        for tid in range(cfg.n_trajectories):
            live.acquire()             # an environment slot must be free before acquiring
            bump("live", 1)
            rec = TrajectoryRecord(tid)
            records[tid] = rec
            rec.t["queued"] = time.perf_counter()
            acquire.submit(stage_acquire, rec, trajectory_plan(cfg, tid))

    feed = threading.Thread(target=feeder, daemon=True)
    feed.start()
    done.wait()
    wall = time.perf_counter() - t_start
    feed.join(timeout=5)
    for ex in (acquire, run, evaluate):
        ex.shutdown(wait=True)
    if errors:
        raise errors[0]
    gen_tokens = sum(len(r.sampled) for r in records.values())
    return dict(records=records, wall_s=wall, tokens=gen_tokens, tokens_per_s=gen_tokens / wall,
                engine_busy=engine.busy_s / wall, engine_steps=engine.steps,
                mean_batch=float(np.mean(engine.batch_hist)) if engine.batch_hist else 0.0, **counters)


def sweep(gen, run_workers=(24, 48, 64, 96, 120), **kw) -> List[dict]:
    """The per-stage concurrency sweep: acquire fixed, run workers varied,
    in-flight capacity fixed; one engine reused across the settings."""
    rows = []
    for rw in run_workers:
        cfg = RolloutConfig(run_workers=rw, **kw)
        eng = Engine(gen)
        try:
            res = run_pipeline(cfg, eng)
        finally:
            eng.close()
        rows.append(dict(run_workers=rw, acquire_workers=cfg.acquire_workers, in_flight=cfg.in_flight,
                         tokens_per_s=round(res["tokens_per_s"], 1), wall_s=round(res["wall_s"], 2),
                         engine_busy=round(res["engine_busy"], 3), mean_batch=round(res["mean_batch"], 1),
                         max_running=res["max_running"], max_live=res["max_live"]))
    return rows


if __name__ == "__main__":  # pragma: no cover - the GPU sweep
    import argparse
    import json

    import torch

    from paper_2608_22167_amd import workload as W
    from paper_2608_22167_amd.generate import GenSpec, Generator

    ap = argparse.ArgumentParser(description="per-stage concurrency sweep of the rollout pipeline on one GPU")
    ap.add_argument("--layers", type=int, default=24)
    ap.add_argument("--trajectories", type=int, default=240)
    ap.add_argument("--turns", type=int, default=4)
    ap.add_argument("--tokens-per-turn", type=int, default=32)
    ap.add_argument("--run-workers", default="24,48,64,96,120")
    args = ap.parse_args()
    torch.cuda.set_device(0)
    spec = GenSpec(n_layers=args.layers, base=W.GPT_OSS_20B, vocab=W.GPT_OSS_VOCAB, pages_full=16384, pages_sw=4096,
                   max_ctx=8192)
    gen = Generator(spec, max_tokens_per_step=8192)
    rows = sweep(gen, run_workers=[int(x) for x in args.run_workers.split(",")], n_trajectories=args.trajectories,
                 turns=args.turns, tokens_per_turn=args.tokens_per_turn, vocab=spec.vocab,
                 prompt_tokens=(256, 1024), obs_tokens=(64, 512), acquire_s=(0.5, 1.5), tool_s=(0.5, 2.0),
                 eval_s=(0.05, 0.2))
    for r in rows:
        print(json.dumps(r), flush=True)
