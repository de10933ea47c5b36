"""Continuous-batching generation over the decoder stack (argument
marshalling and host bookkeeping around the C ABI; every step of the model
runs in libmcpu.so's kernels).

The Run stage of the paper's rollout pipeline keeps many multi-turn
trajectories in flight on one policy replica: each turn the policy generates
tokens at the rollout temperature, the trajectory then waits on a tool, and
the tool's observation joins the context before the next turn (Sec. 1 and
Sec. 3.2; temperature 0.7 in the training-details appendix). `Generator`
serves that pattern. Every call to `step()` advances all sequences that have
input: a prompt or observation chunk is prefilled (chunked prefill through
the same decode_layer call), a decoding sequence feeds its last sampled token,
and every sequence that reached the end of its input samples one new token.

Pages are allocated per step as sequences grow (kv_pages_alloc, one pool id
space per attention kind: the same page ids index every layer of that kind),
pages of sliding-window layers are freed once they fall wholly left of the
window, and all of a sequence's pages are freed when it is released.
`score()` recomputes the log-probabilities of whole trajectories (the GRPO
update's log-prob pass): a long causal prefill with targets, no sampling.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np
import torch

from paper_2608_22167_amd import mcpu, workload as W

PAGE = 16


@dataclass
class GenSpec:
    """A decoder stack with its generation ends. Layer i uses the window if i
    is even (0-based) and full attention if odd, like the 24-layer stack."""
    n_layers: int
    base: W.LayerShape            # bf16 layer shape (experts MXFP4)
    vocab: int
    seed: int = 3001
    window: int = 128
    pages_full: int = 4096        # pages per full-attention layer pool
    pages_sw: int = 1024          # pages per sliding-window layer pool
    max_ctx: int = 65536          # positions the RoPE table covers
    temperature: float = float(np.float32(0.7))

    def stack_spec(self) -> W.StackSpec:
        full = W.replace(self.base, expert_fmt="mxfp4", window=0)
        sw = W.replace(full, window=self.window)
        z = np.zeros((0, 1), np.int32)
        return W.StackSpec(name="generator", seed=self.seed, n_layers=self.n_layers, shape_full=full, shape_sw=sw,
                           seq_lens=np.zeros(0, np.int32), page_table_full=z, n_pages_full=self.pages_full,
                           page_table_sw=z, n_pages_sw=self.pages_sw, rope_max_pos=self.max_ctx)


@dataclass
class _Seq:
    sid: int
    length: int = 0                                     # tokens in the cache
    pending: List[int] = field(default_factory=list)    # input not yet fed
    pages_full: List[int] = field(default_factory=list)  # logical page i -> physical id
    pages_sw: Dict[int, int] = field(default_factory=dict)
    history: List[int] = field(default_factory=list)    # every token fed so far


class Generator:
    """The stack's weights, one K/V pool pair per layer, the embedding and the
    vocabulary head, all resident on the GPU; sequences come and go."""

    def __init__(self, spec: GenSpec, device="cuda", max_tokens_per_step: int = 8192):
        self.spec = spec
        self.ss = ss = spec.stack_spec()
        self.device = device
        self.weights, self.k, self.v, self.pools = [], [], [], []
        for i in range(spec.n_layers):
            s = ss.shape(i)
            self.weights.append(mcpu.DeviceWeights(s, W.stack_weights_device(ss, i, device), device))
            n = ss.n_pages(i)
            self.k.append(torch.zeros((n, s.n_kv_heads, PAGE, s.head_dim), dtype=torch.bfloat16, device=device))
            self.v.append(torch.zeros_like(self.k[-1]))
            self.pools.append(mcpu.KVPool(s, self.k[-1], self.v[-1]))
        # page ids are handed out by the first pool of each kind and used in every layer of that kind
        self.alloc_full = self.pools[1] if spec.n_layers > 1 else None
        self.alloc_sw = self.pools[0]
        lm = W.lm_weights_device(spec.seed, ss.shape_full.hidden, spec.vocab, device)
        self.embed = lm["embed"]
        self.head = mcpu.DeviceLmHead(lm["g_final"], lm["w_lm"], ss.shape_full.rms_eps, device)
        self.max_tokens = max_tokens_per_step
        s0 = ss.shape_full
        self.ws = mcpu.workspace(max(mcpu.decode_layer_workspace_size(ss.shape(i), max_tokens_per_step,
                                                                      max_tokens_per_step)
                                     for i in range(min(2, spec.n_layers))), device)
        self.lm_ws = mcpu.workspace(mcpu.lm_head_workspace_size(s0.hidden, spec.vocab, max_tokens_per_step), device)
        self.seqs: Dict[int, _Seq] = {}
        self.held: Dict[int, List[int]] = {}   # a sequence's sampled token kept back while its turn waits
        self.steps = 0

    # ------------------------------------------------------------------ sequences

    def add(self, sid: int, tokens: Sequence[int]) -> None:
        """Queue input for sequence sid (a new trajectory's prompt, or a tool
        observation appended to a waiting one)."""
        if not len(tokens):
            return
        s = self.seqs.setdefault(sid, _Seq(sid))
        s.pending.extend(int(t) for t in tokens)

    def release(self, sid: int) -> None:
        """Free every page of sequence sid and forget it."""
        s = self.seqs.pop(sid)
        self.held.pop(sid, None)
        if self.alloc_full is not None and s.pages_full:
            mcpu.kv_pages_free(self.alloc_full, np.array(s.pages_full, np.int32))
        if s.pages_sw:
            mcpu.kv_pages_free(self.alloc_sw, np.array(list(s.pages_sw.values()), np.int32))

    def free_pages(self):
        return (self.alloc_full.free_pages() if self.alloc_full is not None else 0, self.alloc_sw.free_pages())

    def _grow(self, s: _Seq, q: int) -> None:
        """Pages for positions s.length .. s.length + q - 1: every full-layer
        page up to the last, and every window page the new tokens can see."""
        last = s.length + q - 1
        if self.alloc_full is not None:
            need = last // PAGE + 1 - len(s.pages_full)
            if need > 0:
                s.pages_full.extend(int(p) for p in mcpu.kv_pages_alloc(self.alloc_full, need))
        lo = max(0, s.length - self.spec.window + 1) // PAGE
        missing = [lp for lp in range(lo, last // PAGE + 1) if lp not in s.pages_sw]
        if missing:
            for lp, p in zip(missing, mcpu.kv_pages_alloc(self.alloc_sw, len(missing))):
                s.pages_sw[lp] = int(p)

    def _shrink(self, s: _Seq) -> None:
        """Free window pages wholly left of the next token's window."""
        lo = max(0, s.length - self.spec.window + 1) // PAGE
        old = [lp for lp in s.pages_sw if lp < lo]
        if old:
            mcpu.kv_pages_free(self.alloc_sw, np.array([s.pages_sw.pop(lp) for lp in old], np.int32))

    # ------------------------------------------------------------------ one step

    def _tables(self, batch: List[_Seq], q_lens: List[int]):
        max_lp = max((s.length + q - 1) // PAGE + 1 for s, q in zip(batch, q_lens))
        pt_f = -np.ones((len(batch), max_lp), np.int32)
        pt_s = -np.ones((len(batch), max_lp), np.int32)
        for b, s in enumerate(batch):
            pt_f[b, :len(s.pages_full)] = s.pages_full
            for lp, p in s.pages_sw.items():
                pt_s[b, lp] = p
        return pt_f, pt_s

    def _forward(self, batch: List[_Seq], q_lens: List[int], tokens: np.ndarray):
        """Embeds the step's input tokens and runs every layer; returns the
        final residual rows [T, H] and cu_q."""
        T = int(sum(q_lens))
        dev = self.device
        cu = np.zeros(len(batch) + 1, np.int32)
        cu[1:] = np.cumsum(q_lens)
        seq_lens = np.array([s.length for s in batch], np.int32)
        pt_f, pt_s = self._tables(batch, q_lens)
        d_tok = torch.from_numpy(tokens.astype(np.int32)).to(dev)
        d_sl = torch.from_numpy(seq_lens).to(dev)
        d_cu = torch.from_numpy(cu).to(dev)
        d_ptf, d_pts = torch.from_numpy(pt_f).to(dev), torch.from_numpy(pt_s).to(dev)
        H = self.ss.shape_full.hidden
        x = [torch.empty((T, H), device=dev), torch.empty((T, H), device=dev)]
        mcpu.embed_tokens(self.embed, d_tok, x[0], self.ws)
        for i in range(self.spec.n_layers):
            sw = self.ss.is_sw(i)
            mcpu.decode_layer(self.ss.shape(i), self.weights[i], self.pools[i], d_pts if sw else d_ptf, d_sl, d_cu,
                              seq_lens, cu, x[i % 2], x[(i + 1) % 2], workspace=self.ws)
        return x[self.spec.n_layers % 2], cu

    def step(self) -> Dict[int, tuple]:
        """Advance every sequence with pending input by up to its whole input
        (bounded by max_tokens_per_step in total, oldest first). Returns
        {sid: (token, logprob)} for the sequences that sampled a token; a
        sampled token becomes that sequence's next input unless the caller
        calls `hold(sid)` (e.g. a tool call ends the turn)."""
        ready = [s for s in self.seqs.values() if s.pending]
        batch, q_lens, budget = [], [], self.max_tokens
        for s in ready:
            if budget <= 0:
                break
            q = min(len(s.pending), budget)
            batch.append(s)
            q_lens.append(q)
            budget -= q
        if not batch:
            return {}
        for s, q in zip(batch, q_lens):
            self._grow(s, q)
        tokens = np.concatenate([np.array(s.pending[:q], np.int64) for s, q in zip(batch, q_lens)])
        x, cu = self._forward(batch, q_lens, tokens)
        # sample for the sequences whose whole input has been fed
        done = [b for b, (s, q) in enumerate(zip(batch, q_lens)) if q == len(s.pending)]
        out = {}
        if done:
            dev = self.device
            rows = torch.from_numpy(np.array([cu[b + 1] - 1 for b in done], np.int32)).to(dev)
            sids = torch.from_numpy(np.array([batch[b].sid for b in done], np.int32)).to(dev)
            pos = torch.from_numpy(np.array([batch[b].length + q_lens[b] for b in done], np.int32)).to(dev)
            n = len(done)
            tok = torch.empty(n, dtype=torch.int32, device=dev)
            lp = torch.empty(n, device=dev)
            mcpu.lm_head_sample(self.head, x, self.spec.temperature, self.spec.seed, sids, pos, None, tok, lp,
                                workspace=self.lm_ws, x_rows=rows)
            tok_h, lp_h = tok.cpu().numpy(), lp.cpu().numpy()
            for j, b in enumerate(done):
                out[batch[b].sid] = (int(tok_h[j]), float(lp_h[j]))
        for b, (s, q) in enumerate(zip(batch, q_lens)):
            s.history.extend(s.pending[:q])
            del s.pending[:q]
            s.length += q
            self._shrink(s)
            if s.sid in out:
                s.pending.append(out[s.sid][0])
        self.steps += 1
        return out

    def hold(self, sid: int) -> None:
        """Drop the sequence's pending sampled token (its turn ended); the
        token is still part of the trajectory: it is fed with the next input."""
        s = self.seqs[sid]
        self.held[sid] = s.pending[:]
        s.pending.clear()

    def resume(self, sid: int, observation: Sequence[int]) -> None:
        """Append a tool observation after the held token."""
        held = self.held.pop(sid, [])
        self.add(sid, list(held) + list(observation))

    def check_errors(self) -> int:
        return mcpu.mcpu_check_device_errors(self.ws) | mcpu.mcpu_check_device_errors(self.lm_ws)

    # ------------------------------------------------------------------ trajectory scoring

    def score(self, trajectories: Sequence[Sequence[int]], sid_base: int = 1 << 20,
              temperature: Optional[float] = None) -> List[np.ndarray]:
        """Log-probability of every token of each trajectory given its prefix
        (token 0 has none), under softmax(logits / temperature): the whole
        trajectories are prefilled in chunks of at most max_tokens_per_step
        tokens in all, with the next tokens as targets. Pages are taken from
        and returned to the pools."""
        tau = self.spec.temperature if temperature is None else temperature
        trajectories = [np.asarray(t, np.int64) for t in trajectories]
        res = [np.zeros(max(len(t) - 1, 0), np.float64) for t in trajectories]
        states = [_Seq(sid_base + i) for i in range(len(trajectories))]
        try:
            while True:
                batch, q_lens, idx, budget = [], [], [], self.max_tokens
                for i, (s, tr) in enumerate(zip(states, trajectories)):
                    left = len(tr) - s.length
                    if left > 0 and budget > 0:
                        q = min(left, budget)
                        batch.append(s)
                        q_lens.append(q)
                        idx.append(i)
                        budget -= q
                if not batch:
                    break
                for s, q in zip(batch, q_lens):
                    self._grow(s, q)
                tokens = np.concatenate([trajectories[i][s.length:s.length + q]
                                         for i, s, q in zip(idx, batch, q_lens)])
                x, cu = self._forward(batch, q_lens, tokens)
                # targets: the token after each row (the last row of a trajectory has none)
                rows, tgts, spans = [], [], []
                for b, (i, s, q) in enumerate(zip(idx, batch, q_lens)):
                    n_t = min(q, len(trajectories[i]) - 1 - s.length)
                    if n_t > 0:
                        rows.append(cu[b] + np.arange(n_t, dtype=np.int32))
                        tgts.append(trajectories[i][s.length + 1:s.length + 1 + n_t])
                        spans.append((i, s.length, n_t))
                if rows:
                    dev = self.device
                    rows, tgts = np.concatenate(rows), np.concatenate(tgts).astype(np.int32)
                    tlp = torch.empty(len(rows), device=dev)
                    mcpu.lm_head_sample(self.head, x, tau, 0, None, None, torch.from_numpy(tgts).to(dev), None, None,
                                        tlp, workspace=self.lm_ws, x_rows=torch.from_numpy(rows).to(dev))
                    vals = tlp.cpu().numpy()
                    at = 0
                    for i, p, n_t in spans:
                        res[i][p:p + n_t] = vals[at:at + n_t]
                        at += n_t
                for s, q in zip(batch, q_lens):
                    s.length += q
                    self._shrink(s)
        finally:
            for s in states:
                if self.alloc_full is not None and s.pages_full:
                    mcpu.kv_pages_free(self.alloc_full, np.array(s.pages_full, np.int32))
                if s.pages_sw:
                    mcpu.kv_pages_free(self.alloc_sw, np.array(list(s.pages_sw.values()), np.int32))
        return res
