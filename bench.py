"""Decode-step benchmark on one MI355X.

One step = one decoder-layer step (RMSNorm, QKV + RoPE + KV append, paged
attention with sinks, O-projection, router, expert permutation, expert
GEMMs, combine) for every sequence of the batch, through the C ABI; for the
stack workload, that step through all 24 layers. Inputs are seeded synthetic
tensors already resident in HBM when timing starts.

Prints one JSON line: tokens/s, the roofline of the dominant kernel (the one
with the most time per step in an untimed breakdown pass), whose launch
durations are measured with HIP events on its own stream inside the timed
region, a per-kernel breakdown, and the CPU reference timed on a bounded
sample of the same workload.
"""
import argparse
import ctypes
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
# dense matrix-core peaks; products with MXFP8 activations run at the fp8 rate
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3, "mxfp8": 5000.0}
METRIC = "decode tokens/s on 1 MI355X (gpt-oss-20b-shape layer); % of HBM / MFMA peak"
PREFILL_MIN_Q = 16  # chunks of this many new tokens or more go to the prefill kernel

STACK_WORKLOADS = ("stack24",)


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def make_workload(name):
    from paper_2608_22167_amd import workload as W
    makers = {"full_b64": W.full_b64, "sliding_b256": W.sliding_b256, "tiny_f32": W.tiny_f32,
              "mixed_prefill": W.mixed_prefill, "stack24": W.stack24,
              "mixed_prefill_mxfp4": lambda: W.mixed_prefill(expert_fmt="mxfp4_native")}
    if name not in makers:
        raise SystemExit(f"unknown workload {name}; one of {sorted(makers)}")
    return makers[name]()


def _visible_sum(L0, q, window):
    """Sum over a sequence's new tokens (positions L0 .. L0+q-1) of the keys each sees."""
    p = np.arange(L0, L0 + q, dtype=np.int64)
    return int(np.minimum(p + 1, window).sum() if window else (p + 1).sum())


def layer_work(s, seq_lens, q_lens, idx):
    """Algorithmic (HBM bytes, flops) of each kernel of one layer step: weights
    read once, the visible K/V once per sequence, activations in and out; MXFP4
    experts count their codes (half a byte per weight) and scales (one byte per
    32). Attention flops are 4 Hq d per (query, visible key) pair."""
    eb = 4 if s.dtype == "f32" else 2
    H, D, Hq, Hkv, I, k = s.hidden, s.head_dim, s.n_q_heads, s.n_kv_heads, s.ffn_dim, s.top_k
    A = Hq * D
    T = int(np.sum(q_lens))
    kvb = Hkv * D * 2 * eb
    dec_pairs = pre_pairs = pre_keys = 0
    t_dec = t_pre = 0
    for L0, q in zip(np.asarray(seq_lens, np.int64), np.asarray(q_lens, np.int64)):
        vis = _visible_sum(int(L0), int(q), s.window)
        if q >= PREFILL_MIN_Q:
            pre_pairs += vis
            t_pre += int(q)
            last = int(L0 + q - 1)
            lo = max(0, int(L0) - s.window + 1) if s.window else 0
            pre_keys += last - lo + 1
        else:
            dec_pairs += vis
            t_dec += int(q)
    rows = T * k
    touched = len(np.unique(idx))
    wb = (lambda r, c: r * c // 2 + r * c // 32) if s.expert_fmt != "dense" else (lambda r, c: r * c * eb)
    work = {
        "attn_split": (dec_pairs * kvb + t_dec * A * eb, 4 * A * dec_pairs),
        "qkv": (s.qkv_dim * H * eb + T * H * eb + T * s.qkv_dim * eb, 2 * T * s.qkv_dim * H),
        "oproj": (H * A * eb + T * A * eb + 2 * T * H * 4, 2 * T * H * A),
        "expert_gu": (touched * wb(2 * I, H) + rows * (H + I) * eb, 2 * rows * 2 * I * H),
        "expert_down": (touched * wb(H, I) + rows * (I * eb + H * 4), 2 * rows * H * I),
    }
    if t_pre:
        work["attn_prefill"] = (pre_keys * kvb + 2 * t_pre * A * eb, 4 * A * pre_pairs)
    return work, t_dec, t_pre


def peak_key(kernel, shape):
    """The matrix-core peak a kernel's products run against."""
    if shape.expert_fmt == "mxfp4_native" and kernel in ("expert_gu", "expert_down"):
        return "mxfp8"
    return shape.dtype


def roofline_of(work_bytes, work_flops, seconds, dtype):
    """The binding resource of a kernel: HBM below the ridge point, MFMA above."""
    peak_tf = MFMA_PEAK_TFLOPS[dtype]
    ridge = peak_tf * 1e12 / (HBM_PEAK_GBS * 1e9)
    if work_flops > ridge * work_bytes:
        a = work_flops / seconds / 1e12
        return {"bound": "mfma", "achieved": round(a, 1), "peak": peak_tf, "unit": "TFLOP/s",
                "frac": round(a / peak_tf, 4)}
    a = work_bytes / seconds / 1e9
    return {"bound": "hbm", "achieved": round(a, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(a / HBM_PEAK_GBS, 4)}


def source_hash(kernel):
    """sha256[:16] over the sources the kernel is built from, in a fixed order."""
    h = hashlib.sha256()
    for name in KERNEL_SOURCES.get(kernel, ATTN_SOURCES):
        h.update(open(os.path.join(ROOT, "paper_2608_22167_amd", "csrc", name), "rb").read())
    return h.hexdigest()[:16]


def traffic_from_profile(kernel, workload_name):
    """HBM bytes per launch from a committed rocprofv3 counter summary, if it
    was taken on the current sources of the kernel; else None."""
    path = os.path.join(ROOT, "profiles", f"{kernel}_{workload_name}_counters.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    m = re.search(r"sources sha256\[:16\]:\s*([0-9a-f]{16})", text)
    t = re.search(r"hbm bytes per launch:\s*([0-9.eE+]+)", text)
    if not m or not t or m.group(1) != source_hash(kernel):
        return None
    return float(t.group(1))


ATTN_SOURCES = ("attention.hip", "device.h", "kernels.h")
GEMM_SOURCES = ("gemm.hip", "gemm_tiled.hip", "gemm_pipe.hip", "gemm_slab.hip", "gemm_mx.hip", "gemm_epilogue.h", "device.h",
                "kernels.h")
KERNEL_SOURCES = {"attn_split": ATTN_SOURCES, "attn_prefill": ATTN_SOURCES, "qkv": GEMM_SOURCES,
                  "oproj": GEMM_SOURCES, "expert_gu": GEMM_SOURCES, "expert_down": GEMM_SOURCES,
                  "lm_head": GEMM_SOURCES + ("lm_head.hip", "kernels_lm.h")}


class StepEvents:
    """Event pairs around the timed steps, recorded without the system-scope
    fence (hipEventDisableSystemFence): a fenced record writes back and
    invalidates the caches, a stall of about 6 us that torch's events add to
    the end of every measured step. The HIP runtime is the one already loaded
    into the process (found by path, so no second copy is opened); if it cannot
    be used, torch's events are."""
    DISABLE_SYSTEM_FENCE = 0x20000000

    def __init__(self, n, stream):
        import torch
        self.stream, self.hip, self.pairs = stream, None, []
        try:
            path = next(l.split()[-1] for l in open("/proc/self/maps") if "libamdhip64.so" in l)
            hip = ctypes.CDLL(path)
            for _ in range(n):
                pair = []
                for _ in range(2):
                    ev = ctypes.c_void_p()
                    if hip.hipEventCreateWithFlags(ctypes.byref(ev), ctypes.c_uint(self.DISABLE_SYSTEM_FENCE)):
                        raise OSError("hipEventCreateWithFlags")
                    pair.append(ev)
                self.pairs.append(pair)
            self.hip = hip
        except (OSError, StopIteration):
            self.pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                          for _ in range(n)]

    def record(self, i, which):
        ev = self.pairs[i][which]
        if self.hip is None:
            ev.record(self.stream)
        elif self.hip.hipEventRecord(ev, ctypes.c_void_p(self.stream.cuda_stream)):
            raise SystemExit("hipEventRecord failed")

    def elapsed_ms(self):
        if self.hip is None:
            return np.array([a.elapsed_time(b) for a, b in self.pairs], np.float64)
        out = []
        for a, b in self.pairs:
            ms = ctypes.c_float()
            if self.hip.hipEventSynchronize(b) or self.hip.hipEventElapsedTime(ctypes.byref(ms), a, b):
                raise SystemExit("hipEventElapsedTime failed")
            out.append(ms.value)
        for pair in self.pairs:
            for ev in pair:
                self.hip.hipEventDestroy(ev)
        return np.array(out, np.float64)


def timed_passes(fn, min_seconds=10.0, max_passes=50):
    """Runs fn until at least min_seconds have passed (at least once, at most
    max_passes times): (passes, seconds)."""
    passes, t0 = 0, time.perf_counter()
    while True:
        fn()
        passes += 1
        dt = time.perf_counter() - t0
        if dt >= min_seconds or passes >= max_passes:
            return passes, dt


def cpu_cores():
    return int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))


def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo), for the CPU baseline."""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


# Reading this many bytes between timed steps evicts the previous step's data
# from the L2 caches and the 256 MB memory-side cache (MALL), so every step
# reads its weights and cache pages from HBM. A read leaves clean lines
# behind; a write would leave dirty ones whose write-back then competes with
# the next step's first kernels.
FLUSH_BYTES = 1 << 30


class LayerBench:
    """One decoder layer over a batch (decode_layer once per step)."""

    def __init__(self, wl):
        from paper_2608_22167_amd import mcpu
        self.wl, self.shape = wl, wl.shape
        self.step = mcpu.DeviceStep(wl)
        self.tokens = wl.n_tokens
        self.launches = 1

    def run(self):
        self.step.run()

    def errors(self):
        return self.step.device_errors()

    def work(self):
        """[launch in a step] -> {kernel: (bytes, flops)}; decode and prefill token counts."""
        w, t_dec, t_pre = layer_work(self.shape, self.wl.seq_lens, self.wl.q_lens,
                                     self.step.topk_idx.cpu().numpy())
        return [w], t_dec, t_pre

    def dominant_launches(self, kernel):
        return [0]

    def config(self):
        wl, s = self.wl, self.shape
        c = {"workload": wl.name, "batch": wl.batch, "tokens": wl.n_tokens,
             "context": f"{int(wl.seq_lens.min())}..{int(wl.seq_lens.max())} (mean {float(wl.seq_lens.mean()):.0f})",
             "layer": f"hidden {s.hidden}, {s.n_q_heads}/{s.n_kv_heads} heads, d {s.head_dim}, "
                      f"{s.n_experts} experts top-{s.top_k}, ffn {s.ffn_dim}",
             "attention": "sliding window %d + sinks" % s.window if s.window else "full + sinks",
             "parallelism": "single GPU"}
        if wl.q_lens.max() > 1:
            pre = wl.q_lens[wl.q_lens > 1]
            c["prefill_chunks"] = f"{len(pre)} chunks of {int(pre.min())}..{int(pre.max())} tokens"
        return c

    def cpu_baseline(self, n_seq=64):
        """The CPU reference on n_seq seeded sequences (decode steps) or on the
        decode sequences plus the shortest prefill chunk (mixed steps)."""
        from oracle import oracle as O
        from paper_2608_22167_amd import workload as W
        wl = self.wl
        rng = np.random.default_rng(wl.seed + 99)
        dec = np.nonzero(wl.q_lens == 1)[0]
        seqs = rng.choice(dec, size=min(n_seq if len(dec) == wl.batch else 8, len(dec)), replace=False)
        if len(dec) < wl.batch:
            pre = np.nonzero(wl.q_lens > 1)[0]
            seqs = np.append(seqs, pre[np.argmin(wl.q_lens[pre])])
        seqs = np.sort(seqs)
        sub, _ = W.restrict(wl, seqs)
        weights = O.Weights(sub.shape, sub.weights)
        passes, dt = timed_passes(lambda: O.decode_layer(sub, weights))
        return {"value": round(passes * sub.n_tokens / dt, 3), "unit": "tokens/s (all tokens of the sample)",
                "cores": cpu_cores(), "cpu": cpu_model(), "kind": "oracle",
                "sample": f"{len(seqs)} of {wl.batch} sequences (seeded), {sub.n_tokens} tokens, one layer step, "
                          f"{passes} passes in {dt:.2f} s wall"}


class StackBench:
    """The whole layer stack over a batch (decode_layer once per layer per step)."""

    def __init__(self, spec):
        from paper_2608_22167_amd import mcpu
        self.spec, self.shape = spec, spec.shape_full
        self.stack = mcpu.DeviceStack(spec)
        self.tokens = spec.batch
        self.launches = spec.n_layers

    def run(self):
        self.stack.run()

    def errors(self):
        return self.stack.device_errors()

    def work(self):
        idx = self.stack.topk_idx.cpu().numpy()
        q = np.ones(self.spec.batch, np.int64)
        per = [layer_work(self.spec.shape(i), self.spec.seq_lens, q, idx[i])[0] for i in range(self.spec.n_layers)]
        return per, self.spec.batch, 0

    def dominant_launches(self, kernel):
        # the full-attention layers read over 99% of the stack's K/V
        if kernel == "attn_split":
            return [i for i in range(self.spec.n_layers) if not self.spec.is_sw(i)]
        return list(range(self.spec.n_layers))

    def config(self):
        sp, s = self.spec, self.shape
        return {"workload": sp.name, "batch": sp.batch, "tokens": sp.batch, "layers": sp.n_layers,
                "context": f"{int(sp.seq_lens.min())}..{int(sp.seq_lens.max())} "
                           f"(mean {float(sp.seq_lens.mean()):.0f}, log-normal median 8192, cap 65536)",
                "layer": f"hidden {s.hidden}, {s.n_q_heads}/{s.n_kv_heads} heads, d {s.head_dim}, "
                         f"{s.n_experts} MXFP4 experts top-{s.top_k}, ffn {s.ffn_dim}",
                "attention": f"alternating sliding window {sp.shape_sw.window} / full, + sinks",
                "kv_resident_gb": round(sum(p.numel() * 2 for p in self.stack.k + self.stack.v) / 1e9, 1),
                "parallelism": "single GPU"}

    def cpu_baseline(self, n_seq=2):
        """The CPU reference of the layer stack on n_seq seeded sequences, all layers."""
        from oracle import stack as OS
        spec = self.spec
        rng = np.random.default_rng(spec.seed + 99)
        seqs = np.sort(rng.choice(spec.batch, size=min(n_seq, spec.batch), replace=False))
        t0 = time.perf_counter()
        OS.reference_stack(spec, seqs)
        dt = time.perf_counter() - t0
        return {"value": round(len(seqs) / dt, 4), "unit": "tokens/s", "cores": cpu_cores(), "cpu": cpu_model(),
                "kind": "oracle",
                "sample": f"{len(seqs)} of {spec.batch} sequences (seeded, contexts "
                          f"{', '.join(str(int(spec.seq_lens[i])) for i in seqs)}) through all {spec.n_layers} "
                          f"layers, pages and used experts regenerated on the host, {dt:.2f} s wall"}


class HeadBench:
    """The vocabulary head of a generation step at batch 256: final RMSNorm,
    the projection onto the 201,088-entry vocabulary with the sampling
    epilogue (temperature 0.7, Gumbel-max draws), and the per-row reduction:
    one lm_head_sample call per step."""

    def __init__(self, T=256, seed=3001):
        import torch
        from paper_2608_22167_amd import mcpu, workload as W
        self.shape = W.GPT_OSS_20B
        H, V = self.shape.hidden, W.GPT_OSS_VOCAB
        lm = W.lm_weights_device(seed, H, V)
        del lm["embed"]
        self.head = mcpu.DeviceLmHead(lm["g_final"], lm["w_lm"], self.shape.rms_eps)
        self.lm_host = None
        self.seed, self.T, self.H, self.V = seed, T, H, V
        self.x = W.synth_normal(seed, 77, (T, H)).cuda()
        self.seq = torch.arange(T, dtype=torch.int32, device="cuda")
        self.pos = torch.full((T,), 4096, dtype=torch.int32, device="cuda")
        self.tok = torch.empty(T, dtype=torch.int32, device="cuda")
        self.lp = torch.empty(T, device="cuda")
        self.ws = mcpu.workspace(mcpu.lm_head_workspace_size(H, V, T))
        self.temperature = float(np.float32(0.7))
        self.tokens, self.launches = T, 1

    def run(self):
        from paper_2608_22167_amd import mcpu
        mcpu.lm_head_sample(self.head, self.x, self.temperature, seed=self.seed, seq_ids=self.seq,
                            positions=self.pos, tokens=self.tok, logprob=self.lp, workspace=self.ws)

    def errors(self):
        from paper_2608_22167_amd import mcpu
        return mcpu.mcpu_check_device_errors(self.ws)

    def work(self):
        # the head's weights once, the normalised rows, the per-slice records written
        T, H, V = self.T, self.H, self.V
        slots = (V + 63) // 64
        return [{"lm_head": (V * H * 2 + T * H * 2 + T * slots * 32, 2 * T * V * H)}], T, 0

    def dominant_launches(self, kernel):
        return [0]

    def config(self):
        return {"workload": "lm_head_b256", "batch": self.T, "tokens": self.T, "vocab": self.V, "hidden": self.H,
                "temperature": self.temperature, "sampling": "Gumbel-max over Philox4x32-10 draws",
                "parallelism": "single GPU"}

    def cpu_baseline(self, n_rows=4):
        """The reference head (float64 logits, the same draws) on n_rows rows."""
        from oracle import oracle as O
        from paper_2608_22167_amd import workload as W
        lm = W.lm_weights_host(self.seed, self.H, self.V, embed=False)
        x = W.synth_normal(self.seed, 77, (self.T, self.H))[:n_rows]
        seq = np.arange(n_rows, dtype=np.int32)
        pos = np.full(n_rows, 4096, np.int32)
        passes, dt = timed_passes(lambda: O.lm_head(x, lm["g_final"], lm["w_lm"], self.shape.rms_eps, self.temperature,
                                                    seed=self.seed, seq_ids=seq, positions=pos))
        return {"value": round(passes * n_rows / dt, 3), "unit": "tokens/s", "cores": cpu_cores(), "cpu": cpu_model(),
                "kind": "oracle", "sample": f"{n_rows} of {self.T} rows, {passes} passes in {dt:.2f} s wall"}


class ScoreBench:
    """The log-probability pass of the policy update over whole trajectories
    (8 seeded trajectories of 4096 tokens): embedding, one causal prefill of
    every trajectory through the 24-layer stack (MXFP4 experts), and the
    vocabulary head scoring each next token; one Generator.score call per
    step, host marshalling of the targets and the copy of the log-probs back
    included."""

    metric = "scored tokens/s on 1 MI355X (trajectory log-prob recompute, gpt-oss-20b-shape stack)"

    def __init__(self, n_traj=8, length=4096, seed=3001):
        from paper_2608_22167_amd import workload as W
        from paper_2608_22167_amd.generate import GenSpec, Generator
        pages = n_traj * length // 16 + 64
        self.spec = GenSpec(n_layers=24, base=W.GPT_OSS_20B, vocab=W.GPT_OSS_VOCAB, seed=seed,
                            pages_full=pages, pages_sw=pages, max_ctx=length + 64)
        self.gen = Generator(self.spec, max_tokens_per_step=n_traj * length)
        self.ss = self.gen.ss
        self.shape = self.ss.shape_full
        rng = np.random.default_rng(seed)
        self.traj = [rng.integers(0, self.spec.vocab, length) for _ in range(n_traj)]
        self.n_traj, self.length = n_traj, length
        self.tokens = n_traj * (length - 1)  # scored tokens per step
        self.launches = self.spec.n_layers

    def run(self):
        self.gen.score(self.traj)

    def errors(self):
        return self.gen.check_errors()

    def work(self):
        z = np.zeros(self.n_traj, np.int64)
        q = np.full(self.n_traj, self.length, np.int64)
        # 131,072 routed rows reach every expert of every layer
        idx = np.arange(self.shape.n_experts)
        per = [layer_work(self.ss.shape(i), z, q, idx)[0] for i in range(self.spec.n_layers)]
        V, H, T = self.spec.vocab, self.shape.hidden, self.tokens
        per[0]["lm_head"] = (V * H * 2 + T * H * 2 + T * ((V + 63) // 64) * 32, 2 * T * V * H)
        return per, self.tokens, 0

    def dominant_launches(self, kernel):
        return [0] if kernel == "lm_head" else list(range(self.spec.n_layers))

    def config(self):
        s = self.shape
        return {"workload": "score_8x4096", "trajectories": self.n_traj, "tokens_per_trajectory": self.length,
                "scored_tokens": self.tokens, "layers": self.spec.n_layers, "vocab": self.spec.vocab,
                "temperature": self.spec.temperature,
                "layer": f"hidden {s.hidden}, {s.n_q_heads}/{s.n_kv_heads} heads, d {s.head_dim}, "
                         f"{s.n_experts} MXFP4 experts top-{s.top_k}, ffn {s.ffn_dim}",
                "attention": f"alternating sliding window {self.ss.shape_sw.window} / full, + sinks",
                "parallelism": "single GPU"}

    def cpu_baseline(self, n=16, n_layers=2):
        """The reference on the first n tokens of one trajectory: the first
        n_layers layers (one sliding-window, one full) as one causal prefill,
        then the head with targets on the n - 1 scored rows. The experts the
        sample routes to are drawn once, before timing. Per scored token:
        (n_layers-layer time x 24 / n_layers + head time) / (n - 1)."""
        import torch
        from oracle import oracle as O
        from oracle import stack as OS
        from paper_2608_22167_amd import workload as W
        ss, s0 = self.ss, self.shape
        tr = np.asarray(self.traj[0][:n], np.int64)
        lm = W.lm_weights_host(self.spec.seed, s0.hidden, self.spec.vocab)
        x0 = lm["embed"][torch.from_numpy(tr[:-1])].double()
        n_pages = (n - 2) // 16 + 1
        layers = []
        for i in range(n_layers):
            s = ss.shape(i)
            ex = OS._Experts(ss)
            Wd = W.stack_weights_host(ss, i, experts=[])
            Wd["w_gu"], Wd["w_d"] = ex.w_gu, ex.w_d
            wl = W.Workload(name="score_sample", shape=s, seed=ss.seed, seq_lens=np.zeros(1, np.int32),
                            q_lens=np.array([n - 1], np.int32), page_table=np.arange(n_pages, dtype=np.int32)[None],
                            n_pages=n_pages, weights=Wd)
            wl.k_pool = torch.zeros((n_pages, s.n_kv_heads, 16, s.head_dim), dtype=torch.bfloat16)
            wl.v_pool = torch.zeros_like(wl.k_pool)
            layers.append((wl, O.Weights(s, Wd), ex))
        x = x0
        for i, (wl, wt, ex) in enumerate(layers):  # routing pass, then draw the experts it picked
            wl.x_in = x
            ex.draw(ss, i, O.decode_layer(wl, wt)["idx"])
            x = torch.from_numpy(O.decode_layer(wl, wt)["out"])

        def stack():
            x = x0
            for wl, wt, _ in layers:
                wl.x_in = x
                x = torch.from_numpy(O.decode_layer(wl, wt)["out"])
            return x.numpy()
        rows = stack()
        p_l, t_l = timed_passes(stack, min_seconds=6.0, max_passes=20)
        tg = tr[1:].astype(np.int32)
        zero = np.zeros(n - 1, np.int32)
        p_h, t_h = timed_passes(lambda: O.lm_head(rows, lm["g_final"], lm["w_lm"], s0.rms_eps, self.spec.temperature,
                                                  seq_ids=zero, positions=zero, targets=tg),
                                min_seconds=6.0, max_passes=20)
        per_tok = (t_l / p_l * self.spec.n_layers / n_layers + t_h / p_h) / (n - 1)
        return {"value": round(1.0 / per_tok, 3), "unit": "scored tokens/s", "cores": cpu_cores(), "cpu": cpu_model(),
                "kind": "oracle",
                "sample": f"the first {n} tokens of one trajectory: layers 0-{n_layers - 1} as one prefill "
                          f"({p_l} passes in {t_l:.2f} s, scaled to {self.spec.n_layers} layers) and the head on "
                          f"{n - 1} rows with targets ({p_h} passes in {t_h:.2f} s)"}


HEAD_WORKLOADS = ("lm_head_b256",)
SCORE_WORKLOADS = ("score_8x4096",)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed steps (default 50; 5 for a stack or mixed step)")
    ap.add_argument("--warmup", type=int, default=None, help="untimed steps (default 10; 2 for a stack or mixed step)")
    ap.add_argument("--workload", default="sliding_b256")
    ap.add_argument("--no-flush", action="store_true", help="do not evict the caches between timed steps")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="after the benchmark, run 5 device-to-device copies of MIB MiB, the "
                         "reference kernel for scaling hardware byte counters")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU; the decode step is not sharded "
                                   "across GPUs in this build", "n_gpus": args.gpus}))
        raise SystemExit(2)
    heavy = args.workload in STACK_WORKLOADS + SCORE_WORKLOADS or args.workload.startswith("mixed_prefill")
    K = args.steps if args.steps is not None else (5 if heavy else 50)
    warmup = args.warmup if args.warmup is not None else (2 if heavy else 10)

    import torch
    from paper_2608_22167_amd import mcpu

    torch.cuda.set_device(0)
    log(f"generating workload {args.workload}")
    if args.workload in HEAD_WORKLOADS:
        bench = HeadBench()
    elif args.workload in SCORE_WORKLOADS:
        bench = ScoreBench()
    else:
        wl = make_workload(args.workload)
        bench = StackBench(wl) if args.workload in STACK_WORKLOADS else LayerBench(wl)
    torch.cuda.synchronize()
    log(f"resident: {torch.cuda.memory_allocated() / 1e9:.1f} GB; {bench.tokens} tokens per step")

    for _ in range(warmup):
        bench.run()
    torch.cuda.synchronize()
    if bench.errors():
        raise SystemExit("device error during warm-up")

    flush = None if args.no_flush else torch.ones(FLUSH_BYTES // 2, dtype=torch.float16, device="cuda")

    def evict(i):
        if flush is not None:
            torch.sum(flush)

    # per-kernel breakdown (microseconds per step, all launches), untimed pass
    nb = min(K, 20)
    cap = 4 * nb * bench.launches
    for k in mcpu.KERNELS:
        mcpu.mcpu_timing_start(k, cap)
    for i in range(nb):
        evict(i)
        bench.run()
    torch.cuda.synchronize()
    breakdown = {}
    for k in mcpu.KERNELS:
        ms = mcpu.mcpu_timing_read(k, cap)
        mcpu.mcpu_timing_start(k, 0)
        if len(ms):
            breakdown[k] = round(float(np.sum(ms)) / nb * 1e3, 2)
    per_launch, t_dec, t_pre = bench.work()
    work = {}
    for w in per_launch:
        for k, (b, f) in w.items():
            work[k] = (work.get(k, (0, 0))[0] + b, work.get(k, (0, 0))[1] + f)
    dominant = max((k for k in breakdown if k in work), key=lambda k: breakdown[k])
    log(f"dominant kernel {dominant} ({breakdown[dominant]} us per step)")

    # timed region: HIP events around the dominant kernel's launches
    n_launch = K * bench.launches
    mcpu.mcpu_timing_start(dominant, n_launch)
    # each step between its own event pair; the cache eviction runs between
    # steps, outside the events
    stream = torch.cuda.current_stream()
    evs = StepEvents(K, stream)
    log("step events: " + ("HIP, without the system-scope fence" if evs.hip else "torch"))
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(K):
        evict(i)
        evs.record(i, 0)
        bench.run()
        evs.record(i, 1)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    step_ms = evs.elapsed_ms()
    ms_step = float(step_ms.mean())
    dom_ms = np.asarray(mcpu.mcpu_timing_read(dominant, n_launch), np.float64)
    mcpu.mcpu_timing_start(dominant, 0)
    if bench.errors():
        raise SystemExit("device error during timing")
    log(f"timed {K} steps: {ms_step * 1e3:.1f} us/step mean, median {np.median(step_ms) * 1e3:.1f} "
        f"(wall {wall / K * 1e6:.1f} us/step with cache eviction)")

    cols = bench.dominant_launches(dominant)
    per = dom_ms.reshape(K, -1)[:, cols]
    launch_bytes = float(np.mean([per_launch[c][dominant][0] for c in cols]))
    launch_flops = float(np.mean([per_launch[c][dominant][1] for c in cols]))
    dom_us = float(per.mean()) * 1e3
    roofline = {"kernel": dominant + (" (full-attention layers)" if cols != list(range(bench.launches)) else "")}
    roofline.update(roofline_of(launch_bytes, launch_flops, dom_us * 1e-6, peak_key(dominant, bench.shape)))
    roofline.update({"traffic": traffic_from_profile(dominant, args.workload), "avg_us": round(dom_us, 2),
                     "algorithmic_bytes": round(launch_bytes), "algorithmic_flops": round(launch_flops)})
    kernels_util = {k: roofline_of(b, f, breakdown[k] * 1e-6, peak_key(k, bench.shape))
                    for k, (b, f) in work.items() if breakdown.get(k)}
    kernels_util = {k: f"{v['achieved']} {v['unit']} ({100 * v['frac']:.1f}% {v['bound']})"
                    for k, v in kernels_util.items()}

    if args.copy_calibration > 0:
        n = args.copy_calibration << 20
        src_t = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src_t)
        for _ in range(5):
            dst.copy_(src_t)
        torch.cuda.synchronize()
        log(f"copy calibration: 5 copies of {n} bytes")

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU reference on a sample")
        cpu = bench.cpu_baseline()

    decode_tokens = t_dec if t_pre else bench.tokens
    out = {
        "metric": getattr(bench, "metric", METRIC), "value": round(decode_tokens / (ms_step * 1e-3), 1),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": K, "warmup": warmup, "ms_per_step": round(ms_step, 4),
        "ms_per_step_p10_p50_p90": [round(float(np.percentile(step_ms, p)), 4) for p in (10, 50, 90)],
        "caches_evicted_between_steps": flush is not None, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": bench.shape.dtype, "data": "synthetic",
        "config": bench.config(),
        "roofline": roofline,
        "cpu_baseline": cpu,
        "kernels_us": breakdown,
        "kernels_roofline": kernels_util,
    }
    if t_pre:
        out["prefill_tokens_per_s"] = round(t_pre / (ms_step * 1e-3), 1)
        out["all_tokens_per_s"] = round((t_dec + t_pre) / (ms_step * 1e-3), 1)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
