"""Decode-step benchmark on one MI355X.

One step = one decoder-layer step (RMSNorm, QKV + RoPE + KV append, paged
attention with sinks, O-projection, router, expert permutation, expert
GEMMs, combine) for every sequence of the batch, through the C ABI. Inputs
are seeded synthetic tensors already resident in HBM when timing starts.
Prints one JSON line: decode tokens/s, the roofline of the dominant kernel
(paged attention) measured with HIP events over the timed region, a
per-kernel breakdown from a separate pass, and the CPU reference timed on a
bounded sample of the same workload.
"""
import argparse
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
BF16_PEAK_TFLOPS = 2500.0
METRIC = "decode tokens/s on 1 MI355X (gpt-oss-20b-shape layer); % of HBM / MFMA peak"


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


STACK_WORKLOADS = ("stack24",)


def make_workload(name):
    from paper_2608_22167_amd import workload as W
    if name == "full_b64":
        return W.full_b64()
    if name == "sliding_b256":
        return W.sliding_b256()
    if name == "tiny_f32":
        return W.tiny_f32()
    if name == "stack24":
        return W.stack24()
    raise SystemExit(f"unknown workload {name}")


def kernel_bytes(s, T, visible_keys, idx):
    """Algorithmic HBM bytes per launch of each kernel of one layer (weights
    read once, the visible K/V once, activations in and out). MXFP4 experts
    count their codes (half a byte per weight) and scales (one byte per 32)."""
    eb = 4 if s.dtype == "f32" else 2
    H, D, Hq, Hkv, I = s.hidden, s.head_dim, s.n_q_heads, s.n_kv_heads, s.ffn_dim
    touched = len(np.unique(idx))
    wb = (lambda r, c: r * c // 2 + r * c // 32) if s.expert_fmt == "mxfp4" else (lambda r, c: r * c * eb)
    kv = visible_keys * Hkv * D * 2 * eb
    return {
        "attn_split": kv + T * Hq * D * eb,
        "qkv": s.qkv_dim * H * eb + T * H * eb + T * s.qkv_dim * eb,
        "oproj": H * Hq * D * eb + T * Hq * D * eb + 2 * T * H * 4,
        "expert_gu": touched * wb(2 * I, H) + T * s.top_k * (H + I) * eb,
        "expert_down": touched * wb(H, I) + T * s.top_k * (I * eb + H * 4),
    }


def stack_visible_keys(spec, layer):
    lens = spec.seq_lens.astype(np.int64) + 1
    return int(np.minimum(lens, spec.shape_sw.window).sum() if spec.is_sw(layer) else lens.sum())


def traffic_from_profile(kernel_src, workload_name):
    """HBM bytes per launch from a committed rocprofv3 counter summary, if it
    was taken on the current source of the kernel; else None."""
    path = os.path.join(ROOT, "profiles", f"attn_split_{workload_name}_counters.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    src_hash = hashlib.sha256(open(kernel_src, "rb").read()).hexdigest()[:16]
    m = re.search(r"source sha256\[:16\]:\s*([0-9a-f]{16})", text)
    t = re.search(r"hbm bytes per launch:\s*([0-9.eE+]+)", text)
    if not m or not t or m.group(1) != src_hash:
        return None
    return float(t.group(1))


def cpu_baseline(wl, n_seq=64):
    """The CPU reference on `n_seq` seeded sequences of the same workload."""
    from oracle import oracle as O
    from paper_2608_22167_amd import workload as W
    rng = np.random.default_rng(wl.seed + 99)
    seqs = np.sort(rng.choice(wl.batch, size=min(n_seq, wl.batch), replace=False))
    sub, _ = W.restrict(wl, seqs)
    weights = O.Weights(sub.shape, sub.weights)
    t0 = time.perf_counter()
    O.decode_layer(sub, weights)
    dt = time.perf_counter() - t0
    cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return {"value": round(sub.n_tokens / dt, 3), "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": f"{len(seqs)} of {wl.batch} sequences (seeded), one full layer step, "
                      f"{dt:.2f} s wall"}


def cpu_baseline_stack(spec, n_seq=2):
    """The CPU reference of the layer stack on `n_seq` seeded sequences, all layers."""
    from oracle import stack as OS
    rng = np.random.default_rng(spec.seed + 99)
    seqs = np.sort(rng.choice(spec.batch, size=min(n_seq, spec.batch), replace=False))
    t0 = time.perf_counter()
    OS.reference_stack(spec, seqs)
    dt = time.perf_counter() - t0
    cores = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    return {"value": round(len(seqs) / dt, 4), "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "sample": f"{len(seqs)} of {spec.batch} sequences (seeded, contexts "
                      f"{', '.join(str(int(spec.seq_lens[i])) for i in seqs)}) through all {spec.n_layers} "
                      f"layers, pages and used experts regenerated on the host, {dt:.2f} s wall"}


class LayerBench:
    """One decoder layer over a batch (decode_layer once per step)."""

    def __init__(self, wl):
        from paper_2608_22167_amd import mcpu
        self.wl, self.shape = wl, wl.shape
        self.step = mcpu.DeviceStep(wl)
        self.tokens = wl.n_tokens
        self.attn_per_step = 1

    def run(self):
        self.step.run()

    def errors(self):
        return self.step.device_errors()

    def bytes(self):
        """(per-step bytes of each kernel, bytes of each attn_split launch in a step)."""
        kb = kernel_bytes(self.shape, self.tokens, self.wl.visible_keys(), self.step.topk_idx.cpu().numpy())
        return kb, [kb["attn_split"]]

    def config(self):
        wl, s = self.wl, self.shape
        return {"workload": wl.name, "batch": wl.batch, "tokens": wl.n_tokens,
                "context": f"{int(wl.seq_lens.min())}..{int(wl.seq_lens.max())} "
                           f"(mean {float(wl.seq_lens.mean()):.0f})",
                "layer": f"hidden {s.hidden}, {s.n_q_heads}/{s.n_kv_heads} heads, d {s.head_dim}, "
                         f"{s.n_experts} experts top-{s.top_k}, ffn {s.ffn_dim}",
                "attention": "sliding window %d + sinks" % s.window if s.window else "full + sinks",
                "parallelism": "single GPU"}

    def cpu_baseline(self):
        return cpu_baseline(self.wl)


class StackBench:
    """The whole layer stack over a batch (decode_layer once per layer per step)."""

    def __init__(self, spec):
        from paper_2608_22167_amd import mcpu
        self.spec, self.shape = spec, spec.shape_full
        self.stack = mcpu.DeviceStack(spec)
        self.tokens = spec.batch
        self.attn_per_step = spec.n_layers

    def run(self):
        self.stack.run()

    def errors(self):
        return self.stack.device_errors()

    def bytes(self):
        idx = self.stack.topk_idx.cpu().numpy()
        total, attn = {}, []
        for layer in range(self.spec.n_layers):
            kb = kernel_bytes(self.spec.shape(layer), self.tokens, stack_visible_keys(self.spec, layer), idx[layer])
            for k, v in kb.items():
                total[k] = total.get(k, 0) + v
            attn.append(kb["attn_split"])
        return total, attn

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

    def cpu_baseline(self):
        return cpu_baseline_stack(self.spec)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed steps (default 50; 5 for a stack)")
    ap.add_argument("--warmup", type=int, default=None, help="untimed steps (default 10; 2 for a stack)")
    ap.add_argument("--workload", default="full_b64")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="after the benchmark, run 5 device-to-device copies of MIB MiB, the "
                         "reference kernel for scaling hardware byte counters")
    args = ap.parse_args()
    if args.gpus != 1:
        print(json.dumps({"error": "this benchmark runs on one GPU; the decode step is not sharded "
                                   "across GPUs in this build", "n_gpus": args.gpus}))
        raise SystemExit(2)
    is_stack = args.workload in STACK_WORKLOADS
    K = args.steps if args.steps is not None else (5 if is_stack else 50)
    warmup = args.warmup if args.warmup is not None else (2 if is_stack else 10)

    import torch
    from paper_2608_22167_amd import mcpu

    torch.cuda.set_device(0)
    log(f"generating workload {args.workload}")
    wl = make_workload(args.workload)
    bench = StackBench(wl) if is_stack else LayerBench(wl)
    torch.cuda.synchronize()
    log(f"resident: {torch.cuda.memory_allocated() / 1e9:.1f} GB; {bench.tokens} tokens per step")

    for _ in range(warmup):
        bench.run()
    torch.cuda.synchronize()
    if bench.errors():
        raise SystemExit("device error during warm-up")

    n_attn = K * bench.attn_per_step
    mcpu.mcpu_timing_start("attn_split", n_attn)
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(K):
        bench.run()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = ev0.elapsed_time(ev1) / K
    attn_ms = mcpu.mcpu_timing_read("attn_split", n_attn)
    mcpu.mcpu_timing_start("attn_split", 0)
    log(f"timed {K} steps: {ms_step * 1e3:.1f} us/step (wall {wall / K * 1e6:.1f} us/step)")

    # per-kernel breakdown (microseconds per step, all launches), separate pass
    nb = min(K, 20)
    n_launch = nb * bench.attn_per_step
    for k in mcpu.KERNELS:
        mcpu.mcpu_timing_start(k, 4 * n_launch)
    for _ in range(nb):
        bench.run()
    torch.cuda.synchronize()
    breakdown = {}
    for k in mcpu.KERNELS:
        ms = mcpu.mcpu_timing_read(k, 4 * n_launch)
        mcpu.mcpu_timing_start(k, 0)
        if len(ms):
            breakdown[k] = round(float(np.sum(ms)) / nb * 1e3, 2)
    if bench.errors():
        raise SystemExit("device error during timing")

    kb, attn_launch_bytes = bench.bytes()
    # dominant kernel: attention over the full-context layers (every launch for a
    # single layer; the full-attention layers of a stack, which read >99% of its K/V)
    per = np.asarray(attn_ms, np.float64).reshape(K, bench.attn_per_step)
    if is_stack:
        cols = [i for i in range(bench.attn_per_step) if not wl.is_sw(i)]
        kernel_label = "attn_split (full-attention layers)"
    else:
        cols = [0]
        kernel_label = "attn_split"
    launch_bytes = float(np.mean([attn_launch_bytes[c] for c in cols]))
    attn_us = float(per[:, cols].mean()) * 1e3
    achieved = launch_bytes / (attn_us * 1e-6) / 1e9
    traffic = traffic_from_profile(os.path.join(ROOT, "paper_2608_22167_amd", "csrc", "attention.hip"),
                                   args.workload)
    roofline = {"kernel": kernel_label, "bound": "hbm", "achieved": round(achieved, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": traffic, "avg_us": round(attn_us, 2), "algorithmic_bytes": round(launch_bytes)}
    per_kernel_gbs = {k: round(kb[k] / (breakdown[k] * 1e-6) / 1e9, 1) for k in kb if k in breakdown}
    step_bytes = sum(kb.values())

    if args.copy_calibration > 0:
        n = args.copy_calibration << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copy calibration: 5 copies of {n} bytes")

    cpu = None
    if not args.no_cpu_baseline:
        log("timing the CPU reference on a sample")
        cpu = bench.cpu_baseline()

    value = bench.tokens / (ms_step * 1e-3)
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": K,
        "warmup": warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": bench.shape.dtype, "data": "synthetic",
        "config": bench.config(),
        "roofline": roofline,
        "step_hbm_gbs": round(step_bytes / (ms_step * 1e-3) / 1e9, 1),
        "cpu_baseline": cpu,
        "kernels_us": breakdown,
        "kernels_gbs": per_kernel_gbs,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
