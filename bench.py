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


def make_workload(name):
    from paper_2608_22167_amd import workload as W
    if name == "full_b64":
        return W.full_b64()
    if name == "sliding_b256":
        return W.sliding_b256()
    if name == "tiny_f32":
        return W.tiny_f32()
    raise SystemExit(f"unknown workload {name}")


def kernel_bytes(wl, idx):
    """Algorithmic HBM bytes per launch of each kernel (weights read once,
    the visible K/V once, activations in and out)."""
    s = wl.shape
    eb = 4 if s.dtype == "f32" else 2
    T = wl.n_tokens
    H, D, Hq, Hkv, E, I = s.hidden, s.head_dim, s.n_q_heads, s.n_kv_heads, s.n_experts, s.ffn_dim
    touched = len(np.unique(idx))
    kv = wl.visible_keys() * Hkv * D * 2 * eb
    return {
        "attn_split": kv + T * Hq * D * eb,
        "qkv": s.qkv_dim * H * eb + T * H * eb + T * s.qkv_dim * eb,
        "oproj": H * Hq * D * eb + T * Hq * D * eb + 2 * T * H * 4,
        "expert_gu": touched * 2 * I * H * eb + T * s.top_k * (H + I) * eb,
        "expert_down": touched * H * I * eb + T * s.top_k * (I * eb + H * 4),
    }


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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
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

    import torch
    from paper_2608_22167_amd import mcpu

    torch.cuda.set_device(0)
    log(f"generating workload {args.workload}")
    wl = make_workload(args.workload)
    log(f"uploading: batch {wl.batch}, tokens {wl.n_tokens}, pages {wl.n_pages}")
    step = mcpu.DeviceStep(wl)
    torch.cuda.synchronize()

    for _ in range(args.warmup):
        step.run()
    torch.cuda.synchronize()
    if step.device_errors():
        raise SystemExit("device error during warm-up")

    K = args.steps
    mcpu.mcpu_timing_start("attn_split", K)
    stream = torch.cuda.current_stream()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record(stream)
    for _ in range(K):
        step.run()
    ev1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = ev0.elapsed_time(ev1) / K
    attn_ms = mcpu.mcpu_timing_read("attn_split", K)
    mcpu.mcpu_timing_start("attn_split", 0)
    log(f"timed {K} steps: {ms_step * 1e3:.1f} us/step (wall {wall / K * 1e6:.1f} us/step)")

    # per-kernel breakdown, separate pass
    nb = min(K, 20)
    for k in mcpu.KERNELS:
        mcpu.mcpu_timing_start(k, nb)
    for _ in range(nb):
        step.run()
    torch.cuda.synchronize()
    breakdown = {}
    for k in mcpu.KERNELS:
        ms = mcpu.mcpu_timing_read(k, nb)
        mcpu.mcpu_timing_start(k, 0)
        if len(ms):
            breakdown[k] = round(float(np.mean(ms)) * 1e3, 2)
    if step.device_errors():
        raise SystemExit("device error during timing")

    idx = step.topk_idx.cpu().numpy()
    kb = kernel_bytes(wl, idx)
    attn_us = float(np.mean(attn_ms)) * 1e3
    achieved = kb["attn_split"] / (attn_us * 1e-6) / 1e9
    traffic = traffic_from_profile(os.path.join(ROOT, "paper_2608_22167_amd", "csrc", "attention.hip"),
                                   args.workload)
    roofline = {"kernel": "attn_split", "bound": "hbm", "achieved": round(achieved, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": traffic, "avg_us": round(attn_us, 2),
                "algorithmic_bytes": kb["attn_split"]}
    per_kernel_gbs = {k: round(kb[k] / (breakdown[k] * 1e-6) / 1e9, 1) for k in kb if k in breakdown}

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
        cpu = cpu_baseline(wl)

    s = wl.shape
    value = wl.n_tokens / (ms_step * 1e-3)
    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": K,
        "warmup": args.warmup, "ms_per_step": round(ms_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": s.dtype, "data": "synthetic",
        "config": {"workload": wl.name, "batch": wl.batch, "tokens": wl.n_tokens,
                   "context": f"{int(wl.seq_lens.min())}..{int(wl.seq_lens.max())} "
                              f"(mean {float(wl.seq_lens.mean()):.0f})",
                   "layer": f"hidden {s.hidden}, {s.n_q_heads}/{s.n_kv_heads} heads, d {s.head_dim}, "
                            f"{s.n_experts} experts top-{s.top_k}, ffn {s.ffn_dim}",
                   "attention": "sliding window %d + sinks" % s.window if s.window else "full + sinks",
                   "parallelism": "single GPU"},
        "roofline": roofline,
        "cpu_baseline": cpu,
        "kernels_us": breakdown,
        "kernels_gbs": per_kernel_gbs,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
