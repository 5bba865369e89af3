"""Benchmark of the tiered-memory decode path on one MI355X.

Default workload: the Llama-3-8B-shaped decode weight chain at batch 1
(32 layers x [fused qkv 6144x4096, o 4096x4096, fused gate_up 28672x4096,
down 4096x14336] + lm_head 128256x4096, bf16 ~N(0, 0.02), random init).  Every
weight tensor is placed on its own by modulo page placement at the modulus
derived from the host/HBM read-bandwidth ratio measured at start-up; a second,
all-HBM copy of the same weights is the HBM-only baseline.  One step = the 129
GEMVs of one decode token, launched back to back on one stream.

Prints ONE JSON line (rank 0, N = 1).  Only one GPU is used: --gpus above 1
exits with a message.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = ("effective GB/s (HBM+host) and decode-step ms vs HBM-only, "
          "% combined roofline")
HBM_PEAK_GBPS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--layers", type=int, default=32)
    p.add_argument("--modulus", type=int, default=0,
                   help="override the modulus derived from the measured alpha")
    p.add_argument("--host-workers", type=int, default=0)
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=15.0)
    p.add_argument("--graph", action="store_true",
                   help="replay each step as a captured HIP graph")
    p.add_argument("--pmc-ref", action="store_true",
                   help="also run a plain 1 GiB device copy (counter scale reference)")
    return p.parse_args()


# ---------------------------------------------------------------- workload
class Chain:
    """The placed weight chain plus its activations."""

    def __init__(self, bd, ctx, torch, layers, M):
        import synth
        self.bd, self.ctx, self.torch = bd, ctx, torch
        per_layer, head = synth.chain_shapes(synth.LLAMA8B)
        self.ops = []            # (boost handle, hbm-only handle, N, K, x, y)
        self.alg_bytes = 0
        self.host_pages = 0
        self.pages = 0
        rng = np.random.default_rng(7)
        xs = {}
        for K in sorted({k for _, _, _, k in per_layer} | {head[3]}):
            xs[K] = torch.from_numpy(synth.normal_bf16(rng, (1, K), 1.0).view(np.int16)).cuda()
        specs = [(l, kind, n, k) for l in range(layers) for _, kind, n, k in per_layer]
        specs.append((0, head[1], head[2], head[3]))
        for (l, kind, N, K) in specs:
            w = synth.chain_weight_torch(l, kind, N, K, "cuda").view(torch.int16)
            nbytes = N * K * 2
            t = bd.boost_place_weights(ctx, w, nbytes, M)
            n = (nbytes + bd.PAGE_BYTES - 1) // bd.PAGE_BYTES
            h = bd.boost_place_weights_map(ctx, w, nbytes, np.zeros(n, np.uint8))
            tiers = bd.boost_tensor_tiers(t)
            self.host_pages += int(tiers.sum())
            self.pages += n
            del w
            y = torch.empty((1, N), dtype=torch.float32, device="cuda")
            self.ops.append((t, h, N, K, xs[K], y))
            self.alg_bytes += nbytes + K * 2 + N * 4
        torch.cuda.synchronize()
        torch.cuda.empty_cache()

    def run(self, which, stream, events=None):
        bd = self.bd
        for i, (t, h, N, K, x, y) in enumerate(self.ops):
            if events is not None:
                events[i][0].record()
            bd.boost_decode_gemv(self.ctx, t if which == "boost" else h, N, K, x, 1,
                                 y, bd.DTYPE_F32, stream)
            if events is not None:
                events[i][1].record()

    def free(self):
        for t, h, *_ in self.ops:
            self.bd.boost_tensor_free(t)
            self.bd.boost_tensor_free(h)


def time_steps(torch, fn, steps):
    """Per-step milliseconds from events on the launching stream."""
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    for a, b in ev:
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    return np.array([a.elapsed_time(b) for a, b in ev])


# ----------------------------------------------------------- CPU baseline
def cpu_baseline(seconds: float):
    """The oracle GEMV (fp32 accumulation over bf16 weights decoded on the
    fly) over layer 0 of the same chain, repeated until about `seconds` of
    CPU work; reported as effective GB/s of algorithmic bytes."""
    import synth
    from oracle import gemv as og
    per_layer, _ = synth.chain_shapes(synth.LLAMA8B)
    rng = np.random.default_rng(7)
    tensors = [(synth.chain_weight(0, kind, N, K), synth.normal_bf16(rng, (1, K), 1.0))
               for _, kind, N, K in per_layer]
    done_bytes, spent, passes = 0, 0.0, 0
    while spent < seconds:
        for w, x in tensors:
            t0 = time.perf_counter()
            og.gemv_f32(w, x)
            spent += time.perf_counter() - t0
            done_bytes += w.nbytes + x.nbytes + w.shape[0] * 4
        passes += 1
    try:
        from threadpoolctl import threadpool_info
        cores = max((i.get("num_threads") or 1) for i in threadpool_info()) or 1
    except Exception:
        cores = os.cpu_count() or 1
    return {"value": round(done_bytes / spent / 1e9, 3), "unit": "GB/s",
            "cores": int(cores), "kind": "oracle",
            "sample": f"oracle fp32 GEMV over layer 0 of the same chain (4 tensors, "
                      f"{passes} passes, {done_bytes / 1e9:.2f} GB), "
                      f"{spent:.1f} s of compute"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); "
              "this build has no multi-GPU path.", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2609_13592_amd import binding as bd
    torch.cuda.init()
    ctx = bd.boost_init(0)
    log("step: calibrate")
    bw_hbm, bw_host, alpha = bd.boost_calibrate(ctx, 4 << 30, 1 << 30, 5)
    M = args.modulus or bd.boost_modulus_from_alpha(alpha)
    log(f"  hbm {bw_hbm:.1f} GB/s host {bw_host:.2f} GB/s alpha {alpha:.5f} M {M}")
    bd.boost_gemv_set_schedule(ctx, bd.SCHED_CAP, args.host_workers)

    log("step: place weights")
    chain = Chain(bd, ctx, torch, args.layers, M)
    log(f"  {len(chain.ops)} tensors, {chain.pages} pages, {chain.host_pages} on host")
    stream = torch.cuda.current_stream()
    sp = stream.cuda_stream

    graphs = {}
    if args.graph:
        for which in ("boost", "hbm"):
            chain.run(which, sp)
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                chain.run(which, torch.cuda.current_stream().cuda_stream)
            graphs[which] = g

    def step(which):
        if args.graph:
            graphs[which].replay()
        else:
            chain.run(which, sp)

    log("step: warmup")
    for _ in range(args.warmup):
        step("boost")
        step("hbm")
    torch.cuda.synchronize()

    log("step: timed")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    boost_ms, hbm_ms = [], []
    for i in range(args.steps):
        # interleaved A/B so both see the same clocks and thermal state
        boost_ms.append(time_steps(torch, lambda: step("boost"), 1)[0])
        hbm_ms.append(time_steps(torch, lambda: step("hbm"), 1)[0])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    boost_ms, hbm_ms = np.array(boost_ms), np.array(hbm_ms)
    ms = float(np.median(boost_ms))
    ms_hbm = float(np.median(hbm_ms))

    # per-launch durations of the GEMV kernel (roofline of the dominant kernel)
    log("step: per-launch timing")
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in chain.ops]
    kern_ms = []
    for _ in range(max(3, min(args.steps, 10))):
        chain.run("boost", sp, ev)
        torch.cuda.synchronize()
        kern_ms.append(sum(a.elapsed_time(b) for a, b in ev))
    launches = len(chain.ops)
    avg_launch_ms = float(np.median(kern_ms)) / launches
    bytes_per_launch = chain.alg_bytes / launches
    achieved = bytes_per_launch / (avg_launch_ms * 1e-3) / 1e9

    if args.pmc_ref:
        a = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        del a, b

    eff = chain.alg_bytes / (ms * 1e-3) / 1e9
    eff_hbm = chain.alg_bytes / (ms_hbm * 1e-3) / 1e9
    host_share = chain.host_pages / chain.pages
    cpu = None
    if not args.no_cpu_baseline:
        log("step: cpu baseline (oracle)")
        cpu = cpu_baseline(args.cpu_seconds)
    chain.free()
    bd.boost_shutdown(ctx)

    out = {
        "metric": METRIC,
        "value": round(eff, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded random-init weights and activations)",
        "config": {
            "workload": "Llama-3-8B-shaped decode weight chain, batch 1, "
                        "modulo placement at the measured bandwidth ratio",
            "layers": args.layers, "d": 4096, "ffn": 14336, "q_heads": 32,
            "kv_heads": 8, "head_dim": 128, "vocab": 128256, "batch": 1,
            "gemvs_per_step": launches, "modulus": M,
            "host_pages": chain.host_pages, "pages": chain.pages,
            "host_byte_share": round(host_share, 6),
            "schedule": "cap", "graph": bool(args.graph),
        },
        "tokens_per_s": round(1000.0 / ms, 2),
        "calibration": {"hbm_gbps": round(bw_hbm, 1), "host_gbps": round(bw_host, 2),
                        "alpha": round(alpha, 6)},
        "pct_combined_roofline": round(100 * eff / (bw_hbm + bw_host), 2),
        "hbm_only": {"ms_per_step": round(ms_hbm, 4), "value": round(eff_hbm, 2),
                     "pct_of_hbm_roofline": round(100 * eff_hbm / bw_hbm, 2)},
        "speedup_vs_hbm_only": round(ms_hbm / ms, 4),
        "step_ms_iqr": [round(float(np.percentile(boost_ms, 25)), 4),
                        round(float(np.percentile(boost_ms, 75)), 4)],
        "roofline": {"bound": "hbm", "kernel": "gemv_kernel<1,2,4>",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": None,
                     "avg_launch_us": round(avg_launch_ms * 1e3, 3),
                     "bytes_per_launch": int(bytes_per_launch)},
        "cpu_baseline": cpu,
        "timed_wall_s": round(wall, 3),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
