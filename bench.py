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
    p.add_argument("--ab-pairs", type=int, default=200,
                   help="interleaved tiered / all-HBM step pairs after the timed steps")
    p.add_argument("--graph", action="store_true",
                   help="replay each step as a captured HIP graph")
    p.add_argument("--pmc-ref", action="store_true",
                   help="also run a plain 1 GiB device copy (counter scale reference)")
    p.add_argument("--cap-quick", action="store_true",
                   help="cap_probe: only a handful of points, for counter runs")
    p.add_argument("--summarize-pmc", default="",
                   help="summarise the rocprofv3 counter CSVs under this directory "
                        "(per kernel and grid) as JSON on stdout, then exit")
    p.add_argument("--part", default="chain", choices=("chain", "single", "attention"),
                   help="tier_counters: which part runs its one tiered call")
    p.add_argument("--summarize-trace", default="",
                   help="summarise a rocprofv3 --kernel-trace --stats directory as "
                        "markdown tables (per kernel; per kernel and grid), then exit")
    p.add_argument("--traffic-profile", default="",
                   help="FETCH_DIR,WRITE_DIR: rocprofv3 FETCH_SIZE / WRITE_SIZE runs of the "
                        "default bench with --pmc-ref; write profiles/traffic_counters.json "
                        "and print its table, then exit")
    p.add_argument("--tier-profile", default="",
                   help="directory holding <part>/ (rocprofv3 counter CSVs of a "
                        "tier_counters run) and <part>.json (its output) for the parts "
                        "chain, single, attention: write profiles/tier_counters.json "
                        "and print its table, then exit")
    p.add_argument("--workload", default="chain8b",
                   choices=("chain8b", "llama70b", "throughput8b", "host_share_sweep",
                            "cap_probe", "batch_sweep", "placements", "dsr_churn",
                            "tier_counters", "gemm_shapes"),
                   help="chain8b: decode weight chain (default); llama70b: full 70B-"
                        "shaped decode step under a 120 GB HBM weight budget; "
                        "throughput8b: 8B-shaped decode at up to 256 requests under a "
                        "40 GB HBM KV budget; host_share_sweep, batch_sweep, "
                        "placements, dsr_churn, cap_probe: the follow-up experiments "
                        "(modulus sweep, batch sensitivity, contrast placements, "
                        "allocator under Poisson arrivals, concurrent streaming "
                        "probe); tier_counters: one tiered call of --part for a "
                        "counter run; gemm_shapes: the 8B layer matrices all-HBM at "
                        "--batches")
    p.add_argument("--batches", default="16,32,64,128,256",
                   help="gemm_shapes: batch sizes (comma-separated, 1..256)")
    p.add_argument("--host-pin-gib", type=float, default=56.0,
                   help="throughput8b: pinned host memory the capacity-limited literal "
                        "variant may give its KV overflow (a process pins at most ~64 GiB "
                        "on the measured box)")
    p.add_argument("--no-literal", action="store_true",
                   help="throughput8b: skip the 256-request variant (~115 GB of "
                        "pinned host KV)")
    args = p.parse_args()
    if args.cpu_seconds <= 0:  # no time for the oracle: no CPU leg
        args.no_cpu_baseline = True
    return args


# ---------------------------------------------------------------- workload
class Chain:
    """The placed weight chain plus its activations."""

    def __init__(self, bd, ctx, torch, layers, M):
        import synth
        self.bd, self.ctx, self.torch = bd, ctx, torch
        per_layer, head = synth.chain_shapes(synth.LLAMA8B)
        self.ops = []            # (boost handle, hbm-only handle, N, K, x, y)
        self.views = {}          # op index -> staged view (prefetch baseline)
        self.alg_bytes = 0
        self.host_pages = 0
        self.pages = 0
        self.hbm_weight_bytes = 0
        self.host_weight_bytes = 0
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
            a, b = tensor_tier_bytes(bd, t, nbytes)
            self.hbm_weight_bytes += a
            self.host_weight_bytes += b
            del w
            y = torch.empty((1, N), dtype=torch.float32, device="cuda")
            self.ops.append((t, h, N, K, xs[K], y))
            self.alg_bytes += nbytes + K * 2 + N * 4
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        # prefetch baseline: a ring of two staging areas, one staged tensor
        # copied ahead of its use on a second stream
        self.staged = [i for i, op in enumerate(self.ops)
                       if bd.boost_tensor_tiers(op[0]).sum()]
        most = max([int(bd.boost_tensor_tiers(self.ops[i][0]).sum()) for i in self.staged],
                   default=0)
        self.ring = [torch.empty(max(1, most) * bd.PAGE_BYTES, dtype=torch.uint8,
                                 device="cuda") for _ in range(2)]
        for k, i in enumerate(self.staged):
            buf = self.ring[k % 2]
            self.views[i] = bd.boost_staged_view(ctx, self.ops[i][0], buf, buf.numel())
        self.copy_stream = torch.cuda.Stream()
        self.ev_ready = {i: torch.cuda.Event() for i in self.staged}
        self.ev_free = [torch.cuda.Event(), torch.cuda.Event()]
        self.staged_bytes = most * len(self.staged) and sum(
            int(bd.boost_tensor_tiers(self.ops[i][0]).sum()) for i in self.staged) * bd.PAGE_BYTES

    def _issue_prefetch(self, k):
        i = self.staged[k]
        cs = self.copy_stream
        cs.wait_event(self.ev_free[k % 2])
        self.bd.boost_prefetch(self.ctx, self.views[i], cs.cuda_stream)
        self.ev_ready[i].record(cs)

    def run_prefetch(self, stream_obj):
        """One step of the prefetch baseline: staged tensors are read from
        HBM staging after their host pages were copied in (one ahead)."""
        bd, torch = self.bd, self.torch
        sp = stream_obj.cuda_stream
        for k in range(min(2, len(self.staged))):
            self._issue_prefetch(k)
        pos = {i: k for k, i in enumerate(self.staged)}
        for i, (t, h, N, K, x, y) in enumerate(self.ops):
            if i in pos:
                k = pos[i]
                stream_obj.wait_event(self.ev_ready[i])
                bd.boost_decode_gemv(self.ctx, self.views[i], N, K, x, 1, y,
                                     bd.DTYPE_F32, sp)
                self.ev_free[k % 2].record(stream_obj)
                if k + 2 < len(self.staged):
                    self._issue_prefetch(k + 2)
            else:
                bd.boost_decode_gemv(self.ctx, t, N, K, x, 1, y, bd.DTYPE_F32, sp)
        stream_obj.wait_stream(self.copy_stream)

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
        for v in self.views.values():
            self.bd.boost_tensor_free(v)
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


def ab_pairs(torch, fn_a, fn_b, pairs):
    """Interleaved A/B: `pairs` pairs of single steps, the order alternating
    from pair to pair, each step timed by events on the launching stream.
    Returns the geometric mean of b/a over the pairs (a's speedup over b)
    with a 95 % interval (t interval on the log ratios) and the medians."""
    ta, tb = [], []
    for i in range(pairs):
        first, second = (fn_a, fn_b) if i % 2 == 0 else (fn_b, fn_a)
        t1 = time_steps(torch, first, 1)[0]
        t2 = time_steps(torch, second, 1)[0]
        ta.append(t1 if i % 2 == 0 else t2)
        tb.append(t2 if i % 2 == 0 else t1)
    ta, tb = np.array(ta), np.array(tb)
    lr = np.log(tb / ta)
    half = 1.96 * float(np.std(lr, ddof=1)) / np.sqrt(len(lr))
    m = float(np.mean(lr))
    return {"pairs": int(pairs), "speedup_geomean": round(float(np.exp(m)), 5),
            "ci95": [round(float(np.exp(m - half)), 5), round(float(np.exp(m + half)), 5)],
            "a_ms_median": round(float(np.median(ta)), 4),
            "b_ms_median": round(float(np.median(tb)), 4),
            "speedup_of_medians": round(float(np.median(tb) / np.median(ta)), 5)}


def tier_counter_entry(part: str):
    """The committed counter summary of one tiered call of `part` (chain step,
    single layer, config-3 attention) from profiles/tier_counters.json, or
    None when the kernel source changed since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "tier_counters.json")
    try:
        ent = json.load(open(path))[part]
        src = open(os.path.join(ROOT, "paper_2609_13592_amd", "csrc", ent["source"]),
                   "rb").read()
    except (OSError, KeyError, ValueError):
        return None
    if hashlib.sha256(src).hexdigest() != ent["source_sha256"]:
        return None
    return ent


def per_tier(part, ms, placement_hbm, placement_host, modulus=None):
    """Per-tier achieved GB/s of one call taking `ms`.  Bytes: the committed
    counters (TCC_EA0_RDREQ_DRAM_32B / TCC_EA0_RDREQ_IO_32B) when they were
    taken on the current kernel source at the same placement; at another
    modulus the placement's bytes scaled by the counters' ratio to the
    placement; without current counters the placement's bytes."""
    ent = tier_counter_entry(part)
    if ent and (modulus is None or ent["modulus"] == modulus):
        hbm, host = ent["hbm_bytes"], ent["host_bytes"]
        src = f"counters (modulus {ent['modulus']})"
    elif ent:
        hbm = placement_hbm * ent["hbm_over_placement"]
        host = placement_host * (ent["host_over_placement"] or 1.0)
        src = f"placement x counter ratio taken at modulus {ent['modulus']}"
    else:
        hbm, host, src = placement_hbm, placement_host, "placement"
    return {"hbm_bytes": int(hbm), "host_bytes": int(host),
            "hbm_gbps": round(hbm / (ms * 1e-3) / 1e9, 1),
            "host_gbps": round(host / (ms * 1e-3) / 1e9, 3), "bytes_from": src}


# ------------------------------------------------------------ single layer
def single_layer_bench(bd, ctx, torch, bw_hbm, bw_host, reps=200):
    """One bf16 layer W[4096 x 4096] (16 pages) with page 15 on host (M = 16),
    batch 1: tiered vs all-HBM vs prefetch-then-GEMV, each rotating over 16
    placed copies (512 MiB) so the last-level cache does not serve the HBM
    pages."""
    import synth
    w, x = synth.single_layer_inputs()
    N = K = 4096
    nbytes = w.nbytes
    copies = 16
    tiered = [bd.boost_place_weights(ctx, w, nbytes, 16) for _ in range(copies)]
    hbm = [bd.boost_place_weights_map(ctx, w, nbytes, np.zeros(16, np.uint8))
           for _ in range(copies)]
    stage = torch.empty(bd.PAGE_BYTES, dtype=torch.uint8, device="cuda")
    views = [bd.boost_staged_view(ctx, t, stage, stage.numel()) for t in tiered]
    xd = torch.from_numpy(x.view(np.int16)).cuda()
    y = torch.empty((1, N), dtype=torch.float32, device="cuda")
    sp = torch.cuda.current_stream().cuda_stream

    def run(handles, pre=False):
        for i in range(copies):
            if pre:
                bd.boost_prefetch(ctx, views[i], sp)
            bd.boost_decode_gemv(ctx, handles[i], N, K, xd, 1, y, bd.DTYPE_F32, sp)
    out = {}
    for name, fn in (("boost", lambda: run(tiered)), ("hbm", lambda: run(hbm)),
                     ("prefetch", lambda: run(views, True))):
        fn()
        torch.cuda.synchronize()
        us = float(np.median(time_steps(torch, fn, max(5, reps // copies)))) * 1e3 / copies
        out[name] = {"us": round(us, 2), "gbps": round(nbytes / (us * 1e-6) / 1e9, 1)}
    for t in views + tiered + hbm:
        bd.boost_tensor_free(t)
    bound_us = max(15 * bd.PAGE_BYTES / (bw_hbm * 1e9), bd.PAGE_BYTES / (bw_host * 1e9)) * 1e6
    out["placement_bound_us"] = round(bound_us, 2)
    out["pct_of_placement_bound"] = round(100 * bound_us / out["boost"]["us"], 2)
    out["per_tier"] = per_tier("single", out["boost"]["us"] * 1e-3, 15 * bd.PAGE_BYTES,
                               bd.PAGE_BYTES)
    out["host_pages"] = [15]
    return out


# --------------------------------------------------------------- attention
def attention_setup(bd, ctx, torch, M):
    """Config-3 inputs: batch 64, 32/8 heads, head_dim 128, context lengths
    U[512, 4096] (seed 0), K/V ~N(0, 1) bf16, blocks from the wave-aware pool
    (linear placement at modulus M) and from an all-HBM pool."""
    import synth
    B, Hq, H, D = 64, 32, 8, 128
    lengths = synth.context_lengths(0, B, 512, 4096)
    need = [(int(L) + 15) // 16 for L in lengths]
    mb = max(need)
    g = torch.Generator(device="cuda")
    g.manual_seed(1)
    total = int(lengths.sum())
    k = torch.randn((total, H, D), generator=g, device="cuda").to(torch.bfloat16)
    v = torch.randn((total, H, D), generator=g, device="cuda").to(torch.bfloat16)
    q = torch.randn((B, Hq, D), generator=g, device="cuda").to(torch.bfloat16)
    lens = torch.from_numpy(lengths.astype(np.int32)).cuda()
    sp = torch.cuda.current_stream().cuda_stream
    pools = {}
    for name, mode, m in (("boost", bd.KV_LPP, M), ("hbm", bd.KV_ALL_HBM, 0)):
        pool = bd.boost_kv_pool_create(ctx, 1, H, D, sum(need), m, mode, q_heads=Hq,
                                       max_batch=B, max_blocks_per_seq=mb)
        tables = np.full((B, mb), -1, np.int32)
        slots = []
        for b in range(B):
            tables[b, :need[b]] = bd.boost_kv_alloc(pool, b, need[b])
            t = np.arange(int(lengths[b]))
            slots.append(tables[b, t // 16] * 16 + t % 16)
        sl = torch.from_numpy(np.concatenate(slots).astype(np.int32)).cuda()
        bd.boost_kv_write(ctx, pool, 0, sl, k, v, total, sp)
        st = bd.boost_kv_stats(pool)
        pools[name] = (pool, torch.from_numpy(tables).cuda(), st)
    del k, v
    out = torch.empty((B, Hq, D), dtype=torch.float32, device="cuda")

    def call(name):
        pool, td, _ = pools[name]
        bd.boost_paged_attn_decode(ctx, pool, 0, q, B, Hq, td, mb, lens, 0.0, out,
                                   bd.DTYPE_F32, sp)
    alg = total * H * D * 2 * 2 + B * Hq * D * 2 + B * Hq * D * 4
    st = pools["boost"][2]
    return {"call": call, "pools": pools, "alg": alg, "stats": st, "B": B, "H": H,
            "D": D, "lengths": lengths, "out": out}


def attention_bench(bd, ctx, torch, M, steps, warmup):
    """Paged-attention decode on the config-3 inputs (attention_setup): the
    wave-aware pool against the all-HBM pool, interleaved."""
    A = attention_setup(bd, ctx, torch, M)
    call, pools, alg, st = A["call"], A["pools"], A["alg"], A["stats"]
    H = A["H"]
    res = {}
    for _ in range(warmup):
        call("boost")
        call("hbm")
    ms = {"boost": [], "hbm": []}
    for _ in range(steps):
        for name in ("boost", "hbm"):
            a = torch.cuda.Event(enable_timing=True)
            b_ = torch.cuda.Event(enable_timing=True)
            a.record()
            call(name)
            b_.record()
            torch.cuda.synchronize()
            ms[name].append(a.elapsed_time(b_))
    for name in ("boost", "hbm"):
        t = float(np.median(ms[name]))
        res[name] = {"ms": round(t, 4), "gbps": round(alg / (t * 1e-3) / 1e9, 1)}
    res["host_share"] = round(st["used_host_head_blocks"] / (H * st["used_blocks"]), 5)
    res["shh_requests"] = int(st["shh_requests"])
    res["alg_bytes"] = int(alg)
    host_kv = int(st["used_host_head_blocks"]) * 16 * A["D"] * 2 * 2   # K and V
    res["per_tier"] = per_tier("attention", res["boost"]["ms"], alg - host_kv, host_kv, M)
    res["speedup_vs_hbm_only"] = round(res["hbm"]["ms"] / res["boost"]["ms"], 4)
    ach = alg / (res["boost"]["ms"] * 1e-3) / 1e9
    res["roofline"] = {"bound": "hbm", "kernel": "attn_partition + attn_merge",
                       "achieved": round(ach, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                       "frac": round(ach / HBM_PEAK_GBPS, 4),
                       "traffic": counter_traffic("attn_partition", "attn.hip")}
    for pool, _, _ in pools.values():
        bd.boost_kv_pool_destroy(pool)
    return res


# ------------------------------------------------------------ traffic data
def counter_traffic(kernel: str, source: str):
    """HBM bytes per launch from the committed FETCH_SIZE / WRITE_SIZE summary
    (profiles/traffic_counters.json), or None when the kernel source changed
    since the counters were taken."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "traffic_counters.json")
    try:
        data = json.load(open(path))[kernel]
        src = open(os.path.join(ROOT, "paper_2609_13592_amd", "csrc", source), "rb").read()
    except (OSError, KeyError, ValueError):
        return None
    if hashlib.sha256(src).hexdigest() != data["source_sha256"]:
        return None
    return int(data["traffic_bytes_per_launch"])


def summarize_pmc(directory: str):
    """Per-kernel sums of rocprofv3 counter CSVs (every `*counter_collection.csv`
    under `directory`): for each (kernel name, grid size) the number of
    dispatches and, per counter, the mean value per dispatch."""
    import csv
    import glob
    acc = {}
    for path in sorted(glob.glob(os.path.join(directory, "**", "*counter_collection.csv"),
                                 recursive=True)):
        with open(path, newline="") as fh:
            for row in csv.DictReader(fh):
                name = row.get("Kernel_Name", "?").replace("(anonymous namespace)::", "")
                name = name[5:] if name.startswith("void ") else name
                name = name.split("(")[0].strip()
                key = f"{name} grid={row.get('Grid_Size', '?')}"
                ent = acc.setdefault(key, {"dispatches": set(), "sums": {}})
                ent["dispatches"].add(row.get("Dispatch_Id"))
                c = row.get("Counter_Name", "?")
                ent["sums"][c] = ent["sums"].get(c, 0.0) + float(row.get("Counter_Value", 0) or 0)
    out = {}
    for key, ent in sorted(acc.items()):
        n = len(ent["dispatches"])
        out[key] = {"dispatches": n,
                    "per_dispatch": {c: round(v / n, 1) for c, v in sorted(ent["sums"].items())}}
    return out


def _short_kernel(name: str) -> str:
    name = name.replace("(anonymous namespace)::", "")
    name = name[5:] if name.startswith("void ") else name
    return name.split("(")[0].strip()


def summarize_trace(directory: str) -> str:
    """Markdown tables of a rocprofv3 kernel-trace run: per kernel (calls,
    average, minimum, maximum, total) and, for this library's kernels, per
    launch shape (grid size in threads: dispatches, median, mean)."""
    import csv
    import glob
    trace = [r for path in sorted(glob.glob(os.path.join(directory, "**", "*kernel_trace.csv"),
                                            recursive=True))
             for r in csv.DictReader(open(path, newline=""))]
    per, shape = {}, {}
    for r in trace:
        k = _short_kernel(r["Kernel_Name"])
        d = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        per.setdefault(k, []).append(d)
        if not (k.startswith("at::") or "rocclr" in k):
            g = int(r.get("Grid_Size_X") or r.get("Grid_Size") or 0)
            shape.setdefault((k, g), []).append(d)
    out = ["| kernel | calls | avg us | min us | max us | total ms |",
           "|---|---:|---:|---:|---:|---:|"]
    for k, v in sorted(per.items(), key=lambda kv: -sum(kv[1])):
        out.append(f"| `{k[:60]}` | {len(v)} | {np.mean(v):.2f} | {min(v):.2f} | "
                   f"{max(v):.2f} | {sum(v) / 1e3:.2f} |")
    out += ["", "| kernel | grid (threads) | dispatches | median us | mean us | total ms |",
            "|---|---:|---:|---:|---:|---:|"]
    for (k, g), v in sorted(shape.items(), key=lambda kv: -sum(kv[1])):
        out.append(f"| `{k[:60]}` | {g} | {len(v)} | {np.median(v):.2f} | {np.mean(v):.2f} | "
                   f"{sum(v) / 1e3:.2f} |")
    return "\n".join(out)


# launch shapes (grid in threads) of one tiered step of the 8B chain at batch 1
CHAIN_GRIDS = {"qkv": (393216, 32), "o": (262144, 32), "gate_up": (1835008, 32),
               "down": (530432, 32)}


def write_traffic_profile(dirs: str, out_dir: str = ""):
    """HBM traffic per launch from FETCH_SIZE and WRITE_SIZE runs of the default
    bench (with --pmc-ref), each scaled by what the counter reads for the
    plain 1 GiB device copy: the GEMV averaged over one tiered chain step
    (the 128 layer launches by grid, the head's tiered launch as the largest
    gemv grid not in the layers) and one config-3 attention call (partition
    and merge kernels).  Written to profiles/traffic_counters.json."""
    import hashlib
    fetch_dir, write_dir = dirs.split(",")
    f, w = summarize_pmc(fetch_dir), summarize_pmc(write_dir)

    def get(summ, name, grid, counter):
        for key, ent in summ.items():
            if key.startswith(name) and key.endswith(f"grid={grid}"):
                return ent["per_dispatch"].get(counter, 0.0), ent["dispatches"]
        return None, 0

    # scale references: FETCH_SIZE of the calibration's HBM stream with 2048
    # workgroups (4 GiB read per dispatch), WRITE_SIZE of the 1 GiB fill
    # that --pmc-ref adds
    def ref_fetch():
        for key, ent in f.items():
            if key.startswith("stream_read") and key.endswith("grid=524288"):
                return ent["per_dispatch"]["FETCH_SIZE"], 4 << 30
        raise SystemExit("no 4 GiB calibration stream in the FETCH_SIZE run")

    def ref_write():
        best = 0.0
        for key, ent in w.items():
            if "Fill" in key or "fill" in key:
                best = max(best, ent["per_dispatch"].get("WRITE_SIZE", 0.0))
        if best <= 0:
            raise SystemExit("no fill in the WRITE_SIZE run (run the bench with --pmc-ref)")
        return best, 1 << 30

    fk_ref, fb_ref = ref_fetch()
    wk_ref, wb_ref = ref_write()
    fscale = fb_ref / (fk_ref * 1024)
    wscale = wb_ref / (wk_ref * 1024)
    gemv_grids = sorted({int(k.split("grid=")[1]) for k in f if k.startswith("gemv_kernel")})
    layer_grids = {g for g, _ in CHAIN_GRIDS.values()}
    # the head's launches: every gemv grid that is neither a layer's nor the
    # single-layer leg's (tiered and all-HBM legs differ by the host workers)
    heads = [g for g in gemv_grids if g not in layer_grids and g != 249856]
    fsum = wsum = 0.0
    launches = 0
    rows = []
    for name, (grid, n) in CHAIN_GRIDS.items():
        fk, _ = get(f, "gemv_kernel", grid, "FETCH_SIZE")
        wk, _ = get(w, "gemv_kernel", grid, "WRITE_SIZE")
        fsum += n * fk * 1024 * fscale
        wsum += n * wk * 1024 * wscale
        launches += n
        rows.append(f"| gemv {name} | {grid} | {n} | {fk:.1f} | {wk:.1f} |")
    hf = hw = hn = 0.0
    for g in heads:
        fk, nd = get(f, "gemv_kernel", g, "FETCH_SIZE")
        wk, _ = get(w, "gemv_kernel", g, "WRITE_SIZE")
        hf, hw, hn = hf + fk * nd, hw + wk * nd, hn + nd
        rows.append(f"| gemv lm_head | {g} | 1 | {fk:.1f} | {wk:.1f} |")
    fsum += hf / hn * 1024 * fscale
    wsum += hw / hn * 1024 * wscale
    launches += 1
    attn_f = attn_w = 0.0
    for kname in ("attn_partition", "attn_merge"):
        for key, ent in f.items():
            if key.startswith(kname):
                attn_f += ent["per_dispatch"].get("FETCH_SIZE", 0.0) * 1024 * fscale
                rows.append(f"| {key} | | {ent['dispatches']} | "
                            f"{ent['per_dispatch'].get('FETCH_SIZE', 0.0):.1f} | |")
        for key, ent in w.items():
            if key.startswith(kname):
                attn_w += ent["per_dispatch"].get("WRITE_SIZE", 0.0) * 1024 * wscale

    def sha(src):
        return hashlib.sha256(open(os.path.join(ROOT, "paper_2609_13592_amd", "csrc", src),
                                   "rb").read()).hexdigest()
    prof = {"gemv": {"source_sha256": sha("gemv.hip"),
                     "traffic_bytes_per_launch": int((fsum + wsum) / launches),
                     "fetch_bytes_per_step": int(fsum), "write_bytes_per_step": int(wsum),
                     "launches_per_step": launches},
            "attn_partition": {"source_sha256": sha("attn.hip"),
                               "traffic_bytes_per_launch": int(attn_f + attn_w),
                               "fetch_bytes": int(attn_f), "write_bytes": int(attn_w)},
            "fetch_scale": round(fscale, 4), "write_scale": round(wscale, 4)}
    with open(os.path.join(out_dir or os.path.join(ROOT, "profiles"), "traffic_counters.json"),
              "w") as fh:
        json.dump(prof, fh, indent=1)
        fh.write("\n")
    print("| launch | grid | per step | FETCH KiB / dispatch | WRITE KiB / dispatch |")
    print("|---|---:|---:|---:|---:|")
    print("\n".join(rows))
    print(json.dumps(prof, indent=1))


TIER_KERNELS = {"chain": (("gemv_kernel", "split_fixup"), "gemv.hip"),
                "single": (("gemv_kernel", "split_fixup"), "gemv.hip"),
                "attention": (("attn_partition", "attn_merge"), "attn.hip")}


def write_tier_profile(directory: str, out_dir: str = ""):
    """Per-tier bytes of the tiered calls of a tier_counters run, summed over
    the part's kernels, against the placement's bytes; written to
    profiles/tier_counters.json with the kernel source's hash."""
    import hashlib
    prof = {}
    lines = ["| part | modulus | kernels | DRAM bytes (counter) | host bytes (counter) | "
             "HBM bytes (placement) | host bytes (placement) | DRAM / placement | "
             "host / placement |", "|---|---:|---|---:|---:|---:|---:|---:|---:|"]
    for part, (names, source) in TIER_KERNELS.items():
        try:
            meta = json.load(open(os.path.join(directory, part + ".json")))
        except OSError:
            continue
        summ = summarize_pmc(os.path.join(directory, part))
        dram = io = 0.0
        used = set()
        for key, ent in summ.items():
            if key.split(" grid=")[0].split("<")[0] in names:
                used.add(key.split(" grid=")[0].split("<")[0])
                pd = ent["per_dispatch"]
                dram += pd.get("TCC_EA0_RDREQ_DRAM_32B", 0.0) * 32 * ent["dispatches"]
                io += pd.get("TCC_EA0_RDREQ_IO_32B", 0.0) * 32 * ent["dispatches"]
        if part == "attention":
            host_p = meta["kv_host_bytes_upper"]
            hbm_p = meta["kv_bytes"] - host_p
        else:
            hbm_p, host_p = meta["weight_hbm_bytes"], meta["weight_host_bytes"]
        sha = hashlib.sha256(open(os.path.join(ROOT, "paper_2609_13592_amd", "csrc", source),
                                  "rb").read()).hexdigest()
        prof[part] = {"source": source, "source_sha256": sha, "modulus": meta["modulus"],
                      "hbm_bytes": int(round(dram)), "host_bytes": int(round(io)),
                      "placement_hbm_bytes": int(hbm_p), "placement_host_bytes": int(host_p),
                      "hbm_over_placement": round(dram / hbm_p, 5),
                      "host_over_placement": round(io / host_p, 5) if host_p else None}
        lines.append(f"| {part} | {meta['modulus']} | {', '.join(sorted(used))} | {dram:,.0f} | "
                     f"{io:,.0f} | {hbm_p:,} | {host_p:,} | {dram / hbm_p:.5f} | "
                     + (f"{io / host_p:.5f} |" if host_p else "- |"))
    with open(os.path.join(out_dir or os.path.join(ROOT, "profiles"), "tier_counters.json"),
              "w") as fh:
        json.dump(prof, fh, indent=1)
        fh.write("\n")
    print("\n".join(lines))


# ----------------------------------------------------------- CPU baseline
def host_topology():
    """Logical CPUs and the sockets x cores x threads of the host (lscpu)."""
    import subprocess
    topo = {"logical_cpus": os.cpu_count()}
    try:
        txt = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        keys = {"Socket(s)": "sockets", "Core(s) per socket": "cores_per_socket",
                "Thread(s) per core": "threads_per_core", "Model name": "model"}
        for line in txt.splitlines():
            k, _, v = line.partition(":")
            if k.strip() in keys:
                v = v.strip()
                topo[keys[k.strip()]] = int(v) if v.isdigit() else v
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        topo["affinity_cpus"] = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        pass
    return topo


def _oracle_gemv_rate(seconds: float):
    """The oracle GEMV (fp32 accumulation over bf16 weights decoded on the
    fly) over layer 0 of the chain, repeated until about `seconds` of CPU
    work: (GB/s of algorithmic bytes, passes, bytes, seconds)."""
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
    return done_bytes / spent / 1e9, passes, done_bytes, spent


def cpu_baseline(seconds: float):
    """The oracle on the host cores: the same chain's layer 0 (4 tensors) with
    every BLAS thread the process gets, then with one thread; reported as
    effective GB/s of algorithmic bytes."""
    from threadpoolctl import threadpool_info, threadpool_limits
    threads = max([(i.get("num_threads") or 1) for i in threadpool_info()] or [1])
    rate, passes, nbytes, spent = _oracle_gemv_rate(seconds)
    with threadpool_limits(limits=1):
        rate1, passes1, nbytes1, spent1 = _oracle_gemv_rate(seconds / 3)
    return {"value": round(rate, 3), "unit": "GB/s", "cores": int(threads), "kind": "oracle",
            "sample": f"oracle fp32 GEMV over layer 0 of the same chain (4 tensors, "
                      f"{passes} passes, {nbytes / 1e9:.2f} GB), {spent:.1f} s of compute "
                      f"on {threads} BLAS threads",
            "single_thread": {"value": round(rate1, 3), "unit": "GB/s", "cores": 1,
                              "sample": f"{passes1} passes, {nbytes1 / 1e9:.2f} GB, "
                                        f"{spent1:.1f} s"},
            "host": host_topology()}


# ------------------------------------------------------ 70B full decode step
# ------------------------------------------------- full decode-step workloads
def model_names(dims, synth):
    """(name, N, K, seed) of every matrix of a Llama-style model: embedding and
    lm_head, then the four fused matrices of every layer."""
    return [("embed", dims.vocab, dims.d, 9998), ("lm_head", dims.vocab, dims.d, 9999)] + \
        [(f"{n}.{l}", N, K, synth.chain_seed(l, i)) for l in range(dims.layers)
         for i, (n, N, K) in enumerate(dims.shapes())]


def place_model(bd, torch, names, tier_fn):
    """Generate every matrix on the GPU (seeded, bf16 ~N(0, 0.02), embedding
    ~N(0, 1)) and place it with tier_fn(w, bytes).  Returns (handles, host
    pages)."""
    mats, host = {}, 0
    for name, N, K, seed in names:
        g = torch.Generator(device="cuda")
        g.manual_seed(seed)
        w = torch.randn((N, K), generator=g, device="cuda")
        w.mul_(1.0 if name == "embed" else 0.02)
        w = w.to(torch.bfloat16).view(torch.int16)
        mats[name] = tier_fn(w, N * K * 2)
        host += int(bd.boost_tensor_tiers(mats[name]).sum())
        del w
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return mats, host


def all_hbm(bd, ctx):
    return lambda w, n: bd.boost_place_weights_map(
        ctx, w, n, np.zeros((n + bd.PAGE_BYTES - 1) // bd.PAGE_BYTES, np.uint8))


def model_norms(torch, dims, synth):
    rng = np.random.default_rng(4)
    norms = {}
    for k in ["norm_f"] + [f"norm{j}.{l}" for l in range(dims.layers) for j in (1, 2)]:
        v = synth.round_bf16((1 + 0.1 * rng.standard_normal(dims.d)).astype(np.float32))
        norms[k] = torch.from_numpy(v.view(np.int16)).cuda()
    return norms


def fill_kv(bd, ctx, torch, pool, dims, tables, lens):
    """K/V of the context before each request's new token, ~N(0, 1) bf16,
    generated on the GPU per (layer, request) so a request's content does not
    depend on the batch it is in."""
    sp = torch.cuda.current_stream().cuda_stream
    for i, L in enumerate(lens):
        n = int(L) - 1
        if n <= 0:
            continue
        t = np.arange(n)
        slots = torch.from_numpy((tables[i, t // 16] * 16 + t % 16).astype(np.int32)).cuda()
        for l in range(dims.layers):
            g = torch.Generator(device="cuda")
            g.manual_seed(1_000_003 * l + i)
            k = torch.randn((n, dims.hkv, dims.hd), generator=g, device="cuda").to(torch.bfloat16)
            v = torch.randn((n, dims.hkv, dims.hd), generator=g, device="cuda").to(torch.bfloat16)
            bd.boost_kv_write(ctx, pool, l, slots, k, v, n, sp)
    torch.cuda.synchronize()


class LayerPrefetch:
    """Prefetch-to-HBM baseline for a full decode step: the host pages of
    every layer's matrices are copied into one of two HBM staging slots on a
    copy stream, one layer ahead, and the layer's GEMVs read staged views
    (all HBM).  lm_head's host pages have a staging area of their own, copied
    after the last layer's; the embedding stays tiered (a step reads B rows of
    it)."""

    def __init__(self, bd, ctx, torch, dims, mats):
        self.bd, self.ctx, self.torch, self.dims = bd, ctx, torch, dims
        kinds = [k for k, _, _ in dims.shapes()]
        host = lambda name: int(bd.boost_tensor_tiers(mats[name]).sum())
        per_layer = max(sum(host(f"{k}.{l}") for k in kinds) for l in range(dims.layers))
        self.slots = [torch.empty(max(1, per_layer) * bd.PAGE_BYTES, dtype=torch.uint8,
                                  device="cuda") for _ in range(2)]
        self.head = torch.empty(max(1, host("lm_head")) * bd.PAGE_BYTES, dtype=torch.uint8,
                                device="cuda")
        self.views = {}             # name -> staged view
        self.layer_views = []       # per layer: views to copy
        for l in range(dims.layers):
            off, vs = 0, []
            buf = self.slots[l % 2]
            for k in kinds:
                name = f"{k}.{l}"
                n = host(name) * bd.PAGE_BYTES
                if n == 0:
                    continue
                v = bd.boost_staged_view(ctx, mats[name], buf[off:off + n], n)
                self.views[name] = v
                vs.append(v)
                off += n
            self.layer_views.append(vs)
        self.head_views = []
        if host("lm_head"):
            v = bd.boost_staged_view(ctx, mats["lm_head"], self.head, self.head.numel())
            self.views["lm_head"] = v
            self.head_views.append(v)
        self.mats = dict(mats)
        self.mats.update(self.views)
        self.staged_bytes = sum(host(n) for n in self.views) * bd.PAGE_BYTES
        self.copy = torch.cuda.Stream()
        self.ready = [torch.cuda.Event() for _ in range(dims.layers + 1)]
        self.free = [torch.cuda.Event(), torch.cuda.Event()]

    def _issue(self, l):
        cs = self.copy
        if l < self.dims.layers:
            cs.wait_event(self.free[l % 2])
            for v in self.layer_views[l]:
                self.bd.boost_prefetch(self.ctx, v, cs.cuda_stream)
        else:
            for v in self.head_views:
                self.bd.boost_prefetch(self.ctx, v, cs.cuda_stream)
        self.ready[l].record(cs)

    def begin(self, stream_obj):
        self.main = stream_obj
        for l in range(min(2, self.dims.layers)):
            self._issue(l)
        return self

    def before_layer(self, l):
        self.main.wait_event(self.ready[l])

    def after_layer(self, l):
        self.free[l % 2].record(self.main)
        nxt = l + 2
        if nxt < self.dims.layers:
            self._issue(nxt)
        elif nxt == self.dims.layers:
            self._issue(self.dims.layers)       # lm_head

    def before_head(self):
        if self.dims.layers < 2:
            self._issue(self.dims.layers)
        self.main.wait_event(self.ready[self.dims.layers])

    def close(self):
        self.main.wait_stream(self.copy)
        for v in self.views.values():
            self.bd.boost_tensor_free(v)


def llama70b(args, bd, ctx, torch, bw_hbm, bw_host, alpha):
    """Llama-3-70B-shaped full decode step (80 layers, d 8192, FFN 28672,
    GQA 64/8, head_dim 128, vocab 128256, bf16 ~N(0, 0.02) random init),
    batch 8, context 2048, weights placed by modulo placement at the modulus
    that fits a 120e9-byte HBM weight budget; KV in HBM.  Timed against the
    same step with every weight in HBM (uncapped)."""
    import synth
    from paper_2609_13592_amd.step import DecodeModel, Dims
    dims = Dims(layers=args.layers, d=8192, hq=64, hkv=8, hd=128, ffn=28672, vocab=128256)
    B, L = 8, 2048
    M_alpha = bd.boost_modulus_from_alpha(alpha)
    sizes = [N * K * 2 for _, N, K in dims.shapes()] * dims.layers + \
        [dims.vocab * dims.d * 2] * 2
    M = args.modulus or bd.boost_modulus_from_budget(sizes, 120 * 10 ** 9, M_alpha)
    log(f"  M_alpha {M_alpha} budget modulus {M}")
    names = model_names(dims, synth)
    norms = model_norms(torch, dims, synth)
    need = L // 16
    pool = bd.boost_kv_pool_create(ctx, dims.layers, dims.hkv, dims.hd, B * need, 0,
                                   bd.KV_ALL_HBM, q_heads=dims.hq, max_batch=B,
                                   max_blocks_per_seq=need)
    tables = np.zeros((B, need), np.int32)
    for b in range(B):
        tables[b] = bd.boost_kv_alloc(pool, b, need)
    fill_kv(bd, ctx, torch, pool, dims, tables, np.full(B, L))
    sp = torch.cuda.current_stream().cuda_stream
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()
    tokens = dev(synth.context_lengths(5, B, 0, dims.vocab - 1))
    lens = dev(np.full(B, L))
    pos = dev(np.full(B, L - 1))
    td = dev(tables)

    def run(mats, steps, warmup, pre=None):
        model = DecodeModel(ctx, dims, B, need, pool, mats if pre is None else pre.mats, norms)
        main = torch.cuda.current_stream()

        def one():
            if pre is None:
                model.step(tokens, pos, lens, td, sp)
            else:
                model.step(tokens, pos, lens, td, sp, hooks=pre.begin(main))
                main.wait_stream(pre.copy)
        for _ in range(warmup):
            one()
        torch.cuda.synchronize()
        ms = time_steps(torch, one, steps)
        return float(np.median(ms)), model.ids.cpu().numpy().tolist()

    log("step: place weights (tiered)")
    mats, host_pages = place_model(bd, torch, names,
                                   lambda w, n: bd.boost_place_weights(ctx, w, n, M))
    log(f"  host pages {host_pages} ({host_pages * 2 / 1024:.2f} GiB)")
    log("step: timed (tiered)")
    ms_boost, ids_boost = run(mats, args.steps, args.warmup)
    log("step: timed (prefetch to HBM)")
    pre = LayerPrefetch(bd, ctx, torch, dims, mats)
    ms_pre, ids_pre = run(mats, args.steps, args.warmup, pre)
    pre.close()
    staged_bytes = pre.staged_bytes
    del pre
    for t_ in mats.values():
        bd.boost_tensor_free(t_)
    log("step: place weights (all HBM)")
    mats, _ = place_model(bd, torch, names, all_hbm(bd, ctx))
    log("step: timed (HBM-only)")
    ms_hbm, ids_hbm = run(mats, max(args.steps, 10), args.warmup)
    model = DecodeModel(ctx, dims, B, need, pool, mats, norms)
    alg = model.bytes_per_step(np.full(B, L))
    for t_ in mats.values():
        bd.boost_tensor_free(t_)
    bd.boost_kv_pool_destroy(pool)
    host_bytes = host_pages * bd.PAGE_BYTES
    hbm_bytes = alg - host_bytes
    bound_ms = max(hbm_bytes / (bw_hbm * 1e9), host_bytes / (bw_host * 1e9)) * 1e3
    return {
        "metric": METRIC, "value": round(alg / (ms_boost * 1e-3) / 1e9, 2), "unit": "GB/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_boost, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded random-init weights, K/V and tokens)",
        "config": {"workload": "Llama-3-70B-shaped full decode step, batch 8, context 2048, "
                               "120 GB HBM weight budget (overflow pages on host by modulo "
                               "placement), KV in HBM",
                   "layers": dims.layers, "d": 8192, "ffn": 28672, "q_heads": 64,
                   "kv_heads": 8, "head_dim": 128, "vocab": 128256, "batch": B,
                   "context": L, "modulus": M, "modulus_from_alpha": M_alpha,
                   "host_weight_bytes": host_bytes},
        "tokens_per_s": round(B * 1000.0 / ms_boost, 3),
        "calibration": {"hbm_gbps": round(bw_hbm, 1), "host_gbps": round(bw_host, 2),
                        "alpha": round(alpha, 6)},
        "placement_bound_ms": round(bound_ms, 3),
        "pct_of_placement_bound": round(100 * bound_ms / ms_boost, 2),
        "hbm_only": {"ms_per_step": round(ms_hbm, 3),
                     "tokens_per_s": round(B * 1000.0 / ms_hbm, 2),
                     "value": round(alg / (ms_hbm * 1e-3) / 1e9, 2)},
        "prefetch": {"ms_per_step": round(ms_pre, 3),
                     "tokens_per_s": round(B * 1000.0 / ms_pre, 3),
                     "staged_bytes_per_step": int(staged_bytes),
                     "argmax_equal": ids_pre == ids_boost},
        "argmax_equal": ids_boost == ids_hbm,
        "bytes_per_step": int(alg),
    }


def throughput8b(args, bd, ctx, torch, bw_hbm, bw_host, alpha):
    """High-throughput Llama-3-8B-shaped decode: up to 256 requests with
    contexts uniform in [1024, 8192] (seed 0), an HBM KV budget of 40e9 bytes.

      literal -- all 256 requests; the pool keeps the budget's share of every
                 K/V tensor in HBM and the overflow on host (BOOST_KV_BUDGET);
      paper   -- the largest batch prefix whose pool, split by LPP at the
                 modulus from the measured ratio, keeps its HBM part within the
                 budget (host share ~ alpha / (1 + alpha));
      hbm     -- HBM-only: the largest prefix whose whole pool fits the budget.

    Weights: modulo placement at the measured ratio for literal/paper, all
    HBM for the baseline.  Each variant times the full decode step."""
    import synth
    from paper_2609_13592_amd.step import DecodeModel, Dims
    dims = Dims(layers=args.layers, d=4096, hq=32, hkv=8, hd=128, ffn=14336, vocab=128256)
    B_max, budget = 256, 40 * 10 ** 9
    lens_all = synth.context_lengths(0, B_max, 1024, 8192)
    M = args.modulus or bd.boost_modulus_from_alpha(alpha)
    mb = 8192 // 16
    bpp = bd.PAGE_BYTES // (16 * dims.hd * 2)
    blocks = np.cumsum([(int(L) + 15) // 16 for L in lens_all])

    def pages(b):          # pages of one K (or V) tensor of a pool for b requests
        nb = -(-int(blocks[b - 1]) // bpp) * bpp
        return dims.hkv * nb // bpp

    per = 2 * dims.layers * bd.PAGE_BYTES
    b_hbm = max(b for b in range(1, B_max + 1) if pages(b) * per <= budget)
    b_paper = max(b for b in range(1, B_max + 1) if (pages(b) - pages(b) // M) * per <= budget)
    # literal reading under the pinned-memory cap: the largest prefix whose
    # KV beyond the HBM budget fits in --host-pin-gib of pinned host memory
    # (the budget pool keeps the budget's share of every K/V tensor in HBM,
    # rounded down to whole pages, and the rest on host)
    cap = int(args.host_pin_gib * (1 << 30))
    b_cap = max(b for b in range(1, B_max + 1) if pages(b) * per - budget <= cap)
    log(f"  batches: hbm-only {b_hbm}, paper-style {b_paper}, literal {B_max}, "
        f"literal under the pin cap {b_cap}; M {M}")
    names = model_names(dims, synth)
    norms = model_norms(torch, dims, synth)
    sp = torch.cuda.current_stream().cuda_stream
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).cuda()
    tokens_all = synth.context_lengths(5, B_max, 0, dims.vocab - 1)

    def variant(tag, b, mode, mats, host_w_pages):
        lens = lens_all[:b]
        need = int(blocks[b - 1])
        log(f"step: {tag}: pool for {b} requests ({need} blocks)")
        pool = bd.boost_kv_pool_create(ctx, dims.layers, dims.hkv, dims.hd, need,
                                       M if mode == bd.KV_LPP else 0, mode,
                                       q_heads=dims.hq, max_batch=b, max_blocks_per_seq=mb,
                                       hbm_budget_bytes=budget)
        try:
            info = bd.boost_kv_pool_info(pool)
            tables = np.zeros((b, mb), np.int32)
            for i, L in enumerate(lens):
                ids = bd.boost_kv_alloc(pool, i, (int(L) + 15) // 16)
                assert ids != bd.EAGAIN
                tables[i, :len(ids)] = ids
            st = bd.boost_kv_stats(pool)
            log(f"step: {tag}: fill K/V")
            fill_kv(bd, ctx, torch, pool, dims, tables, lens)
            model = DecodeModel(ctx, dims, b, mb, pool, mats, norms)
            args_ = (dev(tokens_all[:b]), dev(lens - 1), dev(lens), dev(tables), sp)
            log(f"step: {tag}: timed")
            for _ in range(args.warmup):
                model.step(*args_)
            torch.cuda.synchronize()
            steps = args.steps if mode != bd.KV_BUDGET else max(2, min(args.steps, 3))
            ms = float(np.median(time_steps(torch, lambda: model.step(*args_), steps)))
            alg = model.bytes_per_step(lens)
            kv_bytes = int(sum(int(L) for L in lens)) * dims.hkv * dims.hd * 2 * 2 * dims.layers
            host_kv = st["used_host_head_blocks"] / max(1, st["used_blocks"] * dims.hkv)
            host_bytes = host_w_pages * bd.PAGE_BYTES + host_kv * kv_bytes
            bound = max((alg - host_bytes) / (bw_hbm * 1e9), host_bytes / (bw_host * 1e9)) * 1e3
            return {"batch": b, "ms_per_step": round(ms, 3),
                    "tokens_per_s": round(b * 1000.0 / ms, 1),
                    "gbps": round(alg / (ms * 1e-3) / 1e9, 1),
                    "bytes_per_step": int(alg), "kv_host_share": round(host_kv, 5),
                    "kv_host_pages_per_tensor": int(info["host_pages_per_tensor"]),
                    "host_weight_pages": int(host_w_pages),
                    "placement_bound_ms": round(bound, 3),
                    "pct_of_placement_bound": round(100 * bound / ms, 2),
                    "ids": model.ids.cpu().numpy().tolist()}
        finally:
            bd.boost_kv_pool_destroy(pool)

    out = {}
    log("step: place weights (all HBM)")
    mats, _ = place_model(bd, torch, names, all_hbm(bd, ctx))
    out["hbm"] = variant("hbm-only", b_hbm, bd.KV_ALL_HBM, mats, 0)
    for t_ in mats.values():
        bd.boost_tensor_free(t_)
    log("step: place weights (modulo placement)")
    mats, host_w = place_model(bd, torch, names,
                               lambda w, n: bd.boost_place_weights(ctx, w, n, M))
    out["paper"] = variant("paper-style", b_paper, bd.KV_LPP, mats, host_w)
    if not args.no_literal:
        try:
            out["literal_capacity_limited"] = variant("literal (pin cap)", b_cap, bd.KV_BUDGET,
                                                      mats, host_w)
            out["literal_capacity_limited"]["host_pin_cap_gib"] = args.host_pin_gib
        except bd.BoostError as e:
            out["literal_capacity_limited"] = {"skipped": str(e)}
        if b_cap < B_max:
            out["literal"] = {"skipped": f"{B_max} requests need "
                                         f"{(pages(B_max) * per - budget) / 2**30:.1f} GiB of "
                                         f"pinned host KV, above the {args.host_pin_gib} GiB "
                                         "a process can pin here"}
        else:
            try:
                out["literal"] = variant("literal", B_max, bd.KV_BUDGET, mats, host_w)
            except bd.BoostError as e:        # e.g. pinned host memory exhausted
                out["literal"] = {"skipped": str(e)}
    for t_ in mats.values():
        bd.boost_tensor_free(t_)
    common = min(b_hbm, b_paper)
    same = out["hbm"]["ids"][:common] == out["paper"]["ids"][:common]
    for v in out.values():
        v.pop("ids", None)
    p = out["paper"]
    return {
        "metric": METRIC, "value": p["gbps"], "unit": "GB/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": p["ms_per_step"], "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded random-init weights, K/V and tokens)",
        "config": {"workload": "Llama-3-8B-shaped high-throughput decode, contexts uniform "
                               "in [1024, 8192], 40e9-byte HBM KV budget, overflow KV on host "
                               "through the wave-aware pool",
                   "layers": dims.layers, "d": 4096, "ffn": 14336, "q_heads": 32,
                   "kv_heads": 8, "head_dim": 128, "vocab": 128256, "max_batch": B_max,
                   "modulus": M, "kv_budget_bytes": budget},
        "tokens_per_s": p["tokens_per_s"],
        "calibration": {"hbm_gbps": round(bw_hbm, 1), "host_gbps": round(bw_host, 2),
                        "alpha": round(alpha, 6)},
        "variants": out,
        "throughput_vs_hbm_only": round(p["tokens_per_s"] / out["hbm"]["tokens_per_s"], 4),
        "argmax_equal_on_common_prefix": same,
    }


# ------------------------------------------------------------ experiments
def _gemv_us(bd, ctx, torch, handles, N, K, x, B, y, reps):
    """Median microseconds of one GEMV over a rotation of placed copies."""
    sp = torch.cuda.current_stream().cuda_stream

    def run():
        for h in handles:
            bd.boost_decode_gemv(ctx, h, N, K, x, B, y, bd.DTYPE_F32, sp)
    run()
    torch.cuda.synchronize()
    return float(np.median(time_steps(torch, run, reps))) * 1e3 / len(handles)


def _seeded_weight(torch, N, K, seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    w = torch.randn((N, K), generator=g, device="cuda").mul_(0.02)
    return w.to(torch.bfloat16).view(torch.int16)


def gemm_shapes(args, bd, ctx, torch, bw_hbm, bw_host, alpha, M):
    """All-HBM time of the Llama-3-8B layer matrices (fused qkv, o, fused
    gate_up, down) at the batches of --batches, each call on the next of
    enough placed copies to cover 512 MiB, so no call finds its weights in
    the 256 MB memory-side cache.  Roofline fraction: algorithmic bytes
    (weights, x, y) over the call time against 8 TB/s, or flops against the
    2.5 PFLOP/s dense bf16 peak, whichever is higher.  Beside each: the
    vendor BLAS (torch's linear on plain contiguous copies, bf16 out) on the
    same shape, as a reference point for the kernel."""
    shapes = [("qkv", 6144, 4096), ("o", 4096, 4096), ("gate_up", 28672, 4096),
              ("down", 4096, 14336)]
    batches = [int(b) for b in args.batches.split(",")]
    if not batches or min(batches) < 1 or max(batches) > 256:
        raise SystemExit("--batches: sizes in 1..256")
    rows = []
    for si, (name, N, K) in enumerate(shapes):
        nbytes = N * K * 2
        n = -(-nbytes // bd.PAGE_BYTES)
        w = _seeded_weight(torch, N, K, 501 + si)
        n_copies = -(-(512 << 20) // nbytes)
        copies = [bd.boost_place_weights_map(ctx, w, nbytes, np.zeros(n, np.uint8))
                  for _ in range(n_copies)]
        plain = [w.view(torch.bfloat16).clone() for _ in range(n_copies)]
        del w
        torch.cuda.empty_cache()
        g = torch.Generator(device="cuda")
        g.manual_seed(11)
        xs = torch.randn((max(batches), K), generator=g, device="cuda").to(
            torch.bfloat16).view(torch.int16)
        y = torch.empty((max(batches), N), dtype=torch.float32, device="cuda")
        for B in batches:
            log(f"step: gemm_shapes {name} B={B}")
            x = xs[:B].contiguous()
            us = _gemv_us(bd, ctx, torch, copies, N, K, x, B, y, max(3, args.steps))
            alg = nbytes + B * K * 2 + B * N * 4
            gbps, tflops = alg / us / 1e3, 2 * N * K * B / us / 1e6
            xb = x.view(torch.bfloat16)

            def blas():
                for wp in plain:
                    torch.nn.functional.linear(xb, wp)
            blas()
            torch.cuda.synchronize()
            us_blas = float(np.median(time_steps(torch, blas, max(3, args.steps)))) * 1e3 / len(plain)
            rows.append({"matrix": name, "N": N, "K": K, "B": B, "us": round(us, 2),
                         "gbps": round(gbps, 1), "tflops": round(tflops, 1),
                         "frac": round(max(gbps / 8000.0, tflops / 2500.0), 4),
                         "vendor_blas_us": round(us_blas, 2)})
        for h in copies:
            bd.boost_tensor_free(h)
        del plain
        del xs, y
        torch.cuda.empty_cache()
    fr = [r["frac"] for r in rows]
    return {"metric": "skinny GEMM roofline fraction of the 8B layer matrices (all-HBM)",
            "value": round(float(np.exp(np.mean(np.log(fr)))), 4), "unit": "frac (geomean)",
            "n_gpus": 1, "higher_is_better": True, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": "Llama-3-8B layer matrices [6144|4096|28672|4096 x "
                                   "4096|4096|4096|14336], all pages in HBM",
                       "batches": batches},
            "calibration": {"hbm_gbps": round(bw_hbm, 1), "host_gbps": round(bw_host, 2),
                            "alpha": round(alpha, 6)},
            "rows": rows}


def host_share_sweep(args, bd, ctx, torch, bw_hbm, bw_host, alpha, M_alpha):
    """Speedup of a tiered GEMV over all-HBM as the host share grows (the
    host-share sweep of §3): one 2 GiB bf16 matrix [131072 x 8192] (1024
    pages), batch 1, modulo placement at a range of moduli; the best one is
    the measured-optimal modulus, set beside the one from the measured alpha."""
    N, K = 131072, 8192
    nbytes = N * K * 2
    n = nbytes // bd.PAGE_BYTES
    w = _seeded_weight(torch, N, K, 4242)
    x = torch.from_numpy(np.random.default_rng(7).standard_normal(
        (1, K)).astype(np.float32)).cuda().to(torch.bfloat16).view(torch.int16)
    y = torch.empty((1, N), dtype=torch.float32, device="cuda")
    hbm = bd.boost_place_weights_map(ctx, w, nbytes, np.zeros(n, np.uint8))
    mods = sorted({1025, 512, 400, 300, 250, 200, 160, 140, M_alpha, 120, 111, 100,
                   90, 80, 64, 50, 32}, reverse=True)
    placed = {m: bd.boost_place_weights(ctx, w, nbytes, m) for m in mods}
    del w
    torch.cuda.empty_cache()
    rows = {m: [] for m in mods}
    ref = []
    for _ in range(max(3, args.steps // 5)):
        ref.append(_gemv_us(bd, ctx, torch, [hbm], N, K, x, 1, y, 5))
        for m in mods:
            rows[m].append(_gemv_us(bd, ctx, torch, [placed[m]], N, K, x, 1, y, 5))
    t_hbm = float(np.median(ref))
    out = []
    for m in mods:
        h = int(bd.boost_tensor_tiers(placed[m]).sum())
        t = float(np.median(rows[m]))
        f = h / n
        bound = max((1 - f) * nbytes / (bw_hbm * 1e3), f * nbytes / (bw_host * 1e3))
        out.append({"M": m, "host_pages": h, "host_share": round(f, 5), "us": round(t, 2),
                    "speedup_vs_hbm_only": round(t_hbm / t, 4),
                    "placement_bound_us": round(bound, 2),
                    "ideal_combined_us": round(nbytes / ((bw_hbm + bw_host) * 1e3), 2)})
        bd.boost_tensor_free(placed[m])
    bd.boost_tensor_free(hbm)
    best = max(out, key=lambda r: (r["speedup_vs_hbm_only"], r["M"]))
    return {"metric": "tiered GEMV speedup over all-HBM vs host share (modulus sweep)",
            "value": best["speedup_vs_hbm_only"], "unit": "x", "n_gpus": 1,
            "higher_is_better": True, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": "host-share sweep: bf16 GEMV [131072 x 8192] (2 GiB, "
                                   "1024 pages), batch 1, modulo placement, CAP schedule"},
            "calibration": {"hbm_gbps": round(bw_hbm, 1), "host_gbps": round(bw_host, 2),
                            "alpha": round(alpha, 6), "M_from_alpha": M_alpha},
            "hbm_only_us": round(t_hbm, 2), "best_M": best["M"], "sweep": out}


def cap_measured_optimum(out):
    """The measured-optimal host share of a CAP sweep `out` (its
    `hbm_stream_modes` and `concurrent*` layouts, each with `hbm_only_us`,
    `hbm_only_spread` and `points`).  Every point is also timed against the
    fastest all-HBM launch of any layout (added to the points and to `out`):
    host reads gain only if they beat the best way to stream HBM alone, by
    more than the spread of their layout's all-HBM reference (at least
    0.2 %).  Without a gain the optimum is "no host page" (share 0)."""
    tags = [t for t in out if t.startswith("concurrent")]
    fastest = min([v["us"] for v in out["hbm_stream_modes"].values()] +
                  [out[t]["hbm_only_us"] for t in tags])
    out["fastest_hbm_only_us"] = round(fastest, 2)
    for t in tags:
        for r in out[t]["points"]:
            r["speedup_vs_fastest_hbm_only"] = round(fastest / r["us"], 4)
    cands = [(tag, r) for tag in tags for r in out[tag]["points"]]
    tag, best = max(cands, key=lambda c: c[1]["speedup_vs_fastest_hbm_only"])
    noise = out[tag]["hbm_only_spread"]
    gain = best["speedup_vs_fastest_hbm_only"] > 1.0 + max(noise, 0.002)
    return {"host_share": best["host_share"] if gain else 0.0,
            "host_workgroups": best["host_workgroups"] if gain else 0,
            "speedup_vs_hbm_only": best["speedup_vs_fastest_hbm_only"] if gain else 1.0,
            "best_host_point": dict(best, layout=tag), "reference_spread": noise,
            "modulus": int(round(1 / best["host_share"])) if gain else None}


def cap_probe(args, bd, ctx, torch, bw_hbm, bw_host, alpha, M_alpha):
    """The streaming-probe bound of concurrent access (§3 "CAP": the paper
    sweeps the host share of a streaming kernel whose workgroups read host
    memory and HBM at once, and §6.1 notes the compute units must be able to
    saturate both tiers together).  Sweeps of one kernel (`boost_cap_sweep`):
      * HBM alone, 2 GiB, over the number of workgroups (how many compute
        units it takes to saturate HBM);
      * host alone, 256 MiB, over workgroups x loads in flight per lane x
        cache policy (what the host link needs);
      * both at once: 2 GiB in total with a share f on host, read by h host
        workgroups beside 8192 HBM workgroups of 256 KiB (more than fit at
        once, so the dispatcher balances them over the compute units),
        against the same 2 GiB from HBM alone; and the one-wave layouts (2048
        HBM workgroups with static slices), coherent and non-coherent pages;
      * persistent HBM workers with chunks dealt round robin, one workgroup
        per compute unit (each holds most of the LDS), so the host workgroups
        run on compute units of their own;
      * the host share moved by the copy engine instead (host -> HBM copy on a
        second stream beside the HBM-only launch).
    Each point gives the combined rate, each tier's rate inside the launch
    (workgroup clocks) and the HBM bandwidth lost per GB/s of host bandwidth
    gained, against the all-HBM launch of its own layout and against the
    fastest all-HBM launch of any layout.  The measured-optimal host share is
    the best point against the fastest; its modulus (1/f) is what the
    placement should use when it beats all-HBM, and "no host page" otherwise."""
    T = 2 << 30
    HOST = 256 << 20
    iters = 15
    n_cu = bd.boost_ctx_info(ctx)[1]
    if args.cap_quick:
        # distinct grids per point, so a counter run can tell the launches apart
        hb = int(T / M_alpha) // 16 * 16
        pts = {"hbm_only": dict(hbm_bytes=T, hbm_wgs=8192),
               "host_only_8wg": dict(host_bytes=HOST, host_wgs=8),
               "alpha_share_spread_8wg": dict(hbm_bytes=T - hb, hbm_wgs=8192, host_bytes=hb,
                                              host_wgs=8),
               "hbm_only_queue": dict(hbm_bytes=T, hbm_wgs=n_cu * 8 - 16, hbm_chunk_kib=256),
               "alpha_share_queue_one_xcd_8wg": dict(hbm_bytes=T - hb, hbm_wgs=n_cu * 8 - 8,
                                                     host_bytes=hb, host_wgs=8, host_stride=8,
                                                     hbm_chunk_kib=256),
               # one and two workgroups short of a CU each, so that their grids
               # differ from each other and from calibration's (one per CU)
               "hbm_only_one_per_cu": dict(hbm_bytes=T, hbm_wgs=n_cu - 1, hbm_chunk_kib=256,
                                           chunk_static=3),
               "alpha_share_one_per_cu_spread_8wg": dict(hbm_bytes=T - hb, hbm_wgs=n_cu - 10,
                                                         host_bytes=hb, host_wgs=8,
                                                         hbm_chunk_kib=256, chunk_static=3)}
        res = bd.boost_cap_sweep(ctx, T, HOST, list(pts.values()), 3)
        return {"metric": "CAP probe points for counter runs", "unit": "us",
                "points": {k: {"grid": v.get("hbm_wgs", 0) + v.get("host_wgs", 0),
                               "hbm_bytes": v.get("hbm_bytes", 0),
                               "host_bytes": v.get("host_bytes", 0),
                               "us": round(float(r[1]), 2),
                               "hbm_in_launch_gbps": round(float(r[2]), 1),
                               "host_in_launch_gbps": round(float(r[3]), 2)}
                           for (k, v), r in zip(pts.items(), res)}}

    def run(points, coherent=1):
        bd.boost_set_host_coherent(ctx, coherent)
        try:
            return bd.boost_cap_sweep(ctx, T, HOST, points, iters)
        finally:
            bd.boost_set_host_coherent(ctx, 1)

    def r16(x):
        return int(x) // 16 * 16

    out = {}
    # how the HBM stream is handed to the workgroups, all-HBM: static slices
    # (one per workgroup, 8192 or 2048 of them), persistent workers with
    # 256 KiB chunks dealt round robin, from a queue, and from a queue after a
    # first chunk of their own (the claim of the next chunk overlapping the
    # current one)
    n_slots = bd.boost_ctx_info(ctx)[1] * 8
    modes = {"static_8192": dict(hbm_bytes=T, hbm_wgs=8192),
             "static_one_wave": dict(hbm_bytes=T, hbm_wgs=n_slots),
             "persistent_round_robin_256k": dict(hbm_bytes=T, hbm_wgs=n_slots,
                                                 hbm_chunk_kib=256, chunk_static=1),
             "persistent_queue_256k": dict(hbm_bytes=T, hbm_wgs=n_slots, hbm_chunk_kib=256),
             "persistent_queue_first_own_256k": dict(hbm_bytes=T, hbm_wgs=n_slots,
                                                     hbm_chunk_kib=256, chunk_static=2),
             "persistent_queue_first_own_64k": dict(hbm_bytes=T, hbm_wgs=n_slots,
                                                    hbm_chunk_kib=64, chunk_static=2),
             # one workgroup per compute unit (each holds most of the LDS)
             "persistent_round_robin_one_per_cu_256k": dict(hbm_bytes=T, hbm_wgs=n_cu,
                                                            hbm_chunk_kib=256, chunk_static=3),
             "persistent_round_robin_one_per_cu_64k": dict(hbm_bytes=T, hbm_wgs=n_cu,
                                                           hbm_chunk_kib=64, chunk_static=3)}
    res = run(list(modes.values()))
    out["hbm_stream_modes"] = {k: {"us": round(float(r[1]), 2),
                                   "in_launch_gbps": round(float(r[2]), 1),
                                   "last_end_by_xcd_us": [round(float(v), 1) for v in r[8:16]]}
                               for k, r in zip(modes, res)}
    grids = [64, 128, 256, 512, 1024, 2048, 4096, 8192]
    res = run([dict(hbm_bytes=T, hbm_wgs=g) for g in grids])
    out["hbm_by_workgroups"] = [{"workgroups": g, "gbps": round(float(r[0]), 1),
                                 "in_launch_gbps": round(float(r[2]), 1)}
                                for g, r in zip(grids, res)]
    host_pts = [(h, d, 0) for d in (1, 2, 4, 8) for h in (1, 2, 4, 8, 16, 32, 64)]
    host_pts += [(h, 8, pol) for pol in (1, 2) for h in (4, 16)]
    host_pts += [(h, 8, 0) for h in (128, 256)]
    res = run([dict(host_bytes=HOST, host_wgs=h, host_depth=d, host_policy=pol)
               for h, d, pol in host_pts])
    out["host_by_workgroups"] = [
        {"workgroups": h, "depth": d, "policy": pol, "gbps": round(float(r[0]), 2),
         "in_launch_gbps": round(float(r[3]), 2),
         "bytes_in_flight": h * 256 * 16 * d}
        for (h, d, pol), r in zip(host_pts, res)]

    shares = [1 / 1024, 1 / 256, 1 / M_alpha, 1 / 64]
    BAL = 8192                   # HBM workgroups of 256 KiB, balanced by the dispatcher
    ONE_WAVE = bd.boost_ctx_info(ctx)[1] * 8   # every slot once, static slices

    def with_refs(g_hbm, pts, coherent=1, chunk=0, cs=0):
        """Run the points each right after an all-HBM reference launch set (and
        one more at the end); per point, the mean of the two references
        around it."""
        ref = dict(hbm_bytes=T, hbm_wgs=g_hbm, hbm_chunk_kib=chunk, chunk_static=cs)
        seq = [ref]
        for q in pts:
            seq += [q, ref]
        res = run(seq, coherent)
        refs = res[0::2]
        rows = res[1::2]
        t_ref = [(refs[k][1] + refs[k + 1][1]) / 2 for k in range(len(pts))]
        h_ref = [(refs[k][2] + refs[k + 1][2]) / 2 for k in range(len(pts))]
        spread = float(np.std(refs[:, 1]) / np.mean(refs[:, 1]))
        return rows, t_ref, h_ref, float(np.median(refs[:, 1])), float(np.median(refs[:, 2])), spread

    def sweep(tag, g_hbm, combos, coherent=1, stride=1, chunk=0, cs=0):
        pts, keys = [], []
        for f in shares:
            hb = r16(f * T)
            for h, d, pol in combos:
                # persistent queue workers: the host workgroups take slots of
                # the one wave
                g = g_hbm - h if chunk else g_hbm
                pts.append(dict(hbm_bytes=T - hb, hbm_wgs=g, host_bytes=hb, host_wgs=h,
                                host_stride=stride, host_depth=d, host_policy=pol,
                                hbm_chunk_kib=chunk, chunk_static=cs))
                keys.append((f, h, d, pol))
        res, t_refs, h_refs, t_med, h_med, spread = with_refs(g_hbm, pts, coherent, chunk, cs)
        rows = []
        for key, r, t_ref, h_ref in zip(keys, res, t_refs, h_refs):
            f, h, d, pol = key
            hb = r16(f * T)
            bound_us = max((T - hb) / (bw_hbm * 1e3), hb / (bw_host * 1e3))
            host_g = float(r[3])
            rows.append({"host_share": round(f, 6), "host_workgroups": h, "depth": d,
                         "policy": pol, "us": round(float(r[1]), 2),
                         "ref_us": round(t_ref, 2),
                         "speedup_vs_hbm_only": round(t_ref / float(r[1]), 4),
                         "gbps": round(float(r[0]), 1),
                         "hbm_in_launch_gbps": round(float(r[2]), 1),
                         "ref_hbm_in_launch_gbps": round(h_ref, 1),
                         "host_in_launch_gbps": round(host_g, 2),
                         "hbm_median_end_us": round(float(r[5]), 2),
                         "hbm_last_end_us": round(float(r[7]), 2),
                         "hbm_last_end_by_xcd_us": [round(float(v), 1) for v in r[8:16]],
                         "hbm_lost_per_host_gbps": round((h_ref - float(r[2])) / host_g, 2)
                         if host_g > 0 else None,
                         "bound_us": round(bound_us, 2),
                         "bound_speedup": round(t_ref / bound_us, 4)})
        out[tag] = {"hbm_workgroups": g_hbm, "host_stride": stride, "coherent": bool(coherent),
                    "hbm_chunk_kib": chunk, "chunk_mode": cs, "hbm_only_us": round(t_med, 2), "hbm_only_in_launch_gbps": round(h_med, 1),
                    "hbm_only_spread": round(spread, 4), "points": rows}

    combos = [(h, d, 0) for d in (2, 8) for h in (4, 8, 16)]
    sweep("concurrent_balanced", BAL, combos + [(8, 8, 1), (8, 8, 2)])
    sweep("concurrent_balanced_one_xcd", BAL, combos, stride=8)
    # persistent HBM workers fed by a queue of 256 KiB chunks (a slower XCD
    # takes fewer chunks), host workgroups spread or on one XCD
    sweep("concurrent_queue", ONE_WAVE, [(h, 8, 0) for h in (4, 8, 16)], chunk=256)
    sweep("concurrent_queue_one_xcd", ONE_WAVE, combos, stride=8, chunk=256)
    # persistent HBM workers dealt chunks round robin, every workgroup on a
    # compute unit of its own (the host workgroups' loads never wait in the
    # vector L1 of a CU that streams HBM), host workgroups spread over the
    # XCDs or on one
    sweep("concurrent_one_per_cu_spread", n_cu, [(h, 8, 0) for h in (4, 8, 16)], chunk=256,
          cs=3)
    sweep("concurrent_one_per_cu_one_xcd", n_cu, [(h, 8, 0) for h in (4, 8, 16, 32)], stride=8,
          chunk=256, cs=3)
    sweep("concurrent_one_per_cu_spread_64k", n_cu, [(8, 8, 0)], chunk=64, cs=3)
    sweep("concurrent_one_wave", ONE_WAVE, [(8, 8, 0)])
    sweep("concurrent_one_wave_noncoherent", ONE_WAVE, [(8, 8, 0)], coherent=0)
    sweep("concurrent_balanced_noncoherent", BAL, [(8, 8, 0)], coherent=0)

    # the host share moved by the copy engine beside the HBM-only launch
    pts = []
    for f in shares:
        hb = r16(f * T)
        pts.append(dict(hbm_bytes=T - hb, hbm_wgs=BAL, host_bytes=hb, dma=1))
    res, t_refs, h_refs, t_med, _, spread = with_refs(BAL, pts)
    out["dma_beside_hbm"] = {
        "hbm_only_us": round(t_med, 2), "hbm_only_spread": round(spread, 4),
        "points": [{"host_share": round(f, 6), "kernel_us": round(float(r[1]), 2),
                    "copy_us": round(float(r[6]), 2), "ref_us": round(t_ref, 2),
                    "speedup_vs_hbm_only": round(t_ref / max(float(r[1]), float(r[6])), 4),
                    "hbm_in_launch_gbps": round(float(r[2]), 1),
                    "copy_gbps": round(float(r[3]), 2),
                    "hbm_lost_per_host_gbps": round((h_ref - float(r[2])) / float(r[3]), 2)
                    if r[3] > 0 else None}
                   for f, r, t_ref, h_ref in zip(shares, res, t_refs, h_refs)]}

    out["measured_optimum"] = cap_measured_optimum(out)
    return {"metric": "concurrent HBM + host streaming vs HBM alone (CAP bound)",
            "value": out["measured_optimum"]["speedup_vs_hbm_only"], "unit": "x",
            "n_gpus": 1, "higher_is_better": True, "dtype": "u8", "data": "synthetic",
            "config": {"workload": "streaming read of 2 GiB split between HBM and pinned "
                                   "host memory, 16-byte loads",
                       "iters": iters},
            "calibration": {"hbm_gbps": round(bw_hbm, 1), "host_gbps": round(bw_host, 2),
                            "alpha": round(alpha, 6), "M_from_alpha": M_alpha},
            "results": out}


def tensor_tier_bytes(bd, t, nbytes):
    """(HBM bytes, host bytes) of a placed tensor, from its tier map."""
    tiers = bd.boost_tensor_tiers(t)
    sizes = np.minimum(bd.PAGE_BYTES, nbytes - np.arange(len(tiers)) * bd.PAGE_BYTES)
    host = int(sizes[tiers == 1].sum())
    return nbytes - host, host


def tier_counters_run(args, bd, ctx, torch, M):
    """One tiered call of one part of the default bench, for a counter run
    (rocprofv3 --pmc TCC_EA0_RDREQ_DRAM_32B TCC_EA0_RDREQ_IO_32B): `chain` one
    step of the 129 GEMVs, `single` the 4096 x 4096 layer with page 15 on
    host, `attention` the config-3 paged attention on the wave-aware pool.
    Prints the placement's bytes per tier, which the counters must match."""
    sp = torch.cuda.current_stream().cuda_stream
    out = {"part": args.part, "modulus": M}
    if args.part == "chain":
        chain = Chain(bd, ctx, torch, args.layers, M)
        hbm = host = 0
        for t, h, N, K, x, y in chain.ops:
            a, b = tensor_tier_bytes(bd, t, N * K * 2)
            hbm, host = hbm + a, host + b
        torch.cuda.synchronize()
        chain.run("boost", sp)
        torch.cuda.synchronize()
        out.update(weight_hbm_bytes=hbm, weight_host_bytes=host, launches=len(chain.ops))
        chain.free()
    elif args.part == "single":
        import synth
        w, x = synth.single_layer_inputs()
        t = bd.boost_place_weights(ctx, w, w.nbytes, 16)
        xd = torch.from_numpy(x.view(np.int16)).cuda()
        y = torch.empty((1, 4096), dtype=torch.float32, device="cuda")
        a, b = tensor_tier_bytes(bd, t, w.nbytes)
        torch.cuda.synchronize()
        bd.boost_decode_gemv(ctx, t, 4096, 4096, xd, 1, y, bd.DTYPE_F32, sp)
        torch.cuda.synchronize()
        bd.boost_tensor_free(t)
        out.update(weight_hbm_bytes=a, weight_host_bytes=b, launches=1)
    else:
        A = attention_setup(bd, ctx, torch, M)
        st = A["stats"]
        torch.cuda.synchronize()
        A["call"]("boost")
        torch.cuda.synchronize()
        # K and V bytes on host: host head-blocks in use, 16 tokens of D bf16
        # each, for K and for V (upper bound: a request's last block is
        # partly empty)
        host = int(st["used_host_head_blocks"]) * 16 * A["D"] * 2 * 2
        out.update(kv_bytes=A["alg"], kv_host_bytes_upper=host, launches=1)
        for pool, _, _ in A["pools"].values():
            bd.boost_kv_pool_destroy(pool)
    return out


def batch_sweep(args, bd, ctx, torch, bw_hbm, bw_host, alpha, M):
    """Tiered (modulo placement at the measured modulus) vs all-HBM GEMV/GEMM
    time as the batch grows (the batch sensitivity study of §5.10): the
    tensors of the 8B and 70B shapes large enough to hold host pages at this
    modulus, batches 1..256."""
    shapes = {"8b_lm_head": (128256, 4096), "70b_gate_up": (57344, 8192),
              "70b_down": (8192, 28672), "70b_lm_head": (128256, 8192)}
    batches = [1, 2, 4, 8, 16, 32, 64, 128, 256]
    res = {}
    for si, (name, (N, K)) in enumerate(shapes.items()):
        nbytes = N * K * 2
        n = -(-nbytes // bd.PAGE_BYTES)
        w = _seeded_weight(torch, N, K, 777 + si)
        hbm = bd.boost_place_weights_map(ctx, w, nbytes, np.zeros(n, np.uint8))
        tiered = bd.boost_place_weights(ctx, w, nbytes, M)
        host = int(bd.boost_tensor_tiers(tiered).sum())
        del w
        torch.cuda.empty_cache()
        g = torch.Generator(device="cuda")
        g.manual_seed(9)
        xs = torch.randn((max(batches), K), generator=g, device="cuda").to(
            torch.bfloat16).view(torch.int16)
        y = torch.empty((max(batches), N), dtype=torch.float32, device="cuda")
        rows = []
        for B in batches:
            x = xs[:B].contiguous()
            a, b = [], []
            for _ in range(max(3, args.steps // 5)):
                a.append(_gemv_us(bd, ctx, torch, [hbm], N, K, x, B, y, 3))
                b.append(_gemv_us(bd, ctx, torch, [tiered], N, K, x, B, y, 3))
            ta, tb = float(np.median(a)), float(np.median(b))
            alg = nbytes + B * K * 2 + B * N * 4
            rows.append({"B": B, "hbm_us": round(ta, 2), "tiered_us": round(tb, 2),
                         "speedup_vs_hbm_only": round(ta / tb, 4),
                         "tiered_gbps": round(alg / tb / 1e3, 1),
                         "tiered_tflops": round(2 * N * K * B / tb / 1e6, 2),
                         "path": "gemv" if B < 7 else "mfma"})
        res[name] = {"N": N, "K": K, "pages": n, "host_pages": host, "rows": rows}
        bd.boost_tensor_free(hbm)
        bd.boost_tensor_free(tiered)
        del xs, y
        torch.cuda.empty_cache()
    sp = [r["speedup_vs_hbm_only"] for v in res.values() for r in v["rows"]]
    return {"metric": "tiered vs all-HBM GEMV/GEMM speedup by batch size",
            "value": round(float(np.exp(np.mean(np.log(sp)))), 4), "unit": "x (geomean)",
            "n_gpus": 1, "higher_is_better": True, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": "batch sweep 1..256 of the 8B/70B tensors that hold host "
                                   "pages at the measured modulus", "modulus": M},
            "calibration": {"hbm_gbps": round(bw_hbm, 1), "host_gbps": round(bw_host, 2),
                            "alpha": round(alpha, 6)},
            "shapes": res}


def _window_stats(tiers, P):
    """Host-page fraction of every full window of P consecutive pages of the
    chain in launch order: mean, standard deviation and largest deviation."""
    t = np.asarray(tiers, dtype=np.float64)
    nw = len(t) // P
    if nw == 0:
        return {"windows": 0}
    f = t[:nw * P].reshape(nw, P).mean(axis=1)
    return {"windows": nw, "pages_per_window": P, "mean": round(float(f.mean()), 6),
            "sd": round(float(f.std()), 6), "max_dev": round(float(np.abs(f - f.mean()).max()), 6)}


def placements_bench(args, bd, ctx, torch, bw_hbm, bw_host, alpha, M):
    """The 8B decode weight chain (batch 1) under the contrast placements
    (§2.6, §5.6, §5.7): all-HBM, modulo placement restarted per tensor (the
    method), modulo pattern continued across tensors (an interleave blind to
    kernel boundaries), a linear split per tensor, and random placement
    (BAPP-R, seeded draws); each with the CAP and the address-order
    schedule."""
    import synth
    per_layer, head = synth.chain_shapes(synth.LLAMA8B)
    specs = [(l, kind, n, k) for l in range(args.layers) for _, kind, n, k in per_layer]
    specs.append((0, head[1], head[2], head[3]))
    kinds = {"hbm": None, "mpp": bd.PLACE_MPP, "mpp_global": bd.PLACE_MPP_GLOBAL,
             "linear": bd.PLACE_LINEAR, "bapp_r": bd.PLACE_RANDOM}
    rng = np.random.default_rng(7)
    xs = {K: torch.from_numpy(synth.normal_bf16(rng, (1, K), 1.0).view(np.int16)).cuda()
          for K in sorted({s[3] for s in specs})}
    ops = {k: [] for k in kinds}
    tiers = {k: [] for k in kinds}
    phase = 0
    for t, (l, kind, N, K) in enumerate(specs):
        w = synth.chain_weight_torch(l, kind, N, K, "cuda").view(torch.int16)
        nbytes = N * K * 2
        n = -(-nbytes // bd.PAGE_BYTES)
        for name, pk in kinds.items():
            if pk is None:
                tm = np.zeros(n, np.uint8)
            else:
                tm = bd.boost_plan_contrast(pk, nbytes, M, phase,
                                            synth.uniforms(5000 + t, n))
            ops[name].append((bd.boost_place_weights_map(ctx, w, nbytes, tm), N, K))
            tiers[name].append(tm)
        phase += n
        del w
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    ys = {N: torch.empty((1, N), dtype=torch.float32, device="cuda")
          for N in {s[2] for s in specs}}
    sp = torch.cuda.current_stream().cuda_stream
    alg = sum(N * K * 2 + K * 2 + N * 4 for _, _, N, K in specs)

    def step(name):
        for h, N, K in ops[name]:
            bd.boost_decode_gemv(ctx, h, N, K, xs[K], 1, ys[N], bd.DTYPE_F32, sp)
    res = {}
    scheds = {"cap": bd.SCHED_CAP, "address": bd.SCHED_ADDRESS}
    for sc in scheds.values():
        bd.boost_gemv_set_schedule(ctx, sc, args.host_workers)
        for name in kinds:
            step(name)
    torch.cuda.synchronize()
    # every (schedule, placement) pair once per round, the schedules' order
    # alternating from round to round, so that a drift of the box over the
    # run (clocks, temperature) falls on all of them alike
    ms = {(name, sc): [] for name in kinds for sc in scheds}
    for r in range(max(5, args.steps // 2)):
        for sched in (("cap", "address") if r % 2 == 0 else ("address", "cap")):
            bd.boost_gemv_set_schedule(ctx, scheds[sched], args.host_workers)
            for name in kinds:
                ms[(name, sched)].append(time_steps(torch, lambda: step(name), 1)[0])
    for (name, sched), v in ms.items():
        t = float(np.median(v))
        res.setdefault(name, {})[sched] = {"ms_per_step": round(t, 4),
                                           "gbps": round(alg / (t * 1e-3) / 1e9, 1)}
    bd.boost_gemv_set_schedule(ctx, bd.SCHED_CAP, args.host_workers)
    # one grid wave of the batch-1 GEMV covers about 2048 workgroups x 32 KiB
    wave_pages = 32
    for name in kinds:
        shares = [float(tm.mean()) for tm in tiers[name]]
        res[name].update({
            "host_pages": int(sum(int(tm.sum()) for tm in tiers[name])),
            "tensors_with_host_pages": int(sum(1 for tm in tiers[name] if tm.any())),
            "max_tensor_host_share": round(max(shares), 5),
            "waves": _window_stats(np.concatenate(tiers[name]), wave_pages)})
        for sched in ("cap", "address"):
            res[name][sched]["speedup_vs_hbm_only"] = round(
                res["hbm"][sched]["ms_per_step"] / res[name][sched]["ms_per_step"], 4)
        for h, _, _ in ops[name]:
            bd.boost_tensor_free(h)
    return {"metric": "decode weight-chain step ms by placement (contrast placements)",
            "value": res["mpp"]["cap"]["ms_per_step"], "unit": "ms",
            "n_gpus": 1, "higher_is_better": False, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": "Llama-3-8B-shaped decode weight chain, batch 1, under "
                                   "all-HBM / modulo (per tensor) / modulo across tensors / "
                                   "linear / random placement", "modulus": M,
                       "layers": args.layers, "bytes_per_step": int(alg)},
            "calibration": {"hbm_gbps": round(bw_hbm, 1), "host_gbps": round(bw_host, 2),
                            "alpha": round(alpha, 6)},
            "placements": res}


def run_churn(trace, steps, max_batch, alloc, free, stats, on_step=None):
    """Decode-serving loop over a request trace, driving a KV block allocator.

    trace: (arrival step, prompt tokens, output tokens) per request, request id =
    index.  Each step: arrivals join a FIFO queue; queued requests are admitted
    in order while fewer than max_batch run, each allocating the blocks of its
    prompt (a refusal leaves it and everything behind it queued: the call is
    handed back to the scheduler, §4.3); every running request then appends
    one token, allocating one more block when its last block is full (when
    the pool is out of blocks the latest admitted request is preempted: freed
    and queued again in front, to be recomputed); requests that produced their
    output are freed.  alloc(rid, n) returns block ids or None, free(rid) releases a
    request, stats() returns (used blocks, used host head-blocks, SHH
    requests).  on_step(step, running) may time the step's batch.  Returns
    per-step rows (used blocks, host head-blocks, running, queued, SHH
    requests) and counters."""
    queue, running = [], []
    tokens, made, blocks = {}, {}, {}
    nxt = 0
    rows = []
    refused = preempted = done = 0
    for step in range(steps):
        while nxt < len(trace) and trace[nxt][0] <= step:
            queue.append(nxt)
            nxt += 1
        while queue and len(running) < max_batch:
            rid = queue[0]
            prompt = trace[rid][1]
            ids = alloc(rid, (prompt + 15) // 16)
            if ids is None:
                refused += 1
                break
            queue.pop(0)
            running.append(rid)
            tokens[rid], made[rid], blocks[rid] = prompt, 0, list(ids)
        i = 0
        while i < len(running):
            rid = running[i]
            if tokens[rid] % 16 == 0:
                ids = alloc(rid, 1)
                while ids is None:
                    # out of blocks: preempt the latest admitted request (its
                    # blocks are freed and it is queued again in front, to be
                    # recomputed), then retry unless it was this one
                    victim = running.pop()
                    free(victim)
                    del tokens[victim], made[victim], blocks[victim]
                    queue.insert(0, victim)
                    preempted += 1
                    if victim == rid:
                        break
                    ids = alloc(rid, 1)
                if ids is None:
                    continue
                blocks[rid].extend(ids)
            tokens[rid] += 1
            made[rid] += 1
            i += 1
        if on_step is not None and running:
            on_step(step, running, tokens, blocks)
        keep = []
        for rid in running:
            if made[rid] >= trace[rid][2]:
                free(rid)
                done += 1
                del tokens[rid], made[rid], blocks[rid]
            else:
                keep.append(rid)
        running = keep
        used, host, shh = stats()
        rows.append((used, host, len(running), len(queue), shh))
    return np.array(rows, dtype=np.int64), {"refused_admissions": refused,
                                            "preemptions": preempted, "finished": done,
                                            "arrived": nxt}


def _rolling_median(x, w):
    if len(x) < w:
        return np.array([np.median(x)]) if len(x) else np.array([])
    v = np.lib.stride_tricks.sliding_window_view(x, w)
    return np.median(v, axis=1)


def dsr_churn(args, bd, ctx, torch, bw_hbm, bw_host, alpha, M):
    """The wave-aware KV allocator under Poisson arrivals (the realized host
    ratio study of §5.11, with a synthetic arrival trace in place of the
    paper's LongWriter requests): the realized host share of the KV in use per
    step, its rolling median and range, against the pool's target; twice: at
    the paper's setting (4 KV heads, modulus 12) and at this GPU's (8 KV
    heads, measured modulus).  On the GPU, the paged-attention time of the
    running batch (one layer, 32/8 heads) on sampled steps, wave-aware pool vs
    an all-HBM pool fed the same trace."""
    import synth
    steps, warm, window = 20000, 2000, 100
    trace = synth.poisson_arrivals(11, steps, 0.03, 256, 2048, 512, 4096)
    NB, max_batch = 16000, 256
    out = {}
    for tag, H, m in (("paper_h4_m12", 4, 12), ("this_gpu", 8, M)):
        plan = bd.boost_init(-1)
        pool = bd.boost_kv_pool_create(plan, 1, H, 128, NB, m, bd.KV_LPP, q_heads=4 * H)
        info = bd.boost_kv_pool_info(pool)

        def alloc(rid, n):
            ids = bd.boost_kv_alloc(pool, rid, n)
            return None if ids == bd.EAGAIN else ids

        def stats():
            s = bd.boost_kv_stats(pool)
            return s["used_blocks"], s["used_host_head_blocks"], s["shh_requests"]
        rows, cnt = run_churn(trace, steps, max_batch, alloc,
                              lambda rid: bd.boost_kv_free(pool, rid), stats)
        bd.boost_kv_pool_destroy(pool)
        bd.boost_shutdown(plan)
        used, host = rows[warm:, 0].astype(np.float64), rows[warm:, 1].astype(np.float64)
        share = np.where(used > 0, host / np.maximum(used * H, 1), 0.0)
        rm = _rolling_median(share, window)
        nb = int(info["nb_pool"])
        target = (info["n_shh"] * info["shh_host_heads"] +
                  (nb - info["n_shh"]) * info["local_host_heads"]) / (nb * H)
        out[tag] = {"kv_heads": H, "modulus": m, "pool_blocks": nb,
                    "shh_blocks": int(info["n_shh"]), "ideal_share": round(1 / m, 5),
                    "pool_share": round(float(target), 5), "tau": round(info["tau"], 5),
                    "mean_share": round(float(share.mean()), 5),
                    "rolling_median_min": round(float(rm.min()), 5),
                    "rolling_median_max": round(float(rm.max()), 5),
                    "min_share": round(float(share.min()), 5),
                    "max_share": round(float(share.max()), 5),
                    "mean_running": round(float(rows[warm:, 2].mean()), 1),
                    "mean_blocks_in_use": round(float(used.mean()), 1),
                    "steps": steps, "warmup_steps": warm, "window": window, **cnt}
    # GPU: attention time of the running batch on sampled steps
    Hq, H, D = 32, 8, 128
    mb = (2048 + 4096 + 15) // 16 + 1
    g = torch.Generator(device="cuda")
    g.manual_seed(3)
    q = torch.randn((max_batch, Hq, D), generator=g, device="cuda").to(torch.bfloat16)
    o = torch.empty((max_batch, Hq, D), dtype=torch.float32, device="cuda")
    sp = torch.cuda.current_stream().cuda_stream
    times = {}
    for tag, mode, m in (("boost", bd.KV_LPP, M), ("hbm", bd.KV_ALL_HBM, 0)):
        pool = bd.boost_kv_pool_create(ctx, 1, H, D, NB, m, mode, q_heads=Hq,
                                       max_batch=max_batch, max_blocks_per_seq=mb)
        ms = []

        def alloc(rid, n):
            ids = bd.boost_kv_alloc(pool, rid, n)
            return None if ids == bd.EAGAIN else ids

        def stats():
            s = bd.boost_kv_stats(pool)
            return s["used_blocks"], s["used_host_head_blocks"], s["shh_requests"]

        def on_step(step, running, tokens, blocks):
            if step < warm or step % 20:
                return
            B = len(running)
            tab = np.full((B, mb), -1, np.int32)
            for i, rid in enumerate(running):
                tab[i, :len(blocks[rid])] = blocks[rid]
            lens = np.array([tokens[rid] for rid in running], np.int32)
            td = torch.from_numpy(tab).cuda()
            ld = torch.from_numpy(lens).cuda()
            a = torch.cuda.Event(enable_timing=True)
            b = torch.cuda.Event(enable_timing=True)
            a.record()
            bd.boost_paged_attn_decode(ctx, pool, 0, q, B, Hq, td, mb, ld, 0.0, o,
                                       bd.DTYPE_F32, sp)
            b.record()
            torch.cuda.synchronize()
            ms.append(a.elapsed_time(b))
        run_churn(trace, steps, max_batch, alloc, lambda rid: bd.boost_kv_free(pool, rid),
                  stats, on_step)
        bd.boost_kv_pool_destroy(pool)
        times[tag] = np.array(ms)
    ratio = times["hbm"] / times["boost"]
    out["attention_steps"] = {
        "sampled_steps": int(len(ratio)),
        "boost_ms_p50": round(float(np.percentile(times["boost"], 50)), 4),
        "boost_ms_p99": round(float(np.percentile(times["boost"], 99)), 4),
        "hbm_ms_p50": round(float(np.percentile(times["hbm"], 50)), 4),
        "hbm_ms_p99": round(float(np.percentile(times["hbm"], 99)), 4),
        "median_speedup_vs_hbm_only": round(float(np.median(ratio)), 4)}
    p = out["paper_h4_m12"]
    return {"metric": "realized KV host share under Poisson arrivals (wave-aware pool)",
            "value": p["mean_share"], "unit": "fraction of KV bytes in use",
            "n_gpus": 1, "higher_is_better": None, "dtype": "bf16", "data": "synthetic",
            "config": {"workload": "Poisson arrivals 0.03 per step over 20000 decode steps, "
                                   "prompts U[256, 2048], outputs U[512, 4096], at most 256 "
                                   "running, 16000-block pool",
                       "modulus": M},
            "calibration": {"hbm_gbps": round(bw_hbm, 1), "host_gbps": round(bw_host, 2),
                            "alpha": round(alpha, 6)},
            "results": out}


def main():
    args = parse()
    if args.summarize_pmc:
        print(json.dumps(summarize_pmc(args.summarize_pmc), indent=1))
        return
    if args.tier_profile:
        write_tier_profile(args.tier_profile)
        return
    if args.traffic_profile:
        write_traffic_profile(args.traffic_profile)
        return
    if args.summarize_trace:
        print(summarize_trace(args.summarize_trace))
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); "
              "the library has no multi-GPU path.", file=sys.stderr)
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
    if args.pmc_ref:      # a plain 1 GiB device fill: write reference of the counters
        a = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        a.fill_(1)
        torch.cuda.synchronize()
        del a
    exp = {"host_share_sweep": lambda: host_share_sweep(args, bd, ctx, torch, bw_hbm,
                                                        bw_host, alpha, M),
           "cap_probe": lambda: cap_probe(args, bd, ctx, torch, bw_hbm, bw_host, alpha, M),
           "gemm_shapes": lambda: gemm_shapes(args, bd, ctx, torch, bw_hbm, bw_host,
                                              alpha, M),
           "batch_sweep": lambda: batch_sweep(args, bd, ctx, torch, bw_hbm, bw_host,
                                              alpha, M),
           "placements": lambda: placements_bench(args, bd, ctx, torch, bw_hbm, bw_host,
                                                  alpha, M),
           "dsr_churn": lambda: dsr_churn(args, bd, ctx, torch, bw_hbm, bw_host, alpha, M)}
    if args.workload in exp:
        out = exp[args.workload]()
        bd.boost_shutdown(ctx)
        print(json.dumps(out), flush=True)
        return
    if args.workload == "tier_counters":
        out = tier_counters_run(args, bd, ctx, torch, M)
        bd.boost_shutdown(ctx)
        print(json.dumps(out), flush=True)
        return
    if args.workload in ("llama70b", "throughput8b"):
        if args.workload == "llama70b":
            if args.layers == 32:
                args.layers = 80
            out = llama70b(args, bd, ctx, torch, bw_hbm, bw_host, alpha)
        else:
            out = throughput8b(args, bd, ctx, torch, bw_hbm, bw_host, alpha)
        bd.boost_shutdown(ctx)
        print(json.dumps(out), flush=True)
        return

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
    boost_ms, hbm_ms, pre_ms = [], [], []
    for i in range(args.steps):
        # interleaved A/B/C so all see the same clocks and thermal state
        boost_ms.append(time_steps(torch, lambda: step("boost"), 1)[0])
        hbm_ms.append(time_steps(torch, lambda: step("hbm"), 1)[0])
        pre_ms.append(time_steps(torch, lambda: chain.run_prefetch(stream), 1)[0])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    boost_ms, hbm_ms, pre_ms = np.array(boost_ms), np.array(hbm_ms), np.array(pre_ms)
    ms = float(np.median(boost_ms))
    ms_hbm = float(np.median(hbm_ms))
    ms_pre = float(np.median(pre_ms))

    # roofline of the dominant kernel: the timed region's HIP events (on the
    # launching stream) over the step's GEMV launches, back to back, so each
    # launch's share includes its kernel boundary.  (A pair of events around
    # every launch reads ~2 us more per launch than this: the events' own
    # packets between the kernels cost about as much as a boundary.)
    launches = len(chain.ops)
    avg_launch_ms = ms / launches
    bytes_per_launch = chain.alg_bytes / launches
    achieved = bytes_per_launch / (avg_launch_ms * 1e-3) / 1e9

    log("step: A/B pairs")
    ab = ab_pairs(torch, lambda: step("boost"), lambda: step("hbm"), args.ab_pairs)
    # the tensors that hold host pages, timed alone (tiered and all-HBM): the
    # host tier's rate over the launches that read it
    host_ops = [op for op in chain.ops if tensor_tier_bytes(bd, op[0], op[2] * op[3] * 2)[1]]
    host_ops_t = None
    if host_ops:
        def run_ops(which):
            for t, h, N, K, x, y in host_ops:
                bd.boost_decode_gemv(ctx, t if which == "boost" else h, N, K, x, 1, y,
                                     bd.DTYPE_F32, sp)
        lh = ab_pairs(torch, lambda: run_ops("boost"), lambda: run_ops("hbm"), 50)
        hb = sum(tensor_tier_bytes(bd, op[0], op[2] * op[3] * 2)[0] for op in host_ops)
        hh = sum(tensor_tier_bytes(bd, op[0], op[2] * op[3] * 2)[1] for op in host_ops)
        host_ops_t = {"tensors": len(host_ops), "ms": lh["a_ms_median"],
                      "hbm_only_ms": lh["b_ms_median"],
                      "speedup_vs_hbm_only": lh["speedup_geomean"], "ci95": lh["ci95"],
                      "hbm_gbps": round(hb / (lh["a_ms_median"] * 1e-3) / 1e9, 1),
                      "host_gbps": round(hh / (lh["a_ms_median"] * 1e-3) / 1e9, 2),
                      "host_bytes": int(hh)}

    log("step: attention")
    attn = attention_bench(bd, ctx, torch, M, max(10, args.steps), 3)
    log("step: single layer")
    single = single_layer_bench(bd, ctx, torch, bw_hbm, bw_host)
    eff = chain.alg_bytes / (ms * 1e-3) / 1e9
    eff_hbm = chain.alg_bytes / (ms_hbm * 1e-3) / 1e9
    host_share = chain.host_pages / chain.pages
    cpu = None
    if not args.no_cpu_baseline:
        log("step: cpu baseline (oracle)")
        cpu = cpu_baseline(args.cpu_seconds)
    host_numa = bd.boost_host_numa_info(ctx)
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
                        "alpha": round(alpha, 6),
                        "host_numa": host_numa},
        "pct_combined_roofline": round(100 * eff / (bw_hbm + bw_host), 2),
        "hbm_only": {"ms_per_step": round(ms_hbm, 4), "value": round(eff_hbm, 2),
                     "pct_of_hbm_roofline": round(100 * eff_hbm / bw_hbm, 2)},
        "speedup_vs_hbm_only": ab["speedup_geomean"],
        "speedup_vs_hbm_only_ci95": ab["ci95"],
        "ab_pairs": ab,
        "speedup_vs_hbm_only_timed_region": round(ms_hbm / ms, 4),
        "per_tier": {"step": per_tier("chain", ms, chain.hbm_weight_bytes,
                                      chain.host_weight_bytes, M),
                     "tensors_with_host_pages": host_ops_t},
        "prefetch": {"ms_per_step": round(ms_pre, 4),
                     "value": round(chain.alg_bytes / (ms_pre * 1e-3) / 1e9, 2),
                     "staged_tensors": len(chain.staged),
                     "staged_bytes_per_step": int(chain.staged_bytes)},
        "attention": attn,
        "single_layer": single,
        "step_ms_iqr": [round(float(np.percentile(boost_ms, 25)), 4),
                        round(float(np.percentile(boost_ms, 75)), 4)],
        "roofline": {"bound": "hbm", "kernel": "gemv_kernel (batch 1)",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBPS, 4),
                     "traffic": counter_traffic("gemv", "gemv.hip"),
                     "avg_launch_us": round(avg_launch_ms * 1e3, 3),
                     "bytes_per_launch": int(bytes_per_launch)},
        "cpu_baseline": cpu,
        "timed_wall_s": round(wall, 3),
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
