"""Decode-attention bench: split-KV GQA sweep + LSE combine over every layer of a workload.

One step = for every layer: qf_attn_decode_split (sweep of all cached K/V, per-shard (O, ln Z))
then qf_attn_combine (merge to bf16 out + fp32 lse); with --one-launch both in one launch
(qf_attn_decode).  All layers' inputs are resident in HBM before the timed region.  Prints ONE
JSON line.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

With ``--stage NAME`` it instead times a decode step of a stack of Q-First blocks (synthetic
weights) at the context where the feed-forward's weight bytes equal the sweep's cache bytes, with
the sweep in the serial order and on its own stream beside the feed-forward (both captured in HIP
graphs), and prints one JSON line for that.
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0           # MI355X HBM3E, 8 TB/s
INFINITY_CACHE_BYTES = 256 << 20  # MI355X last-level (Infinity) cache
WARMUP_SECONDS = 0.3              # default warm-up: the first tens of ms of a run are slower
TIMED_SECONDS = 0.25              # default timed work
DEFAULT_WORKLOAD = "qwen3-0.6b_b32_n32768_s64_l28"


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def algorithmic_bytes(case):
    """Minimal HBM bytes of one sweep launch and one combine launch.

    sweep: every cached position's K and V (2 * Hkv * D * 2 B), the block-table entry of every
    used page (4 B), the queries (B * Hq * D * 2 B), the two int32 per request, and the partials
    written for non-empty shards (Hq * (D + 1) * 4 B each).
    combine: those partials read once, plus the bf16 out and fp32 lse written.
    """
    import numpy as np

    B, Hq, Hkv, D = case.shape
    n = case.ctx_lens.cpu().numpy().astype(np.int64)
    S = case.n_shards.cpu().numpy().astype(np.int64)
    pages = -(-n // 16)
    per = np.where(pages > 0, -(-pages // np.maximum(S, 1)), 0)
    live = np.where(per > 0, -(-pages // np.maximum(per, 1)), 0)   # non-empty shards
    kv = int(n.sum()) * 2 * Hkv * D * 2
    partials = int(live.sum()) * Hq * (D + 1) * 4
    sweep = kv + int(pages.sum()) * 4 + B * Hq * D * 2 + B * 8 + partials
    combine = partials + B * Hq * (D * 2 + 4)
    return dict(kv=kv, sweep=sweep, combine=combine, attended=int(n.sum()))


def committed_traffic(workload, two_launch=True):
    """HBM bytes per launch of the timed kernel (the one-launch sweep + merge, or the sweep of
    the two-launch step) from the committed rocprofv3 counter summary of this workload, or None
    when there is none or the kernel's sources changed since it was taken."""
    kind = "decode_split" if two_launch else "decode_fused"
    path = os.path.join(ROOT, "profiles", f"{kind}_{workload}_hbm_traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if kernel_source_digest() != rec.get("kernel_source_sha256"):
        return None
    return rec["traffic_bytes_per_launch"]


KERNEL_SOURCES = ("decode_split.hip", "merge.hip", "linear_body.h", "merge_body.h", "qf_internal.h")


def kernel_source_digest():
    """sha256 over the sweep's kernel sources with comments removed and white space collapsed, so
    that committed counters stay attached to the code they measured and to nothing else."""
    import hashlib
    import re

    h = hashlib.sha256()
    for name in KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2608_15473_amd", "csrc", name)) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
        h.update(b"\0")
    return h.hexdigest()


def cpu_model():
    """The host CPU's model name (what lscpu reports), from /proc/cpuinfo."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def env_info():
    """Where and on what a result was measured: git commit (when the tree has git metadata, else
    QF_GIT_SHA from the environment), source digest, ROCm / HIP / torch versions, GPU, host CPU
    model and the cores this process may use."""
    import subprocess

    import torch

    sha = None
    try:
        r = subprocess.run(["git", "rev-parse", "HEAD"], cwd=ROOT, capture_output=True, text=True,
                           timeout=10)
        sha = r.stdout.strip() or None
    except (OSError, subprocess.SubprocessError):
        pass
    rocm = None
    try:
        with open(os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), ".info", "version")) as f:
            rocm = f.read().strip()
    except OSError:
        pass
    props = torch.cuda.get_device_properties(0)
    import platform

    from paper_2608_15473_amd.report import source_digest

    return {"git_sha": sha or os.environ.get("QF_GIT_SHA"), "source_sha256": source_digest(),
            "rocm": rocm, "hip": torch.version.hip, "torch": torch.__version__,
            "gpu": props.name, "gpu_arch": getattr(props, "gcnArchName", None),
            "gpu_compute_units": props.multi_processor_count, "cpu_model": cpu_model(),
            "host_cores": len(os.sched_getaffinity(0)), "host": platform.node(),
            "time": int(time.time())}


def write_record(path, result):
    """Append one result line to the run record of its workload (a JSON file holding a list of
    runs), creating it if needed."""
    runs = []
    if os.path.exists(path):
        with open(path) as f:
            runs = json.load(f)["runs"]
    runs.append(result)
    d = os.path.dirname(path)
    if d:
        os.makedirs(d, exist_ok=True)
    with open(path, "w") as f:
        json.dump({"workload": result["config"]["workload"], "runs": runs}, f, indent=1)
        f.write("\n")


def cpu_baseline(cases, budget_s=15.0):
    """The fp64 oracle (sweep per shard + pairwise merge) timed on the host over a bounded sample:
    whole requests, layer after layer, added until about ``budget_s`` of CPU work.  Device-to-host
    copies are excluded from the timing."""
    import numpy as np
    import torch
    from threadpoolctl import threadpool_info

    import oracle

    B, Hq, Hkv, D = cases[0].shape
    done_bytes, spent, reqs, layers, passes = 0, 0.0, 0, 0, 0
    while spent < budget_s:         # a workload smaller than the budget is timed again
        before = spent
        passes += 1
        for case in cases:
            layers += passes == 1
            ctx = case.ctx_lens.cpu().numpy()
            S = case.n_shards.cpu().numpy()
            bt = case.block_table.cpu().numpy()
            q = case.q.double().cpu().numpy()
            for b in np.argsort(ctx)[::-1]:
                npg = -(-int(ctx[b]) // 16)
                idx = torch.as_tensor(bt[b, :npg], dtype=torch.long, device=case.k_cache.device)
                k = case.k_cache.index_select(0, idx).float().cpu().numpy()
                v = case.v_cache.index_select(0, idx).float().cpu().numpy()
                table = np.arange(npg)[None, :]
                t0 = time.perf_counter()
                po, pl = oracle.decode_split(q[b:b + 1], k, v, table, ctx[b:b + 1], S[b:b + 1],
                                             case.scale, int(S[b]))
                oracle.fold_combine(po, pl)
                spent += time.perf_counter() - t0
                done_bytes += int(ctx[b]) * 2 * Hkv * D * 2
                reqs += 1
                if spent >= budget_s:
                    break
            if spent >= budget_s:
                break
        if spent == before:
            break
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    return {"value": done_bytes / max(spent, 1e-9) / 1e9, "unit": "GB/s", "cores": int(threads),
            "kind": "oracle", "cpu_model": cpu_model(),
            "host_cores": len(os.sched_getaffinity(0)),
            "sample": f"{reqs} whole request(s) from the first {layers} layer(s) in {passes} "
                      f"pass(es) "
                      f"({done_bytes / 1e6:.0f} MB of KV, all "
                      f"{Hq} heads, per-shard partials + pairwise merge), {spent:.1f} s; host has "
                      f"{len(os.sched_getaffinity(0))} usable cores"}


def run_stage(args, dev):
    """Decode steps of a stack of Q-First blocks in the three orders of the same launches (one
    stream; the sweep on a second stream; the sweep and W_gate|W_up in one launch), each captured
    in a HIP graph, plus the attention side alone.  Each replay appends one position per layer,
    so the caches get room for every replay."""
    import torch

    from paper_2608_15473_amd.stage import MODES, LayerCache, QFirstStack
    from workloads import (BLOCKS, SCALE, STAGE_WORKLOADS, block_input, block_weights,
                           kv_bytes_per_position, make_case)

    w = STAGE_WORKLOADS[args.stage]
    shape = BLOCKS[w.block]
    L = args.layers or shape.layers
    K = args.steps if args.steps is not None else 10
    W = args.warmup if args.warmup is not None else 3
    order = list(MODES) + ["sweep_only"] + list(MODES)   # each mode twice, best kept
    room = 2 * len(MODES) * (K + W) + len(MODES) + 8
    log(f"[stage] generating {L} block(s) of {w.name}")
    layers, caches = [], []
    for l in range(L):
        layers.append(block_weights(shape, seed=1000 * w.index + l, device=dev))
        c = make_case(w.batch, shape.n_q_heads, shape.n_kv_heads, w.ctx + room, w.shards,
                      seed=1000 * w.index + 500 + l, device=dev)
        c.ctx_lens -= room
        caches.append(LayerCache(c.k_cache, c.v_cache, c.block_table, c.ctx_lens, c.n_shards))
    stack = QFirstStack(layers, caches, shape.n_q_heads, shape.n_kv_heads, w.shards, SCALE)
    u = block_input(w.batch, shape.hidden, seed=1000 * w.index + 999, device=dev)

    side = torch.cuda.Stream()                  # warm the libraries up before capturing
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        for mode in MODES:
            stack.step(u, mode=mode)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graphs = {mode: stack.capture(u, mode=mode)[0] for mode in MODES}
    sweep_graph = torch.cuda.CUDAGraph()        # the attention side alone, every layer
    with torch.cuda.graph(sweep_graph):
        for c in stack.caches:
            stack._sweep(c)
    graphs["sweep_only"] = sweep_graph

    ms = {}
    for name in order:
        g = graphs[name]
        for _ in range(W):
            g.replay()
        torch.cuda.synchronize()
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record()
        for _ in range(K):
            g.replay()
        t1.record()
        torch.cuda.synchronize()
        ms[name] = min(ms.get(name, float("inf")), t0.elapsed_time(t1) / K)
        log(f"[stage] {name}: {t0.elapsed_time(t1) / K:.4f} ms/step")
    kernels = stage_kernel_times(stack, u, w, shape)
    if int(stack.status.item()) != 0:
        raise RuntimeError("a cache ran out of room during the stage bench")
    top = max(kernels, key=lambda k: kernels[k]["avg_us"] * kernels[k]["per_block"])
    result = {
        "metric": "Q-First decode step, sweep beside the feed-forward (one shared launch)",
        "value": round(w.batch / (ms["fused"] * 1e-3), 1), "unit": "tokens/s",
        "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": round(ms["fused"], 4), "higher_is_better": True, "dtype": "bf16",
        "data": "synthetic",
        "serial_ms_per_step": round(ms["serial"], 4),
        "streams_ms_per_step": round(ms["streams"], 4),
        "fused_ms_per_step": round(ms["fused"], 4),
        "sweep_only_ms_per_step": round(ms["sweep_only"], 4),
        "speedup_vs_serial": round(ms["serial"] / ms["fused"], 4),
        "sweep_hidden_frac": round((ms["serial"] - ms["fused"]) / ms["sweep_only"], 4),
        "config": {"workload": w.name, "block": shape.name, "layers": L, "batch": w.batch,
                   "context": w.ctx, "shards": w.shards, "hidden": shape.hidden,
                   "inter": shape.inter, "n_q_heads": shape.n_q_heads,
                   "n_kv_heads": shape.n_kv_heads, "ffn_bytes_per_layer": shape.ffn_bytes(),
                   "kv_bytes_per_layer": w.batch * w.ctx * kv_bytes_per_position(shape.n_kv_heads),
                   "graphs": True},
        "kernels": kernels,
        "roofline": {"bound": "hbm", "achieved": kernels[top]["GB/s"], "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(kernels[top]["GB/s"] / HBM_PEAK_GBS, 4),
                     "kernel": top, "launch_avg_us": kernels[top]["avg_us"],
                     "algorithmic_bytes": kernels[top]["bytes"], "traffic": None},
    }
    if not args.no_cpu_baseline:
        log("[stage] cpu_baseline: timing the fp64 block oracle on a bounded sample")
        result["cpu_baseline"] = stage_cpu_baseline(stack, u, w, shape)
    result["env"] = env_info()
    if args.record:
        write_record(args.record, result)
    print(json.dumps(result), flush=True)


def stage_kernel_times(stack, u, w, shape, passes=2):
    """Average GPU time of each launch of a block (shared-launch order), from HIP events around
    every launch of an eager pass queued behind a GPU-side sleep (so the host's launch gaps are
    not inside the events), with each launch's algorithmic bytes."""
    import collections

    import torch

    spans = collections.defaultdict(list)

    class Span:
        def __init__(self, name):
            self.name = name

        def __enter__(self):
            self.e0 = torch.cuda.Event(enable_timing=True)
            self.e0.record()

        def __exit__(self, *exc):
            e1 = torch.cuda.Event(enable_timing=True)
            e1.record()
            spans[self.name].append((self.e0, e1))

    n = int(stack.caches[0].ctx_lens.float().mean().item()) + passes // 2  # positions swept
    stack.recorder = Span
    try:
        for _ in range(passes):
            torch.cuda._sleep(200_000_000)          # ~0.1 s of GPU time to queue behind
            stack.step(u, mode="fused")
            torch.cuda.synchronize()
    finally:
        stack.recorder = None
    B, H, I = w.batch, shape.hidden, shape.inter
    Hq, Hkv, D, S = shape.n_q_heads, shape.n_kv_heads, 128, w.shards

    def lin(N, K, xk=None, gain=True, res=False):
        xk = K if xk is None else xk
        return N * K * 2 + B * xk * 2 + (K * 2 if gain else 0) + B * N * 2 * (2 if res else 1)

    partials = B * S * Hq * (D + 1) * 4
    sweep = B * n * Hkv * D * 4 + B * (-(-n // 16)) * 4 + B * Hq * D * 2 + partials
    nbytes = {
        "W_q": lin(Hq * D, H),
        "sweep + W_gate,W_up": sweep + lin(2 * I, H) - B * I * 2,    # writes the activation
        "W_down": lin(H, I, gain=False, res=True),
        "W_k,W_v": lin(2 * Hkv * D, H),
        # partials, q, k_j and v_j read; out and lse written; k_j and v_j written to the cache and
        # ctx_lens read and advanced
        "merge, current-token fold + cache append": partials + B * Hq * D * 2
        + 2 * B * Hkv * D * 2 + B * Hq * (D * 2 + 4) + 2 * B * Hkv * D * 2 + 8 * B,
        "W_o": lin(H, Hq * D, gain=False, res=True),
    }
    out = {}
    for name, ev in spans.items():
        avg_s = sum(a.elapsed_time(b) for a, b in ev) / len(ev) / 1e3
        out[name] = {"avg_us": round(avg_s * 1e6, 2), "per_block": 1, "bytes": nbytes[name],
                     "GB/s": round(nbytes[name] / avg_s / 1e9, 1)}
    return out


def stage_cpu_baseline(stack, u, w, shape, budget_s=10.0):
    """The fp64 block oracle (oracle.qfirst_block) on the host, block after block from the same
    seeded input, until about ``budget_s`` of CPU work; decode tokens per second of the stack."""
    import numpy as np
    from threadpoolctl import threadpool_info

    import oracle

    x = u.double().cpu().numpy()
    blocks, spent = 0, 0.0
    while spent < budget_s:
        l = blocks % len(stack.layers)
        c = stack.caches[l]
        wts = {k: t.double().cpu().numpy() for k, t in stack.layers[l].items()
               if k not in ("w_gu", "w_kv")}
        kc, vc = c.k_cache.double().cpu().numpy(), c.v_cache.double().cpu().numpy()
        bt, ctx = c.block_table.cpu().numpy(), np.full(w.batch, w.ctx)
        t0 = time.perf_counter()
        x = oracle.qfirst_block(x, wts, kc, vc, bt, ctx, shape.n_q_heads, shape.n_kv_heads,
                                stack.scale)["y"]
        spent += time.perf_counter() - t0
        blocks += 1
    threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    steps = blocks / len(stack.layers)
    return {"value": round(w.batch * steps / spent, 4), "unit": "tokens/s", "cores": int(threads),
            "kind": "oracle", "cpu_model": cpu_model(),
            "host_cores": len(os.sched_getaffinity(0)),
            "sample": f"{blocks} block(s) of the stack at context {w.ctx} (fp64 numpy, q/k/v, "
                      f"feed-forward and attention over the cache plus the current token), "
                      f"{spent:.1f} s; host has {len(os.sched_getaffinity(0))} usable cores"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps (default: at least 10 and at least 0.25 s of work)")
    ap.add_argument("--warmup", type=int, default=None,
                    help="untimed steps first (default: at least 3 and at least 0.3 s; short "
                         "runs measure a slower cold phase of the GPU)")
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--layers", type=int, default=None,
                    help="resident layers (default: the workload's own count)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--one-launch", action="store_true",
                    help="sweep and merge in one launch (qf_attn_decode): faster only where "
                         "launches dominate (small steps)")
    ap.add_argument("--stage", default=None,
                    help="time the [MLP || Attn] decode stage of this block workload instead")
    ap.add_argument("--record", default=None,
                    help="also append the result line to this run-record file (JSON)")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="instead of the bench: one plain device copy of this many MiB (the "
                         "known-size reference that scales the FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path "
              "(position sharding across GPUs is a design note, not code).", file=sys.stderr)
        sys.exit(2)

    import torch

    import paper_2608_15473_amd as qf
    from workloads import WORKLOADS, workload_case

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    qf.load_library()
    dev = torch.device("cuda:0")
    if args.copy_calibration_mib:
        n = args.copy_calibration_mib << 20
        src = torch.ones(n // 4, dtype=torch.int32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n, "read_bytes": n, "write_bytes": n}))
        return
    if args.stage:
        run_stage(args, dev)
        return
    w = WORKLOADS[args.workload]
    L = args.layers or w.layers
    # Cold reads only: a workload whose layers fit the Infinity Cache twice over gets that many
    # distinct resident copies, and each step reads the next L of them in turn.
    first = workload_case(w.name, layer=0, device=dev)
    copies = max(L, -(-2 * INFINITY_CACHE_BYTES // max(1, first.kv_bytes())))
    log(f"[bench] generating {copies} layer(s) of {w.name} on {torch.cuda.get_device_name(0)}")
    t0 = time.time()
    cases = [first] + [workload_case(w.name, layer=l, device=dev) for l in range(1, copies)]
    torch.cuda.synchronize()
    log(f"[bench] inputs resident in {time.time() - t0:.1f} s")
    B, Hq, Hkv, D = cases[0].shape
    S = cases[0].max_shards
    ab = [algorithmic_bytes(c) for c in cases]

    desc = qf.make_desc(cases[0].q, cases[0].k_cache, cases[0].block_table, S, cases[0].scale)
    # The two-launch step leaves a chunked shape's sub-shard chunks as slots of the partials (the
    # combine merges them directly: no chunk fold launch), so it needs S * C slots, no workspace.
    C = 1 if args.one_launch else qf.split_chunks(desc)
    po = torch.empty((B, S * C, Hq, D), dtype=torch.float32, device=dev)
    pl = torch.empty((B, S * C, Hq), dtype=torch.float32, device=dev)
    out = torch.empty((B, Hq, D), dtype=torch.bfloat16, device=dev)
    lse = torch.empty((B, Hq), dtype=torch.float32, device=dev)
    need = qf.decode_workspace_size(desc) if args.one_launch else 0
    ws = torch.empty(max(need, 16), dtype=torch.uint8, device=dev)
    counters = torch.zeros(B * Hkv, dtype=torch.int32, device=dev)  # zero-filled once

    turn = [0]
    # The two-launch step of each resident copy, checked and converted once (the host then does
    # two foreign calls per layer; the small single-layer workload is otherwise host-bound).
    # Every launch goes to one stream of our own (default priority): the legacy null stream
    # synchronises implicitly with other streams, which costs launch-bound steps a few percent.
    run_stream = torch.cuda.Stream(dev)
    plans = [] if args.one_launch else [
        qf.DecodeStepPlan(c.q, c.k_cache, c.v_cache, c.block_table, c.ctx_lens, c.n_shards,
                          max_shards=S, scale=c.scale, part_out=po, part_lse=pl, out=out, lse=lse,
                          fold_chunks=False, stream=run_stream.cuda_stream) for c in cases]
    torch.cuda.synchronize()

    # The sweep's launch duration is timed with HIP events on a sample of the timed region's
    # launches: every EVERY-th sweep (one layer per step for a model of 8+ layers; for fewer
    # layers every 8th to 64th step, at least ~32 launches in all).  Events around every launch
    # would add their cost to each step, which on the launch-bound workloads (one small layer, the
    # per-GPU share) is a large part of a step: on the small single layer one pair per 8 steps
    # still added ~0.7 us to an ~11 us step.
    EVERY = L
    launches = [0]

    def step(events=None):
        base = turn[0]
        turn[0] += L
        for l in range(L):
            c = cases[(base + l) % copies]
            timed = events is not None and launches[0] % EVERY == 0
            launches[0] += 1
            if timed:
                pair = (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                events.append(pair)
                pair[0].record()
            if not args.one_launch:
                plans[(base + l) % copies].split()
            else:
                qf.attn_decode(c.q, c.k_cache, c.v_cache, c.block_table, c.ctx_lens,
                               c.n_shards, max_shards=S, scale=c.scale, out=out, lse=lse,
                               workspace=ws, counters=counters)
            if timed:
                pair[1].record()
            if not args.one_launch:
                plans[(base + l) % copies].combine()

    with torch.cuda.stream(run_stream):
        # Warm-up: the same steps back to back, so that the GPU is busy throughout and reaches
        # its steady clocks before the timed region.  Without --warmup: three synchronized steps
        # estimate the step time, then back-to-back steps for >= WARMUP_SECONDS, synchronized
        # after every ~10 ms of work so that the host never runs far ahead of the GPU.  (A
        # synchronization after every warm-up step left the GPU idle between steps, and the small
        # single layer then timed ~15 us per step instead of ~11.)
        warm, t_w = 0, time.perf_counter()
        if args.warmup is not None:
            for _ in range(args.warmup):
                step()
            warm = args.warmup
        else:
            for _ in range(3):
                step()
                torch.cuda.synchronize()
            warm = 3
            batch = max(1, int(0.01 * warm / max(time.perf_counter() - t_w, 1e-6)))
            while time.perf_counter() - t_w < WARMUP_SECONDS:
                for _ in range(batch):
                    step()
                torch.cuda.synchronize()
                warm += batch
        torch.cuda.synchronize()
        per_step = (time.perf_counter() - t_w) / max(1, warm)
        if args.steps is None:
            args.steps = max(10, int(TIMED_SECONDS / max(per_step, 1e-6)) + 1)
        if L < 8:
            EVERY = max(8, min(64, args.steps // 32)) * L
        args.warmup = warm
        log(f"[bench] warmup done ({warm} steps); timing {args.steps} steps")
        ev = []
        launches[0] = 0
        torch.cuda.synchronize()
        t_start = time.perf_counter()
        for k in range(args.steps):
            step(ev)
        torch.cuda.synchronize()
        elapsed = time.perf_counter() - t_start
    ms_per_step = elapsed * 1e3 / args.steps
    sweep_ms = [a.elapsed_time(b) for a, b in ev]
    sweep_avg_s = sum(sweep_ms) / len(sweep_ms) / 1e3
    log(f"[bench] {ms_per_step:.3f} ms/step, sweep launch avg {sweep_avg_s * 1e6:.1f} us "
        f"({len(sweep_ms)} timed launches)")

    ab = ab[:L]                     # every copy has the same lengths, so the same bytes
    kv_step = sum(a["kv"] for a in ab)
    value = kv_step / (ms_per_step / 1e3) / 1e9
    attended = sum(a["attended"] for a in ab) / L
    sweep_bytes = sum(a["sweep"] + (a["combine"] if args.one_launch else 0) for a in ab) / L
    achieved = sweep_bytes / sweep_avg_s / 1e9
    result = {
        "metric": "decode-attention KV GB/s (and % of HBM peak); attended tokens/s per layer",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": w.name, "launches_per_layer": 1 if args.one_launch else 2,
                   "batch": B, "n_q_heads": Hq, "n_kv_heads": Hkv,
                   "head_dim": D, "page": 16, "layers": L, "max_shards": S,
                   "context": w.ctx if w.ctx else "ragged", "kv_dtype": "bf16",
                   "kv_bytes_per_step": kv_step, "workspace_bytes": need,
                   "chunks_per_shard": C,
                   "resident_layer_copies": copies},
        "hbm_peak_frac": round(value / HBM_PEAK_GBS, 4),
        "attended_tokens_per_s_per_layer": round(attended / (ms_per_step / 1e3 / L), 1),
        "roofline": {"bound": "hbm", "achieved": round(achieved, 2), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                     "kernel": "decode_fused_kernel" if args.one_launch else "decode_split_kernel",
                     "launch_avg_us": round(sweep_avg_s * 1e6, 2),
                     "timed_launches": len(sweep_ms),
                     "algorithmic_bytes": int(sweep_bytes),
                     "traffic": committed_traffic(w.name, not args.one_launch)
                     if L == w.layers else None},
    }
    if not args.no_cpu_baseline:
        log("[bench] cpu_baseline: timing the fp64 oracle on a bounded sample")
        result["cpu_baseline"] = cpu_baseline(cases[:L])
    result["env"] = env_info()
    if args.record:
        write_record(args.record, result)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
