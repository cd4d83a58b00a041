"""Benchmark of one SmallKV decode step on one MI355X.

A step is the whole hot path over one batch: stage 1 (small-model decode
attention over all its layers), stage 2 (partition of every small head),
stage 3 (hybrid attention of every large layer).  The default workload is
the largest configuration: the LLaMA-3-8B (32 layers, 32q/8kv, d=128) +
LLaMA-3.2-1B (16 layers, 32q/8kv, d=64) shapes, bf16, batch 16, context
32768, critical 5% / marginal 15%, 5% heavy hitters.  `--workload N` selects
another: 2 the Qwen2-7B + Qwen2-0.5B step at batch 1 and N = 8192; 4 the
ragged batch-64 decode over 256 drifting steps (value = 64 * 256 / the time
of all 256 steps); 5 the Qwen2-72B + Qwen2-0.5B step at N = 65536 whose large
KV is held only for the retained tokens (the compact store is built from the
step's own lists before timing, untimed, and the full cache freed).

Timing: inputs are resident in HBM; each step is a HIP-graph replay (the
drifting workload launches its steps directly, each with its own queries and
lengths).  W warm-up steps, then exactly K timed steps between two
synchronisations (`value` and `ms_per_step`).  Small workloads rotate over
`--rotate` input copies so that a step never finds the previous step's
operands in the 256 MB MALL.  Then three timing passes with HIP events:
  * per step, with the caches flushed before it (a 1 GiB write): the step's
    own kernels through smallkv_step_events, which records events at the
    stage boundaries -- median, p10 and p90 of the step, the stage means,
    and the roofline of the dominant stage (its algorithmic bytes over its
    event time against 8 TB/s);
  * the same without the flush (warm);
  * the per-layer-launch variant: stages 1 and 2 through their single-stage
    calls, then stage 3 as one smallkv_hybrid_attn_layers call per large
    layer, as a model that runs its layers one after another calls it.
The CPU baseline is the oracle on one pinned host core over one sequence's
whole step (the sample is named in the line).

Prints one JSON line.

`--match` benchmarks the prefill similarity matching instead (Eqs. 1-3: the
step before decoding that computes the head map); `--store` the retained-store
maintenance after a step.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time
import types

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, 8 TB/s
FP32_VECTOR_PEAK_TFLOPS = 157.3  # MI355X fp32 vector (packed FMA counted as 4 flops)
DEFAULT_STEPS = {2: 100, 4: 256}  # others: 20
FLUSH_BYTES = 1 << 30  # written before each flushed step: above L2 and the 256 MB MALL


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=None,
                   help="timed steps (default: 256 for the drifting workload, 100 for "
                        "workload 2, else 20)")
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--rotate", type=int, default=4, help="input copies cycled through")
    p.add_argument("--workload", type=int, default=3,
                   help="3: the LLaMA batch-16 step (default, the largest); 2: Qwen2-7B batch 1; "
                        "4: ragged batch 64 over 256 drifting steps; 5: Qwen2-72B on a compact "
                        "store; 1, 6-10: the other workloads")
    p.add_argument("--eager", action="store_true", help="launch without HIP graphs")
    p.add_argument("--cpu-seconds", type=float, default=12.0, help="oracle time budget")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-extra-passes", action="store_true",
                   help="only the timed steps and the stage events (for profiler runs)")
    p.add_argument("--match", action="store_true",
                   help="benchmark the prefill head matching instead of the decode step")
    p.add_argument("--store", action="store_true",
                   help="benchmark the retained-store maintenance after a step")
    p.add_argument("--store-hbm-only", action="store_true",
                   help="with --store: only the timed rebuild from HBM (for counter runs)")
    p.add_argument("--match-batch", type=int, default=1)
    p.add_argument("--match-window", type=int, default=200)
    p.add_argument("--copy-probe-mib", type=int, default=0,
                   help="first run a plain device copy of this many MiB (counter calibration)")
    a = p.parse_args()
    if a.steps is None:
        a.steps = 20 if (a.match or a.store) else DEFAULT_STEPS.get(a.workload, 20)
    return a


def source_hash(name: str) -> str:
    path = os.path.join(ROOT, "paper_2508_02751_amd", "csrc", name)
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def traffic_file(workload: str) -> str:
    return os.path.join(ROOT, "profiles", f"traffic_{workload}.json")


def load_traffic(kernels, workload: str, path: str = None):
    """HBM bytes of one stage (the sum over its kernels) from the committed
    rocprofv3 --pmc summary of this workload, or None when there is none, a
    kernel is missing, or its source changed since the counters were taken."""
    path = path or traffic_file(workload)
    if not os.path.exists(path):
        return None
    try:
        doc = json.load(open(path))
        if doc.get("workload") != workload:
            return None
        t = doc["kernels"]
        total = 0.0
        for k in kernels:
            e = t[k]
            if e.get("source_sha256_16") != source_hash(e["source"]):
                return None
            total += e["hbm_bytes_per_launch"]
        return total
    except (KeyError, ValueError, TypeError):
        return None


def copy_probe(args, dev):
    """A plain device copy of known size, for the counter calibration."""
    import torch
    if args.copy_probe_mib:
        src = torch.ones(args.copy_probe_mib << 18, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst


def shape_text(m) -> str:
    return f"{m.layers} layers, {m.q_heads}q/{m.kv_heads}kv, d={m.head_dim}"


def budget_text(spec) -> str:
    kind, v = spec
    return f"{v}%" if kind == "pct" else f"{v} tokens"


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def stage3_kernels(w, layers=None):
    """Kernels one stage-3 call launches for workload w: the grouped kernel for
    bf16, head_dim 128 and at most 8 query heads per kv head (plus the merge
    of its token splits when it splits, the library's rule), the per-head
    kernel otherwise."""
    L = w.large
    if w.dtype != "bf16" or L.head_dim != 128 or L.group > 8:
        return ["hybrid_kernel"]
    units = w.batch * (layers or L.layers) * L.kv_heads
    n_cap = w.n_cap
    cost = lambda c: -(-units * c // 512) * (-(-n_cap // c) + 384)
    s = 1
    for c in range(2, min(32, -(-n_cap // 256)) + 1):
        if cost(c) < cost(s):
            s = c
    span = -(-(-(-n_cap // s)) // 256) * 256
    return ["hybrid_group_kernel", "hybrid_group_merge"] if -(-n_cap // span) > 1 \
        else ["hybrid_group_kernel"]


def stage_kernels(w):
    """The kernels inside each of smallkv_step_events' three windows."""
    if w.select == 1:
        return [["small_attn_mfma", "small_attn_merge"],
                ["group_zq", "group_scores", "partition_kernel", "group_weights"],
                stage3_kernels(w)]
    if w.select == 2:
        return [["small_attn_mfma", "small_attn_merge"],
                ["group_zq", "accum_scores", "partition_kernel", "group_weights"],
                stage3_kernels(w)]
    s1 = "small_attn_valu" if w.dtype == "f32" else "small_attn_mfma"
    return [[s1], ["partition_kernel"], stage3_kernels(w)]


def pct(xs, q):
    xs = sorted(xs)
    k = (len(xs) - 1) * q
    lo, hi = int(k), min(int(k) + 1, len(xs) - 1)
    return xs[lo] + (xs[hi] - xs[lo]) * (k - lo)


def host_cpu():
    model = None
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count()
    return {"host_cpu": model, "host_nproc": os.cpu_count(), "host_cpus_available": avail}


# ----------------------------------------------------------- inputs --------

def compact_store(w, x, dev):
    """The large model's KV held only for the retained tokens: the step's own
    lists, the store built from them by smallkv_store_update (rows = the
    largest union over the kv heads), the full cache freed.  Untimed."""
    import torch
    from paper_2508_02751_amd import smallkv as S
    from paper_2508_02751_amd.pipeline import prepare_step

    ps = prepare_step(x)
    ps.run()
    nsh = ps.buf.logits.shape[1]
    probe = S.prepare_store(ps.batch, ps.head_map, nsh, ps.buf.crit_idx, ps.buf.marg_idx,
                            x["l_k"], x["l_v"], 1)
    probe.run()
    torch.cuda.synchronize()
    rows = int(probe.counts.max())
    del probe
    st = S.prepare_store(ps.batch, ps.head_map, nsh, ps.buf.crit_idx, ps.buf.marg_idx,
                         x["l_k"], x["l_v"], rows)
    st.run()
    torch.cuda.synchronize()
    k_union = st.counts[..., 0].to(torch.float64).mean().item() / w.n_cap
    v_union = st.counts[..., 1].to(torch.float64).mean().item() / w.n_cap
    store = {"l_k": st.new_k, "l_v": st.new_v, "k_slot": st.k_slot, "v_slot": st.v_slot}
    del ps, st  # (both hold the full cache)
    x.pop("l_k")
    x.pop("l_v")
    torch.cuda.empty_cache()
    log(f"compact store: {rows} rows per kv head of {w.n_cap} (unions: critical "
        f"{k_union:.3f}, critical+marginal {v_union:.3f} of the tokens); full cache freed")
    info = {"large_store": "compact: retained rows only, read through slot maps",
            "store_rows_per_kv_head": rows, "union_frac_k": k_union, "union_frac_v": v_union}
    return store, info


def prepare(x, store):
    from paper_2508_02751_amd.pipeline import prepare_step
    if store is None:
        return prepare_step(x)
    return prepare_step(x, k_slot=store["k_slot"], v_slot=store["v_slot"], l_k=store["l_k"],
                        l_v=store["l_v"])


def bytes_of(ps, store):
    from paper_2508_02751_amd.bytes_model import step_bytes
    x = dict(ps.inputs)
    if store is not None:
        x["l_k"] = store["l_k"]
    return step_bytes(x, ps.buf.crit_idx, ps.buf.marg_idx, ps.batch.km_cap)


# ----------------------------------------------------------- passes --------

def event_pass(preps, K, stream, flush=None):
    """Per step (preps cycled): events at the stage boundaries of the step's
    own kernels; returns per-step stage and step times in ms."""
    import torch
    from paper_2508_02751_amd import smallkv as S
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
    torch.cuda._sleep(50_000_000)  # keep the GPU busy while the host enqueues
    for i in range(K):
        ps = preps[i % len(preps)]
        if flush is not None:
            # read (not write) 1 GiB: L2 and the MALL end up holding clean
            # lines of the flush buffer, so the step pays no write-backs
            flush.sum(dtype=torch.int32)
        S.smallkv_step_events(ps.desc, ps.buf.ws, ev[i], stream)
    torch.cuda.synchronize()
    stages = [[ev[i][s].elapsed_time(ev[i][s + 1]) for i in range(K)] for s in range(3)]
    steps = [ev[i][0].elapsed_time(ev[i][3]) for i in range(K)]
    return stages, steps


def per_layer_variant(ps, K, W, use_graph):
    """Stages 1-2 through the single-stage calls, stage 3 as one call per
    large layer; mean ms per step over K graph replays."""
    import torch
    from paper_2508_02751_amd import smallkv as S
    b = ps.buf
    nsh = b.logits.shape[1]
    L = ps.large.q.shape[1]
    ws = torch.empty(max(1, S.smallkv_hybrid_attn_workspace_size(ps.batch, ps.large, 1, nsh),
                         b.ws.numel() if b.ws is not None else 1), dtype=torch.uint8,
                     device=b.logits.device)

    def run():
        S.smallkv_small_attn(ps.batch, ps.small, b.logits, b.row_max, b.row_sum, ws)
        S.smallkv_partition(ps.batch, nsh, b.logits, b.row_max, b.row_sum, b.crit_idx,
                            b.marg_idx, b.marg_prob, b.mass, None, small=ps.small)
        for layer in range(L):
            S.smallkv_hybrid_attn_layers(ps.batch, ps.large, layer, 1, ps.head_map, nsh,
                                         b.crit_idx, b.marg_idx, b.marg_prob, b.mass, ps.mode,
                                         ws)

    for _ in range(max(W, 1)):
        run()
    torch.cuda.synchronize()
    g = None
    if use_graph:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            run()
        g.replay()
        torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(K):
        g.replay() if g is not None else run()
    torch.cuda.synchronize()
    return (time.perf_counter() - t0) * 1e3 / K, L


def cpu_baseline(args, w, ps, store):
    """The oracle on one pinned host core over sequence 0's whole step (all
    layers of both models): one token of the metric per run."""
    import numpy as np
    import torch
    sys.path.insert(0, os.path.join(ROOT, "oracle"))
    import oracle as O
    from paper_2508_02751_amd.pipeline import softmax_scale

    def h(t):
        t = t[0:1]
        return t.detach().float().cpu().numpy() if t.dtype == torch.bfloat16 else t.cpu().numpy()

    x = ps.inputs
    host = {k: h(x[k]) for k in ("seq_len", "k_crit", "k_marg", "s_q", "s_k", "s_v", "l_q")}
    host["head_map"] = x["head_map"].cpu().numpy()
    host["l_k"] = h(store["l_k"] if store else x["l_k"])
    host["l_v"] = h(store["l_v"] if store else x["l_v"])
    extra = {}
    if store is not None:
        extra["k_slot"], extra["v_slot"] = h(store["k_slot"]), h(store["v_slot"])
    if x.get("k_recent") is not None:
        extra["k_recent"] = h(x["k_recent"])
    if x.get("s_held") is not None:
        extra.update(s_held=h(x["s_held"]), s_row_pos=h(x["s_row_pos"]), n_cap=x["n_cap"])
    if w.select == 1:
        extra["select"] = O.SELECT_GROUP
    if w.select == 2:
        extra["select"] = O.SELECT_ACCUM
        extra["acc"] = np.zeros((1,) + tuple(ps.buf.acc_score.shape[1:]), np.float32)
    cpu_info = host_cpu()  # before pinning
    try:
        os.sched_setaffinity(0, {sorted(os.sched_getaffinity(0))[0]})
    except (AttributeError, OSError):
        pass
    log("timing the CPU oracle")
    reps, spent = 0, 0.0
    while reps < 1 or spent < args.cpu_seconds:
        c0 = time.perf_counter()
        O.step(seq_len=host["seq_len"], k_crit=host["k_crit"], k_marg=host["k_marg"],
               kc_cap=int(x["kc_cap"]), km_cap=int(x["km_cap"]), head_map=host["head_map"],
               mode=O.NORM_REMAINING, s_q=host["s_q"], s_k=host["s_k"], s_v=host["s_v"],
               s_scale=softmax_scale(w.small.head_dim), l_q=host["l_q"], l_k=host["l_k"],
               l_v=host["l_v"], l_scale=softmax_scale(w.large.head_dim), **extra)
        spent += time.perf_counter() - c0
        reps += 1
    n0 = int(host["seq_len"][0])
    what = ("the whole decode step" if w.batch == 1 else
            f"sequence 0 of {w.batch} (N = {n0}): its whole decode step, every layer of both "
            f"models; the step's rate is {w.batch}x this sample's work")
    return {"value": reps / spent, "unit": "tokens/s", "cores": 1, "kind": "oracle",
            "sample": f"{reps} run(s) of {what}, single-threaded C oracle pinned to one core "
                      f"({spent:.1f} s)", **cpu_info}


# ----------------------------------------------------------- main ----------

def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py: the library runs on one GPU; sharding the step over several GPUs "
              "is not implemented, so --gpus must be 1", file=sys.stderr)
        sys.exit(2)
    if args.match:
        return bench_match(args)
    if args.store:
        return bench_store(args)
    import torch
    from paper_2508_02751_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = W.WORKLOADS[args.workload]
    copy_probe(args, dev)
    log(f"generating {w.name}")
    if w.steps > 1:
        return bench_drift(args, w, dev)
    x0 = W.make_step_inputs(w, dev)
    store, store_info = (compact_store(w, x0, dev) if w.compact_large else (None, {}))
    copy_bytes = sum(v.numel() * v.element_size() for v in x0.values() if torch.is_tensor(v))
    if store is not None:
        copy_bytes += sum(v.numel() * v.element_size() for v in store.values())
    if copy_bytes > (16 << 30):  # far beyond the 256 MB MALL already; keep HBM free
        args.rotate = 1
    copies = [x0]
    for _ in range(args.rotate - 1):
        copies.append({k: (v.clone() if torch.is_tensor(v) else v) for k, v in x0.items()})
    preps = [prepare(x, store) for x in copies]
    stream = torch.cuda.current_stream()

    # warm-up (eager), also builds the partitions used for byte accounting
    for i in range(max(args.warmup, 1)):
        preps[i % len(preps)].run()
    torch.cuda.synchronize()
    graphs = None
    if not args.eager:
        graphs = []
        for ps in preps:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                ps.run()
            graphs.append(g)
        for i in range(max(args.warmup, 1)):
            graphs[i % len(graphs)].replay()
        torch.cuda.synchronize()

    # ---- timed region: exactly K steps ------------------------------------
    K = args.steps
    log(f"timing {K} steps")
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(K):
        if graphs is not None:
            graphs[i % len(graphs)].replay()
        else:
            preps[i % len(preps)].run()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / K

    # ---- the step's own kernels, by stage, with HIP events -----------------
    flush = torch.zeros(FLUSH_BYTES, dtype=torch.uint8, device=dev)
    stages, steps = event_pass(preps, K, stream, flush)
    del flush
    extra = {}
    if not args.no_extra_passes:
        _, warm = event_pass(preps[:1], K, stream)  # the same inputs step after step
        extra["warm_no_flush_ms"] = {"median": statistics.median(warm), "p10": pct(warm, 0.1),
                                     "p90": pct(warm, 0.9)}
        del graphs
        if w.select == 0:  # (the single-stage path of per-head selection)
            ml, L = per_layer_variant(preps[0], K, args.warmup, not args.eager)
            extra["per_layer_launch"] = {
                "ms_per_step": ml, "tokens_per_s": w.batch * 1e3 / ml,
                "launches": f"small attention, partition, then {L} stage-3 calls (one per "
                            f"large layer)"}

    ps = preps[0]
    sb = bytes_of(ps, store)
    out = result_line(args, w, K, ms_per_step, stages, steps, sb, store_info)
    out["step"].update(extra)
    out["cpu_baseline"] = None if args.no_cpu_baseline else cpu_baseline(args, w, ps, store)
    print(json.dumps(out), flush=True)


def result_line(args, w, K, ms_per_step, stages, steps, sb, store_info, value=None, n_tok=None):
    stage_ms = [sum(x) / len(x) for x in stages]
    stage_bytes = [sb.stage1, sb.stage2, sb.stage3]
    dom = max(range(3), key=lambda s: stage_ms[s])
    kern = stage_kernels(w)
    achieved = stage_bytes[dom] / (stage_ms[dom] * 1e-3) / 1e9
    step_gbs = sb.step_compulsory / (ms_per_step * 1e-3) / 1e9
    group = w.select == 1
    return {
        "metric": "SmallKV decode-step attention tokens/s at 1 MI355X; % of HBM roofline",
        "value": value if value is not None else w.batch * 1e3 / ms_per_step,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if w.dtype == "bf16" else "f32",
        "data": "synthetic",
        "config": {
            "workload": w.name,
            "large": shape_text(w.large), "small": shape_text(w.small),
            "kv_dtype": w.dtype, "batch": w.batch, "context": w.n_ctx,
            **({"context_range": f"{w.ragged_min}..{w.n_ctx} + {w.steps} decode steps"}
               if w.ragged_min else {}),
            "critical": budget_text(w.crit), "marginal": budget_text(w.marg),
            **({"heavy_hitters": f"{int(100 * w.heavy_frac)}%"} if w.heavy_frac else {}),
            **({"recent": budget_text(w.recent)} if w.recent != ("abs", 0) else {}),
            **({"small_cache_kept": f"{w.slm_keep}%"} if w.slm_keep else {}),
            **({"selection": "one per large kv head (summed)"} if group else {}),
            **({"selection": "accumulated scores (running state)"} if w.select == 2 else {}),
            **store_info,
            "launch": "eager" if (args.eager or w.steps > 1) else "hip-graph",
            "rotated_input_copies": 1 if w.steps > 1 else args.rotate,
        },
        "roofline": {
            "kernel": "+".join(kern[dom]),
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": load_traffic(kern[dom], w.name),
        },
        "step": {
            "compulsory_bytes": sb.step_compulsory,
            "achieved_GBs": step_gbs,
            "hbm_frac": step_gbs / HBM_PEAK_GBS,
            "flushed_event_ms": {"median": statistics.median(steps), "p10": pct(steps, 0.1),
                                 "p90": pct(steps, 0.9)},
            "stage_ms": stage_ms,
            "stage_kernels": ["+".join(k) for k in kern],
            "stage_bytes": stage_bytes,
            "stage_GBs": [stage_bytes[s] / (stage_ms[s] * 1e-3) / 1e9 for s in range(3)],
            "large_rows_per_head_over_union": (sb.large_k_perhead + sb.large_v_perhead)
            / max(1, sb.large_k_union + sb.large_v_union),
            "index_metadata_bytes": sb.index_meta,
        },
    }


def bench_drift(args, w, dev):
    """The ragged batch over its consecutive drifting decode steps: every
    step has its own queries and lengths (one descriptor each, sharing the
    caches, the intermediates and the workspace); value = batch x steps / the
    time of all the steps."""
    import dataclasses

    import torch
    from paper_2508_02751_amd import smallkv as S
    from paper_2508_02751_amd import workloads as W
    from paper_2508_02751_amd.pipeline import prepare_step

    z = W.latents(w, dev)
    x = W.make_step_inputs(w, dev, 0, z=z)
    base = prepare_step(x)
    K = args.steps
    n_steps = min(K, w.steps)
    log(f"queries and lengths of {n_steps} steps")
    descs = []
    for t in range(n_steps):
        s_q, l_q = W.step_queries(w, z, t, dev)
        n, kc, km = W.budgets(w, t)
        batch = dataclasses.replace(base.batch, seq_len=n.to(dev), k_crit=kc.to(dev),
                                    k_marg=km.to(dev))
        small = dataclasses.replace(base.small, q=s_q.contiguous())
        large = dataclasses.replace(base.large, q=l_q.contiguous())
        b = base.buf
        desc = S.make_step(batch, small, large, base.head_map, base.mode, b.logits, b.row_max,
                           b.row_sum, b.crit_idx, b.marg_idx, b.marg_prob, b.mass)
        descs.append(dataclasses.replace(base, batch=batch, small=small, large=large, desc=desc))
    stream = torch.cuda.current_stream()
    for i in range(max(args.warmup, 1)):
        descs[i % n_steps].run()
    torch.cuda.synchronize()
    log(f"timing {K} steps")
    t0 = time.perf_counter()
    for i in range(K):
        descs[i % n_steps].run()
    torch.cuda.synchronize()
    total_ms = (time.perf_counter() - t0) * 1e3
    ms_per_step = total_ms / K
    stages, steps = event_pass(descs, K, stream)  # 9 GB per step: no cache holds it
    # bytes: every step's own partition (recomputed, untimed)
    log("byte accounting of every step")
    comp = s1 = s2 = s3 = kper = kun = meta = 0
    for t in range(n_steps):
        d = descs[t]
        d.run()
        xi = dict(x)
        xi["s_q"], xi["l_q"], xi["seq_len"] = d.small.q, d.large.q, d.batch.seq_len
        sb = bytes_of(dataclasses.replace(d, inputs=xi), None)
        comp += sb.step_compulsory
        s1, s2, s3 = s1 + sb.stage1, s2 + sb.stage2, s3 + sb.stage3
        kper += sb.large_k_perhead + sb.large_v_perhead
        kun += sb.large_k_union + sb.large_v_union
        meta += sb.index_meta
    torch.cuda.synchronize()
    mean = types.SimpleNamespace(
        stage1=s1 / n_steps, stage2=s2 / n_steps, stage3=s3 / n_steps,
        step_compulsory=comp / n_steps, large_k_perhead=kper / n_steps, large_v_perhead=0,
        large_k_union=kun / n_steps, large_v_union=0, index_meta=meta / n_steps)
    value = w.batch * K / (total_ms * 1e-3)
    out = result_line(args, w, K, ms_per_step, stages, steps, mean, {}, value=value)
    out["config"]["timed_steps"] = f"decode steps 0..{n_steps - 1}" + (
        f", cycled to {K}" if K > n_steps else "")
    out["step"]["lengths"] = {"first_step": [int(descs[0].batch.seq_len.min()),
                                             int(descs[0].batch.seq_len.max())],
                              "last_step": [int(descs[-1].batch.seq_len.min()),
                                            int(descs[-1].batch.seq_len.max())]}
    out["cpu_baseline"] = None if args.no_cpu_baseline else cpu_baseline(args, w, descs[0], None)
    print(json.dumps(out), flush=True)


def bench_store(args):
    """Retained-store maintenance after one step of the workload: a rebuild
    from the full store in HBM (the roofline), and the update after a drifted
    step, which reuses the rows the previous store holds and reads only the
    others from the full store (the rows a host-resident full store would
    have to send)."""
    import torch
    from paper_2508_02751_amd import smallkv as S
    from paper_2508_02751_amd import workloads as W
    from paper_2508_02751_amd.pipeline import prepare_step

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = W.WORKLOADS[args.workload]
    copy_probe(args, dev)
    print(f"[bench] generating {w.name}", file=sys.stderr, flush=True)
    x = W.make_step_inputs(w, dev)
    ps = prepare_step(x)
    ps.run()
    L = w.large
    g = L.group
    rows = min(w.n_cap, g * (int(x["kc_cap"]) + int(x["km_cap"])))
    nsh = ps.buf.logits.shape[1]
    K = args.steps
    stream = torch.cuda.current_stream()

    def timed(call):
        for _ in range(max(args.warmup, 1)):
            call.run()
        torch.cuda.synchronize()
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
              for _ in range(K)]
        torch.cuda._sleep(50_000_000)
        for e0, e1 in ev:
            e0.record(stream)
            call.run(stream)
            e1.record(stream)
        torch.cuda.synchronize()
        return sum(a.elapsed_time(b) for a, b in ev) / K

    def store(full_k, full_v, old=None):
        return S.prepare_store(ps.batch, ps.head_map, nsh, ps.buf.crit_idx, ps.buf.marg_idx,
                               full_k, full_v, rows, old=old)

    hbm = store(x["l_k"], x["l_v"])
    ms_hbm = timed(hbm)
    cnt = hbm.counts.to(torch.int64)
    row_b = L.head_dim * x["l_k"].element_size()
    moved = int(cnt.sum()) * row_b                       # rows read once, written once
    units = cnt.shape[0] * cnt.shape[1] * cnt.shape[2]
    n_tok = int(x["seq_len"].to(torch.int64).sum()) // w.batch
    maps = units * n_tok * 8                             # two slot maps written
    lists = ps.buf.crit_idx.numel() * 4 + ps.buf.marg_idx.numel() * 4
    alg = 2 * moved + maps + lists
    achieved = alg / (ms_hbm * 1e-3) / 1e9
    traffic = load_traffic(["store_index", "store_copy"], f"{w.name}-store",
                           os.path.join(ROOT, "profiles", "traffic_store.json"))
    legs = None
    if not args.store_hbm_only:
        legs = store_legs(args, w, x, ps, store, timed, stream, moved, rows)
    out = {
        "metric": "SmallKV retained-store maintenance updates/s at 1 MI355X",
        "value": 1e3 / ms_hbm,
        "unit": "updates/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_hbm,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": f"{w.name}-store", "rows_per_kv_head": rows,
                   "union_rows": int(cnt.sum()), "kv_heads": units},
        "roofline": {"kernel": "store_index+store_copy", "bound": "hbm", "achieved": achieved,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS,
                     "traffic": traffic},
    }
    if legs:
        out.update(legs)
    print(json.dumps(out), flush=True)


def store_legs(args, w, x, ps, store, timed, stream, moved, rows):
    """The store bench's other legs: the oracle on the host, the update after
    a drifted step, the full store in pinned host memory, and the update
    overlapped with the next step."""
    import torch
    from paper_2508_02751_amd import smallkv as S
    from paper_2508_02751_amd import workloads as W

    dev = x["l_k"].device
    K = args.steps
    nsh = ps.buf.logits.shape[1]
    # the oracle's rebuild of the same store on one host core
    cpu = None
    if not args.no_cpu_baseline:
        sys.path.insert(0, os.path.join(ROOT, "oracle"))
        import oracle as O

        def h(t):
            return t.detach().float().cpu().numpy() if t.dtype == torch.bfloat16 else t.cpu().numpy()

        args_h = dict(seq_len=h(x["seq_len"]), head_map=h(x["head_map"]),
                      crit=h(ps.buf.crit_idx), marg=h(ps.buf.marg_idx), full_k=h(x["l_k"]),
                      full_v=h(x["l_v"]), rows=rows, n_small_heads=nsh)
        try:
            os.sched_setaffinity(0, {sorted(os.sched_getaffinity(0))[0]})
        except (AttributeError, OSError):
            pass
        c0 = time.perf_counter()
        reps = 0
        while reps < 1 or time.perf_counter() - c0 < 5.0:
            O.store_update(**args_h)
            reps += 1
        spent = time.perf_counter() - c0
        cpu = {"value": reps / spent, "unit": "updates/s", "cores": 1, "kind": "oracle",
               "sample": f"{reps} whole store rebuild(s) of the same step, single-threaded C "
                         f"oracle pinned to one core ({spent:.1f} s)"}
    # a drifted step: rows the previous store holds are reused, the others read
    old = store(x["l_k"], x["l_v"])
    old.run()
    s_q, l_q = W.step_queries(w, W.latents(w, dev), 1, dev)
    ps.with_query(s_q, l_q)
    ps.run()
    inc = store(x["l_k"], x["l_v"], old=old)
    ms_inc = timed(inc)
    torch.cuda.synchronize()
    ks_new, ks_old = inc.k_slot, old.k_slot
    vs_new, vs_old = inc.v_slot, old.v_slot
    fetched = int(((ks_new >= 0) & (ks_old < 0)).sum() + ((vs_new >= 0) & (vs_old < 0)).sum())
    kept = int(((ks_new >= 0) & (ks_old >= 0)).sum() + ((vs_new >= 0) & (vs_old >= 0)).sum())
    # the full store in pinned host memory (the paper keeps the evicted KV
    # on the host): a whole rebuild, and the update after the drifted step
    print("[bench] full store in pinned host memory", file=sys.stderr, flush=True)
    hk, hv = x["l_k"].cpu().pin_memory(), x["l_v"].cpu().pin_memory()
    host_full = store(hk, hv)
    ms_host_full = timed(host_full)
    host_inc = store(hk, hv, old=old)
    ms_host_inc = timed(host_inc)
    # the update overlapped with the next step's attention on a second
    # stream (its lists copied, so that the step may rewrite its own)
    crit_c, marg_c = ps.buf.crit_idx.clone(), ps.buf.marg_idx.clone()
    ov = S.prepare_store(ps.batch, ps.head_map, nsh, crit_c, marg_c, hk, hv, rows, old=old)
    side = torch.cuda.Stream()
    for _ in range(max(args.warmup, 1)):
        ps.run(stream)
    torch.cuda.synchronize()
    ms_step = timed(ps)

    def overlapped():
        e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
        torch.cuda._sleep(50_000_000)
        e[0].record(stream)
        side.wait_event(e[0])
        for _ in range(K):
            ov.run(side)
            ps.run(stream)
        e[1].record(side)
        stream.wait_event(e[1])
        e[2].record(stream)
        torch.cuda.synchronize()
        return e[0].elapsed_time(e[2]) / K

    overlapped()
    ms_both = overlapped()
    torch.cuda.synchronize()
    return {
        "after_a_drifted_step": {"ms": ms_inc, "rows_new": fetched, "rows_reused": kept,
                                 "new_fraction": fetched / max(1, fetched + kept)},
        "full_store_in_pinned_host_memory": {
            "rebuild_ms": ms_host_full,
            "rebuild_link_GBs": moved / (ms_host_full * 1e-3) / 1e9,
            "after_a_drifted_step_ms": ms_host_inc,
            "overlapped_with_the_next_step": {"step_ms": ms_step, "update_ms": ms_host_inc,
                                              "both_ms": ms_both}},
        "cpu_baseline": cpu,
    }


def bench_match(args):
    """The prefill similarity matching on the Qwen2-7B + Qwen2-0.5B shapes."""
    import dataclasses

    import torch
    from paper_2508_02751_amd import workloads as W
    from paper_2508_02751_amd.pipeline import prepare_match, softmax_scale

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = dataclasses.replace(W.WORKLOADS[2], batch=args.match_batch)
    win = args.match_window
    print(f"[bench] generating the {win}-token matching window", file=sys.stderr, flush=True)
    x = W.match_inputs(w, win, dev)
    mc = prepare_match(x, scores=False, top_bits=False)
    stream = torch.cuda.current_stream()
    for _ in range(max(args.warmup, 1)):
        mc.run()
    torch.cuda.synchronize()
    g = None
    if not args.eager:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            mc.run()
        g.replay()
        torch.cuda.synchronize()
    K = args.steps
    t0 = time.perf_counter()
    for _ in range(K):
        g.replay() if g is not None else mc.run()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / K
    # the matching call's kernels, timed with HIP events on their stream
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(K)]
    torch.cuda._sleep(50_000_000)
    for e0, e1 in ev:
        e0.record(stream)
        mc.run(stream)
        e1.record(stream)
    torch.cuda.synchronize()
    call_ms = sum(a.elapsed_time(b) for a, b in ev) / K
    # algorithmic flops: one d-long FMA chain (2 flops per term) per causal logit
    heads = [(w.large.layers * w.large.q_heads, w.large.head_dim),
             (w.small.layers * w.small.q_heads, w.small.head_dim)]
    flops = w.batch * sum(n * d * win * (win + 1) for n, d in heads)
    achieved = flops / (call_ms * 1e-3) / 1e12
    cpu = None
    if not args.no_cpu_baseline:
        sys.path.insert(0, os.path.join(ROOT, "oracle"))
        import oracle as O

        def h(t):
            return t.detach().float().cpu().numpy() if t.dtype == torch.bfloat16 else t.cpu().numpy()

        hx = {k: h(v) for k, v in x.items()}
        try:
            os.sched_setaffinity(0, {sorted(os.sched_getaffinity(0))[0]})
        except (AttributeError, OSError):
            pass
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        c0 = time.perf_counter()
        O.match(win_len=hx["win_len"], top_k=hx["top_k"], l_q=hx["l_q"], l_k=hx["l_k"],
                l_scale=softmax_scale(w.large.head_dim), s_q=hx["s_q"], s_k=hx["s_k"],
                s_scale=softmax_scale(w.small.head_dim))
        spent = time.perf_counter() - c0
        cpu = {"value": w.batch / spent, "unit": "sequences/s", "cores": 1, "kind": "oracle",
               "sample": f"one whole matching of the same {w.batch} window(s), single-threaded "
                         f"C oracle pinned to one core ({spent:.1f} s)"}
    out = {
        "metric": "SmallKV prefill head matching (Eqs. 1-3) sequences/s at 1 MI355X",
        "value": w.batch * 1e3 / ms,
        "unit": "sequences/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": f"qwen2-7b+0.5b-prefill-window{win}-b{w.batch}-bf16",
            "large": shape_text(w.large), "small": shape_text(w.small),
            "input_dtype": "bf16", "batch": w.batch, "window": win,
            "top_k": int(x["top_k"][0]), "launch": "eager" if args.eager else "hip-graph",
        },
        "roofline": {
            "kernel": "match_logits+match_rowsum+match_scores+match_map",
            "bound": "alu",
            "achieved": achieved,
            "peak": FP32_VECTOR_PEAK_TFLOPS,
            "unit": "TFLOP/s",
            "frac": achieved / FP32_VECTOR_PEAK_TFLOPS,
            "traffic": None,
        },
        "call_ms": call_ms,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
