"""Benchmark of one SmallKV decode step on one MI355X.

A step is the whole hot path over one batch: stage 1 (small-model decode
attention over all its layers), stage 2 (partition of every small head),
stage 3 (hybrid attention of every large layer).  Workload: the Qwen2-7B
(28 layers, 28q/4kv, d=128) + Qwen2-0.5B (24 layers, 14q/2kv, d=64) shapes,
bf16, batch 1, context 8192, critical 10% / marginal 20%.

Timing: inputs are resident in HBM; the step is captured in one HIP graph per
input copy, and consecutive steps rotate over `--rotate` copies so that a
step never finds the previous step's operands in the 256 MB MALL.  W warm-up
steps, then exactly K timed steps between two synchronisations.  A second
pass with HIP events between the stages (enqueued behind a sleep kernel so
the host never starves the GPU) gives per-stage kernel durations for the
roofline.  The CPU baseline is the oracle on one host core over whole steps.

Prints one JSON line.

`--match` benchmarks the prefill similarity matching instead (Eqs. 1-3: the
step before decoding that computes the head map): the Qwen2-7B + Qwen2-0.5B
shapes over a 200-token window, one JSON line of its own.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, 8 TB/s
FP32_VECTOR_PEAK_TFLOPS = 157.3  # MI355X fp32 vector (packed FMA counted as 4 flops)


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=100)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--rotate", type=int, default=4, help="input copies cycled through")
    p.add_argument("--workload", type=int, default=2,
                   help="2: the Qwen2-7B + Qwen2-0.5B headline step; 3-5: the larger shapes")
    p.add_argument("--eager", action="store_true", help="launch without HIP graphs")
    p.add_argument("--cpu-seconds", type=float, default=12.0, help="oracle time budget")
    p.add_argument("--no-cpu-baseline", action="store_true")
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
    return p.parse_args()


def source_hash(name: str) -> str:
    path = os.path.join(ROOT, "paper_2508_02751_amd", "csrc", name)
    return hashlib.sha256(open(path, "rb").read()).hexdigest()[:16]


def load_traffic(kernels, workload: str, name: str = "traffic.json"):
    """HBM bytes of one stage call (the sum over its kernels) from the committed
    rocprofv3 --pmc summary, or None when the counters were taken on another
    workload, a kernel is missing, or its source changed since."""
    path = os.path.join(ROOT, "profiles", name)
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


def stage3_kernels(w):
    """Kernels one stage-3 call launches for workload w: the grouped kernel for
    bf16, head_dim 128 and at most 8 query heads per kv head (plus the merge
    of its token splits when there are fewer than 512 kv-head units, the
    library's rule), the per-head kernel otherwise."""
    L = w.large
    if w.dtype != "bf16" or L.head_dim != 128 or L.group > 8:
        return ["hybrid_kernel"]
    units = w.batch * L.layers * L.kv_heads
    splits = max(1, min(512 // units, (w.n_cap + 255) // 256))
    return ["hybrid_group_kernel", "hybrid_group_merge"] if splits > 1 else ["hybrid_group_kernel"]


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
    from paper_2508_02751_amd import smallkv as S
    from paper_2508_02751_amd import workloads as W
    from paper_2508_02751_amd.bytes_model import step_bytes
    from paper_2508_02751_amd.pipeline import prepare_step

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    w = W.WORKLOADS[args.workload]
    copy_probe(args, dev)
    print(f"[bench] generating {w.name}", file=sys.stderr, flush=True)
    x0 = W.make_step_inputs(w, dev)
    copy_bytes = sum(v.numel() * v.element_size() for v in x0.values() if torch.is_tensor(v))
    if copy_bytes > (16 << 30):  # far beyond the 256 MB MALL already; keep HBM free
        args.rotate = 1
    copies = [x0]
    for _ in range(args.rotate - 1):
        copies.append({k: (v.clone() if torch.is_tensor(v) else v) for k, v in x0.items()})
    preps = [prepare_step(x) for x in copies]
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

    # ---- per-stage kernel durations with HIP events -------------------------
    nsh = w.small.layers * w.small.q_heads
    group = w.select == 1
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(4)] for _ in range(K)]
    torch.cuda._sleep(50_000_000)  # keep the GPU busy while the host enqueues
    for i in range(K):
        ps = preps[i % len(preps)]
        b = ps.buf
        e = ev[i]
        e[0].record(stream)
        S.smallkv_small_attn(ps.batch, ps.small, b.logits, b.row_max, b.row_sum, b.ws, stream)
        e[1].record(stream)
        if group:
            S.smallkv_group_select(ps.batch, ps.small, ps.large, ps.head_map, b.logits, b.row_max,
                                   b.row_sum, b.crit_idx, b.marg_idx, b.marg_prob, b.mass, b.ws,
                                   stream)
        elif w.select == 2:
            S.smallkv_accum_select(ps.batch, ps.small, b.logits, b.row_max, b.row_sum,
                                   b.acc_score, b.crit_idx, b.marg_idx, b.marg_prob, b.mass, b.ws,
                                   stream)
        else:
            S.smallkv_partition(ps.batch, nsh, b.logits, b.row_max, b.row_sum, b.crit_idx,
                                b.marg_idx, b.marg_prob, b.mass, None, stream, small=ps.small)
        e[2].record(stream)
        S.smallkv_hybrid_attn(ps.batch, ps.large, ps.head_map, nsh, b.crit_idx, b.marg_idx,
                              b.marg_prob, b.mass, ps.mode, b.ws, stream,
                              select=S.SELECT_GROUP if group else S.SELECT_HEAD)
        e[3].record(stream)
    torch.cuda.synchronize()
    stage_ms = [sum(ev[i][s].elapsed_time(ev[i][s + 1]) for i in range(K)) / K for s in range(3)]

    # ---- bytes ------------------------------------------------------------
    ps = preps[0]
    sb = step_bytes(ps.inputs, ps.buf.crit_idx, ps.buf.marg_idx, ps.batch.km_cap)
    stage_bytes = [sb.stage1, sb.stage2, sb.stage3]
    # kernels each single-stage call launches for this workload (bf16, large
    # head_dim 128, 7 query heads per kv head, 112 kv-head units: stage 3 is
    # the grouped kernel over token splits plus their merge)
    stage_kernels = [["small_attn_mfma", "small_attn_merge"],
                     ["group_zq", "group_scores", "partition_kernel", "group_weights"] if group
                     else ["group_zq", "accum_scores", "partition_kernel", "group_weights"]
                     if w.select == 2 else ["partition_kernel"], stage3_kernels(w)]
    dom = max(range(3), key=lambda s: stage_ms[s])
    achieved = stage_bytes[dom] / (stage_ms[dom] * 1e-3) / 1e9
    traffic = load_traffic(stage_kernels[dom], w.name)
    step_gbs = sb.step_compulsory / (ms_per_step * 1e-3) / 1e9

    # ---- CPU baseline: the oracle on one core ------------------------------
    cpu = None
    if not args.no_cpu_baseline:
        sys.path.insert(0, os.path.join(ROOT, "oracle"))
        import numpy as np
        import oracle as O
        from paper_2508_02751_amd.pipeline import softmax_scale

        def h(t):
            return t.detach().float().cpu().numpy() if t.dtype == torch.bfloat16 else t.cpu().numpy()

        x = ps.inputs
        host = {k: h(x[k]) for k in ("seq_len", "k_crit", "k_marg", "head_map", "s_q", "s_k",
                                     "s_v", "l_q", "l_k", "l_v")}
        host["k_recent"] = h(x["k_recent"]) if x.get("k_recent") is not None else None
        held = {} if x.get("s_held") is None else dict(
            s_held=h(x["s_held"]), s_row_pos=h(x["s_row_pos"]), n_cap=x["n_cap"])
        if group:
            held["select"] = O.SELECT_GROUP
        if w.select == 2:
            held["select"] = O.SELECT_ACCUM
            held["acc"] = np.zeros(tuple(ps.buf.acc_score.shape), np.float32)
        try:
            os.sched_setaffinity(0, {sorted(os.sched_getaffinity(0))[0]})
        except (AttributeError, OSError):
            pass
        print("[bench] timing the CPU oracle", file=sys.stderr, flush=True)
        reps, spent = 0, 0.0
        while reps < 1 or spent < args.cpu_seconds:
            c0 = time.perf_counter()
            O.step(seq_len=host["seq_len"], k_crit=host["k_crit"], k_marg=host["k_marg"],
                   kc_cap=x["kc_cap"], km_cap=x["km_cap"], head_map=host["head_map"],
                   mode=O.NORM_REMAINING, s_q=host["s_q"], s_k=host["s_k"], s_v=host["s_v"],
                   s_scale=softmax_scale(w.small.head_dim), l_q=host["l_q"], l_k=host["l_k"],
                   l_v=host["l_v"], l_scale=softmax_scale(w.large.head_dim),
                   k_recent=host["k_recent"], **held)
            spent += time.perf_counter() - c0
            reps += 1
        cpu = {"value": w.batch * reps / spent, "unit": "tokens/s", "cores": 1, "kind": "oracle",
               "sample": f"{reps} whole decode step(s) of the same workload, single-threaded C "
                         f"oracle pinned to one core ({spent:.1f} s)"}

    out = {
        "metric": "SmallKV decode-step attention tokens/s at 1 MI355X; % of HBM roofline",
        "value": w.batch * 1e3 / ms_per_step,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": w.name,
            "large": shape_text(w.large), "small": shape_text(w.small),
            "kv_dtype": w.dtype, "batch": w.batch, "context": w.n_ctx,
            "critical": budget_text(w.crit), "marginal": budget_text(w.marg),
            **({"recent": budget_text(w.recent)} if w.recent != ("abs", 0) else {}),
            **({"small_cache_kept": f"{w.slm_keep}%"} if w.slm_keep else {}),
            **({"selection": "one per large kv head (summed)"} if group else {}),
            **({"selection": "accumulated scores (running state)"} if w.select == 2 else {}),
            "launch": "eager" if args.eager else "hip-graph",
            "rotated_input_copies": args.rotate,
        },
        "roofline": {
            "kernel": "+".join(stage_kernels[dom]),
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": traffic,
        },
        "step": {
            "compulsory_bytes": sb.step_compulsory,
            "achieved_GBs": step_gbs,
            "hbm_frac": step_gbs / HBM_PEAK_GBS,
            "stage_ms": stage_ms,
            "stage_bytes": stage_bytes,
            "stage_GBs": [stage_bytes[s] / (stage_ms[s] * 1e-3) / 1e9 for s in range(3)],
            "large_rows_per_head_over_union": (sb.large_k_perhead + sb.large_v_perhead)
            / max(1, sb.large_k_union + sb.large_v_union),
            "index_metadata_bytes": sb.index_meta,
        },
        "cpu_baseline": cpu,
    }
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
    traffic = load_traffic(["store_index", "store_copy"], f"{w.name}-store", "traffic_store.json")
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
