#!/usr/bin/env python3
"""Benchmark of the tree-verification step on one MI355X.

A step = one pass of Llama-3-70B-shaped decoder layers verifying a 32-token
draft tree (8 levels, branching <= 4) over a 4096-token prefix (int4
group-128 weights, fp16 activations and KV cache), replayed from one HIP
graph.  The step runs every layer copy once (several copies of the layer's
weights and KV cache, so the 256 MB Infinity Cache cannot hold the working
set), and the value is per layer.  Inputs are seeded synthetic tensors
already resident in HBM.  The KV commit of the accepted path runs once per
model step for all layers; it is timed separately (one launch over every
layer copy) and reported next to the per-layer value.

Prints one JSON line: value = mean microseconds per layer (lower is better)
with p10/p50/p90 over the replays; per-operation standalone timings with
algorithmic bytes and achieved GB/s (GEMMs with their split-K fix-up,
attention with its merge); the roofline of the dominant operation (the
fused SwiGLU W4A16 GEMM) timed on its own stream with HIP events; the same
per-layer figures (fewer replays) for the other layer configurations
(`configs`: 1B, 8B, 8B at a 32K prefix); and the fp64 CPU reference checker
timed on the host as a baseline (all threads and one thread, median of
three runs each).
"""
import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MALL_BYTES = 256 << 20


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="c3")
    ap.add_argument("--copies", type=int, default=0, help="layer copies rotated (0: auto)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-repeats", type=int, default=3, help="runs of each CPU-baseline leg (median)")
    ap.add_argument("--no-other-configs", action="store_true",
                    help="skip the per-layer sub-results of the other layer configurations (c1, c2, c4)")
    ap.add_argument("--only-kernel", default="", help="launch only this kernel (for counter runs): "
                    "swiglu | qkv | o | down | attention | commit | copy")
    ap.add_argument("--iters", type=int, default=50)
    ap.add_argument("--no-full-step", action="store_true",
                    help="skip the 80-layer step (all layers + final norm + LM head) timing")
    ap.add_argument("--full-step-reps", type=int, default=10)
    ap.add_argument("--no-paper-shard", action="store_true",
                    help="skip the one-GPU share of the paper's 70B TP4 kernel benchmarks")
    ap.add_argument("--no-draft-side", action="store_true",
                    help="skip the draft-model kernels (non-square attention, KV reorganisation)")
    ap.add_argument("--no-tree-loop", action="store_true",
                    help="skip the sequential tree-generation loop (Alg. 1 with synthetic models)")
    ap.add_argument("--gemm-ab", action="store_true",
                    help="only compare the matrix-core and vector-ALU W4A16 GEMMs over M (JSON line per M)")
    return ap.parse_args()


SHAPE_LABEL = {2048: "Llama-3.2-1B", 4096: "Llama-3-8B", 8192: "Llama-3-70B"}


def source_hash(paths):
    """Hash of the code of C++/HIP sources: comments dropped and white space
    collapsed, so an edited comment keeps the hash and any code change alters
    it (the hashed sources hold no string literal with a comment marker)."""
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p)) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", "", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()[:16]


GEMM_SOURCES = ["paper_2506_11309_amd/csrc/w4a16_gemm.hip", "paper_2506_11309_amd/csrc/ss_device.h"]


def read_traffic(kernel_tag, cur_hash):
    """HBM bytes per launch measured by rocprofv3 counters (committed summary),
    or None if absent or taken on a different kernel source."""
    path = os.path.join(ROOT, "profiles", f"{kernel_tag}_traffic.md")
    if not os.path.exists(path):
        return None
    vals = {}
    for line in open(path):
        if line.startswith("- ") and ":" in line:
            k, v = line[2:].split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("source_hash") != cur_hash:
        return None
    try:
        return float(vals["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def setup_layers(cfg_name, args, ss, torch, np, dev):
    """Seeded synthetic inputs of one layer configuration, uploaded: enough
    layer copies (weights and KV cache) to defeat the Infinity Cache."""
    from gen import workloads as wl
    cfg = wl.CONFIGS[cfg_name]
    s = cfg.shape
    T = cfg.T
    t0 = time.time()
    w = wl.make_layer_weights(cfg)
    kc, vc = wl.make_kv_prefix(cfg)
    x = wl.make_activations(cfg)
    parent, acc = wl.make_tree(cfg)
    gen_s = time.time() - t0

    def up(a):
        a = np.ascontiguousarray(a)
        if a.dtype == np.uint16:
            a = a.view(np.int16)
        return torch.from_numpy(a).to(dev)

    layer_bytes = s.w4_bytes() + cfg.kv_bytes_per_layer()
    copies = args.copies or max(2, -(-2 * MALL_BYTES // layer_bytes) + 1)
    dims = ss.make_dims(s.H, s.Hq, s.Hkv, s.D, s.F, cfg.S_max)
    rope = up(ss.rope_table(500000.0, cfg.S_max, s.D))
    dparent = up(parent)
    dacc = up(np.array([acc], np.int32))
    host_w = {n: (w[n]["qweight"], w[n]["scales"], w[n]["zeros"]) for n in ("wqkv", "wo", "wgate", "wup", "wdown")}
    # all copies' caches in one [copies][Hkv][S_max][D] buffer: one commit launch covers every layer
    kc_all = up(np.broadcast_to(kc, (copies,) + kc.shape))
    vc_all = up(np.broadcast_to(vc, (copies,) + vc.shape))
    P_dev = up(np.array([cfg.P], np.int32))
    inst = []
    for c in range(copies):
        keep = {n: tuple(up(a) for a in host_w[n]) for n in host_w}
        w4 = {n: ss.make_w4(*keep[n]) for n in keep}
        packs = {n: ss.prepack_w4(w4[n]) for n in w4}  # kernel-native copies (one-time)
        d = {"keep": keep, "packs": packs, "w4": w4, "an": up(w["attn_norm"]), "mn": up(w["mlp_norm"]),
             "kc": kc_all[c], "vc": vc_all[c], "P": P_dev, "h": up(x)}
        d["layer"] = ss.make_layer(d["an"], d["mn"], w4["wqkv"], w4["wo"], w4["wgate"], w4["wup"],
                                   w4["wdown"], d["kc"], d["vc"])
        d["ws"] = ss.workspace(ss.verify_layer_workspace_bytes(dims, T), dev)
        inst.append(d)
    torch.cuda.synchronize()
    return {"cfg": cfg, "s": s, "T": T, "w": w, "kc": kc, "vc": vc, "x": x, "parent": parent, "acc": acc,
            "gen_s": gen_s, "copies": copies, "dims": dims, "rope": rope, "dparent": dparent, "dacc": dacc,
            "kc_all": kc_all, "vc_all": vc_all, "P_dev": P_dev, "inst": inst, "up": up}


def make_time_op(ss, torch, stream):
    def time_op(fn, iters):
        """Mean microseconds of one fn(i) call: `iters` calls (rotating layer
        copies) captured into a HIP graph, replayed 3 times, timed with HIP
        events on `stream` (no host launch overhead in the timed region)."""
        g = ss.Graph()
        with torch.cuda.stream(stream):
            for i in range(3):
                fn(i)
            g.begin(stream)
            for i in range(iters):
                fn(i)
            g.end(stream)
            g.launch(stream)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(3):
                g.launch(stream)
            e1.record(stream)
        e1.synchronize()
        return e0.elapsed_time(e1) * 1000.0 / (3 * iters)
    return time_op


def time_step(ctx, steps, warmup, ss, torch, stream):
    """The step graph (every layer copy once, in order, like a multi-layer
    model step) replayed `steps` times after `warmup` replays; per-layer
    microseconds of each replay."""
    inst, copies = ctx["inst"], ctx["copies"]
    # shader clock sampled on the idle chip, and over the first millisecond
    # of the timed replays by a one-wave kernel on a second stream (the
    # power management lowers the clock under load within microseconds and
    # raises it again as soon as the load stops, so only a sample taken
    # during the replays shows the clock the kernels run at)
    clk = torch.zeros(8, dtype=torch.int64, device=inst[0]["h"].device)
    side = torch.cuda.Stream()
    step = ss.Graph()
    with torch.cuda.stream(stream):
        ss.clock_sample(clk[0:4], 20, stream=stream)
        step.begin(stream)
        for d in inst:
            ss.verify_layer(d["layer"], ctx["dims"], d["h"], d["P"], ctx["dparent"], ctx["rope"], d["ws"],
                            stream=stream)
        step.end(stream)
        for i in range(warmup):
            step.launch(stream)
    stream.synchronize()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    with torch.cuda.stream(side):
        ss.clock_sample(clk[4:8], 1000, stream=side)
    with torch.cuda.stream(stream):
        ev[0].record(stream)
        for i in range(steps):
            step.launch(stream)
            ev[i + 1].record(stream)
    ev[-1].synchronize()
    side.synchronize()
    torch.cuda.synchronize()
    c = clk.cpu().tolist()
    ctx["clock_ghz"] = {"idle_before_warmup": round(ss.clock_ghz(c[0:4]), 3),
                        "during_timed_steps": round(ss.clock_ghz(c[4:8]), 3)}
    ms_total = ev[0].elapsed_time(ev[-1])
    per = sorted(ev[i].elapsed_time(ev[i + 1]) * 1000.0 / copies for i in range(steps))
    for d in inst:
        err = ss.read_device_error(d["ws"], stream)
        if err:
            raise RuntimeError(f"device error word {err}")
    return ms_total / steps / copies, per


def time_ops(ctx, it, ss, torch, stream, dev):
    """Standalone timings of the layer's operations (GEMMs with their split-K
    fix-up, attention with its merge), algorithmic bytes, GB/s."""
    s, T, copies, inst = ctx["s"], ctx["T"], ctx["copies"], ctx["inst"]
    cfg = ctx["cfg"]
    time_op = make_time_op(ss, torch, stream)
    w4b = lambda K, N: K * N // 2 + (K // 128) * N * 3
    xin = ctx["up"](ctx["x"])
    big_x = torch.zeros((T, max(s.H, s.F, s.Hq * s.D)), dtype=torch.int16, device=dev)
    big_x.copy_(torch.randint(-3000, 3000, big_x.shape, dtype=torch.int16, device=dev) & 0x3BFF)
    y = torch.zeros((T, max(s.F, s.n_qkv)), dtype=torch.int16, device=dev)
    op_ws = ss.workspace(ss.verify_layer_workspace_bytes(ctx["dims"], T), dev)
    preps = {K: torch.zeros(ss.prepared_bytes(T, K), dtype=torch.uint8, device=dev) for K in {s.H, s.F, s.Hq * s.D}}
    with torch.cuda.stream(stream):
        for K, xp in preps.items():
            ss.prepare_activations(big_x[:, :K], xp, stream=stream)
    ops = {}

    def gemm_op(name, wname, K, N, residual):
        res = big_x[:, :N] if residual else None
        us = time_op(lambda i: ss.w4a16_gemm_prepared(inst[i % copies]["w4"][wname], preps[K], T, y[:, :N],
                                                      op_ws, residual=res, stream=stream), it)
        ops[name] = {"us": round(us, 3), "bytes": w4b(K, N)}

    gemm_op("qkv", "wqkv", s.H, s.n_qkv, False)
    gemm_op("o_proj", "wo", s.Hq * s.D, s.H, True)
    sw_us = time_op(lambda i: ss.w4a16_swiglu_prepared(inst[i % copies]["w4"]["wgate"], inst[i % copies]["w4"]["wup"],
                                                       preps[s.H], T, y[:, :s.F], op_ws, stream=stream), it)
    ops["swiglu"] = {"us": round(sw_us, 3), "bytes": 2 * w4b(s.H, s.F)}
    gemm_op("down", "wdown", s.F, s.H, True)
    Hd = s.Hq * s.D
    qkv_t = big_x[:, :s.n_qkv] if s.n_qkv <= big_x.shape[1] else None
    att_us = time_op(lambda i: ss.tree_attention(qkv_t, qkv_t[:, Hd:], qkv_t[:, Hd + s.Hkv * s.D:],
                                                 inst[i % copies]["kc"], inst[i % copies]["vc"], ctx["P_dev"],
                                                 ctx["dparent"], s.Hq, s.Hkv, s.D, ctx["rope"], y[:, :Hd], op_ws,
                                                 stream=stream), it)
    att_bytes = 2 * s.Hkv * (cfg.P + T) * s.D * 2 + T * (s.n_qkv + Hd) * 2
    ops["attention"] = {"us": round(att_us, 3), "bytes": att_bytes}
    rn_us = time_op(lambda i: ss.rmsnorm(xin, inst[0]["an"], y[:, :s.H], stream=stream), it)
    ops["rmsnorm"] = {"us": round(rn_us, 3), "bytes": 2 * T * s.H * 2 + s.H * 2}
    # the norm with the projection that reads it, as the layer runs them (in
    # one kernel where the GEMM plan splits K within workgroups)
    nq_us = time_op(lambda i: ss.rmsnorm_w4a16_gemm(inst[i % copies]["w4"]["wqkv"], xin, inst[0]["an"],
                                                    y[:, :s.n_qkv], op_ws, stream=stream), it)
    ops["rmsnorm_qkv"] = {"us": round(nq_us, 3), "bytes": w4b(s.H, s.n_qkv) + T * s.H * 2 + s.H * 2}
    ns_us = time_op(lambda i: ss.rmsnorm_w4a16_swiglu(inst[i % copies]["w4"]["wgate"], inst[i % copies]["w4"]["wup"],
                                                      xin, inst[0]["an"], y[:, :s.F], op_ws, stream=stream), it)
    ops["rmsnorm_swiglu"] = {"us": round(ns_us, 3), "bytes": 2 * w4b(s.H, s.F) + T * s.H * 2 + s.H * 2}
    for k, v in ops.items():
        v["GBps"] = round(v["bytes"] / (v["us"] * 1e-6) / 1e9, 1)
        v["frac_hbm"] = round(v["GBps"] / HBM_PEAK_GBS, 4)
    g_names = ("qkv", "o_proj", "swiglu", "down")
    g_bytes = sum(ops[n]["bytes"] for n in g_names)
    g_us = sum(ops[n]["us"] for n in g_names)
    gemm_agg = {"bytes": g_bytes, "us": round(g_us, 3), "GBps": round(g_bytes / (g_us * 1e-6) / 1e9, 1),
                "frac_hbm": round(g_bytes / (g_us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4)}
    return ops, gemm_agg


def workload_label(cfg):
    s = cfg.shape
    return (f"{cfg.name}: {SHAPE_LABEL.get(s.H, 'Llama')}-shaped layer, H={s.H}, Hq/Hkv={s.Hq}/{s.Hkv}, "
            f"D={s.D}, F={s.F}, int4 g128; tree T={cfg.T} ({cfg.levels} levels, branching<={cfg.branching}); "
            f"prefix P={cfg.P}")


def other_config(name, args, ss, torch, np, dev, stream):
    """Per-layer latency, GEMM aggregate and attention bandwidth of another
    layer configuration (fewer replays than the headline configuration)."""
    ctx = setup_layers(name, args, ss, torch, np, dev)
    ms, per = time_step(ctx, max(args.steps // 4, 20), max(args.warmup // 2, 5), ss, torch, stream)
    ops, gagg = time_ops(ctx, max(args.steps // 8, 20), ss, torch, stream, dev)
    out = {"workload": workload_label(ctx["cfg"]), "us_per_layer": round(ms * 1000.0, 3),
           "us_per_layer_p50": round(per[len(per) // 2], 3), "layer_copies_rotated": ctx["copies"],
           "gemm_aggregate": gagg, "attention": ops["attention"],
           "ops_us": {k: v["us"] for k, v in ops.items()}}
    del ctx
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    return out


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(ctx, args):
    """The fp64 reference checker on the host: the whole layer step (+ KV
    commit), with every thread it is given and with one thread; median of
    `args.cpu_repeats` runs each (progress on stderr)."""
    import oracle
    cfg, s, w, x = ctx["cfg"], ctx["s"], ctx["w"], ctx["x"]
    odims = {"H": s.H, "Hq": s.Hq, "Hkv": s.Hkv, "D": s.D, "F": s.F, "S_max": cfg.S_max}
    threads_all = oracle.num_threads()

    def run(reps, label):
        times = []
        for r in range(reps):
            okc, ovc = ctx["kc"].copy(), ctx["vc"].copy()
            t1 = time.time()
            oracle.verify_layer(odims, w, okc, ovc, x, cfg.P, ctx["parent"])
            oracle.kv_commit(okc, ovc, cfg.P, ctx["parent"], ctx["acc"])
            times.append(time.time() - t1)
            print(f"cpu baseline ({label}) run {r + 1}/{reps}: {times[-1]:.2f} s", file=sys.stderr, flush=True)
        return times

    reps = max(1, args.cpu_repeats)
    all_t = run(reps, f"{threads_all} threads")
    oracle.set_num_threads(1)
    try:
        one_t = run(reps, "1 thread")
    finally:
        oracle.set_num_threads(threads_all)
    med = lambda v: sorted(v)[len(v) // 2]
    sample = f"one full {cfg.name} layer step (T={cfg.T}, P={cfg.P}) + KV commit, fp64"
    return {"value": round(med(all_t) * 1e6, 1), "unit": "us/layer", "cores": threads_all, "kind": "oracle",
            "sample": f"{sample}, {threads_all} OpenMP threads; median of {reps} runs",
            "repeats_s": [round(t, 3) for t in all_t],
            "single_thread": {"value": round(med(one_t) * 1e6, 1), "unit": "us/layer", "cores": 1,
                              "sample": f"{sample}, 1 thread; median of {reps} runs",
                              "repeats_s": [round(t, 3) for t in one_t]},
            "cpu_model": cpu_model(), "host_cpus_visible": len(os.sched_getaffinity(0))}


def log(msg):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); sharding across GPUs "
              "is not implemented.", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch

    import paper_2506_11309_amd as ss

    if not os.path.exists(ss.LIB_PATH):
        import __graft_entry__
        __graft_entry__.build()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.Stream()
    ctx = setup_layers(args.config, args, ss, torch, np, dev)
    cfg, s, T, copies, inst = ctx["cfg"], ctx["s"], ctx["T"], ctx["copies"], ctx["inst"]
    log(f"{args.config}: {copies} layer copies uploaded")

    if args.gemm_ab:
        gemm_ab(ss, torch, np, inst, cfg, stream, dev)
        return

    # ---------------- counter-run mode: one kernel type only ----------------
    if args.only_kernel:
        run_only(args, ss, torch, np, inst, cfg, ctx["dims"], ctx["dparent"], ctx["dacc"], ctx["rope"], stream, dev)
        return

    # ---------------- step graph: every layer copy once, in order ----------------
    ms_step, per = time_step(ctx, args.steps, args.warmup, ss, torch, stream)
    log(f"step: {ms_step * 1000.0:.1f} us/layer")
    pct = lambda q: round(per[min(len(per) - 1, int(q * len(per)))], 3)
    time_op = make_time_op(ss, torch, stream)

    # ---------------- KV commit: all layer copies in one launch ----------------
    cm_ws = ss.workspace(ss.verify_layer_workspace_bytes(ctx["dims"], T), dev)
    commit_us = time_op(lambda i: ss.kv_commit(ctx["kc_all"], ctx["vc_all"], ctx["P_dev"], ctx["dparent"],
                                               ctx["dacc"], n_layers=copies, advance=False, ws=cm_ws,
                                               stream=stream), 50)
    if ss.read_device_error(cm_ws, stream):
        raise RuntimeError("device error in kv_commit")

    # ---------------- per-operation standalone timings ----------------
    ops, gemm_agg = time_ops(ctx, max(args.steps // 2, 30), ss, torch, stream, dev)
    log("per-operation timings done")

    # ---------------- dominant operation: fused SwiGLU GEMM ----------------
    sw_us = ops["swiglu"]["us"]
    sw_bytes = ops["swiglu"]["bytes"]
    sw_gbs = sw_bytes / (sw_us * 1e-6) / 1e9
    # the counter profile was taken on the 70B layer (c3): other shapes report none
    traffic = read_traffic("swiglu_gemm_c3", source_hash(GEMM_SOURCES)) if args.config == "c3" else None

    full = None if args.no_full_step else full_step(args, ss, torch, np, dev, stream)
    log("80-layer step done")
    draft = None if args.no_draft_side else draft_side(args, ss, torch, np, dev, stream)
    shard = None if args.no_paper_shard else paper_shard(args, ss, torch, np, dev, stream)
    log("draft side and TP4 shard done")
    loop = None if args.no_tree_loop else tree_loop(ss, torch, np, dev, stream)
    log("tree loop done")
    others = {}
    if not args.no_other_configs:
        for name in ("c1", "c2", "c4"):
            if name != args.config:
                others[name] = other_config(name, args, ss, torch, np, dev, stream)
                log(f"{name}: {others[name]['us_per_layer']:.1f} us/layer")

    # ---------------- CPU baseline: the fp64 reference checker ----------------
    cpu = None if args.no_cpu_baseline else cpu_baseline(ctx, args)

    step_bytes = s.w4_bytes() + cfg.kv_bytes_per_layer()
    out = {
        "metric": "tree-verify step latency (us/layer) + achieved HBM GB/s vs peak, 1 MI355X",
        "value": round(ms_step * 1000.0, 3),
        "unit": "us/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step * copies, 6),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16 (int4 weights, fp32 accumulate)",
        "data": "synthetic",
        "config": {"workload": workload_label(cfg) + "; verify_layer per step, KV commit timed separately",
                   "global_batch": T, "seq_len": cfg.P + T, "parallelism": "none (1 GPU)",
                   "layer_copies_rotated": copies, "layers_per_step": copies},
        "us_per_layer_p10_p50_p90": [pct(0.1), pct(0.5), pct(0.9)],
        "shader_clock_ghz": dict(ctx["clock_ghz"], nominal=2.4,
                                 how="s_memtime over s_memrealtime in a one-wave kernel: 20 us on the idle "
                                     "chip; 1 ms on a second stream at the start of the timed replays"),
        "step_hbm_gbs": round(step_bytes / (ms_step * 1e-3) / 1e9, 1),
        "kv_commit_us": {"all_layers": round(commit_us, 3), "layers": copies,
                         "per_layer": round(commit_us / copies, 3)},
        "ops": ops,
        "gemm_aggregate": gemm_agg,
        "roofline": {"kernel": "w4a16_swiglu (fused gate+up W4A16 GEMM)", "bound": "hbm",
                     "achieved": round(sw_gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(sw_gbs / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "algorithmic_bytes_per_launch": sw_bytes, "avg_launch_us": round(sw_us, 3)},
        "cpu_baseline": cpu,
        "configs": others or None,
        "full_step_80_layers": full,
        "draft_side": draft,
        "paper_tp4_shard": shard,
        "tree_loop": loop,
        "input_generation_s": round(ctx["gen_s"], 2),
    }
    print(json.dumps(out), flush=True)


def paper_shard(args, ss, torch, np, dev, stream):
    """One GPU's share of the paper's own kernel benchmarks: Llama-3-70B
    under tensor parallelism 4 at batch 8 (the per-operation table of Sec.
    2.4 and the kernel table of Sec. 5.4, both measured on H800): QKV
    K = 8192, N = 2560 (16 query and 2 KV heads); O K = 2048, N = 8192 (+
    residual); SwiGLU K = 8192, N = 7168; down K = 7168, N = 8192 (+
    residual); attention over 16 query / 2 KV heads, a tree of 8 tokens, at
    the prefix lengths 500, 1000 and 4096.  The all-reduce is not measured
    (one GPU).  Weights rotate over copies totalling >= 512 MB per
    operation; graphs of 50 launches replayed 3 times.  `paper_us` is the
    paper's number for the same operation (its own kernels, H800, BF16
    compute), `speedup` = paper_us / us."""
    from gen import device as gdev
    M, H, Hq, Hkv, D = 8, 8192, 16, 2, 128
    F = 28672 // 4
    shapes = {"qkv": (H, (Hq + 2 * Hkv) * D, False), "o_proj": (Hq * D, H, True), "swiglu": (H, F, False),
              "down": (F, H, True)}
    paper = {"qkv": 16.9, "o_proj": 10.8, "swiglu": 39.3, "down": 18.1}

    def timed(fn, iters=50):
        g = ss.Graph()
        with torch.cuda.stream(stream):
            for i in range(2):
                fn(i)
            g.begin(stream)
            for i in range(iters):
                fn(i)
            g.end(stream)
            g.launch(stream)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(3):
                g.launch(stream)
            e1.record(stream)
        e1.synchronize()
        return e0.elapsed_time(e1) * 1000.0 / (3 * iters)

    x = torch.randint(-3000, 3000, (M, max(H, F)), dtype=torch.int16, device=dev) & 0x3BFF
    y = torch.zeros((M, max(H, F)), dtype=torch.int16, device=dev)
    ops = {}
    for name, (K, N, res) in shapes.items():
        nmat = 2 if name == "swiglu" else 1
        mbytes = nmat * (K * N // 2 + (K // 128) * N * 3)
        copies = max(2, -(-512 * 2 ** 20 // mbytes))
        # one seeded matrix per operand, its kernel-native copy written
        # `copies` times into one allocation (distinct addresses, so the
        # rotation defeats the Infinity Cache)
        pk = -(-ss.packed_bytes(K, N) // 256) * 256
        big = torch.empty(nmat * copies * pk, dtype=torch.uint8, device=dev)
        canon, descs = [], []
        for j in range(nmat):
            q, sc, z = gdev.w4_random_device(9000, j, N, K, device=dev)
            canon.append((q, sc, z))
            row = []
            for c in range(copies):
                d = ss.make_w4(q, sc, z)
                view = big[(j * copies + c) * pk:(j * copies + c) * pk + ss.packed_bytes(K, N)]
                ss.prepack_w4_into(d, view)
                row.append(d)
            descs.append(row)
        xp = torch.zeros(ss.prepared_bytes(M, K), dtype=torch.uint8, device=dev)
        ws = ss.workspace(max(ss.gemm_workspace_bytes(M, K, N), ss.swiglu_workspace_bytes(M, K, N)), dev)
        with torch.cuda.stream(stream):
            ss.prepare_activations(x[:, :K], xp, stream=stream)
        torch.cuda.synchronize()
        if name == "swiglu":
            us = timed(lambda i: ss.w4a16_swiglu_prepared(descs[0][i % copies], descs[1][i % copies], xp, M,
                                                          y[:, :N], ws, stream=stream))
        else:
            r = x[:, :N] if res else None
            us = timed(lambda i: ss.w4a16_gemm_prepared(descs[0][i % copies], xp, M, y[:, :N], ws, residual=r,
                                                        stream=stream))
        ops[name] = {"us": round(us, 2), "bytes": mbytes, "GBps": round(mbytes / (us * 1e-6) / 1e9, 1),
                     "paper_us": paper[name], "speedup": round(paper[name] / us, 2)}
        del big, canon, descs
    # attention: a tree of 8 (spine of 4, branching <= 2), prefix 500 / 1000 / 4096
    import gen as gen_mod
    parent = gen_mod.tree(M, 4, 2, 2506)
    dparent = torch.from_numpy(np.asarray(parent, np.int32)).to(dev)
    Hd = Hq * D
    qkv = torch.randint(-3000, 3000, (M, Hd + 2 * Hkv * D), dtype=torch.int16, device=dev) & 0x3BFF
    out = torch.zeros((M, Hd), dtype=torch.int16, device=dev)
    for P, paper_us in ((500, 9.6), (1000, 13.4), (4096, 18.8)):
        S_max = P + M
        kv_bytes = 2 * Hkv * S_max * D * 2
        copies = max(2, -(-512 * 2 ** 20 // kv_bytes))
        kcs = gdev.normal_f16_device(11, P, (copies, Hkv, S_max, D), device=dev)
        vcs = gdev.normal_f16_device(12, P, (copies, Hkv, S_max, D), device=dev)
        dP = torch.tensor([P], dtype=torch.int32, device=dev)
        rope = torch.from_numpy(ss.rope_table(500000.0, S_max, D)).to(dev)
        ws = ss.workspace(ss.tree_attention_workspace_bytes(M, Hq, Hkv, D, S_max), dev)
        us = timed(lambda i: ss.tree_attention(qkv, qkv[:, Hd:], qkv[:, Hd + Hkv * D:], kcs[i % copies],
                                               vcs[i % copies], dP, dparent, Hq, Hkv, D, rope, out, ws,
                                               stream=stream))
        ops[f"attention_ctx{P}"] = {"us": round(us, 2), "bytes": kv_bytes, "GBps": round(kv_bytes / (us * 1e-6) / 1e9, 1),
                                    "paper_us": paper_us, "speedup": round(paper_us / us, 2)}
        del kcs, vcs
    torch.cuda.empty_cache()
    return {"workload": "Llama-3-70B, tensor parallelism 4, batch 8: one GPU's share of each operation "
                        "(all-reduce not measured)",
            "paper": "per-operation table (Sec. 2.4; attention there at an unstated context, ~4K implied) and the "
                     "attention columns of the kernel table (Sec. 5.4, contexts 500 and 1000); H800, BF16",
            "ops": ops}


def draft_side(args, ss, torch, np, dev, stream):
    """The draft model's kernels at a Llama-3.2-1B-shaped draft (16 layers,
    Hq/Hkv = 32/8, D = 64) next to the 70B target's prefix (P = 4096): one
    tree expansion of w = 8 leaves over a 56-node tree cache (non-square
    attention, one layer), and the KV reorganisation of all 16 layers after
    re-rooting (path of 3 into the prefix, the subtree below it compacted).
    Inputs seeded, timed as graphs of 20 launches replayed 20 times."""
    from gen import device as gdev
    from gen import workloads as wl
    s = wl.LLAMA_1B
    n_layers, P, N, w = 16, 4096, 56, 8
    S_max = P + 64 + w
    rng = np.random.default_rng(2506)
    # forest: a chain of 3 from the prefix, the rest hung on random earlier nodes
    cp = [-1, 0, 1] + [int(rng.integers(0, j)) for j in range(3, N)]
    lp = [int(rng.integers(0, N)) for _ in range(w)]
    dcp = torch.tensor(cp, dtype=torch.int32, device=dev)
    dlp = torch.tensor(lp, dtype=torch.int32, device=dev)
    dP = torch.tensor([P], dtype=torch.int32, device=dev)
    kc = gdev.normal_f16_device(7, 0, (n_layers, s.Hkv, S_max, s.D), device=dev)
    vc = gdev.normal_f16_device(7, 1, (n_layers, s.Hkv, S_max, s.D), device=dev)
    q = gdev.normal_f16_device(7, 2, (w, s.Hq * s.D), device=dev)
    k = gdev.normal_f16_device(7, 3, (w, s.Hkv * s.D), device=dev)
    v = gdev.normal_f16_device(7, 4, (w, s.Hkv * s.D), device=dev)
    out = torch.zeros((w, s.Hq * s.D), dtype=torch.int16, device=dev)
    rope = torch.from_numpy(ss.rope_table(500000.0, S_max, s.D)).to(dev)
    ws = ss.workspace(ss.tree_attention_workspace_bytes(w, s.Hq, s.Hkv, s.D, S_max), dev)
    last = torch.tensor([2], dtype=torch.int32, device=dev)
    keep = torch.tensor([1], dtype=torch.int32, device=dev)
    newp = torch.zeros(N, dtype=torch.int32, device=dev)
    nk = torch.zeros(1, dtype=torch.int32, device=dev)

    def timed(enqueue, reps=20, inner=20):
        g = ss.Graph()
        with torch.cuda.stream(stream):
            g.begin(stream)
            for _ in range(inner):
                enqueue()
            g.end(stream)
            g.launch(stream)
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
            ev[0].record(stream)
            for i in range(reps):
                g.launch(stream)
                ev[i + 1].record(stream)
        ev[-1].synchronize()
        t = sorted(ev[i].elapsed_time(ev[i + 1]) / inner for i in range(reps))
        return t[len(t) // 2] * 1000.0

    attn_us = timed(lambda: ss.draft_tree_attention(q, k, v, kc[0], vc[0], dP, dcp, dlp, s.Hq, s.Hkv, rope, out, ws,
                                                    stream=stream))
    reorg_us = timed(lambda: ss.kv_reorganize(kc, vc, dP, dcp, last, keep, new_parent=newp, n_kept=nk,
                                              n_layers=n_layers, advance=False, ws=ws, stream=stream))
    # expansion: the k = 8 most probable children of each of the w leaves
    # (top-k log-softmax over the draft's 128256-entry vocabulary)
    V, k = 128256, 8
    dlg = gdev.normal_f16_device(7, 5, (w, V), device=dev)
    dtok = torch.zeros((w, k), dtype=torch.int32, device=dev)
    dlp = torch.zeros((w, k), dtype=torch.float32, device=dev)
    ws_k = ss.workspace(ss.topk_logprobs_workspace_bytes(w), dev)
    topk_us = timed(lambda: ss.topk_logprobs(dlg, dtok, dlp, ws_k, stream=stream))
    if ss.read_device_error(ws, stream):
        raise RuntimeError("device error in the draft-side kernels")
    kept = int(nk.item())
    host = draft_tree_host(ss, np, w=w, k=k)
    attn_bytes = 2 * s.Hkv * (P + N + w) * s.D * 2   # K and V rows read (upper bound: every tree row)
    reorg_bytes = n_layers * 2 * s.Hkv * (3 + kept) * s.D * 2 * 2
    return {"workload": f"Llama-3.2-1B-shaped draft ({n_layers} layers, Hq/Hkv={s.Hq}/{s.Hkv}, D={s.D}); "
                        f"prefix P={P}, tree cache N={N}, w={w} leaves expanded; re-rooting path 3, subtree {kept}",
            "draft_attention_us": round(attn_us, 2),
            "draft_attention_gbs": round(attn_bytes / (attn_us * 1e-6) / 1e9, 1),
            "kv_reorganize_all_layers_us": round(reorg_us, 2),
            "kv_reorganize_bytes": reorg_bytes,
            "topk_logprobs_us": round(topk_us, 2),
            "topk_logprobs_gbs": round(w * V * 2 / (topk_us * 1e-6) / 1e9, 1),
            "draft_tree_host": host}


def tree_loop(ss, torch, np, dev, stream, V=128256, iters=40, w=8, k=8, d=3, bs=8, p_agree=0.8, seed=2506,
              check=None):
    """Iterations of the loop of Alg. 1 run one after the other on one GPU,
    with synthetic models in place of the draft and target networks.

    The target's greedy choice after a token context is a seeded hash of
    that context; its logits rows (fp16 N(0, 1), drawn on the device) carry
    10.0 at that token.  A leaf's draft logits carry 8.0 at the target's
    choice with probability p_agree (else at a random token), so paths of
    several tokens get accepted.  Per iteration: d expansion steps (host
    leaf selection, the leaves' draft rows through the top-k kernel, host
    expansion; the draft's tree-cache rows are tagged with their tokens),
    the bs-node subgraph to the target (its rows tagged, the target's
    logits, greedy acceptance and the KV commit on the device), re-rooting
    on the output (host) with the draft-cache reorganisation on the device
    and the pending tokens appended, then growth to bs nodes.  Returns
    timings (wall clock with the host round trips the loop needs) and the
    accepted tokens per iteration; `check(state)` is called after every
    iteration with the host and device state."""
    import time
    rng = np.random.default_rng(seed)
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    M61 = (1 << 61) - 1

    def push(h, t):  # hash of a context extended by one token
        return (h * 1000003 + t + 1) % M61

    def choice(h):  # the target's greedy next token after a context
        return int((h * 0x9E3779B97F4A7C15 >> 17) % V)

    S_max, D, Hkv = 4096, 8, 1
    P0 = 16
    committed = [int(t) for t in rng.integers(0, V, P0)]
    h_prefix = 0
    for t in committed:
        h_prefix = push(h_prefix, t)
    root = int(rng.integers(0, V))
    tree = ss.DraftTree(1 << 14, root)
    tk = torch.zeros((Hkv, S_max, D), dtype=torch.int32, device=dev)  # target cache (tags in element 0)
    dk = torch.zeros((Hkv, S_max, D), dtype=torch.int32, device=dev)  # draft cache
    tk[0, :P0, 0] = torch.tensor(committed, dtype=torch.int32)
    dk[0, :P0 + 1, 0] = torch.tensor(committed + [root], dtype=torch.int32)
    tkv, dkv = tk.view(torch.int16), dk.view(torch.int16)  # the kernels move fp16 rows: 2 x D halves
    tvv, dvv = torch.zeros_like(tkv), torch.zeros_like(dkv)  # value caches (distinct memory)
    P_t = torch.tensor([P0], dtype=torch.int32, device=dev)
    P_d = torch.tensor([P0 + 1], dtype=torch.int32, device=dev)
    p_d = P0 + 1
    ws = ss.workspace(1 << 16, dev)
    ws_k = ss.workspace(ss.topk_logprobs_workspace_bytes(w), dev)
    ws_a = ss.workspace(ss.greedy_accept_workspace_bytes(bs), dev)
    d_tok = torch.zeros((w, k), dtype=torch.int32, device=dev)
    d_lp = torch.zeros((w, k), dtype=torch.float32, device=dev)
    d_am = torch.zeros(bs, dtype=torch.int32, device=dev)
    d_acc, d_bonus, d_len = (torch.zeros(1, dtype=torch.int32, device=dev) for _ in range(3))
    t_draft = t_target = t_reroot = 0.0
    n_steps = 0
    accepted = []

    def node_hashes():
        tok, par, _, row, _ = tree.nodes()
        hs = [0] * len(tok)
        for v in range(len(tok)):  # parents precede children
            hs[v] = push(h_prefix, int(tok[v])) if v == 0 else push(hs[par[v]], int(tok[v]))
        return tok, par, row, hs

    def expand_step():
        leaves, _ = tree.select_leaves(w)
        n = len(leaves)
        if n == 0:
            return
        tok, par, row, hs = node_hashes()
        for v in leaves:
            if v != 0:
                dk[0, p_d + int(row[v]), 0] = int(tok[v])
        lg = torch.randn((n, V), generator=gen, device=dev).half()
        agree = rng.random(n) < p_agree
        cols = [choice(hs[v]) if agree[j] else int(rng.integers(0, V)) for j, v in enumerate(leaves)]
        lg[torch.arange(n, device=dev), torch.tensor(cols, device=dev)] = 8.0
        ss.topk_logprobs(lg.view(torch.int16), d_tok[:n], d_lp[:n], ws_k, stream=stream)
        tree.expand(leaves, d_tok[:n].cpu().numpy(), d_lp[:n].cpu().numpy())

    with torch.cuda.stream(stream):
        for it in range(iters):
            t0 = time.perf_counter()
            for _ in range(d):
                if tree.rows() + w <= 64:
                    expand_step()
                    n_steps += 1
            torch.cuda.synchronize()
            t1 = time.perf_counter()
            # ---- target: verify the bs most probable nodes ----
            nodes, par, toks = tree.select_subgraph(bs)
            T = len(nodes)
            _, _, _, hs = node_hashes()
            p_t = int(P_t.item())
            tk[0, p_t:p_t + T, 0] = torch.from_numpy(toks.astype(np.int32)).to(dev)  # the tree's new rows
            lg_t = torch.randn((T, V), generator=gen, device=dev).half()
            lg_t[torch.arange(T, device=dev), torch.tensor([choice(hs[v]) for v in nodes], device=dev)] = 10.0
            d_par = torch.from_numpy(par.astype(np.int32)).to(dev)
            d_toks = torch.from_numpy(toks.astype(np.int32)).to(dev)
            ss.greedy_accept(lg_t.view(torch.int16), d_toks, d_par, d_am[:T], d_acc, d_bonus, ws_a,
                             path_len=d_len, stream=stream)
            ss.kv_commit(tkv, tvv, P_t, d_par, d_acc, advance=True, ws=ws, stream=stream)
            a, b, L = int(d_acc.item()), int(d_bonus.item()), int(d_len.item())
            path = []
            j = a
            while j >= 0:
                path.append(int(toks[j]))
                j = int(par[j])
            path = path[::-1]
            t2 = time.perf_counter()
            # ---- draft: re-root on the output, reorganise its cache ----
            forest = tree.forest()
            res = tree.reroot(path + [b])
            if len(forest) > 0:
                d_f = torch.from_numpy(forest.astype(np.int32)).to(dev)
                d_last = torch.tensor([res["last"]], dtype=torch.int32, device=dev)
                d_keep = torch.tensor([res["keep"]], dtype=torch.int32, device=dev)
                ss.kv_reorganize(dkv, dvv, P_d, d_f, d_last, d_keep, advance=True, ws=ws, stream=stream)
            p_d += res["path_rows"]
            for t in res["pending"]:
                dk[0, p_d, 0] = t
                p_d += 1
            P_d.fill_(p_d)
            committed += path
            for t in path:
                h_prefix = push(h_prefix, t)
            while tree.size() < bs and tree.rows() + w <= 64:
                expand_step()
                n_steps += 1
            torch.cuda.synchronize()
            t3 = time.perf_counter()
            t_draft += t1 - t0
            t_target += t2 - t1
            t_reroot += t3 - t2
            accepted.append(L)
            if check is not None:
                check({"it": it, "committed": committed, "bonus": b, "path": path, "L": L, "logits": lg_t,
                       "tokens": toks, "parent": par, "argmax": d_am[:T].cpu().numpy(), "accepted": a,
                       "P_t": int(P_t.item()), "p_d": p_d, "tk": tk, "dk": dk, "tree": tree, "res": res})
    if ss.read_device_error(ws, stream):
        raise RuntimeError("device error in the tree loop")
    return {"workload": f"sequential loop of Alg. 1 on one GPU, synthetic draft and target (V={V}, "
                        f"w={w}, k={k}, d={d}, bs={bs}, draft agrees with the target w.p. {p_agree})",
            "iterations": iters,
            "mean_accepted_per_iteration": round(float(np.mean(accepted)), 2),
            "draft_expansion_ms_per_iteration": round(t_draft / iters * 1e3, 3),
            "verify_accept_commit_ms_per_iteration": round(t_target / iters * 1e3, 3),
            "reroot_reorganise_grow_ms_per_iteration": round(t_reroot / iters * 1e3, 3),
            "expansion_steps": n_steps,
            "note": "wall clock with the host round trips of a Python driver; no target or draft network runs"}


def draft_tree_host(ss, np, w=8, k=8, d=3, bs=8, iters=200, vocab=128256):
    """The draft worker's host-side tree (swiftspec_draft_tree_*, through the
    Python binding) over `iters` iterations of the loop of Alg. 1: d
    expansion steps of w leaves with k children each (synthetic
    log-probabilities, seeded), re-rooting on a synthetic target output (the
    root path to a node drawn at random plus one token, a child's 70 % of
    the time), growth to bs nodes, and the bs-node subgraph; tree-cache rows
    capped at 64 (the draft kernels' limit).  Mean microseconds per call."""
    import time
    rng = np.random.default_rng(11309)
    tree = ss.DraftTree(1 << 16, 1)
    t_exp = t_rr = t_sub = 0.0
    n_exp = 0
    sizes = []
    lps = [(-np.sort(-np.log(rng.dirichlet(np.full(64, 0.3))))[:k]).astype(np.float32) for _ in range(64)]
    toks = rng.integers(0, vocab, (4096, k)).astype(np.int32)
    for it in range(iters):
        for _ in range(d):
            if tree.rows() + w > 64:
                break
            t0 = time.perf_counter()
            leaves, _ = tree.select_leaves(w)
            n = len(leaves)
            tree.expand(leaves, toks[(it * 7 + n_exp) % 4000:(it * 7 + n_exp) % 4000 + n],
                        np.stack([lps[(it + j) % 64] for j in range(n)]))
            t_exp += time.perf_counter() - t0
            n_exp += 1
        sizes.append(tree.size())
        tok_h, par_h, _, _, _ = tree.nodes()
        v = int(rng.integers(len(tok_h)))
        path = []
        while v >= 0:
            path.append(v)
            v = int(par_h[v])
        ver = [int(tok_h[u]) for u in path[::-1]]
        kids = np.nonzero(par_h == path[0])[0]
        ver.append(int(tok_h[kids[0]]) if len(kids) and rng.random() < 0.7 else vocab + 1)
        t0 = time.perf_counter()
        tree.reroot(ver)
        t_rr += time.perf_counter() - t0
        while tree.size() < bs and tree.rows() + w <= 64:
            t0 = time.perf_counter()
            leaves, _ = tree.select_leaves(w)
            tree.expand(leaves, toks[:len(leaves)], np.stack([lps[j] for j in range(len(leaves))]))
            t_exp += time.perf_counter() - t0
            n_exp += 1
        t0 = time.perf_counter()
        tree.select_subgraph(bs)
        t_sub += time.perf_counter() - t0
    return {"iterations": iters, "w": w, "k": k, "d": d, "bs": bs,
            "mean_tree_nodes": round(float(np.mean(sizes)), 1),
            "expand_step_us": round(t_exp / max(n_exp, 1) * 1e6, 2),
            "reroot_us": round(t_rr / iters * 1e6, 2),
            "select_subgraph_us": round(t_sub / iters * 1e6, 2)}


def full_step(args, ss, torch, np, dev, stream):
    """The 80-layer Llama-3-70B-shaped verification step (T = 64, P = 8192,
    final RMSNorm + fp16 LM head over 128256 rows) as one HIP graph: every
    layer's own weights and caches (35.8 GB of int4 weights + 2.1 GB LM head
    + 2.7 GB of KV cache, drawn on the device with the workload recipe), the
    graph replayed `full_step_reps` times and timed with HIP events; the
    KV commit of the accepted path over all 80 layers timed as one launch;
    the greedy acceptance alone, and the closed step (verification, greedy
    acceptance and the commit of the path it accepts) as one graph."""
    from gen import device as gdev
    from gen import workloads as wl
    cfg = wl.CONFIGS["c5"]
    s = cfg.shape
    T, nl = cfg.T, cfg.n_layers
    seed, kv_seed = cfg.seeds()["weights"], cfg.seeds()["kv"]
    t0 = time.time()
    shape = (nl, s.Hkv, cfg.S_max, s.D)
    kc = torch.zeros(shape, dtype=torch.int16, device=dev)
    vc = torch.zeros(shape, dtype=torch.int16, device=dev)
    keep, descs = [], []
    for l in range(nl):
        base = l * wl.LAYER_STREAM_STRIDE
        w4 = {}
        for name, K, N in s.gemms():
            q, sc, z = gdev.w4_random_device(seed, base + wl.W_STREAMS[name], N, K, device=dev)
            d = ss.make_w4(q, sc, z)
            keep.append((q, sc, z, ss.prepack_w4(d)))
            w4[name] = d
        an = gdev.normal_f16_device(seed, base + wl.W_STREAMS["attn_norm"], (s.H,), 1.0, 0.02, dev)
        mn = gdev.normal_f16_device(seed, base + wl.W_STREAMS["mlp_norm"], (s.H,), 1.0, 0.02, dev)
        kc[l, :, :cfg.P] = gdev.normal_f16_device(kv_seed, 2 * l, (s.Hkv, cfg.P, s.D), device=dev)
        vc[l, :, :cfg.P] = gdev.normal_f16_device(kv_seed, 2 * l + 1, (s.Hkv, cfg.P, s.D), device=dev)
        keep.append((an, mn))
        descs.append(ss.make_layer(an, mn, w4["wqkv"], w4["wo"], w4["wgate"], w4["wup"], w4["wdown"], kc[l], vc[l]))
    layers = ss.make_layers(descs)
    gamma = gdev.normal_f16_device(seed, wl.FINAL_NORM_STREAM, (s.H,), 1.0, 0.02, dev)
    lm_w = gdev.normal_f16_device(seed, wl.LM_HEAD_STREAM, (cfg.vocab, s.H), 0.0, 0.02, dev)
    x = gdev.normal_f16_device(cfg.seeds()["activations"], 0, (T, s.H), device=dev)
    parent, acc = wl.make_tree(cfg)
    dparent = torch.from_numpy(np.asarray(parent, np.int32)).to(dev)
    dacc = torch.tensor([acc], dtype=torch.int32, device=dev)
    P_dev = torch.tensor([cfg.P], dtype=torch.int32, device=dev)
    rope = torch.from_numpy(ss.rope_table(500000.0, cfg.S_max, s.D)).to(dev)
    dims = ss.make_dims(s.H, s.Hq, s.Hkv, s.D, s.F, cfg.S_max)
    ws = ss.workspace(ss.verify_step_workspace_bytes(dims, T, cfg.vocab), dev)
    hidden = torch.empty_like(x)
    logits = torch.zeros((T, cfg.vocab), dtype=torch.int16, device=dev)
    # draft tokens of the tree nodes (seeded, uniform over the vocabulary)
    tokens = torch.from_numpy(np.random.default_rng(cfg.seeds()["tree"]).integers(0, cfg.vocab, T)
                              .astype(np.int32)).to(dev)
    d_am = torch.zeros(T, dtype=torch.int32, device=dev)
    d_acc, d_bonus, d_len = (torch.zeros(1, dtype=torch.int32, device=dev) for _ in range(3))
    aws = ss.workspace(ss.greedy_accept_workspace_bytes(T), dev)
    torch.cuda.synchronize()
    setup_s = time.time() - t0

    def timed(enqueue, reps, warm=2, inner=1):
        # `inner` back-to-back copies in one graph, per-copy times returned:
        # a launch of a few microseconds alone would time the host's graph
        # submission rather than the kernel
        g = ss.Graph()
        with torch.cuda.stream(stream):
            g.begin(stream)
            for _ in range(inner):
                enqueue()
            g.end(stream)
            for _ in range(warm):
                g.launch(stream)
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(reps + 1)]
            ev[0].record(stream)
            for i in range(reps):
                g.launch(stream)
                ev[i + 1].record(stream)
        ev[-1].synchronize()
        return sorted(ev[i].elapsed_time(ev[i + 1]) / inner for i in range(reps))

    def step():
        hidden.copy_(x)  # the tree tokens' embeddings enter the step
        ss.verify_step(layers, dims, hidden, P_dev, dparent, rope, ws, gamma, lm_w, logits, stream=stream)

    ms = timed(step, args.full_step_reps)
    if ss.read_device_error(ws, stream):
        raise RuntimeError("device error in the 80-layer step")
    head_ms = timed(lambda: ss.lm_head(hidden, gamma, lm_w, logits, ws, stream=stream), args.full_step_reps)
    commit_ms = timed(lambda: ss.kv_commit(kc, vc, P_dev, dparent, dacc, n_layers=nl, advance=False, ws=ws,
                                           stream=stream), args.full_step_reps, inner=20)

    def accept():
        ss.greedy_accept(logits, tokens, dparent, d_am, d_acc, d_bonus, aws, path_len=d_len, stream=stream)

    accept_ms = timed(accept, args.full_step_reps, inner=20)

    def closed_step():
        step()
        accept()
        ss.kv_commit(kc, vc, P_dev, dparent, d_acc, n_layers=nl, advance=False, ws=aws, stream=stream)

    closed_ms = timed(closed_step, args.full_step_reps)
    if ss.read_device_error(aws, stream):
        raise RuntimeError("device error in the closed step")
    med = lambda v: v[len(v) // 2]
    w_bytes = nl * s.w4_bytes()
    kv_bytes = nl * cfg.kv_bytes_per_layer()
    head_bytes = cfg.vocab * s.H * 2 + T * cfg.vocab * 2
    step_bytes = w_bytes + kv_bytes + head_bytes
    mean_ms = sum(ms) / len(ms)
    out = {"workload": f"{cfg.name}: {nl} Llama-3-70B-shaped layers (int4 g128) + final RMSNorm + fp16 LM head "
                       f"V={cfg.vocab}; tree T={T} ({cfg.levels} levels, branching<={cfg.branching}); "
                       f"prefix P={cfg.P}; one HIP graph per step",
           "ms_per_step": round(mean_ms, 4), "ms_p50": round(med(ms), 4),
           "us_per_layer_incl_head": round(mean_ms * 1000.0 / nl, 2),
           "algorithmic_bytes": step_bytes,
           "hbm_gbs": round(step_bytes / (mean_ms * 1e-3) / 1e9, 1),
           "frac_hbm": round(step_bytes / (mean_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
           "lm_head_us": round(med(head_ms) * 1000.0, 2),
           "lm_head_gbs": round((head_bytes + T * s.H * 4) / (med(head_ms) * 1e-3) / 1e9, 1),
           "kv_commit_all_layers_us": round(med(commit_ms) * 1000.0, 2),
           "greedy_accept_us": round(med(accept_ms) * 1000.0, 2),
           "ms_per_step_closed": round(sum(closed_ms) / len(closed_ms), 4),
           "closed_step": "verification + greedy acceptance + commit of the accepted path, one graph",
           "reps": args.full_step_reps, "setup_s": round(setup_s, 1),
           "weights": "drawn on the device with the workload recipe (torch generator, seeded)"}
    del keep, kc, vc, lm_w
    torch.cuda.empty_cache()
    return out


def gemm_ab(ss, torch, np, inst, cfg, stream, dev):
    """Matrix-core against vector-ALU W4A16 GEMM: the layer's four weight
    shapes (gate alone for the SwiGLU width) at M = 1 .. 64, each entry point
    called on rotated weight copies inside a replayed graph; one JSON line
    per M with microseconds, algorithmic GB/s and the VALU / MFMA time ratio."""
    s = cfg.shape
    copies = len(inst)
    shapes = [("qkv", "wqkv", s.H, s.n_qkv), ("o_proj", "wo", s.Hq * s.D, s.H), ("gate", "wgate", s.H, s.F),
              ("down", "wdown", s.F, s.H)]
    w4b = lambda K, N: K * N // 2 + (K // 128) * N * 3
    for M in (1, 2, 4, 8, 16, 32, 64):
        x = (torch.randn((M, max(s.H, s.F)), device=dev) * 1.0).half().view(torch.int16)
        y = torch.zeros((M, max(s.F, s.n_qkv)), dtype=torch.int16, device=dev)
        out = {"gemm_ab_M": M}
        for name, wname, K, N in shapes:
            ws_m = ss.workspace(ss.gemm_workspace_bytes(M, K, N), dev)
            ws_v = ss.workspace(ss.gemm_valu_workspace_bytes(M, K, N), dev)
            res = {}
            for kind, fn in (("mfma", lambda d: ss.w4a16_gemm(d, x[:, :K], y[:, :N], ws_m, stream=stream)),
                             ("valu", lambda d: ss.w4a16_gemm_valu(d, x[:, :K], y[:, :N], ws_v, stream=stream))):
                g = ss.Graph()
                iters = 30
                with torch.cuda.stream(stream):
                    for i in range(3):
                        fn(inst[i % copies]["w4"][wname])
                    g.begin(stream)
                    for i in range(iters):
                        fn(inst[i % copies]["w4"][wname])
                    g.end(stream)
                    g.launch(stream)
                    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                    e0.record(stream)
                    for _ in range(3):
                        g.launch(stream)
                    e1.record(stream)
                e1.synchronize()
                us = e0.elapsed_time(e1) * 1000.0 / (3 * iters)
                res[kind] = {"us": round(us, 2), "GBps": round(w4b(K, N) / (us * 1e-6) / 1e9, 1)}
            res["valu_over_mfma"] = round(res["valu"]["us"] / res["mfma"]["us"], 2)
            out[name] = res
        print(json.dumps(out), flush=True)


def run_only(args, ss, torch, np, inst, cfg, dims, dparent, dacc, rope, stream, dev):
    """Launch a single kernel type `iters` times (rotating layer copies) for
    rocprofv3 counter collection; prints what it ran."""
    s = cfg.shape
    T = cfg.T
    copies = len(inst)
    kind = args.only_kernel
    xin = torch.zeros((T, max(s.H, s.F)), dtype=torch.int16, device=dev)
    xin.copy_(torch.randint(-3000, 3000, xin.shape, dtype=torch.int16, device=dev) & 0x3BFF)
    out = torch.zeros((T, max(s.F, s.n_qkv)), dtype=torch.int16, device=dev)
    ws = ss.workspace(ss.verify_layer_workspace_bytes(dims, T), dev)
    qkv = torch.zeros((T, s.n_qkv), dtype=torch.int16, device=dev)
    big = torch.zeros(256 << 20, dtype=torch.uint8, device=dev)
    big2 = torch.empty_like(big)
    with torch.cuda.stream(stream):
        for i in range(args.iters):
            d = inst[i % copies]
            if kind == "swiglu":
                ss.w4a16_swiglu(d["w4"]["wgate"], d["w4"]["wup"], xin[:, :s.H], out[:, :s.F], ws, stream=stream)
            elif kind == "qkv":
                ss.w4a16_gemm(d["w4"]["wqkv"], xin[:, :s.H], out[:, :s.n_qkv], ws, stream=stream)
            elif kind == "o":
                ss.w4a16_gemm(d["w4"]["wo"], xin[:, :s.Hq * s.D], out[:, :s.H], ws, stream=stream)
            elif kind == "down":
                ss.w4a16_gemm(d["w4"]["wdown"], xin[:, :s.F], out[:, :s.H], ws, stream=stream)
            elif kind == "attention":
                Hd = s.Hq * s.D
                ss.tree_attention(qkv, qkv[:, Hd:], qkv[:, Hd + s.Hkv * s.D:], d["kc"], d["vc"], d["P"], dparent,
                                  s.Hq, s.Hkv, s.D, rope, out[:, :Hd], ws, stream=stream)
            elif kind == "commit":
                ss.kv_commit(d["kc"], d["vc"], d["P"], dparent, dacc, ws=ws, stream=stream)
            elif kind == "copy":
                big2.copy_(big)
            else:
                raise SystemExit(f"unknown kernel {kind}")
    stream.synchronize()
    print(json.dumps({"only_kernel": kind, "iters": args.iters, "copies": copies,
                      "copy_bytes": big.numel() if kind == "copy" else None}), flush=True)


if __name__ == "__main__":
    main()
