#!/usr/bin/env python3
"""Tree-verification benchmark on one MI355X: verify steps/s and achieved HBM bandwidth.

One step = the whole hot path on one batch of synthetic input: tree-masked attention for every layer of the
workload, greedy tree acceptance, and the KV commit where the workload includes it.  Inputs are resident in
HBM before timing starts.  `--rotate-bytes` worth of distinct input sets (default 1.25 GiB, several times the
256 MB Infinity Cache) are cycled so that every step streams its K/V from HBM rather than from cache.  The
timed steps run as HIP-graph replays on one stream (no host launch gaps), bracketed by
torch.cuda.synchronize() and HIP events.

Printed: one JSON line with the step rate, the attention kernel's achieved bandwidth against the 8 TB/s HBM
roofline (HIP events around a graph of attention launches on the same stream), and the CPU oracle timed on
this host's cores over a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import glob
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "tree-verify steps/sec + achieved HBM GB/s (% peak), LLaVA-1.6-7B shape, 1 GPU"
HBM_PEAK_GBPS = 8000.0
BF16_DENSE_PEAK_TFLOPS = 2500.0


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=2000)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--workload", default="llava7b_layer")
    ap.add_argument("--rotate-bytes", type=float, default=1.25 * 2 ** 30)
    ap.add_argument("--num-splits", type=int, default=0, help="key-axis splits (0 = library's choice)")
    ap.add_argument("--attn-launches", type=int, default=400, help="launches in the attention-only timing")
    ap.add_argument("--cpu-seconds", type=float, default=12.0, help="target length of the CPU-oracle sample")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-only", action="store_true", help="skip the CPU baseline and the parity spot check")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the other workloads' sub-objects (full_pass, llava13b_layer, gqa_long, tiny)")
    ap.add_argument("--repeats", type=int, default=30, help="event-timed repeats behind each p10/p50/p90")
    ap.add_argument("--traffic-calibration", action="store_true",
                    help="for rocprofv3 --pmc runs: a plain device copy of known size, then attention launches; "
                         "prints what each launch should move and exits")
    return ap.parse_args()


def attn_bytes_per_layer(wl, kv_len) -> int:
    """Algorithmic bytes of one tree-attention launch: K and V of every prefix slot and of the tree nodes,
    the queries in and the outputs out (2-byte elements)."""
    s = 2 if wl.dtype == "bf16" else 4
    T, D = wl.num_nodes, wl.head_dim
    kv = sum(2 * wl.num_kv_heads * int(L) * D * s for L in kv_len)
    tree = wl.batch * 2 * wl.num_kv_heads * T * D * s
    qo = wl.batch * 2 * wl.num_q_heads * T * D * s
    return kv + tree + qo


def accept_bytes(wl) -> int:
    """Logits of every node, draft tokens and parents in, lengths / paths / bonus tokens out."""
    return wl.batch * (wl.num_nodes * wl.vocab * 4 + 8 * wl.num_nodes + 4 * (wl.num_nodes + 2))


def commit_bytes(wl, path, alen) -> int:
    s = 2 if wl.dtype == "bf16" else 4
    moved = sum(int((path[b, 1:alen[b] + 1] != np.arange(1, alen[b] + 1)).sum()) for b in range(wl.batch))
    return moved * 2 * 2 * wl.num_kv_heads * wl.head_dim * s * wl.num_layers


def kernel_source_hash() -> str:
    """sha256/16 of the attention kernel's source with comments and blank space removed (so that the hash
    changes with the code, not with its comments)."""
    import re
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(ROOT, "paper_2606_00535_amd", "csrc", "tree_attn_bf16.hip"))):
        src = open(f).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        src = re.sub(r"//[^\n]*", "", src)
        src = "\n".join(line.strip() for line in src.splitlines() if line.strip())
        h.update(src.encode())
    return h.hexdigest()[:16]


def measured_traffic(workload: str):
    """HBM bytes per attention launch from the committed rocprofv3 counter summary, if it was taken on the
    current kernel source (its hash is recorded in the summary); else None."""
    path = os.path.join(ROOT, "profiles", "tree_attn_bf16.%s.hbm_traffic.md" % workload)
    if not os.path.exists(path):
        return None
    rec = None
    for line in open(path):
        if line.startswith("RESULT "):
            rec = json.loads(line[len("RESULT "):])
    if not rec or rec.get("kernel_source_sha256_16") != kernel_source_hash():
        return None
    return rec.get("bytes_per_launch")


def attn_flops_per_layer(wl, kv_len, parent) -> float:
    """Algorithmic flops of one tree-attention launch: q.k and p.v over the visible keys of every row,
    4 * D * Hq * sum_b sum_i (L_b + depth_i + 1)."""
    total = 0
    for b in range(wl.batch):
        par = parent[b]
        depth = np.zeros(len(par), dtype=np.int64)
        for i in range(1, len(par)):
            depth[i] = depth[par[i]] + 1
        total += int((int(kv_len[b]) + depth + 1).sum())
    return 4.0 * wl.head_dim * wl.num_q_heads * total


def dist(xs):
    """p10 / p50 / p90 / mean of a list of per-call times (us)."""
    a = np.sort(np.asarray(xs, dtype=np.float64))
    return {"p10": round(float(np.percentile(a, 10)), 3), "p50": round(float(np.percentile(a, 50)), 3),
            "p90": round(float(np.percentile(a, 90)), 3), "mean": round(float(a.mean()), 3), "repeats": int(a.size)}


def replay_times_us(torch, graph, calls_per_replay, repeats):
    """Each of `repeats` replays of `graph` timed alone with HIP events on the capturing (current) stream; the
    time per call in us, one value per replay."""
    graph.replay()
    torch.cuda.synchronize()
    out = []
    for _ in range(repeats):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        graph.replay()
        e1.record()
        torch.cuda.synchronize()
        out.append(e0.elapsed_time(e1) * 1e3 / calls_per_replay)
    return out


def capture(torch, fn):
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    return g


def gpu_clocks():
    """The GPU's current clocks as rocm-smi reports them (read only; nothing is set), or None."""
    import shutil
    import subprocess
    exe = shutil.which("rocm-smi") or ("/opt/rocm/bin/rocm-smi" if os.path.exists("/opt/rocm/bin/rocm-smi") else None)
    if exe is None:
        return None
    try:
        r = subprocess.run([exe, "--showclocks"], capture_output=True, text=True, timeout=30)
    except (OSError, subprocess.SubprocessError):
        return None
    clocks = {}
    for line in r.stdout.splitlines():
        low = line.lower()
        for key in ("sclk", "mclk", "fclk", "socclk"):
            if key + " clock level" in low and "(" in line and ")" in line:
                clocks.setdefault(key, line[line.rindex("(") + 1:line.rindex(")")].strip())
    return clocks or None


def make_sets(torch, dev, wl, rotate_bytes, with_logits=True, min_sets=2):
    """Input sets of workload `wl` resident on the device: topology, lengths, logits and draft tokens from the
    seeded generator; q/k/v drawn on the device with a seeded generator (same N(0,1) distributions).  Enough
    distinct sets (at least min_sets) that `rotate_bytes` are touched before a set comes round again."""
    from paper_2606_00535_amd import workload as W
    NL, B, Hq, Hkv, T, D = wl.num_layers, wl.batch, wl.num_q_heads, wl.num_kv_heads, wl.num_nodes, wl.head_dim
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    host = W.make_batch(wl, layers=[], with_logits=with_logits)
    S = host.k_cache.shape[3]
    gen = torch.Generator(device=dev)
    gen.manual_seed(wl.seed)

    def draw(shape, std=1.0):
        x = torch.randn(shape, generator=gen, device=dev, dtype=torch.float32)
        if std != 1.0:
            x.mul_(std)
        return x.to(tdt)

    per_set = NL * 2 * B * Hkv * S * D * (2 if tdt == torch.bfloat16 else 4) + (host.logits.nbytes if with_logits else 0)
    R = max(min_sets, int(math.ceil(rotate_bytes / per_set)))
    base = dict(q=draw((NL, B, Hq, T, D), wl.q_std), k=draw((NL, B, Hkv, S, D)), v=draw((NL, B, Hkv, S, D)),
                kv=torch.from_numpy(host.kv_len).to(dev), par=torch.from_numpy(host.parent).to(dev))
    if with_logits:
        base["logits"] = torch.from_numpy(host.logits).to(dev)
        base["tok"] = torch.from_numpy(host.tokens).to(dev)
    sets = []
    for r in range(R):
        st = {key: (val if r == 0 else val.clone()) for key, val in base.items()}
        st["out"] = torch.empty((NL, B, Hq, T, D), dtype=tdt, device=dev)
        st["alen"] = torch.empty(B, dtype=torch.int32, device=dev)
        st["path"] = torch.empty((B, T), dtype=torch.int32, device=dev)
        st["next"] = torch.empty(B, dtype=torch.int32, device=dev)
        st["kv_out"] = torch.empty(B, dtype=torch.int32, device=dev)
        sets.append(st)
    return host, sets, R, tdt


def measure_workload(torch, dev, name, args):
    """One other workload's verify step, graph-replayed over rotated input sets: the whole step (every layer's
    attention, acceptance, commit where the workload has it), the attention call alone and acceptance alone,
    each as p10/p50/p90 over `args.repeats` event-timed replays."""
    from paper_2606_00535_amd import dreams
    from paper_2606_00535_amd import workload as W
    wl = W.WORKLOADS[name]
    NL, B, Hq, T = wl.num_layers, wl.batch, wl.num_q_heads, wl.num_nodes
    # (the fp32 case is latency-bound and a few MB: two sets, no cache rotation)
    host, sets, R, tdt = make_sets(torch, dev, wl, args.rotate_bytes if wl.dtype == "bf16" else 0)
    desc = dreams.attn_desc(sets[0]["q"][0], sets[0]["k"][0], 0, wl.max_kv_len)
    ws_attn = torch.zeros(max(1, dreams.tree_verify_attn_workspace_size(desc)), dtype=torch.uint8, device=dev)
    ws_acc = torch.zeros(max(1, dreams.tree_accept_workspace_size(B, T, wl.vocab)), dtype=torch.uint8, device=dev)

    def attention(st):
        for l in range(NL):
            dreams.tree_verify_attn(st["q"][l], st["k"][l], st["v"][l], st["kv"], st["par"], out=st["out"][l],
                                    with_lse=False, max_kv_len=wl.max_kv_len, workspace=ws_attn)

    def accept(st):
        dreams.tree_accept(st["logits"], st["tok"], st["par"], outputs=(st["alen"], st["path"], st["next"], None),
                           workspace=ws_acc)

    def commit(st):
        dreams.kv_commit(st["k"], st["v"], st["kv"], st["path"], st["alen"], kv_len_out=st["kv_out"])

    def step(st):
        attention(st)
        accept(st)
        if wl.commit:
            commit(st)

    for r in range(R):
        step(sets[r])
    torch.cuda.synchronize()
    reps = max(1, args.repeats)
    step_us = replay_times_us(torch, capture(torch, lambda: [step(st) for st in sets]), R, reps)
    attn_us = replay_times_us(torch, capture(torch, lambda: [attention(st) for st in sets]), R * NL, reps)
    acc_us = replay_times_us(torch, capture(torch, lambda: [accept(st) for st in sets]), R, reps)
    a_bytes = attn_bytes_per_layer(wl, host.kv_len)
    a_flops = attn_flops_per_layer(wl, host.kv_len, host.parent)
    acc_b = accept_bytes(wl)
    ok = True
    if ws_attn.numel() >= 65536:
        try:
            dreams.workspace_status(ws_attn)
        except dreams.DreamsError:
            ok = False
    res = {"workload": name, "layers": NL, "batch": B, "q_heads": Hq, "kv_heads": wl.num_kv_heads,
           "head_dim": wl.head_dim, "dtype": wl.dtype, "kv_len": [int(x) for x in host.kv_len],
           "tree_nodes": T, "vocab": wl.vocab, "rotated_input_sets": R,
           "splits": dreams.tree_verify_attn_splits(desc),
           "step_us": dist(step_us), "steps_per_s": round(1e6 / np.median(step_us), 2),
           "attention": {"us_per_launch": dist(attn_us), "bytes_per_launch": a_bytes, "flops_per_launch": a_flops}}
    a50 = np.median(attn_us)
    res["attention"]["GBps"] = round(a_bytes / (a50 * 1e-6) / 1e9, 1)
    res["attention"]["frac_of_hbm_peak"] = round(a_bytes / (a50 * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)
    res["attention"]["TFLOPs"] = round(a_flops / (a50 * 1e-6) / 1e12, 1)
    res["attention"]["frac_of_bf16_dense_peak"] = round(a_flops / (a50 * 1e-6) / 1e12 / BF16_DENSE_PEAK_TFLOPS, 4)
    res["accept"] = {"us_per_launch": dist(acc_us), "bytes_per_launch": acc_b,
                     "GBps": round(acc_b / (np.median(acc_us) * 1e-6) / 1e9, 1)}
    step_bytes = NL * a_bytes + acc_b
    if wl.commit:
        com_b = commit_bytes(wl, sets[0]["path"].cpu().numpy(), sets[0]["alen"].cpu().numpy())
        res["commit_bytes"] = com_b
        step_bytes += com_b
    res["step_algorithmic_bytes"] = step_bytes
    res["step_GBps"] = round(step_bytes / (np.median(step_us) * 1e-6) / 1e9, 1)
    res["step_frac_of_hbm_peak"] = round(step_bytes / (np.median(step_us) * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4)
    res["workspace_flags_clear"] = ok
    del sets, ws_attn, ws_acc
    torch.cuda.empty_cache()
    return res


def measure_prefill(torch, dev, args, N=3136, n_img=2880, H=32, D=128):
    """The prefill statistics at the LLaVA-1.6-7B prompt shape (3136 tokens, the first 2880 visual, 32 heads of
    128): causal lse and entropy of every row, the layer's AE over the prompt, Eq. 2 importance of the visual
    tokens, and the top-r choice (one in five), each verb graph-replayed alone; TFLOP/s of the two matrix-core
    passes against the dense bf16 peak.  Inputs: seeded N(0,1) bf16 q and k drawn on the device."""
    from paper_2606_00535_amd import dreams
    gen = torch.Generator(device=dev)
    gen.manual_seed(7)
    S = (N + 63) // 64 * 64
    sets = []
    for _ in range(2):
        st = {"q": torch.randn((1, H, N, D), generator=gen, device=dev).to(torch.bfloat16),
              "k": torch.randn((1, H, S, D), generator=gen, device=dev).to(torch.bfloat16),
              "pl": torch.full((1,), N, dtype=torch.int32, device=dev)}
        st["lse"] = torch.empty((1, H, N), dtype=torch.float32, device=dev)
        st["ent"] = torch.empty((1, H, N), dtype=torch.float32, device=dev)
        st["ae"] = torch.empty(1, dtype=torch.float32, device=dev)
        st["imp"] = torch.empty((1, n_img), dtype=torch.float32, device=dev)
        st["keep"] = torch.empty((1, n_img // 5), dtype=torch.int32, device=dev)
        sets.append(st)
    ws = torch.zeros(dreams.visual_importance_workspace_size(1, H, n_img), dtype=torch.uint8, device=dev)
    verbs = {
        "stats": lambda st: dreams.prefill_attn_stats(st["q"], st["k"], st["pl"], lse=st["lse"], entropy=st["ent"]),
        "entropy_mean": lambda st: dreams.prefill_attn_entropy_mean(st["ent"], st["pl"], ae=st["ae"]),
        "importance": lambda st: dreams.prefill_visual_importance(st["q"], st["k"], st["pl"], st["lse"], 0, n_img,
                                                                  importance=st["imp"], workspace=ws),
        "topk": lambda st: dreams.visual_topk(st["imp"], n_img // 5, keep=st["keep"]),
    }
    res = {"workload": "llava7b_prompt", "prompt_tokens": N, "image_tokens": n_img, "keep": n_img // 5,
           "q_heads": H, "kv_heads": H, "head_dim": D, "dtype": "bf16"}
    for name in ("stats", "entropy_mean", "importance", "topk"):
        for st in sets:
            verbs[name](st)
        torch.cuda.synchronize()
        g = capture(torch, lambda: [verbs[name](st) for st in sets])
        us = replay_times_us(torch, g, len(sets), max(1, args.repeats))
        res[name + "_us"] = dist(us)
    # algorithmic flops: q.k over the visible keys of every row (stats), over every (row, visual key) pair with
    # key <= row (importance)
    stats_flops = 2.0 * D * H * (N * (N + 1) / 2)
    imp_flops = 2.0 * D * H * sum(N - j for j in range(n_img))
    for name, fl in (("stats", stats_flops), ("importance", imp_flops)):
        t = res[name + "_us"]["p50"] * 1e-6
        res[name + "_flops"] = fl
        res[name + "_TFLOPs"] = round(fl / t / 1e12, 1)
        res[name + "_frac_of_bf16_dense_peak"] = round(fl / t / 1e12 / BF16_DENSE_PEAK_TFLOPS, 4)
    del sets, ws
    torch.cuda.empty_cache()
    return res


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build's verify step runs on a single MI355X and has no "
              "multi-GPU path (asked for --gpus %d, WORLD_SIZE=%d)." % (args.gpus, world), file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_00535_amd import dreams
    from paper_2606_00535_amd import workload as W

    if not torch.cuda.is_available():
        print("bench.py needs a HIP device", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda", 0)
    dreams.lib()
    wl = W.WORKLOADS[args.workload]
    NL, B, Hq, Hkv, T, D = wl.num_layers, wl.batch, wl.num_q_heads, wl.num_kv_heads, wl.num_nodes, wl.head_dim
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32

    # ---- inputs: topology, prefix lengths, logits and draft tokens from the seeded generator; the q/k/v
    # tensors are drawn on the device (same N(0,1) distribution, seeded) so large workloads stay cheap to set up.
    host = W.make_batch(wl, layers=[], with_logits=True)
    S = host.k_cache.shape[3]
    gen = torch.Generator(device=dev)
    gen.manual_seed(wl.seed)

    def draw(shape, std=1.0):
        x = torch.randn(shape, generator=gen, device=dev, dtype=torch.float32)
        if std != 1.0:
            x.mul_(std)
        return x.to(tdt)

    step_bytes_io = NL * 2 * B * Hkv * S * D * (2 if tdt == torch.bfloat16 else 4) + host.logits.nbytes
    R = max(2, int(math.ceil(args.rotate_bytes / step_bytes_io)))
    sets = []
    base = dict(q=draw((NL, B, Hq, T, D), wl.q_std), k=draw((NL, B, Hkv, S, D)), v=draw((NL, B, Hkv, S, D)),
                kv=torch.from_numpy(host.kv_len).to(dev), par=torch.from_numpy(host.parent).to(dev),
                logits=torch.from_numpy(host.logits).to(dev), tok=torch.from_numpy(host.tokens).to(dev))
    for r in range(R):
        st = {key: (val if r == 0 else val.clone()) for key, val in base.items()}
        st["out"] = torch.empty((NL, B, Hq, T, D), dtype=tdt, device=dev)
        st["alen"] = torch.empty(B, dtype=torch.int32, device=dev)
        st["path"] = torch.empty((B, T), dtype=torch.int32, device=dev)
        st["next"] = torch.empty(B, dtype=torch.int32, device=dev)
        st["kv_out"] = torch.empty(B, dtype=torch.int32, device=dev)
        sets.append(st)
    del base

    desc = dreams.attn_desc(sets[0]["q"][0], sets[0]["k"][0], args.num_splits, wl.max_kv_len)
    ws_attn = torch.zeros(max(1, dreams.tree_verify_attn_workspace_size(desc)), dtype=torch.uint8, device=dev)
    ws_acc = torch.zeros(max(1, dreams.tree_accept_workspace_size(B, T, wl.vocab)), dtype=torch.uint8, device=dev)

    def attention(st):
        for l in range(NL):
            dreams.tree_verify_attn(st["q"][l], st["k"][l], st["v"][l], st["kv"], st["par"], out=st["out"][l],
                                    with_lse=False, max_kv_len=wl.max_kv_len, num_splits=args.num_splits,
                                    workspace=ws_attn)

    def step(st):
        attention(st)
        dreams.tree_accept(st["logits"], st["tok"], st["par"], outputs=(st["alen"], st["path"], st["next"], None),
                           workspace=ws_acc)
        if wl.commit:
            dreams.kv_commit(st["k"], st["v"], st["kv"], st["path"], st["alen"], kv_len_out=st["kv_out"])

    # ---- warm-up (eager), then capture R steps (one per input set) and the remainder into HIP graphs
    if args.traffic_calibration:
        calibrate_traffic(torch, dev, sets, attention, R, wl, host)
        return
    for i in range(max(1, args.warmup)):
        step(sets[i % R])
    torch.cuda.synchronize()
    K = args.steps
    g_full = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_full):
        for r in range(R):
            step(sets[r])
    g_rem = None
    if K % R:
        g_rem = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g_rem):
            for r in range(K % R):
                step(sets[r])
    for _ in range(2):
        g_full.replay()
    torch.cuda.synchronize()

    # ---- timed region: exactly K steps
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    e0.record()
    for _ in range(K // R):
        g_full.replay()
    if g_rem is not None:
        g_rem.replay()
    e1.record()
    torch.cuda.synchronize()
    wall_ms = (time.perf_counter() - w0) * 1e3
    ms = e0.elapsed_time(e1)
    ms_per_step = ms / K
    steps_per_s = 1e3 / ms_per_step
    # the same step, as a distribution: each of args.repeats replays of the R-step graph timed alone
    step_dist = dist(replay_times_us(torch, g_full, R, max(1, args.repeats)))

    # ---- attention kernel alone: a graph of attention launches over the rotated sets, HIP events around it
    n_att = max(R, args.attn_launches // (R * NL) * R)
    g_att = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_att):
        for r in range(R):
            attention(sets[r])
    reps = max(1, n_att // R)
    g_att.replay()
    torch.cuda.synchronize()
    a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a0.record()
    for _ in range(reps):
        g_att.replay()
    a1.record()
    torch.cuda.synchronize()
    attn_us = a0.elapsed_time(a1) * 1e3 / (reps * R * NL)
    attn_dist = dist(replay_times_us(torch, g_att, R * NL, max(1, args.repeats)))

    # accept alone, same method
    g_acc = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_acc):
        for r in range(R):
            dreams.tree_accept(sets[r]["logits"], sets[r]["tok"], sets[r]["par"],
                               outputs=(sets[r]["alen"], sets[r]["path"], sets[r]["next"], None), workspace=ws_acc)
    g_acc.replay()
    torch.cuda.synchronize()
    a0.record()
    for _ in range(reps):
        g_acc.replay()
    a1.record()
    torch.cuda.synchronize()
    acc_us = a0.elapsed_time(a1) * 1e3 / (reps * R)

    # sampled acceptance at temperature 1 on the same target logits (draft = target + N(0,1) noise, children drawn
    # from the draft), same method
    smp = W.make_sampled(wl, target_logits=host.logits)
    ws_smp = torch.zeros(max(1, dreams.tree_accept_sampled_workspace_size(B, T, wl.vocab)), dtype=torch.uint8,
                         device=dev)
    for r, st in enumerate(sets):
        st["dlog"] = torch.from_numpy(smp.draft_logits).to(dev)
        st["stok"] = torch.from_numpy(smp.tokens).to(dev)
        st["uni"] = torch.from_numpy(smp.uniforms).to(dev)
        st["salen"] = torch.empty(B, dtype=torch.int32, device=dev)
        st["spath"] = torch.empty((B, T), dtype=torch.int32, device=dev)
        st["snext"] = torch.empty(B, dtype=torch.int32, device=dev)

    def sampled(st):
        dreams.tree_accept_sampled(st["logits"], st["dlog"], st["stok"], st["par"], st["uni"], smp.temperature,
                                   outputs=(st["salen"], st["spath"], st["snext"]), workspace=ws_smp)

    for st in sets:
        sampled(st)
    torch.cuda.synchronize()
    g_smp = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_smp):
        for r in range(R):
            sampled(sets[r])
    g_smp.replay()
    torch.cuda.synchronize()
    a0.record()
    for _ in range(reps):
        g_smp.replay()
    a1.record()
    torch.cuda.synchronize()
    smp_us = a0.elapsed_time(a1) * 1e3 / (reps * R)
    smp_bytes = 2 * B * T * wl.vocab * 4 + B * T * 12
    smp_alen = sets[0]["salen"].cpu().numpy()

    # greedy acceptance from the final hidden states (LM head fused with the argmax: the logits never reach
    # memory): weight [V, Hq*D] ~ N(0, 0.02), bf16, rotated over enough copies to stream from HBM; the library
    # GEMM into fp32 logits (bf16 operands, fp32 output) followed by dreams_tree_accept is timed the same way,
    # as context
    Hd = Hq * D
    lm_gen = torch.Generator(device=dev)
    lm_gen.manual_seed(wl.seed + 1)
    R_lm = max(2, int(math.ceil(args.rotate_bytes / (wl.vocab * Hd * 2))))
    lm_w = [(torch.randn((wl.vocab, Hd), generator=lm_gen, device=dev) * 0.02).to(torch.bfloat16)
            for _ in range(R_lm)]
    lm_h = torch.randn((B, T, Hd), generator=lm_gen, device=dev).to(torch.bfloat16)
    lm_tok = torch.from_numpy(host.tokens).to(dev)
    ws_lm = torch.zeros(max(1, dreams.tree_accept_lm_head_workspace_size(B, T, Hd, wl.vocab)), dtype=torch.uint8,
                        device=dev)
    lm_out = (torch.empty(B, dtype=torch.int32, device=dev), torch.empty((B, T), dtype=torch.int32, device=dev),
              torch.empty(B, dtype=torch.int32, device=dev), None)   # own outputs: set 0's are checked later

    def lm_fused():
        for w in lm_w:
            dreams.tree_accept_lm_head(lm_h, w, lm_tok, sets[0]["par"], outputs=lm_out, workspace=ws_lm)

    def lm_unfused():   # fp32 logits straight from the bf16 operands, as the fused kernel accumulates them
        for w in lm_w:
            lg = torch.mm(lm_h.view(B * T, Hd), w.t(), out_dtype=torch.float32)
            dreams.tree_accept(lg.view(B, T, wl.vocab), lm_tok, sets[0]["par"], outputs=lm_out, workspace=ws_acc)

    lm_us = {}
    for name, fn in (("fused", lm_fused), ("unfused", lm_unfused)):
        fn()
        torch.cuda.synchronize()
        g_lm = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g_lm):
            fn()
        g_lm.replay()
        torch.cuda.synchronize()
        lm_reps = max(1, 60 // R_lm)
        a0.record()
        for _ in range(lm_reps):
            g_lm.replay()
        a1.record()
        torch.cuda.synchronize()
        lm_us[name] = a0.elapsed_time(a1) * 1e3 / (lm_reps * R_lm)
        del g_lm
    lm_bytes = wl.vocab * Hd * 2 + B * T * Hd * 2 + B * T * 12
    lm_flops = 2.0 * B * T * wl.vocab * Hd
    del lm_w

    # the attention call with every row's attention entropy as well (the layer-selection statistic), same method
    ents = [torch.empty((B, Hq, T), dtype=torch.float32, device=dev) for _ in range(NL)]

    def attention_entropy(st):
        for l in range(NL):
            dreams.tree_verify_attn_entropy(st["q"][l], st["k"][l], st["v"][l], st["kv"], st["par"],
                                            out=st["out"][l], with_lse=False, entropy=ents[l],
                                            max_kv_len=wl.max_kv_len, num_splits=args.num_splits,
                                            workspace=ws_attn)

    g_ent = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g_ent):
        for r in range(R):
            attention_entropy(sets[r])
    g_ent.replay()
    torch.cuda.synchronize()
    a0.record()
    for _ in range(reps):
        g_ent.replay()
    a1.record()
    torch.cuda.synchronize()
    ent_us = a0.elapsed_time(a1) * 1e3 / (reps * R * NL)

    # target-aware visual-token selection on the same rows (Eq. 2 importance over the image tokens, keep one
    # in five, gather their K/V): each verb alone, same method; the rows' lse comes from an attention call
    vis = None
    if wl.image_tokens > 0 and tdt == torch.bfloat16:
        n_img, keep_r = wl.image_tokens, max(1, wl.image_tokens // 5)
        for st in sets:
            st["lse0"] = dreams.tree_verify_attn(st["q"][0], st["k"][0], st["v"][0], st["kv"], st["par"],
                                                 max_kv_len=wl.max_kv_len, workspace=ws_attn)[1]
            st["imp"] = torch.empty((B, n_img), dtype=torch.float32, device=dev)
            st["keep"] = torch.empty((B, keep_r), dtype=torch.int32, device=dev)
            st["ko"] = torch.empty((B, Hkv, keep_r, D), dtype=tdt, device=dev)
            st["vo"] = torch.empty((B, Hkv, keep_r, D), dtype=tdt, device=dev)
        vis_ws = torch.zeros(dreams.visual_importance_workspace_size(B, Hkv, n_img), dtype=torch.uint8, device=dev)
        verbs = {
            "importance": lambda st: dreams.visual_importance(st["q"][0], st["k"][0], st["kv"], st["lse0"], 0, n_img,
                                                              importance=st["imp"], workspace=vis_ws),
            "topk": lambda st: dreams.visual_topk(st["imp"], keep_r, keep=st["keep"]),
            "gather": lambda st: dreams.visual_gather(st["k"][0], st["v"][0], 0, st["keep"], k_out=st["ko"],
                                                      v_out=st["vo"]),
        }
        vis = {"image_tokens": n_img, "keep": keep_r}
        for name in ("importance", "topk", "gather"):
            for st in sets:
                verbs[name](st)
            torch.cuda.synchronize()
            g_v = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g_v):
                for r in range(R):
                    verbs[name](sets[r])
            g_v.replay()
            torch.cuda.synchronize()
            a0.record()
            for _ in range(reps):
                g_v.replay()
            a1.record()
            torch.cuda.synchronize()
            vis[name + "_us"] = round(a0.elapsed_time(a1) * 1e3 / (reps * R), 3)
        # importance: the image tokens' keys, every query row and lse, the importances out
        imp_bytes = B * Hkv * n_img * D * 2 + B * Hq * T * (D * 2 + 4) + B * n_img * 4
        vis["importance_bytes"] = imp_bytes
        vis["importance_GBps"] = round(imp_bytes / (vis["importance_us"] * 1e-6) / 1e9, 1)
        gat_bytes = 2 * 2 * B * Hkv * keep_r * D * 2
        vis["gather_GBps"] = round(gat_bytes / (vis["gather_us"] * 1e-6) / 1e9, 1)

    stream = stream_peak(torch, dev)
    try:
        dreams.workspace_status(ws_attn) if ws_attn.numel() >= 65536 else None
        flags_clear = True
    except dreams.DreamsError:
        flags_clear = False

    # the other workloads, each its own sub-object (the 32-layer step with commit, the 13B layer, the
    # matrix-core-bound GQA shape, the tiny fp32 case); the main workload's sets stay resident meanwhile
    extras = {}
    if not (args.no_extras or args.profile_only):
        for key, name in (("full_pass", "llava7b_full"), ("llava13b_layer", "llava13b_layer"),
                          ("gqa_long", "gqa_long"), ("tiny", "tiny")):
            if name != args.workload:
                extras[key] = measure_workload(torch, dev, name, args)
        extras["prefill_select"] = measure_prefill(torch, dev, args)

    kv_len = host.kv_len
    a_bytes = attn_bytes_per_layer(wl, kv_len)
    acc_b = accept_bytes(wl)
    path0 = sets[0]["path"].cpu().numpy()
    alen0 = sets[0]["alen"].cpu().numpy()
    com_b = commit_bytes(wl, path0, alen0) if wl.commit else 0
    step_bytes = NL * a_bytes + acc_b + com_b
    attn_gbps = a_bytes / (attn_us * 1e-6) / 1e9
    traffic = measured_traffic(args.workload)

    splits_used = desc.num_splits
    result = {
        "metric": METRIC,
        "value": round(steps_per_s, 2),
        "unit": "verify-steps/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if tdt == torch.bfloat16 else "f32",
        "data": "synthetic: seeded N(0,1) q/k/v, N(0,%g) target logits, seeded random draft trees" % wl.logit_std,
        "config": {"workload": wl.name, "layers": NL, "batch": B, "q_heads": Hq, "kv_heads": Hkv, "head_dim": D,
                   "kv_len": (list(wl.kv_len) if isinstance(wl.kv_len, tuple) else wl.kv_len),
                   "image_tokens": wl.image_tokens, "tree_nodes": T, "tree_depth": wl.depth,
                   "max_branch": wl.max_branch, "vocab": wl.vocab, "commit": wl.commit,
                   "rotated_input_sets": R, "graph_replay": True},
        "step_algorithmic_bytes": step_bytes,
        "step_GBps": round(step_bytes / (ms_per_step * 1e-3) / 1e9, 1),
        "wall_ms_timed_region": round(wall_ms, 3),
        "step_us": step_dist,
        "attention": {"us_per_launch": round(attn_us, 3), "us_dist": attn_dist, "bytes_per_launch": a_bytes,
                      "GBps": round(attn_gbps, 1), "splits": dreams.tree_verify_attn_splits(desc),
                      "workspace_flags_clear": flags_clear},
        "accept": {"us_per_launch": round(acc_us, 3), "bytes_per_launch": acc_b,
                   "GBps": round(acc_b / (acc_us * 1e-6) / 1e9, 1)},
        "accept_sampled": {"us_per_launch": round(smp_us, 3), "bytes_per_launch": smp_bytes,
                           "GBps": round(smp_bytes / (smp_us * 1e-6) / 1e9, 1), "temperature": smp.temperature,
                           "mean_accept_len": round(float(smp_alen.mean()), 3)},
        "accept_lm_head": {"us_per_launch": round(lm_us["fused"], 3), "hidden": Hd, "bytes_per_launch": lm_bytes,
                           "GBps": round(lm_bytes / (lm_us["fused"] * 1e-6) / 1e9, 1),
                           "frac_of_hbm_peak": round(lm_bytes / (lm_us["fused"] * 1e-6) / 1e9 / HBM_PEAK_GBPS, 4),
                           "TFLOPs": round(lm_flops / (lm_us["fused"] * 1e-6) / 1e12, 1),
                           "library_gemm_then_accept_us": round(lm_us["unfused"], 3)},
        "visual_select": vis,
        "attention_entropy": {"us_per_launch": round(ent_us, 3), "bytes_per_launch": a_bytes + B * Hq * T * 4,
                              "GBps": round((a_bytes + B * Hq * T * 4) / (ent_us * 1e-6) / 1e9, 1)},
        "roofline": {"bound": "hbm", "achieved": round(attn_gbps, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(attn_gbps / HBM_PEAK_GBPS, 4),
                     "traffic": None if traffic is None else int(traffic)},
        "stream_peak": dict(stream, attention_frac_of_read=round(attn_gbps / stream["read_GBps"], 4)),
        "gpu_clocks": gpu_clocks(),
    }
    result.update(extras)

    if not (args.no_cpu_baseline or args.profile_only):
        result["cpu_baseline"], result["parity_spot_check"] = cpu_baseline(wl, sets[0], host, args.cpu_seconds)
    print(json.dumps(result), flush=True)


def stream_peak(torch, dev):
    """This box's plain streaming rates: the library's read-stream helper over 1 GiB (reads 1 GiB) and a 1 GiB
    device copy (reads and writes 1 GiB), each the median of 10 launches timed with HIP events.  The reference
    for the share of the measured peak that the attention call reaches, beside its share of the 8 TB/s figure."""
    from paper_2606_00535_amd import dreams
    n = 1 << 28
    x = torch.ones(n, dtype=torch.float32, device=dev)
    y = torch.empty_like(x)
    sink = torch.empty(dreams.STREAM_READ_SINK_WORDS, dtype=torch.int32, device=dev)
    out = {}
    for name, fn, nbytes in (("read_GBps", lambda: dreams.stream_read(x, sink), 4 * n),
                             ("copy_GBps", lambda: y.copy_(x), 8 * n)):
        fn()
        torch.cuda.synchronize()
        times = []
        for _ in range(10):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1))
        times.sort()
        out[name] = round(nbytes / (times[len(times) // 2] * 1e-3) / 1e9, 1)
    del x, y
    torch.cuda.empty_cache()
    return out


def calibrate_traffic(torch, dev, sets, attention, R, wl, host):
    """Launches for the HBM-traffic counters: 5 copies of a 512 MiB buffer (reads 512 MiB, writes 512 MiB per
    launch: the reference that turns FETCH_SIZE / WRITE_SIZE into bytes), then 2 * R attention calls over
    the rotated input sets.  Eager launches, one stream; the counters are read per dispatch."""
    n = 512 << 20
    src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    for i in range(2 * R):
        attention(sets[i % R])
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_read": n, "copy_bytes_written": n, "copy_launches": 5,
                      "attention_calls": 2 * R, "attention_algorithmic_bytes_per_call":
                      attn_bytes_per_layer(wl, host.kv_len), "workload": wl.name}), flush=True)


def cpu_baseline(wl, st, host, seconds):
    """The CPU oracle (test-side checker, not tuned) timed on this host's cores on a bounded sample of the same
    workload: whole steps (every layer's attention over all heads, then acceptance) of input set 0, repeated
    until about `seconds` have passed.  Also compares set 0's GPU results with it."""
    import torch

    import oracle
    from paper_2606_00535_amd import workload as W

    NL = wl.num_layers
    to_f32 = lambda t: t.float().cpu().numpy() if t.dtype == torch.bfloat16 else t.cpu().numpy()
    layers = list(range(NL)) if NL <= 2 else [0]          # a 32-layer step is sampled on one layer
    q = [to_f32(st["q"][l]) for l in layers]
    k = [to_f32(st["k"][l]) for l in layers]
    v = [to_f32(st["v"][l]) for l in layers]
    scale = 1.0 / math.sqrt(wl.head_dim)
    reps, t0 = 0, time.perf_counter()
    t_attn = t_acc = 0.0
    while True:
        a = time.perf_counter()
        outs = [oracle.tree_attn(q[i], k[i], v[i], host.kv_len, host.parent, scale, wl.num_kv_heads,
                                 with_lse=False)[0] for i in range(len(layers))]
        b = time.perf_counter()
        acc = oracle.tree_accept(host.logits, host.tokens, host.parent)
        c = time.perf_counter()
        t_attn += b - a
        t_acc += c - b
        reps += 1
        if time.perf_counter() - t0 >= seconds:
            break
    per_layer = t_attn / reps / len(layers)
    step_s = per_layer * NL + t_acc / reps
    sample = ("%d repetitions of %s: tree attention of %s over all %d heads x %d nodes, then acceptance over "
              "%d x %d logits" % (reps, "a full step" if len(layers) == NL else "a step sampled on layer 0 "
                                  "(time scaled by %d layers)" % NL, "every layer" if len(layers) == NL else
                                  "layer 0", wl.num_q_heads, wl.num_nodes, wl.num_nodes, wl.vocab))
    base = {"value": round(1.0 / step_s, 4), "unit": "verify-steps/s", "cores": oracle.num_threads(),
            "kind": "oracle", "sample": sample, "seconds": round(time.perf_counter() - t0, 2),
            "affinity_cores": len(os.sched_getaffinity(0))}
    # the same oracle on one thread: a shorter sample of the same step (a quarter of the time budget)
    threads = oracle.num_threads()
    oracle.set_num_threads(1)
    try:
        reps1, t1, a1 = 0, time.perf_counter(), 0.0
        while True:
            a = time.perf_counter()
            for i in range(len(layers)):
                oracle.tree_attn(q[i], k[i], v[i], host.kv_len, host.parent, scale, wl.num_kv_heads, with_lse=False)
            b = time.perf_counter()
            oracle.tree_accept(host.logits, host.tokens, host.parent)
            c = time.perf_counter()
            a1 += (b - a) / len(layers) * NL + (c - b)
            reps1 += 1
            if time.perf_counter() - t1 >= seconds / 4:
                break
    finally:
        oracle.set_num_threads(threads)
    base["one_thread"] = {"value": round(reps1 / a1, 4), "unit": "verify-steps/s", "cores": 1,
                          "sample": "%d repetitions of the same step" % reps1}
    path_ok = bool(np.array_equal(st["path"].cpu().numpy(), acc[1]) and
                   np.array_equal(st["alen"].cpu().numpy(), acc[0]) and np.array_equal(st["next"].cpu().numpy(), acc[2]))
    check = {"accept_bit_exact": path_ok, "attention_tol": 2e-2}
    if wl.commit:
        # the timed steps committed into set 0's caches after its attention ran, so its outputs no longer match
        # the caches; the commit workload's attention parity is covered by the GPU tests
        check["attention_max_abs_err"] = None
    else:
        check["attention_max_abs_err"] = float(np.abs(st["out"][layers[0]].float().cpu().numpy() - outs[0]).max())
    return base, check


if __name__ == "__main__":
    main()
