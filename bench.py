"""Benchmark: translated KV tokens/s for one full MoT cache translation.

One step = one mot_translate call over every unit (target layer x {K, V})
of the workload, inputs resident in HBM.  Default workload: Qwen2.5-1.5B ->
Qwen2.5-7B shapes (28 layers, B=8, T=4096, source rows 2x128, target rows
4x128, E=8 translators Linear(256->2048)-GELU-Linear(2048->512)), bf16.

Prints one JSON line on stdout; progress goes to stderr.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "translated KV tokens/sec (all layers) Qwen2.5-1.5B→7B; MFMA util % of peak"
PEAK_TFLOPS = {"bf16": 2516.6, "f32": 157.3}     # MI355X dense MFMA peaks (AMD spec)
PEAK_HBM_GBS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def measured_traffic(kernel_files, prefix: str, workload_tag: str):
    """HBM bytes per call from the committed rocprofv3 FETCH_SIZE/WRITE_SIZE
    summary `profiles/<prefix>_<workload_tag>_hbm_traffic.md`, or None when
    that summary is missing or was taken on different kernel sources (its
    recorded hash of the concatenated source files no longer matches)."""
    import hashlib
    if isinstance(kernel_files, str):
        kernel_files = [kernel_files]
    srcs = [os.path.join(ROOT, "paper_2607_28979_amd", "csrc", f) for f in kernel_files]
    prof = os.path.join(ROOT, "profiles", "%s_%s_hbm_traffic.md" % (prefix, workload_tag))
    if not (all(os.path.exists(s) for s in srcs) and os.path.exists(prof)):
        return None
    h = hashlib.sha256()
    for s in srcs:
        h.update(open(s, "rb").read())
    digest = h.hexdigest()[:16]
    vals = {}
    for line in open(prof):
        if "=" in line and not line.startswith("|"):
            k, _, v = line.partition("=")
            vals[k.strip()] = v.strip().split()[0] if v.strip() else ""
    if vals.get("kernel_source_sha256_16") != digest:
        return None
    try:
        return float(vals["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


# file-name tags of the five model pairs, in workload order
WORKLOAD_TAGS = ["gpt2-small-opt-125m", "qwen2.5-0.5b-0.5b", "opt-1.3b-qwen2.5-1.5b", "qwen2.5-1.5b-7b",
                 "qwen2.5-7b-7b-32k"]


def host_cpu() -> dict:
    """The host the CPU baseline ran on: its logical CPU count and model
    name.  The oracle uses at most 16 of those threads, the CPU share a
    single-GPU job gets on these machines."""
    model = ""
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"host_cpus": os.cpu_count() or 1, "cpu_model": model}


def oracle_threads() -> int:
    return min(16, os.cpu_count() or 1)


def calibration_copy(mib: int) -> None:
    """One plain device copy of `mib` MiB: a known-size reference for the HBM
    byte counters of a profiler run."""
    if mib <= 0:
        return
    import torch
    n = mib << 20
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    b = torch.empty(n, dtype=torch.uint8, device="cuda")
    a.fill_(1)
    torch.cuda.synchronize()
    b.copy_(a)
    torch.cuda.synchronize()
    log("calibration copy of %d MiB done" % mib)
    del a, b


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", type=int, default=3,
                    help="index into the workload list (default 3: Qwen2.5-1.5B -> 7B)")
    ap.add_argument("--algo", type=int, default=0, help="0 auto, 1 unfused, 2 fused, 3 routed")
    ap.add_argument("--top-k", type=int, default=0,
                    help="translators per token (default: the workload's, i.e. all E); below E "
                         "the auto path is the routed Top-K kernel")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=0, help="oracle sample rows (0 = auto)")
    ap.add_argument("--moth", action="store_true",
                    help="time the activation variant MoT-h instead: one activation stream per "
                         "layer translated (Qwen2.5-1.5B -> 7B widths 1536 -> 3584), then the "
                         "target K/V restored through its key/value projections")
    ap.add_argument("--replay", action="store_true",
                    help="time the context replay after translation instead: Top-S source-guided "
                         "sparse attention over every Qwen2.5-7B target layer of an 8K context "
                         "(the bottom two layers with full causal attention)")
    ap.add_argument("--backbone", action="store_true",
                    help="time the mixture with the backbone translator body (App. C.2) as its experts "
                         "on the Qwen2.5-1.5B -> 7B cache rows")
    ap.add_argument("--slots", type=int, default=1,
                    help="with --backbone: channel-window slots per expert (the recurrent scan over "
                         "N consecutive target layers' source rows)")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="before timing, run one plain device copy of MIB MiB (a known-size "
                         "reference for the HBM byte counters of a profiler run)")
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py measures one GPU: the translation shards with no exchange (by unit or "
              "by token), and this build runs on a single MI355X; --gpus must be 1.",
              file=sys.stderr)
        sys.exit(2)

    if args.moth:
        return bench_moth(args)
    if args.replay:
        return bench_replay(args)
    if args.backbone:
        return bench_backbone(args)

    import torch
    from paper_2607_28979_amd import binding as mb
    from paper_2607_28979_amd.configs import WORKLOADS
    from paper_2607_28979_amd.inputs import generate, bf16_bits

    w = WORKLOADS[args.workload]
    if args.top_k:
        w = w.with_(top_k=args.top_k)
    torch.cuda.set_device(0)
    t0 = time.time()
    inp = generate(w)
    log("inputs generated in %.1f s" % (time.time() - t0))

    def dev(a):
        if w.dtype == "f32":
            return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).cuda()
        return torch.from_numpy(bf16_bits(a).view(np.int16)).cuda().view(torch.bfloat16)

    d = {n: dev(getattr(inp, n)) for n in ("src_k", "src_v", "w1", "b1", "w2", "b2", "wr", "br")}
    tdt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    shape = (w.L_tgt, w.B, w.T, w.H_tgt, w.D_tgt)
    dk = torch.empty(shape, dtype=tdt, device="cuda")
    dv = torch.empty(shape, dtype=tdt, device="cuda")
    lm = (np.arange(w.L_tgt, dtype=np.int32) if w.layer_map == "identity"
          else mb.depth_ratio_map(w.L_src, w.L_tgt))
    shapes = mb.Shapes.from_workload(w, algo=args.algo)
    ws_bytes = mb.workspace_bytes(shapes)
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device="cuda") if ws_bytes else None

    def step():
        mb.translate(d["src_k"], d["src_v"], lm, d["w1"], d["b1"], d["w2"], d["b2"], d["wr"], d["br"],
                     dk, dv, shapes, workspace=ws)

    calibration_copy(args.calibrate_copy)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log("warmup done (%d steps)" % args.warmup)

    # timed region: K steps, HIP events on the stream the kernels run on
    stream = torch.cuda.current_stream()
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_begin = time.perf_counter()
    for k in range(args.steps):
        starts[k].record(stream)
        step()
        ends[k].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_begin
    per_call_ms = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    ms_per_step = wall * 1e3 / args.steps
    avg_call_ms = float(np.mean(per_call_ms))
    med_call_ms = float(np.median(per_call_ms))
    log("timed %d steps: wall %.3f ms/step, event avg %.3f ms, median %.3f ms"
        % (args.steps, ms_per_step, avg_call_ms, med_call_ms))

    n_tok = w.n_tok
    value = n_tok / (ms_per_step / 1e3)
    flops = w.gemm_flops()
    fusable = w.dtype == "bf16" and w.d_in in (128, 256, 512) and w.d_out in (128, 256, 512)
    # the library's rule: Top-K with K < E takes the routed path on bf16 (the
    # fused kernel's routed mode on its shapes, the routed large-tile GEMMs
    # elsewhere)
    routed = w.dtype == "bf16" and (args.algo == 3 or (args.algo == 0 and 0 < w.top_k < w.E))
    fused = not routed and (args.algo == 2 or (args.algo == 0 and fusable))
    # the library's rule for the fp32 matrix-core kernels (else router + vector-ALU GEMMs)
    f32_mfma = w.dtype == "f32" and w.hidden % 64 == 0 and w.d_in % 16 == 0 and w.d_out % 4 == 0
    achieved_tflops = flops / (avg_call_ms / 1e3) / 1e12
    peak = PEAK_TFLOPS[w.dtype]
    roofline = {
        "bound": "mfma",
        "kernel": ("k_bf16_fused" if fused else "k_f32_mfma_gemm1 + k_f32_mfma_gemm2" if f32_mfma else
                   "mot_translate routed (router lists + plan + %s%s)"
                   % ("k_bf16_fused tiles" if fusable else "routed large-tile GEMMs",
                      " + combine" if w.top_k > 1 else "") if routed
                   else "mot_translate (router + gemm1 + gemm2)"),
        "achieved": round(achieved_tflops, 2),
        "peak": peak,
        "unit": "TFLOP/s",
        "frac": round(achieved_tflops / peak, 4),
        "traffic": (None if routed or args.top_k else
                    measured_traffic("k_bf16_fused_kernel.h", "k_bf16_fused", WORKLOAD_TAGS[args.workload]) if fused
                    else measured_traffic(["k_f32_mfma.hip"] if f32_mfma else ["k_router.hip", "k_f32.hip"],
                                          "mot_translate_f32", WORKLOAD_TAGS[args.workload]) if w.dtype == "f32"
                    else measured_traffic(["k_router.hip", "k_bf16_unfused.hip", "k_bf16_gemm256.hip"], "mot_translate_two_gemm",
                                          WORKLOAD_TAGS[args.workload])),
        "alg_flops_per_launch": flops,
        "alg_bytes_per_launch": w.alg_bytes(),
        "hbm_gbs_alg": round(w.alg_bytes() / (avg_call_ms / 1e3) / 1e9, 1),
    }

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, inp, lm, args.cpu_rows)

    out = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic (seeded numpy; shapes and value recipe of the model pair)",
        "config": {"workload": w.name, "L_src": w.L_src, "L_tgt": w.L_tgt, "B": w.B, "T": w.T,
                   "d_in": w.d_in, "hidden": w.hidden, "d_out": w.d_out, "E": w.E,
                   "top_k": w.top_k or w.E, "units": w.units(), "parallelism": "single GPU"},
        "mfma_util_pct": round(100 * achieved_tflops / peak, 2),
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def cpu_baseline(w, inp, lm, rows):
    """The CPU oracle, untuned, on a bounded sample: every unit for the first
    `rows` tokens (each token translated through all layers, K and V)."""
    from oracle import OracleDims, oracle_rows
    threads = oracle_threads()
    od = OracleDims(L_src=w.L_src, L_tgt=w.L_tgt, B=w.B, T=w.T, H_src=w.H_src, D_src=w.D_src,
                    H_tgt=w.H_tgt, D_tgt=w.D_tgt, E=w.E, hidden=w.hidden, top_k=w.top_k)
    units = [(j, x) for j in range(w.L_tgt) if lm[j] >= 0 for x in (0, 1)]
    per_row_flops = w.gemm_flops() / w.n_tok
    if rows <= 0:
        # about 15 s of work at the oracle's ~4 GFLOP/s per thread
        rows = int(max(1, min(w.n_tok, 60e9 * threads / per_row_flops)))
    sample = np.arange(rows, dtype=np.int64)
    t0 = time.perf_counter()
    oracle_rows(od, inp.src_k, inp.src_v, lm, inp.w1, inp.b1, inp.w2, inp.b2, inp.wr, inp.br,
                units=units, rows=sample, nthreads=threads)
    dt = time.perf_counter() - t0
    log("cpu oracle: %d rows x %d units in %.2f s on %d threads" % (rows, len(units), dt, threads))
    return {"value": round(rows / dt, 3), "unit": "tokens/s", "cores": threads, **host_cpu(), "kind": "oracle",
            "sample": "first %d of %d tokens, all %d units (K and V of every layer), fp64"
                      % (rows, w.n_tok, len(units)),
            "seconds": round(dt, 2)}


def bench_moth(args):
    """MoT-h (App. C.5): one step = mot_translate over the activation stream of
    every layer, then mot_restore_kv of every layer's keys and values."""
    import torch
    from paper_2607_28979_amd import binding as mb
    from paper_2607_28979_amd.configs import MOTH
    from paper_2607_28979_amd.inputs import bf16_bits, generate, projection_weights

    w = MOTH.act
    if args.top_k:
        w = w.with_(top_k=args.top_k)
    torch.cuda.set_device(0)
    t0 = time.time()
    inp = generate(w)
    wk, bk, wv, bv = projection_weights(w.L_tgt, w.d_out, MOTH.d_kv, seed=w.seed)
    log("inputs generated in %.1f s" % (time.time() - t0))

    def dev(a):
        return torch.from_numpy(bf16_bits(a).view(np.int16)).cuda().view(torch.bfloat16)

    d = {n: dev(getattr(inp, n)) for n in ("src_k", "w1", "b1", "w2", "b2", "wr", "br")}
    p = {n: dev(a) for n, a in (("wk", wk), ("bk", bk), ("wv", wv), ("bv", bv))}
    act = torch.empty((w.L_tgt, w.B, w.T, 1, w.d_out), dtype=torch.bfloat16, device="cuda")
    kv_shape = (w.L_tgt, w.B, w.T, MOTH.kv_heads, MOTH.head_dim)
    dk = torch.empty(kv_shape, dtype=torch.bfloat16, device="cuda")
    dv = torch.empty(kv_shape, dtype=torch.bfloat16, device="cuda")
    lm = (np.arange(w.L_tgt, dtype=np.int32) if w.layer_map == "identity"
          else mb.depth_ratio_map(w.L_src, w.L_tgt))
    shapes = mb.Shapes.from_workload(w, algo=args.algo)
    ws_bytes = mb.workspace_bytes(shapes)
    ws = torch.empty(max(ws_bytes, 1), dtype=torch.uint8, device="cuda") if ws_bytes else None
    log("workspace %.2f GB" % (ws_bytes / 1e9))

    def translate():
        mb.translate(d["src_k"], None, lm, d["w1"], d["b1"], d["w2"], d["b2"], d["wr"], d["br"],
                     act, None, shapes, workspace=ws)

    def restore():
        mb.restore_kv(act, None, p["wk"], p["bk"], p["wv"], p["bv"], dk, dv, L=w.L_tgt, B=w.B,
                      T=w.T, d_act=w.d_out, H_tgt=MOTH.kv_heads, D_tgt=MOTH.head_dim)

    calibration_copy(args.calibrate_copy)
    for _ in range(args.warmup):
        translate()
        restore()
    torch.cuda.synchronize()
    log("warmup done (%d steps)" % args.warmup)
    stream = torch.cuda.current_stream()
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_begin = time.perf_counter()
    for k in range(args.steps):
        ev[k][0].record(stream)
        translate()
        ev[k][1].record(stream)
        restore()
        ev[k][2].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_begin
    tr_ms = float(np.mean([e[0].elapsed_time(e[1]) for e in ev]))
    rs_ms = float(np.mean([e[1].elapsed_time(e[2]) for e in ev]))
    ms_per_step = wall * 1e3 / args.steps
    log("timed %d steps: wall %.3f ms/step, translate %.3f ms, restore %.3f ms"
        % (args.steps, ms_per_step, tr_ms, rs_ms))
    tr_flops = w.gemm_flops()
    rs_flops = MOTH.restore_flops()
    # the library's restoration kernel: 256 x 256 tiles when d_kv % 256 == 0 and
    # the launch has at least 128 workgroups, else 128 x 128 tiles
    d_kv = MOTH.kv_heads * MOTH.head_dim
    proj_wgs = (2 * d_kv // 256) * ((w.n_tok + 255) // 256) * w.L_tgt
    proj_kernel = "k_bf16_project_256" if d_kv % 256 == 0 and proj_wgs >= 128 else "k_bf16_project"
    peak = PEAK_TFLOPS["bf16"]
    tr_tf = tr_flops / (tr_ms / 1e3) / 1e12
    rs_tf = rs_flops / (rs_ms / 1e3) / 1e12
    cpu = None if args.no_cpu_baseline else cpu_baseline_moth(w, inp, lm, (wk, bk, wv, bv),
                                                              args.cpu_rows)
    out = {
        "metric": "translated and restored KV tokens/sec (all layers, MoT-h) Qwen2.5-1.5B→7B",
        "value": round(w.n_tok / (ms_per_step / 1e3), 1),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded numpy; activation widths of the model pair)",
        "config": {"workload": w.name, "L_src": w.L_src, "L_tgt": w.L_tgt, "B": w.B, "T": w.T,
                   "d_act_src": w.d_in, "hidden": w.hidden, "d_act_tgt": w.d_out, "E": w.E,
                   "top_k": w.top_k or w.E, "kv_heads": MOTH.kv_heads,
                   "head_dim": MOTH.head_dim, "parallelism": "single GPU"},
        "roofline": {"bound": "mfma", "kernel": "mot_translate (streams = 1)",
                     "achieved": round(tr_tf, 2), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(tr_tf / peak, 4), "traffic": None,
                     "alg_flops_per_launch": tr_flops, "ms": round(tr_ms, 3)},
        "restore": {"kernel": proj_kernel, "achieved": round(rs_tf, 2), "peak": peak,
                    "unit": "TFLOP/s", "frac": round(rs_tf / peak, 4), "ms": round(rs_ms, 3),
                    "alg_flops_per_launch": rs_flops},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


def cpu_baseline_moth(w, inp, lm, proj, rows):
    """The CPU oracle on the first `rows` tokens of every layer: translation of
    the activation stream, then the key/value restoration of those rows."""
    from oracle import OracleDims, oracle_restore_kv, oracle_rows
    wk, bk, wv, bv = proj
    threads = oracle_threads()
    od = OracleDims(L_src=w.L_src, L_tgt=w.L_tgt, B=w.B, T=w.T, H_src=w.H_src, D_src=w.D_src,
                    H_tgt=w.H_tgt, D_tgt=w.D_tgt, E=w.E, hidden=w.hidden, top_k=w.top_k,
                    streams=1)
    units = [(j, 0) for j in range(w.L_tgt) if lm[j] >= 0]
    if rows <= 0:
        rows = int(max(1, min(w.n_tok, 60e9 * threads / (w.gemm_flops() / w.n_tok))))
    t0 = time.perf_counter()
    a = oracle_rows(od, inp.src_k, None, lm, inp.w1, inp.b1, inp.w2, inp.b2, inp.wr, inp.br,
                    units=units, rows=np.arange(rows, dtype=np.int64), nthreads=threads)
    from paper_2607_28979_amd.configs import MOTH
    oracle_restore_kv(a.reshape(len(units), 1, rows, w.d_out), None, wk, bk, wv, bv, B=1, T=rows,
                      H_tgt=MOTH.kv_heads, D_tgt=MOTH.head_dim)
    dt = time.perf_counter() - t0
    log("cpu oracle: %d rows x %d layers in %.2f s on %d threads" % (rows, len(units), dt, threads))
    return {"value": round(rows / dt, 3), "unit": "tokens/s", "cores": threads, **host_cpu(), "kind": "oracle",
            "sample": "first %d of %d tokens, all %d layers (translation + K/V restoration), fp64"
                      % (rows, w.n_tok, len(units)),
            "seconds": round(dt, 2)}


def pair_gathered_rows(idx, T: int) -> float:
    """Key rows the two-position sparse kernel gathers per KV head for one
    launch: for each pair (u, u+1) of every batch row, the size of the union
    of their (ascending) sets when it is at most 192, else both sets."""
    import torch
    B, _, S = idx.shape
    tp = T // 2 * 2
    a = idx[:, 0:tp:2].long()
    b = idx[:, 1:tp:2].long()
    na = (a >= 0).sum(-1)
    nb = (b >= 0).sum(-1)
    common = ((a.unsqueeze(-1) == b.unsqueeze(-2)) & (a.unsqueeze(-1) >= 0)).sum((-1, -2))
    union = na + nb - common
    rows = torch.where(union <= 192, union, na + nb).sum().item()
    if T % 2:
        rows += (idx[:, T - 1] >= 0).sum().item()
    return float(rows)


def bench_replay(args):
    """Context replay (App. C.4): one step = for every target layer, either
    the full causal attention (bottom L_full layers) or mot_topS_select on
    the paired source layer's head-averaged attention map followed by
    mot_replay_attention over the selected sets."""
    import torch
    from paper_2607_28979_amd import binding as mb
    from paper_2607_28979_amd.configs import REPLAY
    from paper_2607_28979_amd.inputs import bf16_bits, replay_inputs, source_attention

    w = REPLAY
    torch.cuda.set_device(0)
    pi = mb.depth_ratio_map(w.L_src, w.L_tgt)
    t0 = time.time()

    def dev(a):
        return torch.from_numpy(bf16_bits(a).view(np.int16)).cuda().view(torch.bfloat16)

    layers = []
    for l in range(w.L_tgt):
        q, k, v = replay_inputs(w.B, w.T, w.H_q, w.H_kv, w.D, seed=w.seed + 100 * l)
        layers.append((dev(q), dev(k), dev(v)))
    maps = {}
    for l in range(w.L_full, w.L_tgt):
        i = int(pi[l])
        if i not in maps:
            maps[i] = torch.from_numpy(source_attention(w.B, w.T, seed=w.seed + 1000 * i)).cuda()
    log("inputs generated in %.1f s (%d source maps)" % (time.time() - t0, len(maps)))
    idx = torch.empty((w.B, w.T, w.S), dtype=torch.int32, device="cuda")
    out = torch.empty((w.B, w.T, w.H_q, w.D), dtype=torch.bfloat16, device="cuda")
    stream = torch.cuda.current_stream()
    ev = {"select": [], "sparse": [], "causal": []}

    def step(record):
        for l in range(w.L_tgt):
            q, k, v = layers[l]
            if l < w.L_full:
                e0 = torch.cuda.Event(enable_timing=True) if record else None
                e1 = torch.cuda.Event(enable_timing=True) if record else None
                if record: e0.record(stream)
                mb.replay_attention(q, k, v, None, out, B=w.B, T=w.T, H_q=w.H_q, H_kv=w.H_kv, D=w.D)
                if record:
                    e1.record(stream)
                    ev["causal"].append((e0, e1))
            else:
                es = [torch.cuda.Event(enable_timing=True) for _ in range(3)] if record else None
                if record: es[0].record(stream)
                mb.topS_select(maps[int(pi[l])], idx, w.B, w.T, w.S)
                if record: es[1].record(stream)
                mb.replay_attention(q, k, v, idx, out, B=w.B, T=w.T, H_q=w.H_q, H_kv=w.H_kv, D=w.D, S=w.S)
                if record:
                    es[2].record(stream)
                    ev["select"].append((es[0], es[1]))
                    ev["sparse"].append((es[1], es[2]))

    calibration_copy(args.calibrate_copy)
    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()
    log("warmup done (%d steps)" % args.warmup)
    torch.cuda.synchronize()
    t_begin = time.perf_counter()
    for _ in range(args.steps):
        step(True)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_begin
    ms_per_step = wall * 1e3 / args.steps
    avg = {kk: float(np.mean([a.elapsed_time(b) for a, b in vv])) for kk, vv in ev.items()}
    log("timed %d steps: wall %.3f ms/step; per launch: select %.3f ms, sparse %.3f ms, causal %.3f ms"
        % (args.steps, ms_per_step, avg["select"], avg["sparse"], avg["causal"]))
    # per-launch algorithmic figures
    n_tok = w.B * w.T
    sp_flops = 4.0 * w.H_q * w.D * w.B * sum(min(u + 1, w.S) for u in range(w.T))
    ca_flops = 4.0 * w.H_q * w.D * w.B * w.T * (w.T + 1) / 2
    sel_bytes = 4.0 * w.B * w.T * (w.T + 1) / 2 + 4.0 * n_tok * w.S        # causal half of A once, idx
    # sparse attention: q and o once, idx once, the layer's K and V once; the
    # selected K and V rows it gathers per (query, KV head) are reported beside
    sp_gather_sets = 2.0 * 2 * w.D * w.H_kv * w.B * sum(min(u + 1, w.S) for u in range(w.T))
    sp_gather = sp_gather_sets
    pair = w.D in (64, 128) and w.S <= 128 and 2 * (w.H_q // w.H_kv) <= 16   # the library's rule for that kernel
    if pair:
        # the two-position kernel gathers the union of a pair's sets once (or
        # both sets when the union exceeds its 192-key limit): count the rows
        # on this run's own sets, averaged over the sparse layers
        rows_all = 0.0
        for l in range(w.L_full, w.L_tgt):
            mb.topS_select(maps[int(pi[l])], idx, w.B, w.T, w.S)
            rows_all += pair_gathered_rows(idx, w.T)
        sp_gather = 2.0 * 2 * w.D * w.H_kv * rows_all / (w.L_tgt - w.L_full)
    sp_bytes = 2.0 * 2 * n_tok * w.H_q * w.D + 4.0 * n_tok * w.S + 2.0 * 2 * n_tok * w.H_kv * w.D
    peak_bf16 = PEAK_TFLOPS["bf16"]
    rows = {
        "select": {"bound": "hbm", "achieved": sel_bytes / (avg["select"] / 1e3) / 1e9, "peak": PEAK_HBM_GBS,
                   "unit": "GB/s", "alg_bytes_per_launch": sel_bytes, "ms": avg["select"]},
        "sparse": {"bound": "hbm", "achieved": sp_bytes / (avg["sparse"] / 1e3) / 1e9, "peak": PEAK_HBM_GBS,
                   "unit": "GB/s", "alg_bytes_per_launch": sp_bytes, "ms": avg["sparse"],
                   "gathered_bytes_per_launch": sp_gather,
                   "gathered_bytes_per_launch_one_set_per_position": sp_gather_sets,
                   "gather_gbs": round(sp_gather / (avg["sparse"] / 1e3) / 1e9, 1),
                   "tflops": round(sp_flops / (avg["sparse"] / 1e3) / 1e12, 2)},
        "causal": {"bound": "mfma", "achieved": ca_flops / (avg["causal"] / 1e3) / 1e12, "peak": peak_bf16,
                   "unit": "TFLOP/s", "alg_flops_per_launch": ca_flops, "ms": avg["causal"]},
    }
    for r in rows.values():
        r["achieved"] = round(r["achieved"], 2)
        r["frac"] = round(r["achieved"] / r["peak"], 4)
        r["ms"] = round(r["ms"], 4)
    share = {"select": avg["select"] * (w.L_tgt - w.L_full), "sparse": avg["sparse"] * (w.L_tgt - w.L_full),
             "causal": avg["causal"] * w.L_full}
    dom = max(share, key=share.get)
    kname = {"select": "k_topS_select", "sparse": "k_sparse_attn_pair" if pair else "k_sparse_attn",
             "causal": "k_causal_attn"}
    roof = dict(rows[dom], kernel=kname[dom],
                traffic=measured_traffic("k_replay.hip", "k_replay", "qwen2.5-7b-replay-8k") if dom == "sparse" else None)
    cpu = None if args.no_cpu_baseline else cpu_baseline_replay(w, args.cpu_rows)
    out_line = {
        "metric": "replayed context tokens/sec (all target layers, Top-S source-guided sparse attention)",
        "value": round(n_tok / (ms_per_step / 1e3), 1),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded numpy; Qwen2.5-7B head shapes, structured source attention maps)",
        "config": {"workload": w.name, "L_tgt": w.L_tgt, "L_full": w.L_full, "B": w.B, "T": w.T,
                   "H_q": w.H_q, "H_kv": w.H_kv, "D": w.D, "S": w.S, "parallelism": "single GPU"},
        "roofline": roof,
        "kernels": {kname[k_]: rows[k_] for k_ in rows},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out_line), flush=True)


def cpu_baseline_replay(w, rows):
    """The CPU oracle on the first `rows` query positions of every target
    layer: selection and attention (sparse layers), or full causal attention."""
    from oracle import oracle_replay_attention_rows, oracle_topS_rows
    from paper_2607_28979_amd import binding as mb
    from paper_2607_28979_amd.inputs import replay_inputs, source_attention
    rows = rows if rows > 0 else 256
    pi = mb.depth_ratio_map(w.L_src, w.L_tgt)
    sample = [(0, u) for u in range(rows)]
    dt = 0.0
    maps = {}
    for l in range(w.L_tgt):
        q, k, v = replay_inputs(w.B, w.T, w.H_q, w.H_kv, w.D, seed=w.seed + 100 * l)
        if l < w.L_full:
            t0 = time.perf_counter()
            oracle_replay_attention_rows(q, k, v, None, sample)
            dt += time.perf_counter() - t0
            continue
        i = int(pi[l])
        if i not in maps:
            maps = {i: source_attention(w.B, w.T, seed=w.seed + 1000 * i)}
        t0 = time.perf_counter()
        sets = oracle_topS_rows(maps[i], w.S, sample)
        idx = np.full((w.B, w.T, w.S), -1, np.int32)
        idx[0, :rows] = sets
        oracle_replay_attention_rows(q, k, v, idx, sample)
        dt += time.perf_counter() - t0
    log("cpu oracle: %d positions x %d layers in %.2f s (1 thread)" % (rows, w.L_tgt, dt))
    return {"value": round(rows / dt, 3), "unit": "tokens/s", "cores": 1, **host_cpu(), "kind": "oracle",
            "sample": "first %d of %d query positions, all %d target layers (selection + attention), fp64"
                      % (rows, w.T, w.L_tgt), "seconds": round(dt, 2)}


def bench_backbone(args):
    """One step = one mot_backbone_translate call over every unit."""
    import torch
    from paper_2607_28979_amd import binding as mb
    from paper_2607_28979_amd.configs import BACKBONE
    from paper_2607_28979_amd.inputs import backbone_params, bf16_bits, generate, window_router

    bw = BACKBONE
    w = bw.kv
    N = max(1, args.slots)
    torch.cuda.set_device(0)
    t0 = time.time()
    inp = generate(w)
    params = backbone_params(w, bw.d_h, bw.d_ff, seed=w.seed, n_slots=N)
    log("inputs generated in %.1f s" % (time.time() - t0))

    def dev(a):
        return torch.from_numpy(bf16_bits(a).view(np.int16)).cuda().view(torch.bfloat16)

    d = {n: dev(getattr(inp, n)) for n in ("src_k", "src_v", "wr", "br")}
    if N > 1:
        wr, br = window_router(w, N, seed=w.seed)
        d["wr"], d["br"] = dev(wr), dev(br)
    pr = dev(params)
    shape = (w.L_tgt, w.B, w.T, w.H_tgt, w.D_tgt)
    dk = torch.empty(shape, dtype=torch.bfloat16, device="cuda")
    dv = torch.empty(shape, dtype=torch.bfloat16, device="cuda")
    lm = np.arange(w.L_tgt, dtype=np.int32)
    shapes = mb.Shapes.from_workload(w)

    def step():
        mb.backbone_translate(d["src_k"], d["src_v"], lm, pr, d["wr"], d["br"], dk, dv, shapes, bw.d_h,
                              bw.n_heads, bw.d_ff, n_slots=N)

    calibration_copy(args.calibrate_copy)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log("warmup done (%d steps)" % args.warmup)
    stream = torch.cuda.current_stream()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    t_begin = time.perf_counter()
    for a, b in ev:
        a.record(stream)
        step()
        b.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_begin
    ms_per_step = wall * 1e3 / args.steps
    call_ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    log("timed %d steps: wall %.3f ms/step, event avg %.3f ms" % (args.steps, ms_per_step, call_ms))
    flops = bw.flops(N)
    tf = flops / (call_ms / 1e3) / 1e12
    out = {
        "metric": "translated KV tokens/sec (all layers, backbone-translator experts) Qwen2.5-1.5B→7B",
        "value": round(w.n_tok / (ms_per_step / 1e3), 1),
        "unit": "tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded numpy; shapes of the model pair, random backbone parameters)",
        "config": {"workload": w.name, "L_tgt": w.L_tgt, "B": w.B, "T": w.T, "d_in": w.d_in, "d_out": w.d_out,
                   "E": w.E, "d_h": bw.d_h, "n_heads": bw.n_heads, "d_ff": bw.d_ff, "n_slots": N,
                   "parallelism": "single GPU"},
        "roofline": {"bound": "mfma", "kernel": "mot_backbone_translate (LayerNorm + linear + causal attention chain)",
                     "achieved": round(tf, 2), "peak": PEAK_TFLOPS["bf16"], "unit": "TFLOP/s",
                     "frac": round(tf / PEAK_TFLOPS["bf16"], 4), "traffic": None, "alg_flops_per_launch": flops},
        "cpu_baseline": None,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
