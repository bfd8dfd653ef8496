#!/usr/bin/env python3
"""Benchmark of the integer-only I-LW-DETR encoder on one MI355X.

One step is one forward pass of the whole encoder (every block: LayerNorm,
QKV, attention with Constrained Shiftmax, projection + residual, LayerNorm,
fc1 + SD-ShiftGELU, fc2 + residual) over one batch of seeded synthetic int8
tokens that are already resident in HBM.  The default workload is the
largest single-GPU encoder configuration: the Medium-shaped encoder on a
640x640 image (1600 tokens, dim 384, 6 heads, MLP 1536, 10 blocks alternating
2x2 windows of 400 tokens and global attention, batch 8).

Prints ONE JSON line on stdout:
  value        int8 TOPS: algorithmic GEMM ops (2*M*N*K over QKV, Q K^T, P V,
               projection, fc1, fc2; attention counted per window) / time
  images_per_s batch / time per step
  roofline     the dominant kernel's achieved rate against its peak, timed
               with HIP events on its launch stream
  cpu_baseline the CPU oracle on the same workload: every image of the batch
               over the host's cores (one thread per image), and image 0 on
               one thread; core count and CPU model
  parity       every benchmarked image against the oracle
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "int8 TOPS + images/sec, integer-only encoder block, bit-exact vs oracle"
PEAK_INT8_TOPS = 5000.0      # MI355X dense int8 MFMA, 5.0 POPS
PEAK_HBM_GBS = 8000.0        # MI355X HBM3E, 8 TB/s


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def stage_work(wl, B, launches):
    """Algorithmic work of one forward, per profiling stage, given the number
    of launches per forward of each stage: (kind, amount) with kind 'ops'
    (int8 ops) or 'bytes' (HBM bytes)."""
    T, D, Hm = wl.tokens, wl.dim, wl.mlp_dim
    M = B * T
    nb = len(wl.windows)
    attn = 0
    for wh, ww in wl.windows:
        tw = T if wh == 0 else wh * ww
        attn += 4 * (T // tw) * tw * tw * D * B
    qkv, proj, mlp = 2 * M * 3 * D * D, 2 * M * D * D, 2 * M * Hm * D
    n = lambda k: launches.get(k, 0)
    return {
        "gemm_qkv": ("ops", n("gemm_qkv") * qkv),
        "attention": ("ops", attn),
        "gemm_proj": ("ops", n("gemm_proj") * proj),
        "gemm_fc1": ("ops", n("gemm_fc1") * mlp),
        "gemm_fc2": ("ops", n("gemm_fc2") * mlp),
        # projection, fc1 and fc2 in one launch
        "tail384": ("ops", n("tail384") * (proj + 2 * mlp)),
        # projection, fc1, fc2, and the QKV linear of the next block
        "block_tail": ("ops", n("block_tail") * (proj + 2 * mlp) + (nb - n("gemm_qkv")) * qkv
                       if n("block_tail") else 0),
        # int8 row in and out, plus beta / multiplier / shift per channel
        "layernorm": ("bytes", n("layernorm") * (2 * M * D + 12 * D)),
    }


_INTERNAL = "paper_2607_24981_amd/csrc/ilw_internal.h"
KERNEL_OF_STAGE = {
    "attention": ("attention_kernel", ["paper_2607_24981_amd/csrc/attention.hip", _INTERNAL]),
    "gemm_qkv": ("gemm_i8_kernel", ["paper_2607_24981_amd/csrc/gemm.hip", _INTERNAL]),
    "gemm_proj": ("gemm_i8_kernel", ["paper_2607_24981_amd/csrc/gemm.hip", _INTERNAL]),
    "gemm_fc1": ("gemm_i8_kernel", ["paper_2607_24981_amd/csrc/gemm.hip", _INTERNAL]),
    "gemm_fc2": ("gemm_i8_kernel", ["paper_2607_24981_amd/csrc/gemm.hip", _INTERNAL]),
    "tail384": ("tail384_kernel", ["paper_2607_24981_amd/csrc/tail384.hip", _INTERNAL]),
    "block_tail": ("block_tail_kernel", ["paper_2607_24981_amd/csrc/block_tail.hip", _INTERNAL]),
    "layernorm": ("layernorm_rows_kernel", ["paper_2607_24981_amd/csrc/rowops.hip", _INTERNAL]),
    "split_conv": ("split_conv_kernel", ["paper_2607_24981_amd/csrc/split_conv.hip", _INTERNAL]),
    "patch_embed": ("gemm_i8_kernel", ["paper_2607_24981_amd/csrc/gemm.hip", _INTERNAL]),
    "shiftmax": ("shiftmax_rows_kernel", ["paper_2607_24981_amd/csrc/rowops.hip", _INTERNAL]),
    "sdshiftgelu": ("gelu_kernel", ["paper_2607_24981_amd/csrc/rowops.hip", _INTERNAL]),
    "residual": ("residual_kernel", ["paper_2607_24981_amd/csrc/rowops.hip", _INTERNAL]),
}


def measured_traffic(stage, workload):
    """HBM bytes per launch from the committed rocprofv3 counter summary
    (profiles/traffic.json), only while the kernel's sources are unchanged
    since the counters were taken."""
    from paper_2607_24981_amd.profsum import source_digest
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        table = json.load(f)
    kernel, srcs = KERNEL_OF_STAGE[stage]
    rec = table.get(workload, {}).get(stage)
    if not rec or rec.get("source_sha256_16") != source_digest(srcs):
        return None
    return rec.get("hbm_bytes_per_launch")


def launch_overhead_ms(prof, profile_steps, step_ms):
    """Per-launch overhead of the event-timed profile pass: HIP events around
    each eager launch also time its dispatch, which the graph replay hides.
    Estimated as (event-timed sum per step - graph step time) / launches per
    step and subtracted from every stage's event time, so that the per-launch
    durations agree with rocprofv3's kernel durations."""
    total = sum(ms for ms, n in prof.values()) / profile_steps
    launches = sum(n for ms, n in prof.values()) / profile_steps
    if launches == 0:
        return 0.0
    return max(0.0, (total - step_ms) / launches)


def main():
    ap = argparse.ArgumentParser(description=__doc__,
                                 formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="encoder_t1600_d384_b8")
    ap.add_argument("--batch", type=int, default=None, help="override the batch size")
    ap.add_argument("--seed", type=int, default=2)
    ap.add_argument("--no-graph", action="store_true", help="launch eagerly")
    ap.add_argument("--steps-per-graph", type=int, default=10,
                    help="split convolution: steps captured per graph replay (one kernel "
                         "per step is shorter than a replay's host-side submission)")
    ap.add_argument("--streams", type=int, default=None,
                    help="encoder workloads: split the batch over this many streams "
                         "(default: 2 for the 192-wide encoder at batch >= 14 and the "
                         "384-wide one at batch >= 5, where it measured faster, else 1)")
    ap.add_argument("--profile-steps", type=int, default=20)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--from-image", action="store_true",
                    help="start each step from the int8 640x640x3 image: patch embedding and "
                         "positional embedding, then the encoder")
    ap.add_argument("--mode", type=int, default=0,
                    help="decoder workloads: deformable sampling 0 = nearest, 1 = bilinear-Q8")
    ap.add_argument("--boxes", action="store_true",
                    help="decoder workloads: reference boxes (offsets relative to the box) "
                         "instead of reference points")
    ap.add_argument("--calibration-copy-mib", type=int, default=0,
                    help="first make one plain device-to-device copy of this many MiB "
                         "(the known-size reference for rocprofv3 byte counters)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}, "
              f"WORLD_SIZE={world}); the encoder is not sharded across GPUs",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2607_24981_amd import ilw, synth

    if not os.path.exists(ilw.LIB_PATH):
        from paper_2607_24981_amd import build as hip_build
        hip_build.build()
    if not torch.cuda.is_available():
        print("bench.py needs a ROCm GPU", file=sys.stderr)
        sys.exit(1)

    if args.calibration_copy_mib:
        src = torch.ones(args.calibration_copy_mib << 20, dtype=torch.int8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
        log(f"calibration copy of {args.calibration_copy_mib} MiB done")

    if args.workload in synth.SPLIT_WORKLOADS:
        return bench_split(args, synth.SPLIT_WORKLOADS[args.workload])
    if args.workload in synth.ROWOP_WORKLOADS:
        return bench_rowop(args, synth.ROWOP_WORKLOADS[args.workload])
    if args.workload in synth.DECODER_WORKLOADS:
        return bench_decoder(args, synth.DECODER_WORKLOADS[args.workload])
    wl = synth.WORKLOADS[args.workload]
    B = wl.batch if args.batch is None else args.batch
    log(f"workload {wl.name}: batch {B}, {wl.tokens} tokens, dim {wl.dim}, "
        f"{len(wl.windows)} blocks")
    if args.streams is None:
        # two half-batches on two streams where measured faster: the tiny
        # encoder from batch 14, the 384-wide one from batch 5 (each half's
        # block tails and attention then share the CUs); below those one
        # stream wins (batch 12: 0.53 against 0.64 ms, batch 4: 0.68
        # against 0.70 ms)
        args.streams = 2 if (B >= 14 or (wl.dim == 384 and B >= 5)) else 1
    blocks, x = synth.encoder_inputs(wl, args.seed, "baseline", batch=B)
    enc = ilw.Encoder(blocks, wl.windows, wl.grid_h, wl.grid_w)
    xd = ilw.to_device(x)
    out = torch.empty_like(xd)
    enc.workspace(B)
    pe = None
    if args.from_image:
        pe = synth.patch_embed_inputs(args.seed + 1000, B, wl.dim, wl.grid_h * 16,
                                      wl.grid_w * 16)
        ped = {k: (ilw.to_device(v) if isinstance(v, np.ndarray) else v) for k, v in pe.items()}

    def eager(parts=args.streams):
        if pe is not None:
            ilw.ilw_patch_embed(ped["img"], ped["w"], ped["bias"], ped["mult"], ped["shift"],
                                ped["pos"], pe["pos_mult_a"], pe["pos_mult_b"], pe["pos_shift"],
                                y=xd)
        if parts > 1:
            enc.forward_streams(xd, out, parts)
        else:
            enc.forward(xd, out)

    def capture(parts):
        s = torch.cuda.Stream()
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            for _ in range(3):
                eager(parts)
        torch.cuda.current_stream().wait_stream(s)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            eager(parts)
        return graph.replay

    step = eager
    if not args.no_graph:
        step = capture(args.streams)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record()
    for _ in range(args.steps):
        step()
    ev1.record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    wall_ms = (t1 - t0) * 1e3 / args.steps
    ev_ms = ev0.elapsed_time(ev1) / args.steps
    pe_ops = 2 * B * wl.tokens * wl.dim * 3 * 256 if pe is not None else 0
    ops = wl.gemm_ops() * B // wl.batch + pe_ops
    tops = ops / (wall_ms * 1e-3) / 1e12
    log(f"timed {args.steps} steps: {wall_ms:.4f} ms/step wall, {ev_ms:.4f} ms/step events, "
        f"{tops:.2f} TOPS, {B / (wall_ms * 1e-3):.1f} images/s")
    spread = _step_spread(step)
    log(f"single steps p10 / median / p90: {spread} ms")
    result = out.cpu().numpy()

    # per-stage kernel time, HIP events around each launch (eager pass, one
    # stream, so that the stages do not overlap)
    ilw.profile_enable(True)
    for _ in range(args.profile_steps):
        eager(parts=1)
    torch.cuda.synchronize()
    prof = ilw.profile_read()
    ilw.profile_enable(False)
    work = stage_work(wl, B, {k: v[1] // args.profile_steps for k, v in prof.items()})
    if pe is not None:
        work["patch_embed"] = ("ops", pe_ops)
    one_ms = ev_ms
    if args.streams > 1 and not args.no_graph:
        # the overhead estimate needs the one-stream graph's step time
        one_ms = _timed(capture(1), max(10, args.steps // 5), 5)[1]
    ovh = launch_overhead_ms(prof, args.profile_steps, one_ms)
    stages = {}
    for name, (kind, amount) in work.items():
        ms, n = prof[name]
        if n == 0:
            continue
        per_launch = ms / n - ovh
        per_step_ms = per_launch * n / args.profile_steps
        rate = amount / (per_step_ms * 1e-3)
        stages[name] = {"ms_per_step": round(per_step_ms, 5),
                        "launches_per_step": n // args.profile_steps,
                        "ms_per_launch": round(per_launch, 5),
                        "ms_per_launch_events": round(ms / n, 5),
                        ("TOPS" if kind == "ops" else "GBps"):
                            round(rate / (1e12 if kind == "ops" else 1e9), 2)}
    dom = max(stages, key=lambda k: stages[k]["ms_per_step"])
    kind, amount = work[dom]
    launches = stages[dom]["launches_per_step"]
    achieved = amount / (stages[dom]["ms_per_step"] * 1e-3)
    if kind == "ops":
        roof = {"bound": "mfma", "achieved": round(achieved / 1e12, 3),
                "peak": PEAK_INT8_TOPS, "unit": "TOPS"}
    else:
        roof = {"bound": "hbm", "achieved": round(achieved / 1e9, 2), "peak": PEAK_HBM_GBS,
                "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 5)
    roof["kernel"] = KERNEL_OF_STAGE[dom][0]
    roof["stage"] = dom
    roof["ms_per_launch"] = stages[dom]["ms_per_launch"]
    roof["algorithmic_per_launch"] = amount // (launches * 1)
    roof["traffic"] = measured_traffic(dom, wl.name)
    roof["launch_overhead_ms"] = round(ovh, 5)
    log(f"dominant stage {dom}: {json.dumps(roof)}")
    log("stages: " + json.dumps(stages))

    cpu = None
    parity = None
    if not args.no_cpu_baseline:
        cpu, parity = encoder_cpu_baseline(wl, blocks, x, pe, B, pe_ops, result)

    line = {
        "metric": METRIC,
        "value": round(tops, 3),
        "unit": "TOPS",
        "images_per_s": round(B / (wall_ms * 1e-3), 2),
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall_ms, 5),
        "ms_per_step_p10_p50_p90": spread,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic",
        "config": {"workload": wl.name, "batch": B, "tokens": wl.tokens, "dim": wl.dim,
                   "heads": wl.heads, "mlp_dim": wl.mlp_dim, "blocks": len(wl.windows),
                   "attention": "window 20x20 / global alternating",
                   "launch": "eager" if args.no_graph else "hip graph",
                   "streams": args.streams,
                   "input": ("int8 image 640x640x3: patch + positional embedding, then the "
                             "encoder" if pe is not None else "int8 tokens"),
                   "gemm_ops_per_step": ops},
        "roofline": roof,
        "cpu_baseline": cpu,
        "parity": parity,
        "stages": stages,
    }
    print(json.dumps(line), flush=True)
    if parity not in (None, "bit-exact"):
        sys.exit(1)



def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def encoder_cpu_baseline(wl, blocks, x, pe, B, pe_ops, result):
    """The CPU oracle on the benchmarked workload, as it stands: image 0 on
    one thread, then every image of the batch on a pool of host threads (one
    image per task; the oracle's C calls release the GIL, and images are
    independent, so the results are the same).  Every image is compared with
    the GPU output of the timed run."""
    import concurrent.futures as cf

    import numpy as np

    import oracle
    if not os.path.exists(oracle._SO):
        oracle.build()

    def forward(i):
        y = x[i:i + 1]
        if pe is not None:
            y = oracle.patch_embed(pe["img"][i:i + 1], pe["w"], pe["bias"], pe["mult"],
                                   pe["shift"], pe["pos"], pe["pos_mult_a"], pe["pos_mult_b"],
                                   pe["pos_shift"])
        for p, (wh, ww) in zip(blocks, wl.windows):
            y = oracle.block_forward(p, y, wl.grid_h, wl.grid_w, wh, ww)
        return y

    ops1 = wl.gemm_ops() // wl.batch + pe_ops // B
    log("cpu baseline: oracle on image 0, one thread ...")
    c0 = time.perf_counter()
    ref = {0: forward(0)}
    t1 = time.perf_counter() - c0
    avail = len(os.sched_getaffinity(0))
    threads = max(1, min(avail, B))
    log(f"cpu baseline: oracle on all {B} images, {threads} threads ({avail} cores) ...")
    c0 = time.perf_counter()
    with cf.ThreadPoolExecutor(max_workers=threads) as ex:
        outs = list(ex.map(forward, range(B)))
    tall = time.perf_counter() - c0
    bad_images = [i for i in range(B) if not np.array_equal(result[i:i + 1], outs[i])]
    if not np.array_equal(outs[0], ref[0]):
        bad_images.append("oracle image 0 differs between its two runs")
    model = cpu_model()
    cpu = {"value": round(ops1 * B / tall / 1e12, 6), "unit": "TOPS",
           "images_per_s": round(B / tall, 4), "cores": threads, "kind": "oracle",
           "cpu_model": model, "host_cores_available": avail,
           "sample": f"all {B} images of {wl.name}, the full {len(wl.windows)}-block forward "
                     f"of each ({ops1 / 1e9:.2f} G int8 ops per image), one image per thread "
                     f"on {threads} threads, {tall:.1f} s",
           "single_thread": {"value": round(ops1 / t1 / 1e12, 6), "unit": "TOPS",
                             "images_per_s": round(1 / t1, 4), "cores": 1,
                             "sample": f"image 0, {t1:.1f} s"}}
    parity = ("bit-exact" if not bad_images
              else f"images differing from the oracle: {bad_images}")
    log(f"cpu baseline {cpu['value']} TOPS on {threads} threads, {cpu['single_thread']['value']} "
        f"TOPS on one ({model}); parity of all {B} images: {parity}")
    return cpu, parity


def _timed(step, steps, warmup):
    import torch
    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record()
    for _ in range(steps):
        step()
    ev1.record()
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    return (t1 - t0) * 1e3 / steps, ev0.elapsed_time(ev1) / steps


def _step_spread(step, n=50):
    """p10 / median / p90 of single-step times: one HIP event between
    consecutive steps (a pass of its own, after the timed region)."""
    import numpy as np
    import torch
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    torch.cuda.synchronize()
    evs[0].record()
    for i in range(n):
        step()
        evs[i + 1].record()
    torch.cuda.synchronize()
    t = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(n)])
    return [round(float(v), 5) for v in np.percentile(t, [10, 50, 90])]


def bench_split(args, wl):
    """Stage three: the projector's scale-preserving split convolution."""
    import numpy as np
    import torch

    from paper_2607_24981_amd import ilw, synth
    B = wl.batch if args.batch is None else args.batch
    log(f"workload {wl.name}: batch {B}, {wl.tokens} tokens, branches {wl.branches} -> {wl.out}")
    d = synth.split_conv_inputs(wl, args.seed, batch=B)
    xs = [ilw.to_device(x) for x in d["xs"]]
    ws = [ilw.to_device(w) for w in d["ws"]]
    bm = [ilw.to_device(m) for m in d["branch_mults"]]
    bs = [ilw.to_device(v) for v in d["branch_shifts"]]
    bias, om, os_ = (ilw.to_device(d[k]) for k in ("bias", "out_mult", "out_shift"))
    y = torch.empty((B * wl.tokens, wl.out), dtype=torch.int8, device="cuda")

    def eager():
        ilw.ilw_split_conv(xs, ws, bm, bs, bias, om, os_, y=y)

    # G steps per graph replay (each one the whole split convolution of the
    # batch), so that the timed steps are not paced by the host's replay calls
    G = 1 if args.no_graph or args.steps_per_graph < 1 or args.steps % args.steps_per_graph \
        else args.steps_per_graph
    step = eager
    if not args.no_graph:
        st = torch.cuda.Stream()
        st.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(st):
            for _ in range(3):
                eager()
        torch.cuda.current_stream().wait_stream(st)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for _ in range(G):
                eager()
        step = graph.replay
    wall_ms, ev_ms = _timed(step, args.steps // G, max(1, args.warmup // G))
    wall_ms, ev_ms = wall_ms / G, ev_ms / G
    ops = wl.gemm_ops() * B // wl.batch
    tops = ops / (wall_ms * 1e-3) / 1e12
    log(f"timed {args.steps} steps ({G} per graph replay): {wall_ms:.4f} ms/step wall, "
        f"{ev_ms:.4f} ms/step events, {tops:.2f} TOPS, {B / (wall_ms * 1e-3):.1f} images/s")
    spread = [round(v / G, 5) for v in _step_spread(step)]
    result = y.cpu().numpy()

    ilw.profile_enable(True)
    for _ in range(args.profile_steps):
        eager()
    torch.cuda.synchronize()
    prof = ilw.profile_read()
    ilw.profile_enable(False)
    ms, n = prof["split_conv"]
    ovh = launch_overhead_ms(prof, args.profile_steps, ev_ms)
    per_launch = ms / n - ovh
    roof = {"bound": "mfma", "achieved": round(ops / (per_launch * 1e-3) / 1e12, 3),
            "peak": PEAK_INT8_TOPS, "unit": "TOPS"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 5)
    roof.update({"kernel": "split_conv_kernel", "stage": "split_conv",
                 "ms_per_launch": round(per_launch, 5), "algorithmic_per_launch": ops,
                 "traffic": measured_traffic("split_conv", wl.name),
                 "launch_overhead_ms": round(ovh, 5)})
    log(f"dominant stage split_conv: {json.dumps(roof)}")

    cpu = parity = None
    if not args.no_cpu_baseline:
        import oracle
        if not os.path.exists(oracle._SO):
            oracle.build()
        T = wl.tokens
        c0 = time.perf_counter()
        ref = oracle.split_conv([x[:T] for x in d["xs"]], d["ws"], d["branch_mults"],
                                d["branch_shifts"], d["bias"], d["out_mult"], d["out_shift"])
        c1 = time.perf_counter()
        ops1 = wl.gemm_ops() // wl.batch
        cpu = {"value": round(ops1 / (c1 - c0) / 1e12, 6), "unit": "TOPS",
               "images_per_s": round(1 / (c1 - c0), 4), "cores": 1, "kind": "oracle",
               "sample": f"one image (1 of {B}) of {wl.name}, {ops1 / 1e9:.3f} G int8 ops, "
                         f"{c1 - c0:.2f} s"}
        bad = int(np.count_nonzero(result[:T] != ref))
        parity = "bit-exact" if bad == 0 else f"{bad} of {ref.size} outputs differ"
        log(f"cpu baseline {cpu['value']} TOPS; parity of image 0: {parity}")

    line = {"metric": METRIC, "value": round(tops, 3), "unit": "TOPS",
            "images_per_s": round(B / (wall_ms * 1e-3), 2), "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": round(wall_ms, 5),
            "ms_per_step_p10_p50_p90": spread, "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "int8", "data": "synthetic",
            "config": {"workload": wl.name, "batch": B, "tokens": wl.tokens,
                       "branches": list(wl.branches), "out_channels": wl.out,
                       "launch": "eager" if args.no_graph else f"hip graph, {G} steps per replay",
                       "gemm_ops_per_step": ops},
            "roofline": roof, "cpu_baseline": cpu, "parity": parity}
    print(json.dumps(line), flush=True)
    if parity not in (None, "bit-exact"):
        sys.exit(1)


def bench_rowop(args, wl):
    """A stand-alone row-wise or element-wise operator over the tensor it
    sees in the encoder; reported as achieved HBM GB/s of its algorithmic
    bytes (int8 in and out once) against the 8 TB/s peak."""
    import numpy as np
    import torch

    from paper_2607_24981_amd import ilw, synth
    log(f"workload {wl.name}: {wl.op} over {wl.rows} x {wl.cols} int8")
    d = synth.rowop_inputs(wl, args.seed)
    x = ilw.to_device(d["x"])
    y = torch.empty_like(x)
    if wl.op == "shiftmax":
        call = lambda: ilw.ilw_shiftmax(x, d["I0"], y=y)
    elif wl.op == "sdshiftgelu":
        call = lambda: ilw.ilw_sdshiftgelu(x, d["I0"], d["mult"], d["shift"], y=y)
    elif wl.op == "layernorm":
        beta, mult, shift = (ilw.to_device(d[k]) for k in ("beta", "mult", "shift"))
        call = lambda: ilw.ilw_int_layernorm(x, beta, mult, shift, 10, y=y)
    else:
        b = ilw.to_device(d["b"])
        call = lambda: ilw.ilw_residual_add(x, b, d["mult_a"], d["mult_b"], d["shift"], y=y)
    G = 1 if args.no_graph or args.steps % args.steps_per_graph else args.steps_per_graph
    step = call
    if not args.no_graph:
        st = torch.cuda.Stream()
        st.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(st):
            for _ in range(3):
                call()
        torch.cuda.current_stream().wait_stream(st)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for _ in range(G):
                call()
        step = graph.replay
    wall_ms, ev_ms = _timed(step, args.steps // G, max(1, args.warmup // G))
    wall_ms, ev_ms = wall_ms / G, ev_ms / G
    nbytes = wl.bytes_moved()
    gbs = nbytes / (ev_ms * 1e-3) / 1e9
    log(f"timed {args.steps} calls ({G} per graph replay): {ev_ms * 1e3:.2f} us per call, "
        f"{gbs:.1f} GB/s of {nbytes / 1e6:.2f} MB")
    spread = [round(v / G, 5) for v in _step_spread(step)]
    result = y.cpu().numpy()
    roof = {"bound": "hbm", "achieved": round(gbs, 2), "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": round(gbs / PEAK_HBM_GBS, 5), "kernel": KERNEL_OF_STAGE[wl.op if wl.op
                                                                             != "layernorm"
                                                                             else "layernorm"][0],
            "stage": wl.op, "ms_per_launch": round(ev_ms, 5), "algorithmic_per_launch": nbytes,
            "traffic": measured_traffic(wl.op, wl.name)}

    cpu = parity = None
    if not args.no_cpu_baseline:
        import oracle
        if not os.path.exists(oracle._SO):
            oracle.build()
        n = min(wl.rows, max(1, (64 << 20) // (64 * wl.cols)))  # a sample of whole rows
        xs = d["x"][:n]
        c0 = time.perf_counter()
        if wl.op == "shiftmax":
            ref = oracle.shiftmax_rows(xs, d["I0"])
        elif wl.op == "sdshiftgelu":
            ref = oracle.sdshiftgelu_tensor(xs, d["I0"], d["mult"], d["shift"])
        elif wl.op == "layernorm":
            ref = oracle.int_layernorm(xs, d["beta"], d["mult"], d["shift"], 10)
        else:
            ref = oracle.residual_tensor(xs, d["b"][:n], d["mult_a"], d["mult_b"], d["shift"])
        c1 = time.perf_counter()
        sb = wl.bytes_moved() * n // wl.rows
        cpu = {"value": round(sb / (c1 - c0) / 1e9, 4), "unit": "GB/s", "cores": 1,
               "kind": "oracle", "cpu_model": cpu_model(),
               "sample": f"the first {n} of {wl.rows} rows, {c1 - c0:.2f} s"}
        bad = int(np.count_nonzero(result[:n] != ref))
        parity = "bit-exact" if bad == 0 else f"{bad} of {ref.size} outputs differ"
        log(f"cpu baseline {cpu['value']} GB/s; parity of the sampled rows: {parity}")

    line = {"metric": f"HBM GB/s of the stand-alone {wl.op} operator", "value": round(gbs, 2),
            "unit": "GB/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
            "ms_per_step": round(ev_ms, 5), "ms_per_step_p10_p50_p90": spread,
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "int8",
            "data": "synthetic",
            "config": {"workload": wl.name, "op": wl.op, "rows": wl.rows, "cols": wl.cols,
                       "launch": "eager" if args.no_graph else f"hip graph, {G} calls per replay",
                       "algorithmic_bytes": nbytes},
            "roofline": roof, "cpu_baseline": cpu, "parity": parity}
    print(json.dumps(line), flush=True)
    if parity not in (None, "bit-exact"):
        sys.exit(1)


def bench_decoder(args, wl):
    """The integer deformable decoder layer around the deformable workload."""
    import numpy as np
    import torch

    from paper_2607_24981_amd import ilw, synth
    B = wl.batch if args.batch is None else args.batch
    log(f"workload {wl.name}: batch {B}, {wl.queries} queries, dim {wl.dim}, mode {args.mode}, "
        f"references {'boxes' if args.boxes else 'points'}")
    p, tgt, mem, ref, hw, start = synth.decoder_inputs(wl, args.seed, batch=B, mode=args.mode,
                                                       boxes=args.boxes)
    dd = ilw.DeviceDecoder(p)
    tgt_d, mem_d, ref_d = ilw.to_device(tgt), ilw.to_device(mem), ilw.to_device(ref)
    y = torch.empty_like(tgt_d)
    S = mem.shape[1]
    ws = torch.empty(dd.workspace_bytes(B, wl.queries, S), dtype=torch.int8, device="cuda")

    def eager():
        ilw.ilw_decoder_layer(dd, tgt_d, mem_d, ref_d, hw, start, y=y, workspace=ws)

    step = eager
    if not args.no_graph:
        st = torch.cuda.Stream()
        st.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(st):
            for _ in range(3):
                eager()
        torch.cuda.current_stream().wait_stream(st)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            eager()
        step = graph.replay
    wall_ms, ev_ms = _timed(step, args.steps, args.warmup)
    ops = wl.gemm_ops() * B // wl.batch
    tops = ops / (wall_ms * 1e-3) / 1e12
    log(f"timed {args.steps} steps: {wall_ms:.4f} ms/step wall, {ev_ms:.4f} ms/step events, "
        f"{tops:.2f} TOPS, {B / (wall_ms * 1e-3):.1f} images/s")
    spread = _step_spread(step)
    result = y.cpu().numpy()

    ilw.profile_enable(True)
    for _ in range(args.profile_steps):
        eager()
    torch.cuda.synchronize()
    prof = ilw.profile_read()
    ilw.profile_enable(False)
    Q, D, H, F = wl.queries, wl.dim, wl.heads, wl.ffn_dim
    L, P = len(wl.levels), wl.points
    MQ, MS, NW = B * Q, B * S, H * L * P
    work = {
        "gemm_qkv": ("ops", 2 * MQ * 3 * D * D),
        "attention": ("ops", 4 * B * Q * Q * D),
        "decoder": ("ops", 2 * MQ * D * (2 * D + 3 * NW + 2 * F) + 2 * MS * D * D),
        # gathered head slices, offsets (int8, widened in the sampler), logits, output
        "deform": ("bytes", MQ * NW * (D // H) + MQ * 2 * NW + MQ * NW + MQ * D),
        "layernorm": ("bytes", 3 * (2 * MQ * D + 12 * D)),
    }
    ovh = launch_overhead_ms(prof, args.profile_steps, ev_ms)
    stages = {}
    for name, (kind, amount) in work.items():
        ms, n = prof[name]
        if n == 0:
            continue
        per_launch = ms / n - ovh
        per_step = per_launch * n / args.profile_steps
        stages[name] = {"ms_per_step": round(per_step, 5),
                        "launches_per_step": n // args.profile_steps,
                        "ms_per_launch": round(per_launch, 5),
                        "ms_per_launch_events": round(ms / n, 5),
                        ("TOPS" if kind == "ops" else "GBps"):
                            round(amount / (per_step * 1e-3) / (1e12 if kind == "ops" else 1e9),
                                  2)}
    dom = max(stages, key=lambda k: stages[k]["ms_per_step"])
    kind, amount = work[dom]
    achieved = amount / (stages[dom]["ms_per_step"] * 1e-3)
    if kind == "ops":
        roof = {"bound": "mfma", "achieved": round(achieved / 1e12, 3), "peak": PEAK_INT8_TOPS,
                "unit": "TOPS"}
    else:
        roof = {"bound": "hbm", "achieved": round(achieved / 1e9, 2), "peak": PEAK_HBM_GBS,
                "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 5)
    roof.update({"stage": dom, "ms_per_launch": stages[dom]["ms_per_launch"],
                 "algorithmic_per_step": amount, "traffic": None,
                 "launch_overhead_ms": round(ovh, 5)})
    log(f"dominant stage {dom}: {json.dumps(roof)}")
    log("stages: " + json.dumps(stages))

    cpu = parity = None
    if not args.no_cpu_baseline:
        import oracle
        if not os.path.exists(oracle._SO):
            oracle.build()
        c0 = time.perf_counter()
        ref0 = oracle.decoder_forward(p, tgt[:1], mem[:1], ref[:1], hw, start)
        c1 = time.perf_counter()
        ops1 = wl.gemm_ops() // wl.batch
        cpu = {"value": round(ops1 / (c1 - c0) / 1e12, 6), "unit": "TOPS",
               "images_per_s": round(1 / (c1 - c0), 4), "cores": 1, "kind": "oracle",
               "sample": f"one image (1 of {B}) of {wl.name}, mode {args.mode}: the whole "
                         f"layer, {ops1 / 1e9:.2f} G int8 ops, {c1 - c0:.2f} s"}
        bad = int(np.count_nonzero(result[:1] != ref0))
        parity = "bit-exact" if bad == 0 else f"{bad} of {ref0.size} outputs differ"
        log(f"cpu baseline {cpu['value']} TOPS; parity of image 0: {parity}")

    line = {"metric": METRIC, "value": round(tops, 3), "unit": "TOPS",
            "images_per_s": round(B / (wall_ms * 1e-3), 2), "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": round(wall_ms, 5),
            "ms_per_step_p10_p50_p90": spread, "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "int8", "data": "synthetic",
            "config": {"workload": wl.name, "batch": B, "queries": Q, "dim": D, "heads": H,
                       "ffn_dim": F, "levels": [list(l) for l in wl.levels], "points": P,
                       "sampling": "nearest" if args.mode == 0 else "bilinear-Q8",
                       "references": "boxes" if args.boxes else "points",
                       "launch": "eager" if args.no_graph else "hip graph",
                       "gemm_ops_per_step": ops},
            "roofline": roof, "cpu_baseline": cpu, "parity": parity, "stages": stages}
    print(json.dumps(line), flush=True)
    if parity not in (None, "bit-exact"):
        sys.exit(1)


if __name__ == "__main__":
    main()
