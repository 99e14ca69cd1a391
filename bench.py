#!/usr/bin/env python3
"""MPM merge + unmerge throughput on one MI355X.

One step = the whole hot path over one batch already resident in HBM: MPM
before encoder blocks 2 and 5 (two insertions, identity blocks in between),
map composition and the gather back to the full token grid. Default workload:
ViT-B/16 tokens of 512x512 images (B=64, N=1024, D=768, bfloat16), synthetic.

Prints one JSON line: images/s, per-step time, the roofline of the dominant
kernel (the fused affinity-argmax, MFMA-bound), per-kernel timings, and the
CPU oracle timed on a bounded sample on this host.
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

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_F32_TFLOPS = 157.3     # MI355X dense fp32 matrix
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E

METRIC = "MPM merge+unmerge images/s at ViT-B N=1024 B=64; % MFMA and % HBM peak"

AFFINITY_BATCH = 20  # back-to-back affinity launches between two timing events
AFFINITY_REPS = 5    # such batches per insertion; the median is taken

# HBM traffic of one affinity step (the whole-block launch and, where the schedule
# defers diagonal blocks, the half-block launch; the two insertions averaged) from
# rocprofv3 FETCH_SIZE / WRITE_SIZE runs on each workload, calibrated with a copy
# kernel (profiles/<workload>_rocprof.md). Valid only for the kernel source it was
# measured on, with the default schedule.
TRAFFIC = {"source_sha256": "1dae8e815f91dc3ce104e116133adef4251abc9e32c244ab1520b8269f69403b",
           "bytes_per_launch": {"vit_ti_512": 6556890, "vit_s_512": 25826025, "vit_b_512": 151433431,
                                "vit_l_1024": 510617954, "stress_768": 182226447}}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def kernel_source_hash() -> str:
    """Hash of the affinity kernel's source, to tell whether stored counters still apply."""
    p = os.path.join(ROOT, "paper_2604_05718_amd", "csrc", "affinity_argmax.hip")
    return hashlib.sha256(open(p, "rb").read()).hexdigest()


def executed_affinity_flops(cfg, counts, schedule):
    """Matrix-core flops each affinity launch issues: 2 * w^2 * D per w x w block,
    nb^2 blocks per image of nb = ceil(n / w) blocks under the full schedules
    (w = 256, or 64 for full_64), nb (nb + 1) / 2 under the symmetric one
    (padding rows included)."""
    w = 64 if schedule == "full_64" else 256
    out = []
    n_in = [cfg.N] * cfg.B
    for st in range(cfg.insertions):
        blocks = 0
        for n in n_in:
            nb = (n + w - 1) // w
            blocks += nb * (nb + 1) // 2 if schedule == "symmetric" else nb * nb
        out.append(blocks * 2.0 * w * w * cfg.D)
        n_in = counts[st]
    return out


def algorithmic_work(cfg, counts):
    """Per kernel step of one step: ('flops'|'bytes', amount). counts[s] = per-image
    token counts after insertion s (counts[-1] = N for every image). The affinity step
    carries the compaction (its last workgroup per image); its work is counted as the
    affinity's flops (the compaction's few bytes are not)."""
    s = 2 if cfg.dtype == "bf16" else 4
    D, N, B = cfg.D, cfg.N, cfg.B
    work = []
    n_in = [N] * B
    for st in range(cfg.insertions):
        n_out = counts[st]
        work.append(("flops", sum(2.0 * n * n * D for n in n_in)))
        # average: read every member row once, write every cluster row, read src and the offsets
        work.append(("bytes", sum((n + m) * D * s + 8.0 * m + 4 for n, m in zip(n_in, n_out))))
        n_in = n_out
    # gather: read the composed map, each final row once, write the full grid
    gather = sum(4.0 * N + m * D * s + N * D * s for m in n_in)
    if cfg.insertions == 1:
        work.append(("bytes", gather))
        return work
    # compose: read r* (4N), touch the stage map of the previous survivors (4 n), write r* (4N);
    # the last composition runs inside the gather kernel
    compose = [sum(8.0 * N + 4.0 * m for m in counts[st - 1]) for st in range(1, cfg.insertions)]
    for c in compose[:-1]:
        work.append(("bytes", c))
    work.append(("bytes", compose[-1] + gather))
    return work


def window_candidates(positions, grid: int, window: int) -> int:
    """Sum over tokens of the number of other tokens inside their window (the locality
    constraint): positions = raster indices of one image's tokens on a grid x grid grid."""
    import numpy as np

    occ = np.zeros((grid, grid), np.int64)
    occ.flat[np.asarray(positions)] = 1
    cs = np.zeros((grid + 1, grid + 1), np.int64)
    cs[1:, 1:] = occ.cumsum(0).cumsum(1)
    r, c = np.divmod(np.asarray(positions), grid)
    r0, r1 = np.clip(r - window, 0, grid), np.clip(r + window + 1, 0, grid)
    c0, c1 = np.clip(c - window, 0, grid), np.clip(c + window + 1, 0, grid)
    inside = cs[r1, c1] - cs[r0, c1] - cs[r1, c0] + cs[r0, c0]
    return int((inside - 1).sum())


def algorithmic_work_local(cfg, counts, stage_positions, window):
    """algorithmic_work for locality-constrained insertions: each insertion's affinity
    costs 2 D flops per (token, candidate in its window) pair; the merge_local step
    also holds the compaction and the pair average."""
    work = []
    for st in range(cfg.insertions):
        work.append(("flops", sum(2.0 * cfg.D * window_candidates(p, cfg.G, window) for p in stage_positions[st])))
    dense = algorithmic_work(cfg, counts)
    return work + dense[2 * cfg.insertions:]


def cpu_baseline(cfg, x_cpu, budget_s: float, threads: int | None = None):
    import oracle

    threads = threads or oracle.default_threads()
    t0 = time.perf_counter()
    done = 0
    # Images of the batch in order, starting over after the last one, until the
    # budget is spent (a whole batch can take less than the budget).
    while True:
        b = done % cfg.B
        oracle.schedule(oracle.as_f64(x_cpu[b]), cfg.dtype, insertions=cfg.insertions, threads=threads)
        done += 1
        if time.perf_counter() - t0 >= budget_s:
            break
    el = time.perf_counter() - t0
    return {
        "value": done / el,
        "unit": "images/s",
        "cores": threads,
        "kind": "oracle",
        "cpu": cpu_model(),
        "sample": (f"{done} image schedules over the {cfg.B} images of {cfg.name} in order "
                   f"({min(done, cfg.B)} distinct), full schedule ({cfg.insertions} insertions, "
                   f"compose, gather), float64 brute force, {el:.1f} s"),
    }


def backbone(args, cfg, dev) -> int:
    """The paper's end-to-end setting with this library's kernels: a ViT encoder (random weights, 12
    blocks, the workload's width, 64-wide heads) with MPM before blocks 2 and 5 and the
    gather after the last block, against the same encoder without merging; whole
    forward passes timed, images/s for both."""
    import torch

    from paper_2604_05718_amd import synth
    from paper_2604_05718_amd.encoder import Encoder

    dtype = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    x = synth.make_batch(cfg, seed=0).to(dev)
    heads = cfg.D // 64
    res = {}
    for name, merge_before, attn in (("plain", (), "varlen"), ("mpm_2_5", (2, 5), "varlen"),
                                     ("plain_padded_attention", (), "padded"),
                                     ("mpm_2_5_padded_attention", (2, 5), "padded")):
        enc = Encoder(D=cfg.D, heads=heads, depth=12, merge_before=merge_before, dtype=dtype, device=dev,
                      attn=attn)
        for _ in range(max(2, args.warmup)):
            enc.forward(x)
        torch.cuda.synchronize()
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record()
        for _ in range(args.steps):
            enc.forward(x)
        t1.record()
        torch.cuda.synchronize()
        ms = t0.elapsed_time(t1) / args.steps
        res[name] = {"ms_per_forward": round(ms, 3), "images_per_s": round(cfg.B / (ms * 1e-3), 1)}
        if merge_before:
            res[name]["tokens_after_each_merge_mean"] = [round(sum(c) / len(c), 1) for c in enc.last_counts]
        log(f"bench: backbone {name}: {ms:.2f} ms per forward")
        del enc
        torch.cuda.empty_cache()
    out = {
        "metric": f"ViT encoder forward images/s, MPM before blocks 2 and 5 vs none ({cfg.name} tokens)",
        "value": res["mpm_2_5"]["images_per_s"], "unit": "images/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": res["mpm_2_5"]["ms_per_forward"], "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": cfg.dtype, "data": "synthetic tokens, random weights",
        "config": {"workload": f"{cfg.name}: 12-block ViT encoder, D={cfg.D}, {heads} heads, B={cfg.B}, N={cfg.N}",
                   "global_batch": cfg.B, "seq_len": cfg.N, "parallelism": "none (1 GPU)"},
        "attention": "torch variable-length flash attention on the packed rows",
        "plain": res["plain"], "mpm": res["mpm_2_5"],
        "speedup": round(res["plain"]["ms_per_forward"] / res["mpm_2_5"]["ms_per_forward"], 4),
        "padded_attention": {"plain": res["plain_padded_attention"], "mpm": res["mpm_2_5_padded_attention"],
                             "speedup": round(res["plain_padded_attention"]["ms_per_forward"] /
                                              res["mpm_2_5_padded_attention"]["ms_per_forward"], 4)},
    }
    print(json.dumps(out), flush=True)
    return 0


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--workload", default="vit_b_512")
    ap.add_argument("--cpu-seconds", type=float, default=15.0,
                    help="budget of the CPU oracle baseline (0 skips it)")
    ap.add_argument("--cold-steps", type=int, default=10,
                    help="steps timed after evicting the caches (0 skips them)")
    ap.add_argument("--prewarm-seconds", type=float, default=0.5,
                    help="run steps for this long before the warmup steps, so the device clocks have ramped up")
    ap.add_argument("--cpu-single-seconds", type=float, default=3.0,
                    help="budget of the single-thread CPU oracle figure (0 skips it)")
    ap.add_argument("--schedule", default="auto", choices=["auto", "full", "symmetric", "full_64"],
                    help="affinity work schedule (auto: the library's choice for the batch shape)")
    ap.add_argument("--window", type=int, default=None,
                    help="locality-constrained merging (Sec. 5): candidates within this many grid rows and columns")
    ap.add_argument("--backbone", action="store_true",
                    help="time a random-weight ViT encoder of the workload's width with MPM before blocks 2 and 5 "
                         "against the plain encoder, and print that instead")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="only run 5 device-to-device copies of this many MiB (counter calibration) and exit")
    args = ap.parse_args()

    if args.copy_calibration_mib:
        import torch

        n = args.copy_calibration_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"bench: copied {args.copy_calibration_mib} MiB 5 times")
        return 0

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        log("bench.py: measures one GPU only; the path shards by image with no communication, "
            "so a multi-GPU figure is not produced. Run with --gpus 1.")
        return 2

    import torch

    import paper_2604_05718_amd as mpm  # noqa: F401  (fails loudly without libmpm.so)
    from paper_2604_05718_amd import api, synth

    cfg = synth.config(args.workload)
    dev = torch.device("cuda:0")
    if args.backbone:
        return backbone(args, cfg, dev)
    dtype = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    log(f"bench: {cfg.name} B={cfg.B} N={cfg.N} D={cfg.D} {cfg.dtype}, generating inputs")
    x_cpu = synth.make_batch(cfg, seed=0)
    x = x_cpu.to(dev)
    sched = api.Schedule(cfg.B, cfg.N, cfg.D, dtype, cfg.insertions, schedule=args.schedule,
                         grid_w=cfg.G if args.window is not None else None, window=args.window)

    # Device pre-warm (outside the step count): the clocks of an idle device take a few
    # hundred milliseconds of load to ramp up, longer than a handful of warmup steps.
    prewarm_steps = 0
    t_end = time.perf_counter() + args.prewarm_seconds
    while time.perf_counter() < t_end:
        for _ in range(8):
            sched.run(x)
        prewarm_steps += 8
        torch.cuda.synchronize()
    for _ in range(args.warmup):
        sched.run(x)
    torch.cuda.synchronize()
    log(f"bench: pre-warm {prewarm_steps} steps, warmup {args.warmup} done, timing {args.steps} steps")

    # Timed region: K steps and nothing else on the stream between its two events.
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    start.record()
    for k in range(args.steps):
        sched.run(x)
    end.record()
    torch.cuda.synchronize()
    ms_per_step = start.elapsed_time(end) / args.steps

    # The dominant kernel, timed after the timed region in two ways. (1) Events bound to
    # the affinity launches of every step (start on the first launch, stop on the last):
    # each bound event leaves the device idle for a few microseconds next to its launch,
    # and part of that idle time falls inside the interval (at vit_b_512 this reads
    # 2-4% above (2)). (2) The launches of each insertion back to back on the input the
    # last step gave that insertion, AFFINITY_BATCH at a time between two events, which
    # agrees with the in-step kernel durations of a kernel trace within about 2%. The
    # roofline is computed from (2) where the path has a separate affinity entry point.
    aff_ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(cfg.insertions)] for _ in range(args.steps)]
    for pairs in aff_ev:
        for e0, e1 in pairs:  # torch creates events lazily, at their first record
            e0.record()
            e1.record()
    torch.cuda.synchronize()
    for k in range(args.steps):
        sched.run(x, affinity_events=aff_ev[k])
    torch.cuda.synchronize()
    aff_ms_bound = [sum(aff_ev[k][s][0].elapsed_time(aff_ev[k][s][1]) for k in range(args.steps)) / args.steps
                    for s in range(cfg.insertions)]
    aff_ms = aff_ms_bound
    if args.window is None:
        aff_ms = []
        for s in range(cfg.insertions):
            cur, cur_off, cur_inv = (x, None, None) if s == 0 else (sched.y[s - 1], sched.y_off[s - 1],
                                                                    sched.y_inv[s - 1])
            reps = []
            for _ in range(AFFINITY_REPS):
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                for _ in range(AFFINITY_BATCH):
                    api.affinity(cur, cur_off, N=cfg.N, x_inv=cur_inv, schedule=args.schedule, ws=sched.ws[s])
                e1.record()
                torch.cuda.synchronize()
                reps.append(e0.elapsed_time(e1) / AFFINITY_BATCH)
            aff_ms.append(sorted(reps)[len(reps) // 2])
    log(f"bench: {ms_per_step * 1e3:.1f} us/step, affinity kernels " + ", ".join(f"{m * 1e3:.1f}" for m in aff_ms)
        + " us (launch-bound events: " + ", ".join(f"{m * 1e3:.1f}" for m in aff_ms_bound) + " us)")

    # Per-kernel breakdown, outside the timed region: an event before every kernel
    # (these events add gaps between kernels, so this loop is slower than the timed one).
    nm = sched.n_marks()
    marks = [[torch.cuda.Event(enable_timing=True) for _ in range(nm)] for _ in range(args.steps)]
    start2, end2 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start2.record()
    for k in range(args.steps):
        sched.run(x, marks[k])
    end2.record()
    torch.cuda.synchronize()
    ms_marked = start2.elapsed_time(end2) / args.steps

    names = sched.kernel_names
    per_kernel_ms = [sum(m[i].elapsed_time(m[i + 1]) for m in marks) / args.steps for i in range(len(names))]
    counts = [torch.diff(sched.y_off[s].cpu()).tolist() for s in range(cfg.insertions)]
    if args.window is None:
        work = algorithmic_work(cfg, counts)
    else:
        stage_positions = [[list(range(cfg.N))] * cfg.B]
        for s in range(cfg.insertions - 1):
            off = sched.y_off[s].cpu().tolist()
            yp = sched.y_pos[s].cpu()
            stage_positions.append([yp[off[b]:off[b + 1]].tolist() for b in range(cfg.B)])
        work = algorithmic_work_local(cfg, counts, stage_positions, args.window)

    # Step-time distribution: one event per step boundary (outside the timed region).
    bounds = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    bounds[0].record()
    for k in range(args.steps):
        sched.run(x)
        bounds[k + 1].record()
    torch.cuda.synchronize()
    step_ms = sorted(bounds[k].elapsed_time(bounds[k + 1]) for k in range(args.steps))
    pct = lambda q: step_ms[min(len(step_ms) - 1, int(q * (len(step_ms) - 1) + 0.5))]
    distribution = {"p10_ms": round(pct(0.1), 4), "median_ms": round(pct(0.5), 4), "p90_ms": round(pct(0.9), 4)}

    # Cold caches: before each step a 1 GiB buffer is overwritten, which evicts the token
    # matrix from the 256 MB MALL and the L2s; per-kernel events as in the breakdown loop.
    cold = None
    if args.cold_steps > 0:
        scrub = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        cmarks = [[torch.cuda.Event(enable_timing=True) for _ in range(nm)] for _ in range(args.cold_steps)]
        for k in range(args.cold_steps):
            scrub.fill_(k & 0xFF)
            sched.run(x, cmarks[k])
        torch.cuda.synchronize()
        del scrub
        cold_kernel_ms = [sum(m[i].elapsed_time(m[i + 1]) for m in cmarks) / args.cold_steps
                          for i in range(len(names))]
        cold = {"steps": args.cold_steps,
                "ms_per_step_with_per_kernel_events": round(sum(cold_kernel_ms), 4),
                "kernels": []}
        for name, ms, (kind, amount) in zip(names, cold_kernel_ms, work):
            ent = {"name": name, "us": round(ms * 1e3, 2)}
            if kind == "bytes":
                gbs = amount / (ms * 1e-3) / 1e9
                ent.update({"gbs": round(gbs, 1), "frac_hbm": round(gbs / PEAK_HBM_GBS, 4)})
            cold["kernels"].append(ent)

    # The same step captured once in a HIP graph and replayed.
    graph = None
    try:
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            sched.run(x)
        for _ in range(3):
            g.replay()
        torch.cuda.synchronize()
        gs, ge = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        gs.record()
        for _ in range(args.steps):
            g.replay()
        ge.record()
        torch.cuda.synchronize()
        gms = gs.elapsed_time(ge) / args.steps
        graph = {"ms_per_step": round(gms, 4), "images_per_s": round(cfg.B / (gms * 1e-3), 1)}
        del g
    except Exception as exc:  # reported, not fatal: the eager figures above stand on their own
        graph = {"error": f"{type(exc).__name__}: {exc}"}

    schedule = mpm.affinity_schedule_used(cfg.B, cfg.N, cfg.D, dtype, args.schedule)
    if args.window is not None:
        rows = mpm.local_block_rows(cfg.B, cfg.N, cfg.D, dtype, cfg.G, args.window)
        schedule = f"window {args.window}, {rows}-row blocks"
    executed = executed_affinity_flops(cfg, counts, schedule) if args.window is None else None
    kernels = []
    for name, ms, (kind, amount) in zip(names, per_kernel_ms, work):
        ent = {"name": name, "us": round(ms * 1e3, 2)}
        if kind == "flops":
            tf = amount / (ms * 1e-3) / 1e12
            peak = PEAK_BF16_TFLOPS if cfg.dtype == "bf16" else PEAK_F32_TFLOPS
            ent.update({"gflop": round(amount / 1e9, 3), "tflops": round(tf, 1), "frac_mfma": round(tf / peak, 4)})
            if executed is not None:
                ent["executed_gflop"] = round(executed[int(name[len("affinity+compact"):]) - 1] / 1e9, 3)
        else:
            gbs = amount / (ms * 1e-3) / 1e9
            ent.update({"mbytes": round(amount / 1e6, 3), "gbs": round(gbs, 1), "frac_hbm": round(gbs / PEAK_HBM_GBS, 4)})
        kernels.append(ent)

    # Dominant kernel: the fused affinity-argmax (both insertions' launches).
    a_idx = [i for i, n in enumerate(names) if n.startswith("affinity") or n.startswith("merge_local")]
    a_flops = sum(work[i][1] for i in a_idx)
    a_ms = sum(aff_ms)
    peak = PEAK_BF16_TFLOPS if cfg.dtype == "bf16" else PEAK_F32_TFLOPS
    achieved = a_flops / len(a_idx) / (a_ms / len(a_idx) * 1e-3) / 1e12
    traffic = None
    if (TRAFFIC.get("source_sha256") == kernel_source_hash() and args.schedule == "auto" and
            args.window is None):
        traffic = TRAFFIC["bytes_per_launch"].get(cfg.name)
    roofline = {"bound": "mfma", "achieved": round(achieved, 1), "peak": peak, "unit": "TFLOP/s",
                "frac": round(achieved / peak, 4), "traffic": traffic, "schedule": schedule}
    if executed is not None:
        # The same launches counted by the matrix-core work they issue: below the
        # algorithmic figure under the symmetric schedule, which skips the blocks
        # below the diagonal.
        issued = sum(executed) / len(a_idx) / (a_ms / len(a_idx) * 1e-3) / 1e12
        roofline.update({"issued": round(issued, 1), "frac_issued": round(issued / peak, 4)})

    value = cfg.B / (ms_per_step * 1e-3)
    result = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "images/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": (f"{cfg.name}: ViT token grid {cfg.G}x{cfg.G} (N={cfg.N}), D={cfg.D}, B={cfg.B}, "
                                f"{cfg.insertions} MPM insertions + compose + gather"
                                + ("" if args.window is None else
                                   f", locality-constrained (window {args.window})")),
                   "global_batch": cfg.B, "seq_len": cfg.N, "parallelism": "none (1 GPU)"},
        "tokens_per_s": round(value * cfg.N, 0),
        "prewarm": {"seconds": args.prewarm_seconds, "steps": prewarm_steps},
        "affinity_timing": ({"method": "back to back", "launches": AFFINITY_BATCH * AFFINITY_REPS,
                             "us": [round(m * 1e3, 2) for m in aff_ms],
                             "launch_bound_events_us": [round(m * 1e3, 2) for m in aff_ms_bound]}
                            if args.window is None else
                            {"method": "launch-bound events", "steps": args.steps,
                             "us": [round(m * 1e3, 2) for m in aff_ms]}),
        "ms_per_step_with_per_kernel_events": round(ms_marked, 4),
        "survivors_mean": [round(sum(c) / len(c), 1) for c in counts],
        "roofline": roofline,
        "step_time_distribution": distribution,
        "kernels": kernels,
        "cold_cache": cold,
        "hip_graph": graph,
    }
    if args.cpu_seconds > 0:
        log("bench: timing the CPU oracle baseline")
        result["cpu_baseline"] = cpu_baseline(cfg, x_cpu, args.cpu_seconds)
    if args.cpu_single_seconds > 0:
        log("bench: timing the CPU oracle on one thread")
        result["cpu_baseline_single_thread"] = cpu_baseline(cfg, x_cpu, args.cpu_single_seconds, threads=1)
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
