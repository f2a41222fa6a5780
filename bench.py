"""Benchmark of the MixRT per-pixel rendering path on one MI355X.

One step = one mixrt_render call over one frame of the 1280x720 workload
(every stage of the path: ray setup, Eq. 2 calibration, K samples,
contraction, hash encoding, MLP, compositing), inputs already resident in
HBM.  For mesh workloads (--workload mesh720p) a step computes the G-buffer
from the mesh (rasterised by default, ray cast with --geometry raycast) and
then makes that render call.  Prints one JSON line.
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0          # MI355X HBM3E
MFMA_F16_PEAK_TFLOPS = 2500.0   # MI355X dense fp16 MFMA
PROFILE_COUNTERS = os.path.join(ROOT, "profiles", "render_kernel_view720p.counters.json")
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2312_11841_amd", "csrc", f)
                  for f in ("mixrt_render.hip", "mixrt_device.hpp", "mixrt_common.hpp")]


def kernel_source_digest() -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str):
    """HBM bytes per launch from the committed rocprofv3 FETCH_SIZE / WRITE_SIZE
    passes, each scaled by the same counter's reading for a plain copy of known
    size; None when no such record exists for this workload or the kernel
    sources changed since the counters were taken."""
    try:
        rec = json.load(open(PROFILE_COUNTERS))
    except (OSError, ValueError):
        return None, "no counter record"
    if rec.get("workload") != workload:
        return None, "counters taken on another workload"
    if rec.get("kernel_source_digest") != kernel_source_digest():
        return None, "kernel changed since the counters were taken"
    fetch = rec["FETCH_SIZE_KiB"] * 1024 * rec["fetch_scale"]
    write = rec["WRITE_SIZE_KiB"] * 1024 * rec["write_scale"]
    return int(fetch + write), "rocprofv3 FETCH_SIZE+WRITE_SIZE, copy-calibrated"


def measured_rooflines(cfg):
    """Achievable rates on this GPU from libmixrt_microbench.so: random
    gathers at the working sets of one hash level and of the whole table,
    streaming copy, streaming read, fp16 MFMA."""
    from paper_2312_11841_amd import microbench as mb
    eb = 2 if cfg.table_dtype == "f16" else 4
    entry = cfg.F * eb
    level_bytes = cfg.T * entry
    out = {"gather_random_lane_loads_per_s": {}, "gather_entry_bytes": entry}
    for name, size in (("one_level", level_bytes), ("whole_table", level_bytes * cfg.L)):
        size = 1 << (int(size) - 1).bit_length()
        r = mb.gather(size, 4 if entry <= 4 else (8 if entry <= 8 else 16), 0, iters=128)
        out["gather_random_lane_loads_per_s"][name] = {"bytes": size,
                                                       "value": round(r["lane_loads_per_s"])}
    # streaming rates peak at a few blocks per CU (more blocks contend for
    # DRAM pages): the best of a short sweep, with the block count it took
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    for name, fn, per_cu in (("copy", mb.copy, (2, 3, 4)), ("read", mb.read, (1, 1.5, 2, 3))):
        best = max((fn(1 << 30, blocks=int(k * cus)) for k in per_cu), key=lambda r: r["GBps"])
        out[f"{name}_GBps"] = round(best["GBps"], 1)
        out[f"{name}_blocks"] = int(best.get("blocks") or 0)
    out["mfma_f16_TFLOPs"] = round(mb.mfma()["TFLOPs"], 1)
    return out


def standalone_mlp(cfg, ds, renderer, samples):
    """The MLP stage alone (mixrt_debug_mlp) on `samples` fp16 input rows."""
    import torch
    x = torch.randn((samples, cfg.widths[0]), device="cuda:0").to(torch.float16)
    xi = x.view(torch.int16)
    # half a second of launches first: right after the render loop the first
    # tens of milliseconds of this stage ran up to 20% slower than its steady
    # rate (measured), so a few warm-up launches are not enough
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < 0.5:
        for _ in range(20):
            renderer.mlp(ds.mlp, xi)
        torch.cuda.synchronize()
    sec = time_launches(renderer.stream, lambda: renderer.mlp(ds.mlp, xi), 50) * 1e-3
    flops = samples * 2 * sum(p * q for p, q in zip(cfg.widths[:-1], cfg.widths[1:]))
    in_bytes = cfg.widths[0] * 2
    out = {"samples": samples, "ms": round(sec * 1e3, 4), "TFLOPs": round(flops / sec / 1e12, 1),
           "util_of_peak": round(flops / sec / 1e12 / MFMA_F16_PEAK_TFLOPS, 4),
           "hbm_bytes": samples * (in_bytes + 16),
           "GBps": round(samples * (in_bytes + 16) / sec / 1e9, 1)}
    if in_bytes in (32, 64, 96):
        # the stage's own memory pattern alone (rows in, 16 B per row out),
        # measured now: the most the stage can stream on this GPU
        from paper_2312_11841_amd import microbench as mb
        st = mb.rowstream(samples, in_bytes, blocks_list=(1, 2, 3, 4, 6, 8))
        ceiling_s = samples * (in_bytes + 16) / (st["GBps"] * 1e9)
        out["stream_ceiling"] = {
            "pattern": f"{in_bytes} B read + 16 B written per row, 64-row tiles, coalesced, "
                       "non-temporal (mixrt_mb_rowstream)",
            "GBps": round(st["GBps"], 1), "blocks": st["blocks"],
            "ms": round(ceiling_s * 1e3, 4),
            "util_of_peak": round(flops / ceiling_s / 1e12 / MFMA_F16_PEAK_TFLOPS, 4),
            "stage_frac_of_ceiling": round(ceiling_s / sec, 4)}
    return out


def gather_replay_floor(cfg, ds, renderer):
    """The render kernel's gather stream replayed alone: this frame's own
    sample positions (its ray setup), the kernel's tile order, lane order and
    level batches, loads XOR-folded (mixrt_mb_gather_replay).  The fastest of
    a sweep of grid sizes is the floor for this access stream."""
    import torch
    from paper_2312_11841_amd import microbench as mb
    from paper_2312_11841_amd import mixrt
    x, hit = renderer.ray_setup(ds)
    plan = renderer.launch_plan(ds)
    blocks, stripe, chunk = plan["blocks"], plan["tile_stripe"], plan["chunk"]
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    N = mixrt.level_resolutions(ds.grid)
    grids = sorted({blocks} | {k * cus for k in (1, 2, 3, 4, 6, 8)})
    r = mb.gather_replay(x, hit, cfg.views, cfg.W, cfg.rows_kept, cfg.K, ds.table, N, stripe,
                         grids, chunk=chunk, block_from=plan["block_from"],
                         hash_batch=plan["hash_batch"], claims=bool(plan["claims"]))
    del x, hit
    return {"render_blocks": blocks, "tile_stripe": stripe, "early_stop_chunk": chunk,
            "block_from": plan["block_from"], "hash_batch": plan["hash_batch"],
            "claims": plan["claims"], **r}


def stage_metrics(cfg, ds, out, steps, chunk=0):
    """Where the fused kernel's time goes, two ways, both from builds of the
    same render source with one -D option:
      - phase timer: every wave adds the shader clocks of each phase of each
        tile (s_memtime at the phase boundaries); a phase's share of all
        wave-clocks times the kernel's time is that phase's time;
      - ablation (the paper's own method, Tab. 3): the frame with one stage
        removed; the difference to the full kernel is the stage's marginal
        cost (stages overlap in the fused kernel, so marginal costs need not
        add up to the whole)."""
    import torch
    from paper_2312_11841_amd import mixrt
    stream = torch.cuda.current_stream()
    res = {}
    r = mixrt.Renderer(0, stream=stream, variant="timer", early_stop_chunk=chunk)
    for _ in range(5):
        r.render(ds, out)
    r.phase_cycles(reset=True)
    timer_ms = time_launches(stream, lambda: r.render(ds, out), steps)
    ph = r.phase_cycles(reset=True)
    r.close()
    res["samples_evaluated_per_frame"] = ph["samples"] // steps
    tot = sum(ph[k] for k in ("setup", "hash", "mlp", "composite"))
    res["phase_share"] = {k: round(ph[k] / tot, 4) for k in ("setup", "hash", "mlp", "composite")}
    res["timer_build_ms"] = round(timer_ms, 4)
    abl = {}
    for v in ("split_nodisp", "split_nohash", "split_nomlp"):
        r = mixrt.Renderer(0, stream=stream, variant=v, early_stop_chunk=chunk)
        for _ in range(5):
            r.render(ds, out)
        abl[v.replace("split_", "without_")] = round(time_launches(stream, lambda: r.render(ds, out),
                                                                   steps), 4)
        r.close()
    res["ablation_ms"] = abl
    return res


def algorithmic_work(cfg):
    """Bytes the method must move and MLP flops it must do, per frame.

    Per sample: the 8 corner entries of every level (L * 8 * F * element size).
    Per ray: the G-buffer record read (16 B: t, u, v, pad), the 4 bilinear
    taps of the channels the displacement form reads (4 * channels * element
    size, plus the scale map's 4 taps for Eq. 2 as printed) and the RGBA
    written (16 B).
    MLP: 2 * sum of in*out over layers per sample."""
    eb = 2 if cfg.table_dtype == "f16" else 4
    xb = {"f32": 4, "f16": 2, "u8": 1}[cfg.tex_dtype]
    per_sample_hash = cfg.L * 8 * cfg.F * eb
    # the 4 bilinear taps of the channels the displacement form reads (Eq. 2
    # as printed also reads the scale map's 4 taps)
    tex = 4 * cfg.tex_channels * xb + (4 * xb if cfg.disp == "vec3" else 0)
    per_ray = 16 + tex + 16
    flops_per_sample = 2 * sum(a * b for a, b in zip(cfg.widths[:-1], cfg.widths[1:]))
    return {
        "hash_bytes": cfg.samples * per_sample_hash,
        "ray_bytes": cfg.rays * per_ray,
        "mlp_flops": cfg.samples * flops_per_sample,
        "per_sample_hash_bytes": per_sample_hash,
        "per_ray_bytes": per_ray,
        "flops_per_sample": flops_per_sample,
    }


def cpu_baseline(scene, budget_s: float):
    """The oracle, as it is, on a bounded random sample of the frame's pixels
    (for mesh workloads: its brute-force ray cast of those pixels, then its
    render of them)."""
    import dataclasses
    import oracle
    threads = oracle.max_threads()
    cfg = scene.cfg

    def run(pix, nthreads):
        if scene.mesh is None:
            return oracle.OracleScene(scene).render_pixels(pix, threads=nthreads)
        g0, _, _, _ = oracle.raycast_pixels(scene.cams, cfg.W, cfg.H, scene.mesh, pix,
                                            threads=nthreads)
        flat = scene.g0.reshape(-1, 4).copy()
        flat[pix] = g0.astype(np.float32)
        sc = dataclasses.replace(scene, g0=flat.reshape(scene.g0.shape))
        return oracle.OracleScene(sc).render_pixels(pix, threads=nthreads)

    rng = np.random.default_rng(0)
    # one thread on a small sample first (the single-core rate)
    n1 = 300 if scene.mesh is None else 20
    pix1 = rng.choice(cfg.rays, n1, replace=False)
    t0 = time.perf_counter()
    run(pix1, 1)
    single = n1 / (time.perf_counter() - t0) / 1e6
    n0 = 2000 if scene.mesh is None else 200
    probe = rng.choice(cfg.rays, n0, replace=False)
    t0 = time.perf_counter()
    run(probe, threads)
    dt = time.perf_counter() - t0
    n = int(min(cfg.rays, max(n0, n0 * budget_s / max(dt, 1e-6))))
    pix = rng.choice(cfg.rays, n, replace=False)
    t0 = time.perf_counter()
    run(pix, threads)
    dt = time.perf_counter() - t0
    what = "brute-force ray cast + render" if scene.mesh is not None else "render"
    return {"value": n / dt / 1e6, "unit": "Mpix/s", "cores": threads, "kind": "oracle",
            "sample": f"{n} random pixels of one {cfg.W}x{cfg.H} frame, {what} "
                      f"({dt:.1f} s wall, OpenMP over pixels)",
            "single_thread_value": single, "single_thread_sample": f"{n1} pixels",
            "cpu_model": cpu_model()}


def time_launches(stream, fn, steps):
    """Average ms of fn() over steps launches, HIP events on `stream`."""
    import torch
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record(stream)
    for _ in range(steps):
        fn()
    b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / steps


def launch_stats(stream, fn, launches):
    """Per-launch durations of fn() over `launches` launches, an event on
    `stream` between consecutive launches: (median ms, mean ms)."""
    import torch
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(launches + 1)]
    torch.cuda.synchronize()
    ev[0].record(stream)
    for i in range(launches):
        fn()
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    per = np.array([ev[i].elapsed_time(ev[i + 1]) for i in range(launches)])
    return float(np.median(per)), float(per.mean())


# The paper's profiling points (FPS at 1280x720 on a MacBook M1 Pro in WebGL,
# one query per pixel): Tab. 3 (levels, table size, MLP) and Tab. 6 (with and
# without the displacement map).  Context only: other hardware.
PAPER_FPS = {"tab3_L8_T17_mlp": 27, "tab3_L8_T17": 30, "tab3_L1_T17": 120, "tab3_L8_T5": 35,
             "tab3_L8_T22": 25, "paper720p": 31, "paper720p_novdd": 35}


def time_workload(cfg, steps, warmup):
    import torch
    from paper_2312_11841_amd import mixrt, synth
    scene = synth.make_scene(cfg)
    ds = mixrt.DeviceScene.from_scene(scene, "cuda:0")
    out = torch.empty((cfg.rays, 4), dtype=torch.float32, device="cuda:0")
    stream = torch.cuda.current_stream()
    r = mixrt.Renderer(0, stream=stream)
    for _ in range(warmup):
        r.render(ds, out)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record(stream)
    for _ in range(steps):
        r.render(ds, out)
    b.record(stream)
    torch.cuda.synchronize()
    r.close()
    return a.elapsed_time(b) / steps


def paper_tables(steps, warmup):
    """Tab. 3 and Tab. 6 of the paper re-run on this GPU, plus level and
    table-size sweeps."""
    from paper_2312_11841_amd import synth
    rows = []
    for cfg in (synth.TABLE3 + synth.LEVEL_SWEEP + synth.SIZE_SWEEP +
                [synth.PAPER720P, synth.PAPER720P_NOVDD]):
        if any(r["workload"] == cfg.name for r in rows):
            continue
        ms = time_workload(cfg, steps, warmup)
        row = {"workload": cfg.name, "L": cfg.L, "log2_T": cfg.log2_T, "F": cfg.F,
               "mlp": "-".join(map(str, cfg.widths)) if len(cfg.widths) > 1 else "removed",
               "displacement": cfg.disp, "ms_per_frame": round(ms, 4),
               "fps": round(1e3 / ms, 1), "paper_m1_fps": PAPER_FPS.get(cfg.name)}
        rows.append(row)
        print(json.dumps(row), file=sys.stderr, flush=True)
    print(json.dumps({"paper_tables": rows, "resolution": "1280x720", "queries_per_pixel": 1}),
          flush=True)


def sweep(steps, warmup):
    """The ray x sample sweep: the central 2^16..2^24 rays (whole rows) of a
    coherent 4096x4096 view x K in {1..32}, on view720p's texture, grid and
    MLP.  The view is generated once; each ray count renders its central rows
    as an image of those rows whose camera keeps the full view's focal length
    (tan(fov'/2) = tan(fov/2) rows / 4096), so every pixel's ray is the one it
    has in the full view and the gathers keep the view's coherence."""
    import dataclasses
    import math
    import torch
    from paper_2312_11841_amd import mixrt, synth
    full = synth.sweep_config(1 << 24, 8)
    print("bench: generating the 4096x4096 sweep view (about a minute)", file=sys.stderr,
          flush=True)
    scene = synth.make_scene(full)
    ds = mixrt.DeviceScene.from_scene(scene, "cuda:0")
    stream = torch.cuda.current_stream()
    r = mixrt.Renderer(0, stream=stream)
    rows_out = []
    for log2r in (16, 18, 20, 22, 24):
        rays = 1 << log2r
        rows = rays // full.W
        row0 = (full.H - rows) // 2
        out = torch.empty((rays, 4), dtype=torch.float32, device="cuda:0")
        g0 = ds.g0[:, row0:row0 + rows].contiguous()
        gbuf = mixrt.GBuffer(1, full.W, rows, g0.data_ptr(), 0)
        cams = scene.cams.copy()
        half = math.radians(float(cams[0, 12])) / 2
        cams[:, 12] = math.degrees(2 * math.atan(math.tan(half) * rows / full.H))
        for K in (1, 2, 4, 8, 16, 32):
            d = dataclasses.replace(ds, g0=g0, gbuf=gbuf, rays=rays,
                                    cams=mixrt.make_cameras(cams),
                                    smp=mixrt.make_sampling(K, full.delta, full.t_term))
            n = max(steps, int(2e7 // (rays * K)))   # small launches: more of them
            for _ in range(warmup):
                r.render(d, out)
            ms = time_launches(stream, lambda: r.render(d, out), n)
            samples = rays * K
            c = full.replace(rows=rays // full.W, K=K)
            work = algorithmic_work(c)
            row = {"rays": rays, "K": K, "samples": samples, "launches": n, "ms": round(ms, 4),
                   "ns_per_sample": round(ms * 1e6 / samples, 4),
                   "hash_GBps": round(work["hash_bytes"] / (ms * 1e-3) / 1e9, 1),
                   "mlp_TFLOPs": round(work["mlp_flops"] / (ms * 1e-3) / 1e12, 1)}
            rows_out.append(row)
            print(json.dumps(row), file=sys.stderr, flush=True)
    r.close()
    print(json.dumps({"sweep": rows_out, "view": "central rows of a coherent 4096x4096 view, "
                                                 "each pixel's ray as in the full view",
                      "grid": "L16 T2^19 F2 f16 N 16-4096", "mlp": "48-64-64-4 fp16"}), flush=True)


def environment():
    """What the numbers were measured on.  The compiler version comes from
    the record the build wrote beside the library: no compiler is started
    here (under a counter-collecting profiler a child process would inherit
    its GPU-initialising preload)."""
    import torch
    from paper_2312_11841_amd import build as hip_build
    from paper_2312_11841_amd import microbench as mb
    p = torch.cuda.get_device_properties(0)
    env = {"device": p.name, "hip": torch.version.hip, "torch": torch.__version__}
    env.update(mb.device_info(0))
    env["hipcc"] = hip_build.build_info().get("hipcc")
    return env


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def gather_cost():
    """Cycles per gather instruction per CU as a function of the distinct
    128-byte lines its 64 lanes touch (1 to 64), whether the lanes sharing a
    line are adjacent, the load width (4, 8, 16 bytes) and where the lines
    live (a 16 KiB table stays in the vector L1, a 2 MiB one in the L2).
    One JSON line per point."""
    from paper_2312_11841_amd import microbench as mb
    for kib in (16, 2048):
        for width in (4, 8, 16):
            for lines in (1, 2, 4, 8, 16, 32, 64):
                for adjacent in ((True,) if lines in (1, 64) else (True, False)):
                    cyc = mb.gather_lines(kib * 1024, width, lines, adjacent)
                    print(json.dumps({"table_KiB": kib, "width": width, "lines": lines,
                                      "adjacent": adjacent,
                                      "cycles_per_instruction_per_cu": round(cyc, 2)}),
                          flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1, help="GPUs (one: the only count measured)")
    ap.add_argument("--steps", type=int, default=100, help="timed steps")
    ap.add_argument("--warmup", type=int, default=10, help="untimed warm-up steps")
    from paper_2312_11841_amd import synth as _synth
    ap.add_argument("--workload", default="view720p", choices=sorted(_synth.CONFIGS),
                    metavar="WORKLOAD", help="one of: " + ", ".join(sorted(_synth.CONFIGS)))
    ap.add_argument("--geometry", choices=("raster", "raycast"), default="raster",
                    help="mesh workloads: how each step computes the G-buffer")
    ap.add_argument("--cpu-budget", type=float, default=10.0,
                    help="seconds of oracle work for the CPU baseline (0: skip)")
    ap.add_argument("--sweep", action="store_true",
                    help="time the rays x K sweep (2^16..2^24 rays, K 1..32) instead")
    ap.add_argument("--paper-tables", action="store_true",
                    help="time the paper's Tab. 3 / Tab. 6 profiling points instead")
    ap.add_argument("--no-rooflines", action="store_true",
                    help="skip the microbenchmark rooflines and the standalone MLP leg")
    ap.add_argument("--early-stop-chunk", type=int, default=0, metavar="C",
                    help="render in front-to-back rounds of C samples per ray, dropping rays "
                         "once opaque (0: the library's default, the tile path)")
    ap.add_argument("--gather-cost", action="store_true",
                    help="only measure how the vector L1 charges a gather instruction "
                         "(cycles per instruction by distinct lines, lanes per line, width)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device copy of BYTES bytes per step (the "
                         "reference kernel that scales the FETCH_SIZE / WRITE_SIZE counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build measures one GPU; --gpus {args.gpus} is not supported "
              "(the path would shard by view, with no per-frame collective)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2312_11841_amd import mixrt, synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    if args.copy_calibration:
        n = args.copy_calibration
        src = torch.ones(n, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(args.steps):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes": n, "steps": args.steps}), flush=True)
        return
    if args.gather_cost:
        gather_cost()
        return
    if args.paper_tables:
        paper_tables(args.steps, args.warmup)
        return
    if args.sweep:
        sweep(min(args.steps, 20), min(args.warmup, 3))
        return
    cfg = synth.CONFIGS[args.workload]
    print(f"bench: generating {cfg.name} ({cfg.rays} rays, K={cfg.K})", file=sys.stderr,
          flush=True)
    scene = synth.make_scene(cfg)
    ds = mixrt.DeviceScene.from_scene(scene, "cuda:0")
    out = torch.empty((cfg.rays, 4), dtype=torch.float32, device="cuda:0")
    stream = torch.cuda.current_stream()
    r = mixrt.Renderer(0, stream=stream, early_stop_chunk=args.early_stop_chunk)
    mesh = None
    if scene.mesh is not None:
        # load time, outside the timed region: grid build on the host + upload
        t0 = time.perf_counter()
        mesh = mixrt.DeviceMesh(r, scene.mesh)
        mesh_load_s = time.perf_counter() - t0

    def raycast():
        r.raycast(mesh, ds.cams, cfg.W, cfg.H, g1=False, out=(ds.g0, None))

    def rasterize():
        r.rasterize(mesh, ds.cams, cfg.W, cfg.H, g1=False, out=(ds.g0, None))

    geometry = rasterize if args.geometry == "raster" else raycast
    extra = {}

    def render():
        r.render(ds, out)

    def step():
        if mesh is not None:
            geometry()
        render()

    # The measurements beside the headline (microbenchmark rooflines, the MLP
    # stage alone, the gather replay, the profiling builds) run first: a GPU
    # left idle for some tens of milliseconds drops its clock, and the first
    # ~25 launches after that ran up to 12% slower than the steady rate
    # (measured), so the timed steps come right after this GPU work.
    replay = None
    stages = None
    if mesh is not None:
        geometry()   # the G-buffer the legs below read
    if not args.no_rooflines:
        print("bench: rooflines, replay and stage builds", file=sys.stderr, flush=True)
        extra["rooflines_measured"] = measured_rooflines(cfg)
        extra["mlp_standalone"] = standalone_mlp(cfg, ds, r, cfg.samples)
        replay = gather_replay_floor(cfg, ds, r)
        stages = stage_metrics(cfg, ds, out, max(args.steps, 20), args.early_stop_chunk)

    plan = r.launch_plan(ds)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    # HIP events on the renderer's stream bracket exactly the timed launches.
    t_wall = time.perf_counter()
    ms = time_launches(stream, step, args.steps)
    t_wall = time.perf_counter() - t_wall
    # The roofline's kernel timed on its own (for a render-only step this is
    # the step itself).
    render_ms = ms if mesh is None else time_launches(stream, render, args.steps)
    # ms per frame as the median of at least 100 launches, each timed by the
    # events on either side of it (the K timed steps above give the mean)
    n_med = max(100, args.steps)
    med_ms, med_mean_ms = launch_stats(stream, step, n_med)
    print(f"bench: timed {args.steps} frames ({ms:.4f} ms each), median of {n_med}: "
          f"{med_ms:.4f} ms", file=sys.stderr, flush=True)
    if mesh is not None:
        ray_ms = time_launches(stream, raycast, args.steps)
        ras_ms = time_launches(stream, rasterize, args.steps)
        extra["geometry"] = {
            "route": args.geometry + " (in the timed step)",
            "raster_ms": round(ras_ms, 4),
            "raster_kernels": "clear + raster (wave-balanced triangle x pixel pairs, 64-bit "
                              "atomic min) + resolve",
            "raycast_ms": round(ray_ms, 4),
            "raycast_kernel": "uniform-grid walk with empty-space leaps + fp32 Moller-Trumbore",
            "render_ms": round(render_ms, 4),
            "Mpix_per_s": {"raster": round(cfg.rays / (ras_ms * 1e-3) / 1e6, 1),
                           "raycast": round(cfg.rays / (ray_ms * 1e-3) / 1e6, 1)},
            "mesh_faces": int(len(scene.mesh.faces)), "mesh_bytes": int(scene.mesh.nbytes),
            "grid": mesh.info, "load_s": round(mesh_load_s, 2)}
    if mesh is not None:
        mesh.close()
    r.close()

    work = algorithmic_work(cfg)
    if stages is not None and stages["samples_evaluated_per_frame"] != cfg.samples:
        # misses and rays stopped early evaluate no samples: the work the
        # frame actually has is that of the samples evaluated (counted by
        # the phase-timer build)
        ev = stages["samples_evaluated_per_frame"]
        work["hash_bytes"] = ev * work["per_sample_hash_bytes"]
        work["mlp_flops"] = ev * work["flops_per_sample"]
        work["samples_evaluated"] = ev
    traffic, traffic_src = measured_traffic(cfg.name)
    sec = ms * 1e-3
    rsec = render_ms * 1e-3
    total_bytes = work["hash_bytes"] + work["ray_bytes"]
    achieved = total_bytes / rsec / 1e9
    mpix = cfg.rays / sec / 1e6
    hbm_line = {"achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                "frac": round(achieved / HBM_PEAK_GBPS, 4),
                "note": "algorithmic bytes over the HBM peak; the bytes include gathers "
                        "the L1 and L2 serve, so this is not what binds the kernel"}
    if replay is not None:
        rms = replay["best"]["ms"]
        roofline = {
            "kernel": "render_kernel (fused path" + (", the only kernel of a step)"
                                                     if mesh is None else "; timed alone)"),
            "bound": "vector_l1",
            "achieved": round(achieved, 1),
            "peak": round(total_bytes / (rms * 1e-3) / 1e9, 1),
            "unit": "GB/s",
            "frac": round(rms / render_ms, 4),
            "traffic": traffic,
            "traffic_source": traffic_src,
            "peak_source": "gather replay measured in this run: this frame's own corner "
                           "loads, in the kernel's tile, lane and level-batch order, issued "
                           "alone (mixrt_mb_gather_replay, fastest grid size); the counters "
                           "show the vector L1 as the saturated unit",
            "gather_replay": {"ms": round(rms, 4), "frac": round(rms / render_ms, 4),
                              "early_stop_chunk": replay["early_stop_chunk"],
                              "note": "the render's own order (tile path, or its rounds of "
                                      "early_stop_chunk samples per ray); rounds are replayed as "
                                      "they run when no ray stops, so where rays stop the render "
                                      "gathers fewer samples than the replay",
                              "address_only_ms": round(replay["best"]["address_only_ms"], 4),
                              "blocks": replay["best"]["blocks"],
                              "render_blocks": replay["render_blocks"],
                              "tile_stripe": replay["tile_stripe"],
                              "by_blocks": [{k: (round(v, 4) if isinstance(v, float) else v)
                                             for k, v in row.items()}
                                            for row in replay["by_blocks"]]},
            "hbm": hbm_line,
            "algorithmic_bytes_per_launch": total_bytes,
            "algorithmic_bytes_per_unit": {"sample": work["per_sample_hash_bytes"],
                                           "ray": work["per_ray_bytes"]},
            "samples_per_launch": work.get("samples_evaluated", cfg.samples),
        }
    else:
        roofline = {
            "kernel": "render_kernel",
            "bound": "hbm", **hbm_line, "traffic": traffic, "traffic_source": traffic_src,
            "algorithmic_bytes_per_launch": total_bytes,
            "algorithmic_bytes_per_unit": {"sample": work["per_sample_hash_bytes"],
                                           "ray": work["per_ray_bytes"]},
        }
    stage_fields = {}
    if stages is not None:
        share = stages["phase_share"]
        hash_s = share["hash"] * rsec
        mlp_s = share["mlp"] * rsec
        stage_fields = {
            "stages": {
                "method": "phase-timer build (the render source compiled with "
                          "-DMIXRT_PHASE_TIMER: per-wave shader clocks per phase, a phase's "
                          "time = its share of all wave-clocks x the kernel's time) and "
                          "ablation builds (-DMIXRT_SPLIT_NO_*: one stage removed; full - "
                          "ablated = that stage's marginal cost)",
                **stages,
                "hash_stage_ms": round(hash_s * 1e3, 4),
                "mlp_phase_ms": round(mlp_s * 1e3, 4),
            },
            "hash_encode_GBps": round(work["hash_bytes"] / hash_s / 1e9, 1),
            "hash_encode_GBps_vs_replay": round(
                (work["hash_bytes"] / hash_s) / (work["hash_bytes"] / (replay["best"]["ms"] * 1e-3)),
                4) if replay is not None else None,
            "mlp_mfma_util": round(work["mlp_flops"] / mlp_s / 1e12 / MFMA_F16_PEAK_TFLOPS, 4),
            "mlp_phase_tflops": round(work["mlp_flops"] / mlp_s / 1e12, 1),
            "stage_metric_method": "phase timer (see stages.method)",
        }
    line = {
        "metric": "Mpix/s and ms/frame at 1280x720 (1 GPU); hash-encode GB/s, MLP MFMA util",
        "value": round(mpix, 2),
        "unit": "Mpix/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "ms_per_frame": round(med_ms, 4),
        "ms_per_frame_stat": f"median of {n_med} launches, each bracketed by HIP events",
        "ms_per_frame_mean": round(med_mean_ms, 4),
        "Mpix_per_s_at_median": round(cfg.rays / (med_ms * 1e-3) / 1e6, 2),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32 (fp16 storage, fp16 MFMA with fp32 accumulation)",
        "data": "synthetic",
        "config": {
            "workload": f"{cfg.name}: {cfg.views}x{cfg.W}x{cfg.H} px, K={cfg.K}, "
                        f"hash L={cfg.L} T=2^{cfg.log2_T} F={cfg.F} {cfg.table_dtype} "
                        f"N {cfg.N_min}-{cfg.N_max}, texture {cfg.tex_R}^2x{cfg.tex_V} "
                        f"{cfg.tex_dtype}, MLP {'-'.join(map(str, cfg.widths))} fp16"
                        + (f"; G-buffer computed from a {len(scene.mesh.faces)}-triangle mesh "
                           f"in each step ({args.geometry})" if scene.mesh is not None else ""),
            "rays": cfg.rays,
            "samples": cfg.samples,
            "parallelism": "single GPU",
            "launch": {"blocks": plan["blocks"], "tile_stripe": plan["tile_stripe"],
                       "early_stop_chunk": plan["chunk"], "block_from": plan["block_from"],
                       "hash_batch": plan["hash_batch"], "claims": plan["claims"]},
        },
        "roofline": roofline,
        **stage_fields,
        "hash_lane_loads_per_s": round(cfg.samples * cfg.L * 8 / rsec),
        "wall_s_timed": round(t_wall, 3),
        "kernel_source_digest": kernel_source_digest(),
    }
    line.update(extra)
    rm = extra.get("rooflines_measured")
    if rm:
        g = rm["gather_random_lane_loads_per_s"]
        rate = cfg.samples * cfg.L * 8 / rsec
        line["hash_vs_measured_random_gather"] = {
            k: round(rate / v["value"], 2) for k, v in g.items()}
    line["environment"] = environment()
    if args.cpu_budget > 0:
        line["cpu_baseline"] = cpu_baseline(scene, args.cpu_budget)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
