"""Benchmark: steady-state simulation steps of the headline workload on 1 GPU.

One step = the kinematic bicycle update of every agent followed by rendering
every agent's camera views (class + depth) through the C ABI.  Default
workload: 1024 worlds x 64 agents x 4 cameras at 64x64 (262,144 views per
step), 44.8k static triangles per world on average, far plane 150 m, seeded
synthetic inputs resident in HBM before timing.

Prints one JSON line with agent-steps/s, images/s, the render kernel's HBM
write roofline fraction (HIP events on the launch stream), the write rate a
plain streaming-store kernel reaches on the same device in the same run, and
the CPU oracle timed on a bounded sample of the same workload.

    python bench.py [--steps 100] [--warmup 10] [--config 4] [--no-cpu-baseline]

(--config 6 times the paper's own rig: 2,048 egos x 4 views at 96x54;
--config 7 the same rig over towns with walls, parked cars and traffic lights;
--encoder adds the policy's image encoder on the rendered tensors to every step:
render and encode on one stream, no host round trip;
--instances times pictura_render_instances instead: the owning agent of every
pixel and each agent's footprint and visible pixels, besides class and depth;
--rgb times pictura_render_rgb: the shaded colour image besides class and depth;
--aa with --rgb times pictura_render_rgb_aa: the colour image antialiased.)
"""
import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0   # MI355X HBM3E peak

# HBM bytes per launch of render_views_kernel on the headline workload, from
# rocprofv3 FETCH_SIZE and WRITE_SIZE runs (one counter per run), each scaled
# by what the counter reads for a plain 1 GiB device copy (FETCH_SIZE x1.99994,
# WRITE_SIZE x1.0).  The figures hold only for the kernel sources they were
# measured on (and the workload generator); when the fingerprint differs,
# `traffic` is reported as null.
TRAFFIC = {
    "config": 4,
    "sources_sha256": "5ea88b326a9df7bc350c6b5ef16ea98b3c6baff4c1e50137f15d573cfa7593ec",
    "fetch_bytes": 1.1546e9,
    "write_bytes": 5368709120,
}
TRAFFIC_SOURCES = ["paper_2607_26005_amd/csrc/pictura_render.hip",
                   "paper_2607_26005_amd/csrc/pictura_internal.h",
                   "paper_2607_26005_amd/csrc/pictura_device.h",
                   "paper_2607_26005_amd/csrc/pictura_abi.hip",      # primitive layout in HBM
                   "paper_2607_26005_amd/csrc/pictura_binner.hip",   # cell order of the primitives
                   "paper_2607_26005_amd/build.py",
                   "paper_2607_26005_amd/scenegen.py"]   # the workload (scene, cell size) too


def kernel_fingerprint():
    import hashlib
    h = hashlib.sha256()
    for rel in TRAFFIC_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", type=int, default=4)
    ap.add_argument("--worlds", type=int, default=None, help="use only the first N worlds (testing)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--rgb", action="store_true", help="render the shaded colour image too (pictura_render_rgb)")
    ap.add_argument("--aa", action="store_true", help="with --rgb: antialiased colour (pictura_render_rgb_aa)")
    ap.add_argument("--instances", action="store_true",
                    help="render with instance visibility (pictura_render_instances)")
    ap.add_argument("--encoder", action="store_true",
                    help="also run the image encoder on each step's views (in-loop coupling)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--stats", action="store_true",
                    help="after the timed region, one more launch with the work counters on (debug instantiation); "
                         "prints them per view tile")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="run only a plain device copy of known size (counter calibration)")
    args = ap.parse_args()
    if args.aa and not args.rgb:
        ap.error("--aa needs --rgb")
    return args


def copy_calibration():
    import torch
    n = 1 << 30   # 1 GiB
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    a.fill_(1)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes_per_launch": n, "launches": 3}))


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def cpu_baseline(wl, target_s):
    from oracle import oracle as O
    threads = os.cpu_count() or 1
    env = os.environ.get("OMP_NUM_THREADS")
    if env and env.isdigit():
        threads = min(threads, int(env))
    rng = np.random.default_rng(1234)
    probe = np.sort(rng.choice(wl.num_views, size=min(32 * threads, wl.num_views), replace=False))
    t0 = time.perf_counter()
    O.render(wl.scene, wl.agents, wl.rig, view_ids=probe, want_flags=False, num_threads=threads, lights=wl.lights)
    dt = time.perf_counter() - t0
    n = int(min(wl.num_views, max(len(probe), target_s / max(dt / len(probe), 1e-9))))
    ids = np.sort(rng.choice(wl.num_views, size=n, replace=False))
    t0 = time.perf_counter()
    O.render(wl.scene, wl.agents, wl.rig, view_ids=ids, want_flags=False, num_threads=threads, lights=wl.lights)
    dt = time.perf_counter() - t0
    images_s = n / dt
    C = wl.rig.num_cams
    return {"value": images_s / C, "unit": "agent-steps/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(), "images_per_s": images_s,
            "sample": f"{n} seeded-random views of the same workload (brute force over every triangle of the "
                      f"view's world + every other agent's box), {dt:.1f} s wall on {threads} threads; "
                      f"agent-steps/s = images/s / {C} cameras"}


def main():
    args = parse()
    if args.gpus != 1:
        print(json.dumps({"error": "the benchmark runs on one GPU only: the render path shards by world, "
                                   "but no multi-GPU launch exists; use --gpus 1"}))
        sys.exit(2)
    import torch
    if args.copy_calibration:
        copy_calibration()
        return
    from paper_2607_26005_amd import pictura, scenegen as sg

    t_gen = time.perf_counter()
    wl = sg.make_config(args.config, num_worlds=args.worlds)
    t_gen = time.perf_counter() - t_gen
    K, Wm = args.steps, args.warmup
    A = wl.agents.count
    V = wl.num_views
    H, W = wl.rig.height, wl.rig.width
    print(f"# workload {wl.name}: {wl.scene.num_worlds} worlds, {wl.scene.num_tris} tris, {A} agents, "
          f"{V} views {W}x{H}; generated in {t_gen:.1f} s", file=sys.stderr, flush=True)

    r = pictura.Renderer(0)
    r.upload(wl.scene, wl.cell_size)
    da = pictura.DeviceAgents.from_host(wl.agents)
    if wl.lights is not None:
        r.set_lights(pictura.DeviceLights.from_host(wl.lights))
    steer, accel = sg.controls(A, K + Wm, seed=wl.seed)
    steer_d = torch.as_tensor(steer, device="cuda")
    accel_d = torch.as_tensor(accel, device="cuda")
    out_cls = torch.empty((V, H, W), dtype=torch.uint8, device="cuda")
    out_depth = torch.empty((V, H, W), dtype=torch.float32, device="cuda")
    out_inst = out_counts = out_rgb = None
    if args.rgb:
        out_rgb = torch.empty((V, 3, H, W), dtype=torch.uint8, device="cuda")
    if args.instances:
        out_inst = torch.empty((V, H, W), dtype=torch.int32, device="cuda")
        out_counts = torch.empty((V, wl.agents.agents_per_world, 2), dtype=torch.int32, device="cuda")

    def render():
        if out_rgb is not None:
            fn = pictura.pictura_render_rgb_aa if args.aa else pictura.pictura_render_rgb
            fn(r.ctx, da, wl.rig, out_cls, out_depth, out_rgb)
        elif out_inst is None:
            r.render(da, wl.rig, out_cls, out_depth)
        else:
            pictura.pictura_render_instances(r.ctx, da, wl.rig, out_cls, out_depth, out_inst, out_counts)
    moving = args.config == 4
    enc = None
    if args.encoder:
        from paper_2607_26005_amd.encoder import ViewEncoder
        torch.manual_seed(0)
        enc = ViewEncoder(cams=wl.rig.num_cams).cuda().eval()
    emb = [None]
    torch.cuda.synchronize()

    def encode():
        if enc is not None:
            with torch.no_grad():
                emb[0] = enc(out_cls, out_depth)

    def step(s):
        if moving:
            r.agents_step(da, steer_d[s], accel_d[s], dt=0.1, vmax=20.0)
        render()
        encode()

    for s in range(Wm):
        step(s)
    torch.cuda.synchronize()
    print(f"# warmup done ({Wm} steps)", file=sys.stderr, flush=True)

    stream = torch.cuda.current_stream()
    ev_r0 = [torch.cuda.Event(enable_timing=True) for _ in range(K)]
    ev_r1 = [torch.cuda.Event(enable_timing=True) for _ in range(K)]
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t_start.record(stream)
    for s in range(K):
        if moving:
            r.agents_step(da, steer_d[Wm + s], accel_d[Wm + s], dt=0.1, vmax=20.0)
        ev_r0[s].record(stream)
        render()
        ev_r1[s].record(stream)
        encode()
    t_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    total_ms = t_start.elapsed_time(t_end)
    render_ms = [a.elapsed_time(b) for a, b in zip(ev_r0, ev_r1)]
    ms_step = total_ms / K
    avg_render_ms = float(np.mean(render_ms))
    print(f"# timed {K} steps: {total_ms:.2f} ms (wall {wall * 1e3:.1f} ms); render avg {avg_render_ms:.4f} ms "
          f"min {min(render_ms):.4f} max {max(render_ms):.4f}", file=sys.stderr, flush=True)

    # measured HBM write reference in the same run: the library's store probe
    # (16-byte non-temporal stores of zeros, the write-out's store pattern)
    # over the depth output buffer, timed with events on the same stream
    probe = out_depth.view(torch.uint8).reshape(-1)
    probe = probe[: probe.numel() // 16 * 16]
    for _ in range(2):
        pictura.pictura_store_probe(r.ctx, probe)
    ev_p0, ev_p1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    n_probe = 10
    ev_p0.record(stream)
    for _ in range(n_probe):
        pictura.pictura_store_probe(r.ctx, probe)
    ev_p1.record(stream)
    torch.cuda.synchronize()
    store_gbs = probe.numel() * n_probe / (ev_p0.elapsed_time(ev_p1) * 1e-3) / 1e9
    if args.stats:
        r.set_option(pictura.OPT_STATS, 1)
        render()
        torch.cuda.synchronize()
        st = pictura.pictura_stats_copy(r.ctx, reset=True)
        r.set_option(pictura.OPT_STATS, 0)
        nt = max(st["view_tiles"], 1)
        print("# work per view tile (one more launch, debug instantiation): " +
              ", ".join(f"{k}={v / nt:.1f}" for k, v in st.items() if v), file=sys.stderr, flush=True)
    dev_err = r.device_errors()
    print(f"# store probe: {probe.numel() / 1e9:.2f} GB per launch, {store_gbs:.0f} GB/s; device errors {dev_err:#x}",
          file=sys.stderr, flush=True)

    out_bytes = V * H * W * 5
    if out_rgb is not None:    # + 3 colour bytes per pixel
        out_bytes += V * H * W * 3
    if out_inst is not None:   # + int32 owner per pixel and 2 x uint32 counts per (view, agent)
        out_bytes += V * H * W * 4 + V * wl.agents.agents_per_world * 8
    achieved = out_bytes / (avg_render_ms * 1e-3) / 1e9
    agent_steps_s = A * K / (total_ms * 1e-3)
    images_s = V * K / (total_ms * 1e-3)
    r.close()

    traffic = None
    if (args.config == TRAFFIC["config"] and args.worlds is None and not args.rgb and not args.instances
            and not args.encoder and kernel_fingerprint() == TRAFFIC["sources_sha256"]):
        traffic = TRAFFIC["fetch_bytes"] + TRAFFIC["write_bytes"]

    cpu = None
    if not args.no_cpu_baseline:
        print("# cpu baseline (oracle) ...", file=sys.stderr, flush=True)
        cpu = cpu_baseline(wl, args.cpu_seconds)

    line = {
        "metric": "agent-steps/s",
        "value": agent_steps_s,
        "unit": "agent-steps/s",
        "images_per_s": images_s,
        "n_gpus": 1,
        "steps": K,
        "warmup": Wm,
        "ms_per_step": ms_step,
        "render_ms": avg_render_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic (seeded generator; CARLA/WOMD stand-in)",
        "config": {
            "workload": f"{wl.name}: {wl.scene.num_worlds} worlds x {wl.agents.agents_per_world} agents x "
                        f"{wl.rig.num_cams} cameras, {W}x{H} uint8 class + fp32 depth, "
                        f"{wl.scene.num_tris // wl.scene.num_worlds} static tris/world, far {wl.rig.far:g} m"
                        + (f", {wl.lights.lights_per_world} traffic lights/world" if wl.lights is not None else ""),
            "views_per_step": V,
            "step": "bicycle update + render" if moving else "render",
        },
        "roofline": {
            "bound": "hbm",
            "kernel": "render_views_kernel",
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "algorithmic_bytes_per_launch": out_bytes,
            "traffic": traffic,
            "traffic_source": ("rocprofv3 FETCH_SIZE + WRITE_SIZE per launch, copy-calibrated, profiled on these kernel "
                               "sources (profiles/render_views_kernel_throughput_headline_64x64.md)"
                               if traffic is not None else None),
            "measured_store_gbs": store_gbs,
            "frac_of_measured_store": achieved / store_gbs,
        },
        "device_errors": dev_err,
        "cpu_baseline": cpu,
    }
    if out_rgb is not None:
        line["config"]["step"] += " with the shaded colour image (planar RGB)"
        if args.aa:
            line["config"]["step"] += ", antialiased (analytic coverage, one sample per pixel)"
        line["roofline"]["traffic"] = line["roofline"]["traffic_source"] = None
    if out_inst is not None:
        line["config"]["step"] += " with instance visibility (owner per pixel, footprint and visible pixels per agent)"
        line["roofline"]["traffic"] = line["roofline"]["traffic_source"] = None
    if enc is not None:
        line["config"]["step"] += " + image encoder (5 conv layers, 16 queries x 1 cross-attention per camera, fp32)"
        line["encoder_ms"] = ms_step - avg_render_ms
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
