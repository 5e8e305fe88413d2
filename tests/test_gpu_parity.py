"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Every test renders on the GPU and compares with the oracle on the same seeded
inputs: whole images for the small workloads, seeded samples of views for
the large ones (the GPU renders every view of the batch in the same launch
configuration the benchmark times; the oracle computes the sampled views one
by one).
"""
import dataclasses
import functools

import numpy as np
import pytest

from oracle import oracle as O
from paper_2607_26005_amd import scenegen as sg
from tests.parity import assert_parity, compare
from tests.scenes import make_agents, make_rig, make_scene, quad, walled

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    return torch


@functools.lru_cache(maxsize=None)
def workload(cfg, worlds=None):
    return sg.make_config(cfg, num_worlds=worlds)


@pytest.fixture(scope="module")
def lib():
    _torch()
    from paper_2607_26005_amd import pictura
    return pictura


def render_gpu(pictura, wl_scene, agents, rig, cell, cull=1, tile=0):
    torch = _torch()
    r = pictura.Renderer(0)
    try:
        r.set_option(pictura.OPT_CULL, cull)
        r.set_option(pictura.OPT_TILE, tile)
        r.upload(wl_scene, cell)
        da = pictura.DeviceAgents.from_host(agents)
        c, d = r.render(da, rig)
        torch.cuda.synchronize()
        return c, d
    finally:
        r.close_checked()


def check_views(pictura, wl, view_ids, label, cull=1, tile=0, cell=None):
    cell = wl.cell_size if cell is None else cell
    print(f"[{label}] render {wl.num_views} views {wl.rig.width}x{wl.rig.height} cull={cull} tile={tile}", flush=True)
    c, d = render_gpu(pictura, wl.scene, wl.agents, wl.rig, cell, cull, tile)
    idx = np.asarray(view_ids, np.int64)
    import torch
    ti = torch.as_tensor(idx, device=c.device)
    gc = c.index_select(0, ti).cpu().numpy()
    gd = d.index_select(0, ti).cpu().numpy()
    del c, d
    ora = O.render(wl.scene, wl.agents, wl.rig, view_ids=idx)
    s = assert_parity(gc, gd, ora, label)
    print(f"[{label}] {s}", flush=True)
    return s


def sample_views(n_views, k, seed):
    rng = np.random.default_rng(seed)
    if k >= n_views:
        return np.arange(n_views)
    return np.sort(rng.choice(n_views, size=k, replace=False))


def test_tiny_all_views(lib):
    wl = workload(1)
    s = check_views(lib, wl, np.arange(wl.num_views), "tiny")
    assert s["mismatches"] == 0


def test_small_batch_sampled(lib):
    wl = workload(2)
    check_views(lib, wl, sample_views(wl.num_views, 384, 21), "small_batch")


def test_dense_traffic_sampled(lib):
    wl = workload(3)
    check_views(lib, wl, sample_views(wl.num_views, 384, 22), "dense_traffic")


def test_headline_full_size_sampled(lib):
    # the benchmark's workload and launch: 1024 worlds x 64 agents x 4 cameras
    wl = workload(4)
    check_views(lib, wl, sample_views(wl.num_views, 256, 23), "headline")


def test_headline_after_bench_steps_sampled(lib):
    # the state the benchmark's last timed render sees: the headline agents moved
    # by 110 bicycle updates on the GPU (10 warm-up + 100 timed steps, the same
    # controls), read back, then rendered by both sides from that state
    torch = _torch()
    wl = workload(4)
    steps = 110
    steer, accel = sg.controls(wl.agents.count, steps, seed=wl.seed)
    da = lib.DeviceAgents.from_host(wl.agents)
    r = lib.Renderer(0)
    try:
        for s in range(steps):
            r.agents_step(da, torch.as_tensor(steer[s], device="cuda"), torch.as_tensor(accel[s], device="cuda"),
                          dt=0.1, vmax=20.0)
        torch.cuda.synchronize()
    finally:
        r.close_checked()
    ag = wl.agents.copy()
    for f in ("x", "y", "cos_h", "sin_h", "psi", "speed"):
        setattr(ag, f, getattr(da, f).cpu().numpy().astype(np.float32))
    moved = float(np.median(np.hypot(ag.x - wl.agents.x, ag.y - wl.agents.y)))
    print(f"[headline-stepped] median displacement {moved:.1f} m over {steps} steps", flush=True)
    assert moved > 10.0
    check_views(lib, dataclasses.replace(wl, agents=ag), sample_views(wl.num_views, 256, 29), "headline-stepped")


def test_highres_full_launch_sampled(lib):
    # the whole high-res workload in one launch, as the benchmark times it:
    # 128 worlds x 64 agents x 4 cameras at 128x128 (2x2 tiles per view),
    # ~527k triangles per world; 96 views sampled across all worlds
    wl = sg.make_config(5)
    views = sample_views(wl.num_views, 96, 24)
    assert len(np.unique(views // (64 * 4))) > 48
    check_views(lib, wl, views, "highres")


def test_paper_rig_sampled(lib):
    # the paper's rig (96x54, f = 77.25 px, yaws 0 / +-55 / 180): two tiles per view
    wl = workload(6, 8)
    check_views(lib, wl, sample_views(wl.num_views, 160, 26), "paper-rig")


# ---- invariances: culling, tiling, cell size, permutation, duplication -------

def _small():
    return workload(2, 2)


def test_cull_off_and_forced_tiles_identical(lib):
    wl = _small()
    base = render_gpu(lib, wl.scene, wl.agents, wl.rig, wl.cell_size)
    for cull, tile, cell in ((0, 0, wl.cell_size), (1, 16, wl.cell_size), (1, 24, wl.cell_size),
                             (1, 0, 8.0), (1, 0, 64.0), (0, 32, 32.0)):
        print(f"[invariance] cull={cull} tile={tile} cell={cell}", flush=True)
        c, d = render_gpu(lib, wl.scene, wl.agents, wl.rig, cell, cull, tile)
        assert bool((c == base[0]).all()), (cull, tile, cell)
        assert bool((d == base[1]).all()), (cull, tile, cell)


def test_permutation_duplication_identical(lib):
    wl = _small()
    base = render_gpu(lib, wl.scene, wl.agents, wl.rig, wl.cell_size)
    sc = wl.scene
    rng = np.random.default_rng(3)
    verts, cls, offs = [], [], [0]
    for w in range(sc.num_worlds):
        v, c = sc.world(w)
        p = rng.permutation(len(v))
        dup = rng.choice(len(v), size=len(v) // 10, replace=False)
        verts.append(np.concatenate([v[p], v[dup]]))
        cls.append(np.concatenate([c[p], c[dup]]))
        offs.append(offs[-1] + len(verts[-1]))
    sc2 = sg.Scene(sc.num_worlds, np.ascontiguousarray(np.concatenate(verts)), np.concatenate(cls),
                   np.asarray(offs, np.int64), sc.bounds)
    c, d = render_gpu(lib, sc2, wl.agents, wl.rig, wl.cell_size)
    assert bool((c == base[0]).all())
    assert bool((d == base[1]).all())


# ---- edge cases ----------------------------------------------------------------

def test_ragged_sizes_and_tiles(lib):
    # non-square, not a multiple of 16 (scalar write path), ragged 64x64 tiles
    wl = workload(2, 1)
    for (W, H) in ((40, 24), (100, 70), (17, 129)):
        rig = sg.Rig(width=W, height=H, fx=W / 2.0, fy=W / 2.0, cx=W / 2.0, cy=H / 2.0, near=0.5, far=100.0,
                     mount=wl.rig.mount)
        wl2 = sg.Workload(wl.name, 2, 1, wl.scene, wl.agents, rig, wl.cell_size, wl.world_size)
        check_views(lib, wl2, sample_views(wl2.num_views, 64, W), f"ragged {W}x{H}")


def test_largest_view_full_image(lib):
    # the largest view the ABI accepts, 4096 x 4096 (4,096 tiles of 64 x 64),
    # on the tiny workload's scene: two whole images against the oracle
    wl = workload(1)
    rig = sg.Rig(width=4096, height=4096, fx=2048.0, fy=2048.0, cx=2048.0, cy=2048.0, near=0.5, far=100.0,
                 mount=wl.rig.mount)
    wl2 = sg.Workload(wl.name, 1, 0, wl.scene, wl.agents, rig, wl.cell_size, wl.world_size)
    check_views(lib, wl2, [0, 5], "largest 4096x4096")


def test_eight_cameras(lib):
    # the most cameras a rig may have: eight at 45 degree steps (cos and sin of
    # the odd steps rounded to fp32), with mount offsets and heights
    wl = workload(2, 1)
    c45 = float(np.float32(np.sqrt(0.5)))
    dirs = ((1.0, 0.0), (c45, c45), (0.0, 1.0), (-c45, c45), (-1.0, 0.0), (-c45, -c45), (0.0, -1.0), (c45, -c45))
    mounts = tuple((0.4 * cy, -0.3 * sy, 1.2 + 0.1 * k, cy, sy) for k, (cy, sy) in enumerate(dirs))
    rig = make_rig(res=64, far=100.0, mounts=mounts)
    wl2 = sg.Workload(wl.name, 2, 1, wl.scene, wl.agents, rig, wl.cell_size, wl.world_size)
    assert wl2.num_views == 8 * 32
    check_views(lib, wl2, sample_views(wl2.num_views, 64, 88), "eight cameras")


def test_tiles_above_the_horizon(lib):
    # tiles whose pixel centres all lie above the horizon: the tiny workload's
    # flat world (sky there) and the same world with walls reaching above the
    # cameras, 128 x 128 views in four tiles and in forced 16-pixel tiles
    wl = workload(1)
    rig = sg.Rig(width=128, height=128, fx=64.0, fy=64.0, cx=64.0, cy=64.0, near=0.5, far=100.0,
                 mount=wl.rig.mount)
    for name, scene in (("flat", wl.scene), ("walled", walled(wl.scene))):
        wl2 = sg.Workload(wl.name, 1, 0, scene, wl.agents, rig, wl.cell_size, wl.world_size)
        check_views(lib, wl2, np.arange(wl2.num_views), f"horizon {name}")
        check_views(lib, wl2, np.arange(wl2.num_views), f"horizon {name} tile16", tile=16)


def test_off_grid_principal_point_anisotropic(lib):
    # a principal point off the 1/256-pixel grid (31.3, 23.7) and fx != fy:
    # pixel-centre offsets are no longer exact sums, so the kernel takes its
    # general block raster and centre arithmetic
    wl = workload(2, 1)
    rig = sg.Rig(width=64, height=48, fx=40.0, fy=29.0, cx=31.3, cy=23.7, near=0.5, far=100.0, mount=wl.rig.mount)
    wl2 = sg.Workload(wl.name, 2, 1, wl.scene, wl.agents, rig, wl.cell_size, wl.world_size)
    views = sample_views(wl2.num_views, 64, 313)
    check_views(lib, wl2, views, "off-grid cx/cy")
    check_views(lib, wl2, views[:24], "off-grid cx/cy tile24", tile=24)


def test_extreme_near_and_far(lib):
    # far = 8 km puts 1/far below 2^-12, so the write-out decodes depths with
    # IEEE division instead of the fast reciprocal; near = 0.01 m raises the
    # key's cap to 128 and clips almost nothing; both against the oracle
    wl = workload(2, 1)
    for near, far in ((0.5, 8000.0), (0.01, 100.0)):
        rig = sg.Rig(width=64, height=64, fx=32.0, fy=32.0, cx=32.0, cy=32.0, near=near, far=far,
                     mount=wl.rig.mount)
        wl2 = sg.Workload(wl.name, 2, 1, wl.scene, wl.agents, rig, wl.cell_size, wl.world_size)
        check_views(lib, wl2, sample_views(wl2.num_views, 48, int(far)), f"near {near} far {far}")


def test_random_quad_pairs(lib):
    # quads given as pairs (a, b, c), (a, c, d): convex, darts, slivers, near-plane
    # crossings and quads reaching far to the side, seen by four cameras
    from tests.test_gpu_aa import _random_quads
    for seed in (81, 82):
        tris, cls = _random_quads(seed)
        sc = make_scene(np.asarray(tris, np.float32), cls)
        rng = np.random.default_rng(seed + 100)
        rows = [(0.0, 0.0, 0.0, 1.0, 0.0, 4.5, 1.9, 1.5, 3)]
        for _ in range(5):
            ang = rng.uniform(0, 2 * np.pi)
            rows.append((rng.uniform(-20, 20), rng.uniform(-20, 20), 0.0, float(np.cos(ang)), float(np.sin(ang)),
                         4.5, 1.9, 1.5, 3))
        rig = make_rig(res=64, far=80.0, mounts=((0.0, 0.0, 1.0, 1.0, 0.0), (0.0, 0.0, 1.0, 0.0, 1.0),
                                                  (0.0, 0.0, 1.0, -1.0, 0.0), (0.0, 0.0, 1.0, 0.0, -1.0)))
        wl = sg.Workload("random-quads", 0, seed, sc, make_agents(rows), rig, 16.0, 2000.0)
        check_views(lib, wl, np.arange(wl.num_views), f"random-quads {seed}")


def test_empty_world_and_lone_agent(lib):
    # world 0 has no triangles, world 1 one quad; one agent per world (no boxes)
    q = np.asarray(quad((8.0, -2.0, -2.0), (8.0, 2.0, -2.0), (8.0, 2.0, 2.0), (8.0, -2.0, 2.0)), np.float32)
    scene = sg.Scene(2, np.ascontiguousarray(q.reshape(-1, 9)), np.array([7, 7], np.uint8),
                     np.array([0, 0, 2], np.int64), np.array([[-50, -50, 50, 50]] * 2, np.float32))
    ag = make_agents([(0.0, 0.0, 0.0, 1.0, 0.0, 4.0, 2.0, 1.5, 3), (0.0, 0.0, 0.0, 1.0, 0.0, 4.0, 2.0, 1.5, 3)],
                     num_worlds=2)
    rig = make_rig(mounts=((0.0, 0.0, 0.0, 1.0, 0.0), (0.0, 0.0, 0.0, 0.0, 1.0)))
    wl = sg.Workload("edge", 0, 0, scene, ag, rig, 16.0, 100.0)
    check_views(lib, wl, np.arange(wl.num_views), "empty+lone")


@pytest.mark.parametrize("s,lo,hi", [(1.875, 24, 39), (2.0, 24, 40), (1.87451171875, 24, 39), (1.87548828125, 24, 39)])
def test_fill_rule_and_snap_ties_closed_form(lib, s, lo, hi):
    # A square of half-size s facing the camera 8 m ahead (fx = 32): its edges
    # project to 32 -+ 4 s px.  For s = 1.875 they run through pixel centres
    # (top-left rule: left/top included, right/bottom excluded); the last two
    # sizes put them half a subpixel off the centres, and the snap's ties to
    # even move them onto the centres.  Closed-form pixel set and depth 8 m,
    # and the oracle's images bit for bit.
    pts = [(8.0, a, b) for (a, b) in ((-s, -s), (s, -s), (s, s), (-s, s))]
    scene = make_scene(quad(*pts), [7, 7])
    wl = sg.Workload("pin", 0, 0, scene, make_agents([(0.0, 0.0, 0.0, 1.0, 0.0, 1.0, 1.0, 1.0, 3)]), make_rig(),
                     16.0, 2000.0)
    c, d = render_gpu(lib, wl.scene, wl.agents, wl.rig, 16.0)
    gc, gd = c.cpu().numpy()[0], d.cpu().numpy()[0]
    want = np.zeros((64, 64), bool)
    want[lo:hi, lo:hi] = True
    assert np.array_equal(gc == 7, want)
    assert np.all(np.isinf(gd[~want])) and np.allclose(gd[want], 8.0, rtol=2 ** -20, atol=0)
    check_views(lib, wl, np.arange(1), f"pin s={s}")


def test_far_rule_square_beyond_and_on_far(lib):
    # far = 110: a fronto square (half-size 16) one fp32 step beyond the far
    # plane, where the plane value at its covered centres equals fl(1/110) and
    # passes the per-pixel far test; the triangle-level rule of R4 keeps the
    # image empty.  The same square on the far plane covers the 10 x 10 centres
    # within 32 +- 4.65 px at depth 110.
    D = float(np.nextafter(np.float32(110.0), np.float32(np.inf)))
    rig = make_rig(far=110.0)
    ag = make_agents([(0.0, 0.0, 0.0, 1.0, 0.0, 1.0, 1.0, 1.0, 3)])
    for dist, want_px in ((D, 0), (110.0, 100)):
        pts = [(dist, a, b) for (a, b) in ((-16.0, -16.0), (16.0, -16.0), (16.0, 16.0), (-16.0, 16.0))]
        wl = sg.Workload("far-rule", 0, 0, make_scene(quad(*pts), [7, 7]), ag, rig, 16.0, 2000.0)
        c, d = render_gpu(lib, wl.scene, wl.agents, wl.rig, 16.0)
        gc = c.cpu().numpy()[0]
        want = np.zeros((64, 64), bool)
        if want_px:
            want[27:37, 27:37] = True
        assert np.array_equal(gc == 7, want), (dist, int((gc == 7).sum()))
        check_views(lib, wl, np.arange(1), f"far-rule D={dist!r}")


def test_degenerate_and_non_finite_triangles(lib):
    # Triangles the rules drop or that sit on their boundaries, among ordinary
    # ones: a NaN and an infinite vertex (dropped by the snap's range rule or
    # the depth plane's finiteness rule), zero-area and coincident-vertex
    # triangles (area 0), one lying in the near plane (depth = near, the cap's
    # code), one whose plane holds the camera (delta = 0), one reaching behind
    # the camera, and one with a vertex 100 km away (wide edge values).
    nan, inf = float("nan"), float("inf")
    tris = quad((8.0, -3.0, -2.0), (8.0, 3.0, -2.0), (8.0, 3.0, 2.0), (8.0, -3.0, 2.0))
    tris += [[(6.0, -1.0, 0.5), (6.0, 1.0, nan), (6.0, 0.0, 1.5)],
             [(6.0, -1.0, -0.5), (inf, 1.0, -0.5), (6.0, 0.0, -1.5)],
             [(5.0, -1.0, 0.0), (5.0, 0.0, 0.5), (5.0, 1.0, 1.0)],
             [(5.0, 2.0, 1.0), (5.0, 2.0, 1.0), (5.0, 2.5, 1.5)],
             [(0.5, -0.2, -0.2), (0.5, 0.2, -0.2), (0.5, 0.0, 0.2)],
             [(2.0, -1.0, 0.0), (4.0, 1.0, 0.0), (6.0, 0.0, 0.0)],
             [(-3.0, -1.0, -0.7), (7.0, -1.5, -0.7), (7.0, 1.5, -0.7)],
             [(7.5, -2.0, 1.0), (7.5, -1.0, 1.0), (100000.0, 50000.0, -1.0)]]
    scene = make_scene(tris, [7, 7, 1, 1, 2, 2, 3, 5, 6, 0])
    ag = make_agents([(0.0, 0.0, 0.0, 1.0, 0.0, 1.0, 1.0, 1.0, 3)])
    rig = make_rig(mounts=((0.0, 0.0, 0.0, 1.0, 0.0), (0.0, 0.0, 0.0, 0.0, 1.0)), far=100.0)
    wl = sg.Workload("degenerate", 0, 0, scene, ag, rig, 16.0, 2000.0)
    s = check_views(lib, wl, np.arange(wl.num_views), "degenerate")
    assert s["mismatches"] == 0


def test_camera_inside_box_and_near_clipped_ground(lib):
    G = 1000.0
    tris = quad((-G, -G, 0.0), (G, -G, 0.0), (G, G, 0.0), (-G, G, 0.0))
    scene = make_scene(tris, [0, 0])
    rows = [(0.0, 0.0, 0.0, 1.0, 0.0, 4.5, 1.9, 1.5, 3),
            (1.0, 0.2, 0.0, 0.6, 0.8, 4.5, 1.9, 1.7, 6),   # camera of agent 0 is inside this box
            (12.0, 3.0, 0.0, 0.0, 1.0, 4.5, 1.9, 1.5, 3)]
    ag = make_agents(rows)
    rig = make_rig(mounts=((0.0, 0.0, 1.5, 1.0, 0.0), (0.5, 0.1, 1.2, 0.0, -1.0)), far=100.0)
    wl = sg.Workload("inside", 0, 0, scene, ag, rig, 16.0, 2000.0)
    check_views(lib, wl, np.arange(wl.num_views), "inside-box")


def test_edge_paths_all_exercised(lib):
    """A 2 km ground quad seen from 1.5 m, a mid-size box and small far
    boxes: near-clipped ground triangles reach 2^22 subpixels per edge (fp64
    edge path), the box faces take the int32 record path and the far boxes the
    single-lane raster.  The kernel's own counters show every path ran."""
    torch = _torch()
    G = 1000.0
    tris = quad((-G, -G, 0.0), (G, -G, 0.0), (G, G, 0.0), (-G, G, 0.0))
    scene = make_scene(tris, [0, 0])
    rows = [(0.0, 0.0, 0.0, 1.0, 0.0, 4.5, 1.9, 1.5, 3),
            (9.0, 1.0, 0.0, 1.0, 0.0, 4.5, 1.9, 1.5, 3)] + \
           [(60.0 + 7.0 * k, -20.0 + 9.0 * k, 0.0, 0.6, 0.8, 1.0, 0.8, 1.2, 6) for k in range(6)]
    ag = make_agents(rows)
    rig = make_rig(mounts=((0.0, 0.0, 1.5, 1.0, 0.0),), far=100.0)
    wl = sg.Workload("paths", 0, 0, scene, ag, rig, 16.0, 2000.0)
    r = lib.Renderer(0)
    try:
        r.set_option(lib.OPT_STATS, 1)
        r.upload(wl.scene, 16.0)
        da = lib.DeviceAgents.from_host(wl.agents)
        c, d = r.render(da, wl.rig)
        torch.cuda.synchronize()
        st = lib.pictura_stats_copy(r.ctx)
    finally:
        r.close_checked()
    print(f"[paths] {st}", flush=True)
    assert st["record_tris_fp64"] > 0
    assert st["record_tris"] - st["record_tris_fp64"] > 0
    assert st["lane_tris"] > 0
    ora = O.render(wl.scene, wl.agents, wl.rig)
    s = assert_parity(c.cpu().numpy(), d.cpu().numpy(), ora, "paths")
    print(f"[paths] {s}", flush=True)


def test_random_small_scenes(lib):
    from tests.test_oracle_pins import _random_scene
    for seed in range(12):
        scene, ag = _random_scene(seed)
        rig = make_rig(res=32, near=0.5, far=30.0, mounts=((0.0, 0.0, 1.0, 1.0, 0.0), (0.0, 0.0, 1.0, -1.0, 0.0)))
        wl = sg.Workload("random", 0, seed, scene, ag, rig, 4.0, 2000.0)
        check_views(lib, wl, np.arange(wl.num_views), f"random seed {seed}")


# ---- binner and agent step -----------------------------------------------------

def test_binner_matches_oracle(lib):
    wl = workload(2, 3)
    sc = wl.scene
    print("[binner] 3 worlds", flush=True)
    r = lib.Renderer(0)
    try:
        r.upload(sc, 16.0)
        b = r.bins()
    finally:
        r.close_checked()
    ob = O.bin_scene(sc, 16.0)
    assert np.array_equal(b["dims"], ob["dims"])
    assert np.array_equal(b["cell_base"], ob["cell_base"])
    counts = np.diff(b["cell_start"].astype(np.int64))
    assert np.array_equal(counts, ob["count"].astype(np.int64))
    ne = counts > 0
    assert np.array_equal(b["aabb"][ne], ob["aabb"][ne])
    # the same primitives (triangle pairs), each in the oracle's cell
    perm = b["perm"].astype(np.int64)
    assert np.array_equal(np.sort(perm), np.sort(ob["prims"].astype(np.int64)))
    home_of = dict(zip(ob["prims"].astype(np.int64).tolist(), ob["home"].tolist()))
    cell_of_slot = np.repeat(np.arange(len(counts)), counts)
    assert np.array_equal(np.asarray([home_of[p] for p in perm.tolist()]), cell_of_slot)


def test_agents_step_matches_oracle(lib):
    torch = _torch()
    wl = workload(4, 8)
    ag = wl.agents.copy()
    steer, accel = sg.controls(ag.count, 5, seed=3)
    da = lib.DeviceAgents.from_host(ag)
    r = lib.Renderer(0)
    try:
        for s in range(5):
            print(f"[agents_step] step {s}", flush=True)
            st = torch.as_tensor(steer[s], device="cuda")
            ac = torch.as_tensor(accel[s], device="cuda")
            r.agents_step(da, st, ac, dt=0.1, vmax=20.0)
            out = O.agents_step(ag, steer[s], accel[s], dt=0.1, vmax=20.0)
            torch.cuda.synchronize()
            gx, gy = da.x.cpu().numpy(), da.y.cpu().numpy()
            assert np.max(np.abs(gx - out["x"])) < 2e-4 * (s + 1)
            assert np.max(np.abs(gy - out["y"])) < 2e-4 * (s + 1)
            assert np.max(np.abs(da.speed.cpu().numpy() - out["speed"])) < 1e-5
            dpsi = np.angle(np.exp(1j * (da.psi.cpu().numpy() - out["psi"])))
            assert np.max(np.abs(dpsi)) < 1e-5 * (s + 1)
            assert np.max(np.abs(da.cos_h.cpu().numpy() - out["cos_h"])) < 1e-5 * (s + 1)
            assert np.max(np.abs(da.sin_h.cpu().numpy() - out["sin_h"])) < 1e-5 * (s + 1)
            # continue both sides from their own state
            ag.x, ag.y = out["x"].astype(np.float32), out["y"].astype(np.float32)
            ag.psi, ag.speed = out["psi"].astype(np.float32), out["speed"].astype(np.float32)
    finally:
        r.close_checked()


# ---- C ABI error handling (host-side checks, no kernel launched) ---------------

def test_abi_errors(lib):
    _torch()
    ctx = lib.pictura_create(0)
    try:
        wl = workload(1)
        da = lib.DeviceAgents.from_host(wl.agents)
        import torch
        oc = torch.empty(8 * 64 * 64, dtype=torch.uint8, device="cuda")
        od = torch.empty(8 * 64 * 64, dtype=torch.float32, device="cuda")
        with pytest.raises(lib.PicturaError) as e:
            lib.pictura_render_views(ctx, da, wl.rig, oc, od)
        assert e.value.status == lib.ESTATE
        with pytest.raises(lib.PicturaError) as e:
            lib.pictura_bin_scene(ctx, 16.0)
        assert e.value.status == lib.ESTATE
        lib.pictura_scene_upload(ctx, wl.scene)
        with pytest.raises(lib.PicturaError) as e:
            lib.pictura_bin_scene(ctx, -1.0)
        assert e.value.status == lib.EINVAL
        lib.pictura_bin_scene(ctx, 16.0)
        bad = sg.Rig(64, 64, 32.0, 32.0, 32.0, 32.0, 1.0, 0.5, wl.rig.mount)
        with pytest.raises(lib.PicturaError) as e:
            lib.pictura_render_views(ctx, da, bad, oc, od)
        assert e.value.status == lib.EINVAL
        huge = sg.Rig(64, 64, 32.0, 32.0, 32.0, 32.0, 1e-30, 1e30, wl.rig.mount)
        with pytest.raises(lib.PicturaError) as e:
            lib.pictura_render_views(ctx, da, huge, oc, od)
        assert e.value.status == lib.EINVAL
        with pytest.raises(lib.PicturaError) as e:
            lib.pictura_set_option(ctx, lib.OPT_TILE, 3)
        assert e.value.status == lib.EINVAL
        # the context is still usable after errors
        lib.pictura_render_views(ctx, da, wl.rig, oc, od)
        torch.cuda.synchronize()
        ora = O.render(wl.scene, wl.agents, wl.rig)
        assert_parity(oc.view(8, 64, 64).cpu().numpy(), od.view(8, 64, 64).cpu().numpy(), ora, "after-errors")
    finally:
        lib.pictura_destroy(ctx)


def test_fast_reciprocal_is_correctly_rounded(lib):
    # The kernels replace IEEE division by rcp + one fused Newton step where
    # |argument| lies in [2^-12, 2^20); check every fp32 value there, of
    # both signs (the sign bit is 0x80000000).
    ctx = lib.pictura_create(0)
    try:
        lo = int(np.float32(2.0 ** -12).view(np.uint32))
        hi = int(np.float32(2.0 ** 20).view(np.uint32))
        bad = 0
        for sign in (0, 0x80000000):
            for start in range(lo, hi, 1 << 26):
                bad += lib.pictura_selftest_rcp(ctx, sign | start, min(1 << 26, hi - start))
        assert bad == 0
    finally:
        lib.pictura_destroy(ctx)


def test_store_probe_writes_exactly_its_range(lib):
    # the bench's HBM write reference: zeros over exactly the requested bytes,
    # nothing past them; misaligned sizes and buffers are refused
    torch = _torch()
    buf = torch.full((1 << 20,), 0xAB, dtype=torch.uint8, device="cuda")
    r = lib.Renderer(0)
    try:
        lib.pictura_store_probe(r.ctx, buf[: (1 << 20) - 4096])
        torch.cuda.synchronize()
        assert int(buf[: (1 << 20) - 4096].sum()) == 0
        assert bool((buf[(1 << 20) - 4096:] == 0xAB).all())
        with pytest.raises(lib.PicturaError):
            lib.pictura_store_probe(r.ctx, buf[:100])
        with pytest.raises(lib.PicturaError):
            lib.pictura_store_probe(r.ctx, buf[8:8 + 4096])
    finally:
        r.close_checked()
