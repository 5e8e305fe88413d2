"""GPU parity of instance visibility (render_instances) against the oracle:
the owning agent of every pixel and each agent's footprint and visible pixel
counts are integers, compared exactly."""
import functools

import numpy as np
import pytest

from oracle import oracle as O
from paper_2607_26005_amd import scenegen as sg
from tests.parity import assert_parity

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    return torch


@pytest.fixture(scope="module")
def lib():
    _torch()
    from paper_2607_26005_amd import pictura
    return pictura


@functools.lru_cache(maxsize=None)
def workload(cfg, worlds=None):
    return sg.make_config(cfg, num_worlds=worlds)


def check(lib, wl, views, label, tile=0, cull=1):
    torch = _torch()
    print(f"[{label}] {wl.num_views} views tile={tile} cull={cull}", flush=True)
    r = lib.Renderer(0)
    try:
        r.set_option(lib.OPT_TILE, tile)
        r.set_option(lib.OPT_CULL, cull)
        r.upload(wl.scene, wl.cell_size)
        if wl.lights is not None:
            r.set_lights(lib.DeviceLights.from_host(wl.lights))
        da = lib.DeviceAgents.from_host(wl.agents)
        c, d, inst, counts = r.render_instances(da, wl.rig)
        torch.cuda.synchronize()
        idx = torch.as_tensor(np.asarray(views), device="cuda")
        gc, gd = c[idx].cpu().numpy(), d[idx].cpu().numpy()
        gi = inst[idx].cpu().numpy()
        gk = counts[idx].cpu().numpy().view(np.uint32)
    finally:
        r.close_checked()
    ora = O.render(wl.scene, wl.agents, wl.rig, view_ids=np.asarray(views), lights=wl.lights, want_instances=True)
    s = assert_parity(gc, gd, ora, label)
    assert s["mismatches"] == 0, s
    assert np.array_equal(gi, ora["inst"]), (label, int((gi != ora["inst"]).sum()))
    assert np.array_equal(gk, ora["counts"]), (label, np.argwhere(gk != ora["counts"])[:5])
    owned = int((ora["inst"] >= 0).sum())
    print(f"[{label}] owned px {owned}, agents seen {int((ora['counts'][..., 0] > 0).sum())}", flush=True)
    return owned


def test_instances_tiny_all_views(lib):
    wl = workload(1)
    assert check(lib, wl, np.arange(wl.num_views), "inst-tiny") > 0


def test_instances_dense_traffic_sampled(lib):
    wl = workload(3, 4)   # 128 agents per world, 20 % pedestrians, contacts
    rng = np.random.default_rng(41)
    views = np.sort(rng.choice(wl.num_views, size=96, replace=False))
    assert check(lib, wl, views, "inst-dense") > 0


def test_instances_tiled_and_unculled(lib):
    wl = workload(2, 2)
    rng = np.random.default_rng(42)
    views = np.sort(rng.choice(wl.num_views, size=48, replace=False))
    check(lib, wl, views, "inst-tiles16", tile=16)
    check(lib, wl, views, "inst-tiles48", tile=48)   # 48 x 48 tiles and ragged 16-wide ones
    check(lib, wl, views, "inst-nocull", cull=0)


def test_instances_headline_full_launch_sampled(lib):
    # the benchmark's instance launch: 1024 worlds x 64 agents x 4 cameras
    wl = workload(4)
    views = np.sort(np.random.default_rng(44).choice(wl.num_views, size=64, replace=False))
    assert len(np.unique(views // 256)) > 48
    check(lib, wl, views, "inst-headline")


def test_instances_among_random_quad_pairs(lib):
    # boxes among a soup of quad pairs (convex, darts, slivers, near-plane crossings)
    from tests.test_gpu_aa import _random_quads
    from tests.scenes import make_agents, make_rig, make_scene
    tris, cls = _random_quads(91)
    rng = np.random.default_rng(191)
    rows = [(0.0, 0.0, 0.0, 1.0, 0.0, 4.5, 1.9, 1.5, 3)]
    for _ in range(11):
        ang = rng.uniform(0, 2 * np.pi)
        rows.append((rng.uniform(-15, 15), rng.uniform(-15, 15), 0.0, float(np.cos(ang)), float(np.sin(ang)),
                     4.5, 1.9, 1.5, 3))
    rig = make_rig(res=64, far=80.0, mounts=((0.0, 0.0, 1.0, 1.0, 0.0), (0.0, 0.0, 1.0, 0.0, 1.0),
                                              (0.0, 0.0, 1.0, -1.0, 0.0), (0.0, 0.0, 1.0, 0.0, -1.0)))
    wl = sg.Workload("random-quads", 0, 91, make_scene(np.asarray(tris, np.float32), cls), make_agents(rows), rig,
                     16.0, 2000.0)
    assert check(lib, wl, np.arange(wl.num_views), "inst-random-quads") > 0


def test_instances_town_with_lights(lib):
    wl = workload(7, 2)   # paper rig: two tiles per view; lights and parked cars own no instance
    rng = np.random.default_rng(43)
    views = np.sort(rng.choice(wl.num_views, size=64, replace=False))
    check(lib, wl, views, "inst-town")


def test_instances_faces_behind_near_or_beyond_far(lib):
    # Regression: the instance pass must drop a box triangle with no vertex at
    # zv >= near, or with every vertex beyond far (R4), as the class/depth pass
    # and the oracle do.  Car 1 in the next lane has its rear face 0.25 m ahead
    # of the forward camera (between the camera plane and the near plane);
    # car 2 starts 0.3 m ahead of it in its own lane, so the camera looks into
    # its open rear end; car 3 lies wholly beyond far = 110 m, its rear face one
    # fp32 step beyond the far plane, where the plane value at the covered
    # centres equals fl(1/110) and so passes the per-pixel far test: its
    # footprint must be 0.  The second camera looks right, along car 1's side.
    from tests.scenes import make_agents, make_rig, make_scene, quad
    D = float(np.nextafter(np.float32(110.0), np.float32(np.inf)))
    G = 1000.0
    scene = make_scene(quad((-G, -G, 0.0), (G, -G, 0.0), (G, G, 0.0), (-G, G, 0.0)), [0, 0])
    ag = make_agents([(0.0, 0.0, 0.0, 1.0, 0.0, 4.5, 1.9, 1.5, 3),
                      (2.5, -3.5, 0.0, 1.0, 0.0, 4.5, 1.9, 1.5, 3),
                      (2.55, 0.0, 0.0, 1.0, 0.0, 4.5, 1.9, 1.6, 3),
                      (D + 2.0, 0.0, 0.5, 1.0, 0.0, 4.0, 2.0, 2.0, 3)])
    assert np.float32(ag.x[3]) - np.float32(2.0) == np.float32(D)
    rig = make_rig(mounts=((0.0, 0.0, 1.5, 1.0, 0.0), (0.0, 0.0, 1.5, 0.0, -1.0)), far=110.0)
    wl = sg.Workload("inst-near-far", 0, 0, scene, ag, rig, 16.0, 2000.0)
    check(lib, wl, np.arange(wl.num_views), "inst-near-far")
    ora = O.render(scene, ag, rig, want_instances=True)
    assert ora["counts"][0, 1, 0] > 0 and ora["counts"][0, 2, 0] > 0   # cars 1 and 2 are seen
    assert (ora["counts"][:, 3, 0] == 0).all()                         # car 3 never is


def test_instances_same_class_overlap_and_ties(lib):
    # Two vehicles overlap in view with the farther one listed first: only the
    # full depth key, not the class, names the nearer box as the owner.  Two
    # identical boxes elsewhere tie, and the lower index takes the pixels.
    from tests.scenes import make_agents, make_rig, make_scene, quad
    G = 1000.0
    scene = make_scene(quad((-G, -G, -0.75), (G, -G, -0.75), (G, G, -0.75), (-G, G, -0.75)), [0, 0])
    ag = make_agents([(0.0, 0.0, 0.0, 1.0, 0.0, 4.5, 1.9, 1.5, 3),
                      (18.0, -0.6, -0.75, 1.0, 0.0, 4.5, 1.9, 2.5, 3),
                      (10.0, 0.8, -0.75, 1.0, 0.0, 4.5, 1.9, 1.5, 3),
                      (12.0, -6.0, -0.75, 0.8, 0.6, 4.5, 1.9, 1.5, 3),
                      (12.0, -6.0, -0.75, 0.8, 0.6, 4.5, 1.9, 1.5, 3)])
    rig = make_rig(res=96, mounts=((0.0, 0.0, 0.0, 1.0, 0.0), (0.0, 0.0, 0.0, 0.0, -1.0)))
    wl = sg.Workload("inst-same-class", 0, 0, scene, ag, rig, 16.0, 2000.0)
    check(lib, wl, np.arange(wl.num_views), "inst-same-class")
    c = O.render(scene, ag, rig, view_ids=[0], want_instances=True)["counts"][0]
    assert c[2, 0] == c[2, 1] > 0 and 0 < c[1, 1] < c[1, 0]
    assert c[3, 0] == c[4, 0] == c[3, 1] > 0 and c[4, 1] == 0


def test_instances_largest_view(lib):
    # owners and counts on the largest view the ABI accepts, 4096 x 4096
    # (4,096 tiles per view), two whole images against the oracle
    wl = workload(1)
    rig = sg.Rig(width=4096, height=4096, fx=2048.0, fy=2048.0, cx=2048.0, cy=2048.0, near=0.5, far=100.0,
                 mount=wl.rig.mount)
    wl2 = sg.Workload(wl.name, 1, 0, wl.scene, wl.agents, rig, wl.cell_size, wl.world_size)
    assert check(lib, wl2, [0, 5], "inst-largest") > 0
