"""GPU parity of traffic lights (R10 visibility cone, R11 disks) and the town
workload (walls, parked cars, lights) against the CPU oracle."""
import functools

import numpy as np
import pytest

from oracle import oracle as O
from paper_2607_26005_amd import scenegen as sg
from tests.parity import assert_parity
from tests.scenes import make_agents, make_rig, make_scene
from tests.test_lights import lights_of

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
def town(worlds):
    return sg.make_config(7, num_worlds=worlds)


def render_gpu(pictura, scene, agents, rig, cell, lights, cull=1, tile=0):
    torch = _torch()
    r = pictura.Renderer(0)
    try:
        r.set_option(pictura.OPT_CULL, cull)
        r.set_option(pictura.OPT_TILE, tile)
        r.upload(scene, cell)
        r.set_lights(pictura.DeviceLights.from_host(lights) if lights is not None else None)
        da = pictura.DeviceAgents.from_host(agents)
        c, d = r.render(da, rig)
        torch.cuda.synchronize()
        return c.cpu().numpy(), d.cpu().numpy()
    finally:
        r.close_checked()


def test_town_features_sampled(lib):
    wl = town(6)
    print(f"[town] {wl.num_views} views, {wl.scene.num_tris} tris, {wl.lights.lights_per_world} lights/world",
          flush=True)
    c, d = render_gpu(lib, wl.scene, wl.agents, wl.rig, wl.cell_size, wl.lights)
    rng = np.random.default_rng(31)
    ids = np.sort(rng.choice(wl.num_views, size=192, replace=False))
    ora = O.render(wl.scene, wl.agents, wl.rig, view_ids=ids, lights=wl.lights)
    s = assert_parity(c[ids], d[ids], ora, "town")
    lit = int((ora["cls"] >= sg.LIGHT_RED).sum())
    walls = int((ora["cls"] == sg.WALL).sum())
    print(f"[town] {s} light px {lit} wall px {walls}", flush=True)
    assert lit > 0 and walls > 0


def _light_field(seed, n_agents=6, n_lights=80):
    """Ground plane, agents on it and lights of random orientation and height around them."""
    rng = np.random.default_rng([91, seed])
    g = [[(-200.0, -200.0, 0.0), (200.0, -200.0, 0.0), (200.0, 200.0, 0.0)],
         [(-200.0, -200.0, 0.0), (200.0, 200.0, 0.0), (-200.0, 200.0, 0.0)]]
    rows = []
    for k in range(n_agents):
        a = rng.uniform(-np.pi, np.pi)
        rows.append((rng.uniform(-30, 30), rng.uniform(-30, 30), 0.0, float(np.float32(np.cos(a))),
                     float(np.float32(np.sin(a))), 4.5, 1.9, 1.5, 3))
    lr = []
    for k in range(n_lights):
        a = rng.uniform(-np.pi, np.pi)
        lr.append((rng.uniform(-60, 60), rng.uniform(-60, 60), rng.uniform(0.5, 8.0), float(np.float32(np.cos(a))),
                   float(np.float32(np.sin(a))), rng.uniform(0.2, 2.0), 8 + k % 3))
    mounts = tuple((0.0, 0.0, 1.5, c, s) for c, s in ((1, 0), (0, 1), (-1, 0), (0, -1)))
    return make_scene(g, [0, 0], bounds=(-200.0, -200.0, 200.0, 200.0)), make_agents(rows), \
        lights_of(lr, cos_max=0.4), make_rig(mounts=mounts)


@pytest.mark.parametrize("seed", range(3))
def test_random_lights_all_views_cull_and_tiles(lib, seed):
    sc, ag, L, rig = _light_field(seed)
    ora = O.render(sc, ag, rig, lights=L)
    assert (ora["cls"] >= 8).sum() > 0
    base = None
    for cull, tile in ((1, 0), (0, 0), (1, 16)):
        print(f"[lights {seed}] cull={cull} tile={tile}", flush=True)
        c, d = render_gpu(lib, sc, ag, rig, 16.0, L, cull, tile)
        s = assert_parity(c, d, ora, f"lights-{seed}-{cull}-{tile}")
        assert s["mismatches"] == 0, s
        if base is None:
            base = (c, d)
        else:
            assert np.array_equal(c, base[0]) and np.array_equal(d.view(np.uint32), base[1].view(np.uint32))


def test_lights_detach_and_errors(lib):
    torch = _torch()
    sc, ag, L, rig = _light_field(7, n_lights=40)
    ctx = lib.pictura_create(0)
    try:
        lib.pictura_scene_upload(ctx, sc)
        lib.pictura_bin_scene(ctx, 16.0)
        DL = lib.DeviceLights.from_host(L)
        bad = lib.DeviceLights(**{**DL.__dict__, "cos_max": 1.5})
        with pytest.raises(lib.PicturaError) as e:
            lib.pictura_set_lights(ctx, bad)
        assert e.value.status == lib.EINVAL
        other = lib.DeviceLights(**{**DL.__dict__, "num_worlds": 2, "lights_per_world": 20})
        lib.pictura_set_lights(ctx, other)
        da = lib.DeviceAgents.from_host(ag)
        V = ag.count * rig.num_cams
        oc = torch.empty(V * 64 * 64, dtype=torch.uint8, device="cuda")
        od = torch.empty(V * 64 * 64, dtype=torch.float32, device="cuda")
        with pytest.raises(lib.PicturaError) as e:
            lib.pictura_render_views(ctx, da, rig, oc, od)
        assert e.value.status == lib.EINVAL
        # attached: lights drawn; detached: the plain scene
        lib.pictura_set_lights(ctx, DL)
        lib.pictura_render_views(ctx, da, rig, oc, od)
        torch.cuda.synchronize()
        assert_parity(oc.view(V, 64, 64).cpu().numpy(), od.view(V, 64, 64).cpu().numpy(),
                      O.render(sc, ag, rig, lights=L), "attached")
        lib.pictura_set_lights(ctx, None)
        lib.pictura_render_views(ctx, da, rig, oc, od)
        torch.cuda.synchronize()
        assert_parity(oc.view(V, 64, 64).cpu().numpy(), od.view(V, 64, 64).cpu().numpy(),
                      O.render(sc, ag, rig), "detached")
        # a signal changing state between renders: new class values, same pointers
        DL.cls.copy_(torch.full_like(DL.cls, 9))
        lib.pictura_set_lights(ctx, DL)
        lib.pictura_render_views(ctx, da, rig, oc, od)
        torch.cuda.synchronize()
        L2 = type(L)(**{**L.__dict__, "cls": np.full_like(L.cls, 9)})
        assert_parity(oc.view(V, 64, 64).cpu().numpy(), od.view(V, 64, 64).cpu().numpy(),
                      O.render(sc, ag, rig, lights=L2), "state-change")
    finally:
        lib.pictura_destroy(ctx)
