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
        r.close()
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
    check(lib, wl, views, "inst-nocull", cull=0)


def test_instances_town_with_lights(lib):
    wl = workload(7, 2)   # paper rig: two tiles per view; lights and parked cars own no instance
    rng = np.random.default_rng(43)
    views = np.sort(rng.choice(wl.num_views, size=64, replace=False))
    check(lib, wl, views, "inst-town")
