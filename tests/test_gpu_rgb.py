"""GPU parity of the shaded colour mode (rule R13) against the oracle: classes
and depth as in the plain mode, colour bytes bit-exact wherever the oracle does
not flag the pixel (EDGE / TIE), and at most 1e-4 of the pixels may differ."""
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


def check(lib, wl, views, label, tile=0):
    torch = _torch()
    print(f"[{label}] {wl.num_views} views tile={tile}", flush=True)
    r = lib.Renderer(0)
    try:
        r.set_option(lib.OPT_TILE, tile)
        r.upload(wl.scene, wl.cell_size)
        if wl.lights is not None:
            r.set_lights(lib.DeviceLights.from_host(wl.lights))
        da = lib.DeviceAgents.from_host(wl.agents)
        c, d, rgb = r.render_rgb(da, wl.rig)
        torch.cuda.synchronize()
        idx = torch.as_tensor(np.asarray(views), device="cuda")
        gc, gd, grgb = c[idx].cpu().numpy(), d[idx].cpu().numpy(), rgb[idx].cpu().numpy()
    finally:
        r.close_checked()
    ora = O.render(wl.scene, wl.agents, wl.rig, view_ids=np.asarray(views), lights=wl.lights, want_rgb=True)
    s = assert_parity(gc, gd, ora, label)
    unflag = ora["flags"] == 0
    diff = (grgb != ora["rgb"]).any(1)
    assert not (diff & unflag).any(), (label, int((diff & unflag).sum()))
    assert diff.sum() <= 1e-4 * diff.size, (label, int(diff.sum()))
    boxes = int(((ora["cls"] == 3) | (ora["cls"] == 6)).sum())
    print(f"[{label}] {s} colour mismatches {int(diff.sum())}, box pixels {boxes}", flush=True)
    return boxes


def test_rgb_tiny_all_views(lib):
    wl = workload(1)
    assert check(lib, wl, np.arange(wl.num_views), "rgb-tiny") > 0


def test_rgb_dense_traffic_sampled(lib):
    wl = workload(3, 4)
    views = np.sort(np.random.default_rng(51).choice(wl.num_views, size=96, replace=False))
    assert check(lib, wl, views, "rgb-dense") > 0


def test_rgb_town_paper_rig_and_tiles(lib):
    wl = workload(7, 2)   # two tiles per view, lights
    views = np.sort(np.random.default_rng(52).choice(wl.num_views, size=64, replace=False))
    check(lib, wl, views, "rgb-town")
    check(lib, wl, views, "rgb-town-tile24", tile=24)


@pytest.mark.parametrize("aa", [False, True], ids=["one-sample", "antialiased"])
def test_rgb_unaligned_output_matches_aligned(lib, aa):
    """An output colour image that starts at an odd byte address takes the
    per-pixel byte stores; its bytes equal those of a word-aligned image."""
    torch = _torch()
    wl = workload(1)
    r = lib.Renderer(0)
    try:
        r.upload(wl.scene, wl.cell_size)
        da = lib.DeviceAgents.from_host(wl.agents)
        c0, d0, rgb0 = r.render_rgb(da, wl.rig, antialias=aa)
        n = rgb0.numel()
        buf = torch.full((n + 1,), 7, dtype=torch.uint8, device="cuda")
        out = buf[1:].view(rgb0.shape)
        assert out.data_ptr() % 4 == 1
        c1, d1 = torch.empty_like(c0), torch.empty_like(d0)
        fn = lib.pictura_render_rgb_aa if aa else lib.pictura_render_rgb
        fn(r.ctx, da, wl.rig, c1, d1, out)
        torch.cuda.synchronize()
        assert int(buf[0]) == 7
        assert torch.equal(out, rgb0)
        assert torch.equal(c1, c0) and torch.equal(d1, d0)
    finally:
        r.close_checked()


def test_rgb_headline_full_launch_sampled(lib):
    # the benchmark's one-sample colour launch: 1024 worlds x 64 agents x 4
    # cameras, every view rendered, 64 sampled across the worlds
    wl = workload(4)
    views = np.sort(np.random.default_rng(53).choice(wl.num_views, size=64, replace=False))
    assert len(np.unique(views // 256)) > 48
    assert check(lib, wl, views, "rgb-headline") > 0


def test_rgb_ragged_sizes(lib):
    # 40 x 24 and 96 x 54 (two tiles of 48) take the four-pixel colour
    # stores; 100 x 70 (tiles 50 wide) and 17 x 129 the per-byte ones
    wl = workload(2, 1)
    for (W, H) in ((40, 24), (100, 70), (17, 129), (96, 54)):
        rig = sg.Rig(width=W, height=H, fx=W / 2.0, fy=W / 2.0, cx=W / 2.0, cy=H / 2.0, near=0.5, far=100.0,
                     mount=wl.rig.mount)
        wl2 = sg.Workload(wl.name, 2, 1, wl.scene, wl.agents, rig, wl.cell_size, wl.world_size)
        views = np.sort(np.random.default_rng(W + 1).choice(wl2.num_views, size=32, replace=False))
        check(lib, wl2, views, f"rgb-ragged {W}x{H}")
