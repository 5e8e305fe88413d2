"""Render calls of one context on two streams.  Every render call first packs
its agents into the context's one device buffer and then runs its kernels, so
a call on another stream than the previous one must not pack before that
call's kernels are done; the library orders it after them with an event.
Different agent sets rendered back to back on two streams must give the images
each set gives alone."""
import numpy as np
import pytest

from paper_2607_26005_amd import scenegen as sg

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    return torch


def test_render_calls_on_two_streams_keep_their_agents():
    torch = _torch()
    from paper_2607_26005_amd import pictura
    wl = sg.make_config(2, num_worlds=4)    # small-batch worlds: 512 views per call
    other = wl.agents.copy()
    rng = np.random.default_rng(7)
    # a second agent set: every agent moved and turned, so every view differs
    other.x = (other.x + rng.uniform(-30.0, 30.0, other.x.shape)).astype(np.float32)
    other.y = (other.y + rng.uniform(-30.0, 30.0, other.y.shape)).astype(np.float32)
    h = rng.uniform(-np.pi, np.pi, other.x.shape)
    other.cos_h = np.cos(h).astype(np.float32)
    other.sin_h = np.sin(h).astype(np.float32)
    r = pictura.Renderer(0)
    try:
        r.upload(wl.scene, wl.cell_size)
        sets = [pictura.DeviceAgents.from_host(wl.agents), pictura.DeviceAgents.from_host(other)]
        refs = [tuple(t.clone() for t in r.render(d, wl.rig)) for d in sets]
        torch.cuda.synchronize()
        assert not torch.equal(refs[0][0], refs[1][0])
        streams = [torch.cuda.Stream(), torch.cuda.Stream()]   # default priority
        outs = []
        for rep in range(4):
            for i in (0, 1):
                outs.append((i, r.render(sets[i], wl.rig, stream=streams[i])))
        torch.cuda.synchronize()
        for i, (c, d) in outs:
            assert torch.equal(c, refs[i][0]), f"class image of agent set {i} changed on its stream"
            assert torch.equal(d, refs[i][1]), f"depth image of agent set {i} changed on its stream"
    finally:
        r.close_checked()
