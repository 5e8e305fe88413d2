"""In-loop coupling: the policy's image encoder consumes the rendered views on the
device, on the render stream, with no host round trip (paper Sec. 3.2: rendered
views feed the network on the device)."""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2607_26005_amd import scenegen as sg

pytestmark = pytest.mark.gpu


def _torch():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no HIP device")
    return torch


def test_encoder_on_rendered_views_matches_oracle_views():
    torch = _torch()
    from paper_2607_26005_amd import pictura
    from paper_2607_26005_amd.encoder import ViewEncoder
    wl = sg.make_config(7, num_worlds=2)   # paper rig, walls, parked cars, traffic lights
    r = pictura.Renderer(0)
    try:
        r.upload(wl.scene, wl.cell_size)
        r.set_lights(pictura.DeviceLights.from_host(wl.lights))
        da = pictura.DeviceAgents.from_host(wl.agents)
        V = wl.num_views
        oc = torch.empty((V, wl.rig.height, wl.rig.width), dtype=torch.uint8, device="cuda")
        od = torch.empty((V, wl.rig.height, wl.rig.width), dtype=torch.float32, device="cuda")
        torch.manual_seed(0)
        enc = ViewEncoder(cams=wl.rig.num_cams).cuda().eval()
        torch.cuda.synchronize()
        # render + encode with synchronising calls turned into errors: no host round trip
        torch.cuda.set_sync_debug_mode("error")
        try:
            with torch.no_grad():
                r.render(da, wl.rig, oc, od)
                emb = enc(oc, od)
        finally:
            torch.cuda.set_sync_debug_mode("default")
        torch.cuda.synchronize()
        assert emb.shape == (V // wl.rig.num_cams, wl.rig.num_cams * 128)
        # the same encoder on the oracle's images of a few egos gives the same embedding
        egos = np.array([0, 5, 17, 40, 63])
        views = (egos[:, None] * wl.rig.num_cams + np.arange(wl.rig.num_cams)[None, :]).ravel()
        ora = O.render(wl.scene, wl.agents, wl.rig, view_ids=views, want_flags=False, lights=wl.lights)
        assert np.array_equal(oc[torch.as_tensor(views, device="cuda")].cpu().numpy(), ora["cls"])
        with torch.no_grad():
            ref = enc(torch.as_tensor(ora["cls"], device="cuda"), torch.as_tensor(ora["depth"], device="cuda"))
        got = emb[torch.as_tensor(egos, device="cuda")]
        assert torch.allclose(got, ref, rtol=1e-4, atol=1e-5), (got - ref).abs().max().item()
    finally:
        r.close_checked()
