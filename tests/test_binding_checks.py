"""The Python binding refuses buffers the library could not use safely: the C
ABI takes plain device pointers and cannot see sizes, so a short, mistyped,
strided or host-resident tensor must be stopped before the call.  These
checks run before any library call, so no GPU is needed: a correct tensor
that lives in host memory is refused for its device, every other case for its
dtype, layout or size."""
import numpy as np
import pytest
import torch

from paper_2607_26005_amd import pictura, scenegen as sg


def _agents(nw=2, A=3, **over):
    n = nw * A
    f = {k: torch.zeros(n, dtype=torch.float32) for k in pictura._AGENT_F32 + ("psi", "speed")}
    f["cls"] = torch.zeros(n, dtype=torch.uint8)
    f.update(over)
    return pictura.DeviceAgents(nw, A, f["x"], f["y"], f["z0"], f["cos_h"], f["sin_h"], f["length"], f["width"],
                                f["height"], f["cls"], f["psi"], f["speed"])


RIG = sg.make_rig(4, 16, 100.0)   # 4 cameras, 16x16
V = 2 * 3 * 4


def _out(n=V * 16 * 16):
    return torch.zeros(n, dtype=torch.uint8), torch.zeros(n, dtype=torch.float32)


@pytest.fixture(autouse=True)
def host_is_device(request, monkeypatch):
    # Host tensors stand in for device tensors in the dtype, layout and size
    # checks (the device check would otherwise stop every call first); the
    # tests of the device check itself keep it.
    if "device" not in request.node.name:
        monkeypatch.setattr(pictura, "_check_device", lambda t, name, ctx: None)


def _raises(match, fn, *a):
    with pytest.raises(pictura.PicturaError, match=match) as e:
        fn(*a)
    assert e.value.status == pictura.EINVAL


def test_host_tensors_are_refused_for_their_device():
    oc, od = _out()
    _raises("expected the HIP device", pictura.pictura_render_views, None, _agents(), RIG, oc, od)


def test_numpy_arrays_are_refused():
    oc, od = _out()
    _raises("expected a torch tensor", pictura.pictura_render_views, None, _agents(x=np.zeros(6, np.float32)), RIG,
            oc, od)
    _raises("expected a torch tensor", pictura.pictura_render_views, None, _agents(), RIG, oc.numpy(), od)


@pytest.mark.parametrize("field", pictura._AGENT_F32)
def test_agent_arrays_dtype_and_count(field):
    oc, od = _out()
    _raises("dtype torch.float64", pictura.pictura_render_views, None,
            _agents(**{field: torch.zeros(6, dtype=torch.float64)}), RIG, oc, od)
    _raises("5 elements, at least 6", pictura.pictura_render_views, None,
            _agents(**{field: torch.zeros(5, dtype=torch.float32)}), RIG, oc, od)


def test_agent_classes_must_be_uint8():
    oc, od = _out()
    _raises("agents.cls: dtype torch.int32", pictura.pictura_render_views, None,
            _agents(cls=torch.zeros(6, dtype=torch.int32)), RIG, oc, od)


def test_strided_tensor_is_refused():
    oc, od = _out()
    strided = torch.zeros(12, dtype=torch.float32)[::2]
    assert strided.numel() == 6
    _raises("not contiguous", pictura.pictura_render_views, None, _agents(y=strided), RIG, oc, od)


def test_outputs_dtype_and_size():
    oc, od = _out()
    short_c, short_d = _out(V * 16 * 16 - 1)
    _raises("out_cls: 6143 elements", pictura.pictura_render_views, None, _agents(), RIG, short_c, od)
    _raises("out_depth: 6143 elements", pictura.pictura_render_views, None, _agents(), RIG, oc, short_d)
    _raises("out_depth: dtype torch.float16", pictura.pictura_render_views, None, _agents(), RIG, oc,
            od.to(torch.float16))
    _raises("out_cls: dtype torch.float32", pictura.pictura_render_views, None, _agents(), RIG, od, od)
    # colour: 3 bytes per pixel
    _raises("out_rgb: 18431 elements", pictura.pictura_render_rgb, None, _agents(), RIG, oc, od,
            torch.zeros(3 * V * 256 - 1, dtype=torch.uint8))
    _raises("out_rgb: 18431 elements", pictura.pictura_render_rgb_aa, None, _agents(), RIG, oc, od,
            torch.zeros(3 * V * 256 - 1, dtype=torch.uint8))


def test_antialiased_depth_may_not_overlap_the_other_outputs():
    # the antialiased kernel keeps its edge buffer in out_depth's words
    n = V * 16 * 16
    big = torch.zeros(4 * n + 4 * n, dtype=torch.uint8)
    od = big[: 4 * n].view(torch.float32)
    _raises("out_depth overlaps out_cls", pictura.pictura_render_rgb_aa, None, _agents(), RIG, big[4 * n - 8:][:n], od,
            torch.zeros(3 * n, dtype=torch.uint8))
    _raises("out_depth overlaps out_rgb", pictura.pictura_render_rgb_aa, None, _agents(), RIG,
            torch.zeros(n, dtype=torch.uint8), od, big[8:][: 3 * n])


def test_instance_outputs_dtype_and_size():
    oc, od = _out()
    inst = torch.zeros(V * 256, dtype=torch.int32)
    counts = torch.zeros(V * 3 * 2, dtype=torch.int32)
    _raises("out_inst: dtype torch.int64", pictura.pictura_render_instances, None, _agents(), RIG, oc, od,
            inst.to(torch.int64), counts)
    _raises("out_counts: 143 elements, at least 144", pictura.pictura_render_instances, None, _agents(), RIG, oc,
            od, inst, counts[:-1])


def test_agents_step_arrays():
    st = _agents()
    ok = torch.zeros(6, dtype=torch.float32)
    _raises("steer: 5 elements", pictura.pictura_agents_step, None, st, ok[:5], ok)
    _raises("accel: dtype torch.float64", pictura.pictura_agents_step, None, st, ok, ok.double())
    _raises("state.psi: 4 elements", pictura.pictura_agents_step, None, _agents(psi=torch.zeros(4)), ok, ok)


def test_agents_step_arrays_on_the_device():
    ok = torch.zeros(6, dtype=torch.float32)
    _raises("expected the HIP device", pictura.pictura_agents_step, None, _agents(), ok, ok)


def test_lights_arrays():
    n = 2 * 5
    f = {k: torch.zeros(n, dtype=torch.float32) for k in ("x", "y", "z", "cos_f", "sin_f", "radius")}
    lights = pictura.DeviceLights(2, 5, f["x"], f["y"], f["z"], f["cos_f"], f["sin_f"], f["radius"],
                                  torch.zeros(n, dtype=torch.uint8), 0.5)
    lights.radius = torch.zeros(n - 1)
    _raises("lights.radius: 9 elements", pictura.pictura_set_lights, None, lights)


def test_lights_arrays_on_the_device():
    n = 2 * 5
    f = {k: torch.zeros(n, dtype=torch.float32) for k in ("x", "y", "z", "cos_f", "sin_f", "radius")}
    lights = pictura.DeviceLights(2, 5, f["x"], f["y"], f["z"], f["cos_f"], f["sin_f"], f["radius"],
                                  torch.zeros(n, dtype=torch.uint8), 0.5)
    _raises("expected the HIP device", pictura.pictura_set_lights, None, lights)
