"""Python binding of the HIP rasterizer library (libpictura.so).

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  PyTorch provides device memory and the current HIP stream.  The
functions carry the C ABI's names (include/pictura.h); `Renderer` wraps a
context for convenience.  If the library is not built, importing this module
raises: there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libpictura.so")

OK, EINVAL, ENOMEM, EDEVICE, ESTATE, ERANGE = 0, -1, -2, -3, -4, -5
OPT_CULL, OPT_TILE, OPT_STATS = 1, 2, 3
MAX_CAMS = 8

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build the HIP library first (python __graft_entry__.py build)")

_lib = ctypes.CDLL(LIB_PATH)


class PicturaError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"pictura status {status}: {msg}")
        self.status = status


class _Scene(ctypes.Structure):
    _fields_ = [("num_worlds", ctypes.c_int32), ("tri_offsets", ctypes.c_void_p), ("verts", ctypes.c_void_p),
                ("cls", ctypes.c_void_p), ("bounds", ctypes.c_void_p)]


class _Agents(ctypes.Structure):
    _fields_ = [("num_worlds", ctypes.c_int32), ("agents_per_world", ctypes.c_int32)] + \
               [(n, ctypes.c_void_p) for n in ("x", "y", "z0", "cos_h", "sin_h", "length", "width", "height", "cls")]


class _Rig(ctypes.Structure):
    _fields_ = [("num_cams", ctypes.c_int32), ("width", ctypes.c_int32), ("height", ctypes.c_int32),
                ("fx", ctypes.c_float), ("fy", ctypes.c_float), ("cx", ctypes.c_float), ("cy", ctypes.c_float),
                ("near_m", ctypes.c_float), ("far_m", ctypes.c_float),
                ("mount", (ctypes.c_float * 5) * MAX_CAMS)]


class _Lights(ctypes.Structure):
    _fields_ = [("num_worlds", ctypes.c_int32), ("lights_per_world", ctypes.c_int32)] + \
               [(n, ctypes.c_void_p) for n in ("x", "y", "z", "cos_f", "sin_f", "radius", "cls")] + \
               [("cos_max", ctypes.c_float)]


class _AgentState(ctypes.Structure):
    _fields_ = [("count", ctypes.c_int32)] + \
               [(n, ctypes.c_void_p) for n in ("x", "y", "psi", "speed", "cos_h", "sin_h", "length")]


_P = ctypes.c_void_p
_lib.pictura_create.argtypes = [ctypes.c_int32, ctypes.POINTER(_P)]
_lib.pictura_create.restype = ctypes.c_int32
_lib.pictura_destroy.argtypes = [_P]
_lib.pictura_destroy.restype = None
_lib.pictura_last_error.argtypes = [_P]
_lib.pictura_last_error.restype = ctypes.c_char_p
_lib.pictura_scene_upload.argtypes = [_P, ctypes.POINTER(_Scene), _P]
_lib.pictura_scene_upload.restype = ctypes.c_int32
_lib.pictura_bin_scene.argtypes = [_P, ctypes.c_float, _P]
_lib.pictura_bin_scene.restype = ctypes.c_int32
_lib.pictura_render_views.argtypes = [_P, ctypes.POINTER(_Agents), ctypes.POINTER(_Rig), _P, _P, _P]
_lib.pictura_render_views.restype = ctypes.c_int32
_lib.pictura_agents_step.argtypes = [_P, ctypes.POINTER(_AgentState), _P, _P, ctypes.c_float, ctypes.c_float, _P]
_lib.pictura_agents_step.restype = ctypes.c_int32
_lib.pictura_bins_info.argtypes = [_P, _P, _P, _P, _P]
_lib.pictura_bins_info.restype = ctypes.c_int32
_lib.pictura_bins_copy.argtypes = [_P, _P, _P, _P]
_lib.pictura_bins_copy.restype = ctypes.c_int32
_lib.pictura_set_option.argtypes = [_P, ctypes.c_int32, ctypes.c_int32]
_lib.pictura_set_option.restype = ctypes.c_int32
_lib.pictura_stats_copy.argtypes = [_P, _P, ctypes.c_int32, ctypes.c_int32]
_lib.pictura_stats_copy.restype = ctypes.c_int32
_lib.pictura_render_rgb.argtypes = [_P, ctypes.POINTER(_Agents), ctypes.POINTER(_Rig), _P, _P, _P, _P]
_lib.pictura_render_rgb.restype = ctypes.c_int32
_lib.pictura_render_rgb_aa.argtypes = [_P, ctypes.POINTER(_Agents), ctypes.POINTER(_Rig), _P, _P, _P, _P]
_lib.pictura_render_rgb_aa.restype = ctypes.c_int32
_lib.pictura_render_instances.argtypes = [_P, ctypes.POINTER(_Agents), ctypes.POINTER(_Rig), _P, _P, _P, _P, _P]
_lib.pictura_render_instances.restype = ctypes.c_int32
_lib.pictura_set_lights.argtypes = [_P, ctypes.POINTER(_Lights)]
_lib.pictura_set_lights.restype = ctypes.c_int32
_lib.pictura_selftest_rcp.argtypes = [_P, ctypes.c_uint32, ctypes.c_uint32, _P]
_lib.pictura_selftest_rcp.restype = ctypes.c_int32
_lib.pictura_selftest_rcp_noalloc.argtypes = [_P, ctypes.c_uint32, ctypes.c_uint32, _P]
_lib.pictura_selftest_rcp_noalloc.restype = ctypes.c_int32
_lib.pictura_store_probe.argtypes = [_P, _P, ctypes.c_uint64, _P]
_lib.pictura_store_probe.restype = ctypes.c_int32
_lib.pictura_device_errors.argtypes = [_P, _P, ctypes.c_int32]
_lib.pictura_device_errors.restype = ctypes.c_int32

EXPORTED = ["pictura_create", "pictura_destroy", "pictura_last_error", "pictura_scene_upload",
            "pictura_bin_scene", "pictura_render_views", "pictura_agents_step", "pictura_bins_info",
            "pictura_bins_copy", "pictura_set_option", "pictura_stats_copy", "pictura_selftest_rcp",
            "pictura_set_lights", "pictura_render_instances", "pictura_render_rgb", "pictura_render_rgb_aa",
            "pictura_device_errors", "pictura_selftest_rcp_noalloc", "pictura_store_probe"]
DEVERR_RING_WAIT = 1

STAT_NAMES = ["view_tiles", "cells_in_rect", "cells_prefiltered", "cells_visible", "cand_tris", "boxes_visible",
              "box_tris", "first_pass_survivors", "exact_batches", "clipped", "raster_tris", "lane_tris",
              "lane_px", "record_tris", "record_tris_fp64", "blocks_tested", "blocks_passed", "first_pass_chunks",
              "cyc_prologue", "cyc_sources", "cyc_first_pass", "cyc_exact", "cyc_records", "cyc_writeout",
              "aa_surfaces_packed", "aa_packed_px", "aa_packed_steps", "aa_surfaces_swept", "aa_blocks_swept",
              "aa_fragments"]


_CTX_DEVICE = {}   # context handle -> HIP device index it was created on

_DTYPE_NAMES = {"f32": "float32", "u8": "uint8", "i32": "int32"}


def _torch_dtypes(kind):
    import torch
    return {"f32": (torch.float32,), "u8": (torch.uint8,),
            "i32": (torch.int32,) + ((torch.uint32,) if hasattr(torch, "uint32") else ())}[kind]


def _ctx_key(ctx):
    return ctx.value if isinstance(ctx, ctypes.c_void_p) else ctx


def _dev(t, name: str, kind: str, count: int, ctx=None) -> int:
    """Device address of a caller-owned buffer after checking it: a torch
    tensor of the expected dtype, contiguous, holding at least `count`
    elements, on the HIP device of the context.  The library cannot see buffer
    sizes, so these checks are what keeps a short or mistyped buffer from
    becoming out-of-bounds device accesses.  Raises PicturaError(EINVAL)."""
    import torch
    if not isinstance(t, torch.Tensor):
        raise PicturaError(EINVAL, f"{name}: expected a torch tensor on the HIP device, got {type(t).__name__}")
    if t.dtype not in _torch_dtypes(kind):
        raise PicturaError(EINVAL, f"{name}: dtype {t.dtype}, expected {_DTYPE_NAMES[kind]}")
    if not t.is_contiguous():
        raise PicturaError(EINVAL, f"{name}: tensor is not contiguous")
    if t.numel() < count:
        raise PicturaError(EINVAL, f"{name}: {t.numel()} elements, at least {count} needed")
    _check_device(t, name, ctx)
    return t.data_ptr()


def _check_device(t, name: str, ctx) -> None:
    if t.device.type != "cuda":
        raise PicturaError(EINVAL, f"{name}: tensor on {t.device}, expected the HIP device")
    want = _CTX_DEVICE.get(_ctx_key(ctx))
    if want is not None and t.device.index is not None and t.device.index != want:
        raise PicturaError(EINVAL, f"{name}: tensor on cuda:{t.device.index}, the context renders on cuda:{want}")


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _check(ctx, st):
    if st != OK:
        msg = _lib.pictura_last_error(ctx).decode() if ctx else ""
        raise PicturaError(st, msg)


# --- functions with the C ABI's names ---------------------------------------

def pictura_create(device: int = 0):
    h = _P()
    st = _lib.pictura_create(int(device), ctypes.byref(h))
    if st != OK:
        raise PicturaError(st, "pictura_create failed (no HIP device?)")
    _CTX_DEVICE[h.value] = int(device)
    return h


def pictura_destroy(ctx):
    _CTX_DEVICE.pop(_ctx_key(ctx), None)
    _lib.pictura_destroy(ctx)


def pictura_last_error(ctx) -> str:
    return _lib.pictura_last_error(ctx).decode()


def pictura_scene_upload(ctx, scene, stream=None):
    """scene: object with num_worlds, tri_offsets (int64), verts (float32 [T,9]),
    cls (uint8), bounds (float32 [nw,4]) as host NumPy arrays."""
    offs = np.ascontiguousarray(scene.tri_offsets, np.int64)
    verts = np.ascontiguousarray(scene.verts, np.float32)
    cls = np.ascontiguousarray(scene.cls, np.uint8)
    bounds = np.ascontiguousarray(scene.bounds, np.float32)
    s = _Scene(int(scene.num_worlds), offs.ctypes.data, verts.ctypes.data if verts.size else None,
               cls.ctypes.data if cls.size else None, bounds.ctypes.data)
    _check(ctx, _lib.pictura_scene_upload(ctx, ctypes.byref(s), _stream(stream)))


def pictura_bin_scene(ctx, cell_size_m: float, stream=None):
    _check(ctx, _lib.pictura_bin_scene(ctx, float(cell_size_m), _stream(stream)))


def make_rig(rig) -> _Rig:
    r = _Rig()
    r.num_cams = int(rig.mount.shape[0])
    r.width, r.height = int(rig.width), int(rig.height)
    r.fx, r.fy, r.cx, r.cy = float(rig.fx), float(rig.fy), float(rig.cx), float(rig.cy)
    r.near_m, r.far_m = float(rig.near), float(rig.far)
    m = np.asarray(rig.mount, np.float32)
    for k in range(min(r.num_cams, MAX_CAMS)):
        for q in range(5):
            r.mount[k][q] = float(m[k, q])
    return r


_AGENT_F32 = ("x", "y", "z0", "cos_h", "sin_h", "length", "width", "height")


def _agents(ctx, agents) -> _Agents:
    """The C struct of a DeviceAgents, every array checked (float32 SoA of
    num_worlds * agents_per_world elements, uint8 classes)."""
    n = int(agents.num_worlds) * int(agents.agents_per_world)
    return _Agents(int(agents.num_worlds), int(agents.agents_per_world),
                   *[_dev(getattr(agents, f), f"agents.{f}", "f32", n, ctx) for f in _AGENT_F32],
                   _dev(agents.cls, "agents.cls", "u8", n, ctx))


def _rig(rig) -> _Rig:
    return make_rig(rig) if not isinstance(rig, _Rig) else rig


def _views(agents, r: _Rig) -> int:
    return int(agents.num_worlds) * int(agents.agents_per_world) * int(r.num_cams)


def _outputs(ctx, agents, r: _Rig, out_cls, out_depth):
    npx = _views(agents, r) * r.height * r.width
    return npx, _dev(out_cls, "out_cls", "u8", npx, ctx), _dev(out_depth, "out_depth", "f32", npx, ctx)


def pictura_render_views(ctx, agents, rig, out_cls, out_depth, stream=None):
    """agents: DeviceAgents (torch CUDA tensors); rig: scenegen.Rig-like;
    out_cls uint8 / out_depth float32 CUDA tensors of V*H*W elements."""
    r = _rig(rig)
    a = _agents(ctx, agents)
    _, oc, od = _outputs(ctx, agents, r, out_cls, out_depth)
    _check(ctx, _lib.pictura_render_views(ctx, ctypes.byref(a), ctypes.byref(r), oc, od, _stream(stream)))


def pictura_render_rgb(ctx, agents, rig, out_cls, out_depth, out_rgb, stream=None):
    """As pictura_render_views, plus out_rgb (uint8, V*3*H*W, planar)."""
    r = _rig(rig)
    a = _agents(ctx, agents)
    npx, oc, od = _outputs(ctx, agents, r, out_cls, out_depth)
    orgb = _dev(out_rgb, "out_rgb", "u8", 3 * npx, ctx)
    _check(ctx, _lib.pictura_render_rgb(ctx, ctypes.byref(a), ctypes.byref(r), oc, od, orgb, _stream(stream)))


def _disjoint(name_a: str, a: int, na: int, name_b: str, b: int, nb: int) -> None:
    """Raise PicturaError(EINVAL) if the byte ranges [a, a + na) and [b, b + nb) meet."""
    if a < b + nb and b < a + na:
        raise PicturaError(EINVAL, f"{name_a} overlaps {name_b}")


def pictura_render_rgb_aa(ctx, agents, rig, out_cls, out_depth, out_rgb, stream=None):
    """As pictura_render_rgb, with analytic-coverage antialiasing of out_rgb.
    The kernel keeps its edge buffer in out_depth's words during the call, so
    out_depth may not overlap out_cls or out_rgb."""
    r = _rig(rig)
    a = _agents(ctx, agents)
    npx, oc, od = _outputs(ctx, agents, r, out_cls, out_depth)
    orgb = _dev(out_rgb, "out_rgb", "u8", 3 * npx, ctx)
    _disjoint("out_depth", od, 4 * npx, "out_cls", oc, npx)
    _disjoint("out_depth", od, 4 * npx, "out_rgb", orgb, 3 * npx)
    _check(ctx, _lib.pictura_render_rgb_aa(ctx, ctypes.byref(a), ctypes.byref(r), oc, od, orgb, _stream(stream)))


def pictura_render_instances(ctx, agents, rig, out_cls, out_depth, out_inst, out_counts, stream=None):
    """As pictura_render_views, plus out_inst (int32, V*H*W) and out_counts
    (int32 tensor viewed as uint32, V*A*2: footprint, visible)."""
    r = _rig(rig)
    a = _agents(ctx, agents)
    npx, oc, od = _outputs(ctx, agents, r, out_cls, out_depth)
    oi = _dev(out_inst, "out_inst", "i32", npx, ctx)
    ok = _dev(out_counts, "out_counts", "i32", _views(agents, r) * int(agents.agents_per_world) * 2, ctx)
    _check(ctx, _lib.pictura_render_instances(ctx, ctypes.byref(a), ctypes.byref(r), oc, od, oi, ok,
                                              _stream(stream)))


def pictura_agents_step(ctx, state, steer, accel, dt: float = 0.1, vmax: float = 20.0, stream=None):
    """state: DeviceAgents-like (float32 x, y, psi, speed, cos_h, sin_h,
    length of num_worlds * agents_per_world elements); steer, accel: float32
    tensors of the same count."""
    n = int(state.num_worlds) * int(state.agents_per_world)
    s = _AgentState(n, *[_dev(getattr(state, f), f"state.{f}", "f32", n, ctx) for f in
                         ("x", "y", "psi", "speed", "cos_h", "sin_h", "length")])
    st_, ac_ = _dev(steer, "steer", "f32", n, ctx), _dev(accel, "accel", "f32", n, ctx)
    _check(ctx, _lib.pictura_agents_step(ctx, ctypes.byref(s), st_, ac_, float(dt), float(vmax), _stream(stream)))


def pictura_set_lights(ctx, lights):
    """lights: DeviceLights (torch CUDA tensors) or None (detach).  The context
    keeps the pointers: the tensors must stay alive while it renders."""
    if lights is None:
        _check(ctx, _lib.pictura_set_lights(ctx, None))
        return
    n = int(lights.num_worlds) * int(lights.lights_per_world)
    l = _Lights(int(lights.num_worlds), int(lights.lights_per_world),
                *[_dev(getattr(lights, f), f"lights.{f}", "f32", n, ctx) for f in
                  ("x", "y", "z", "cos_f", "sin_f", "radius")],
                _dev(lights.cls, "lights.cls", "u8", n, ctx), float(lights.cos_max))
    _check(ctx, _lib.pictura_set_lights(ctx, ctypes.byref(l)))


def pictura_bins_info(ctx, num_worlds: int):
    """(dims [nw, 2], cell_base [nw + 1], total cells, total primitives)"""
    dims = np.empty((num_worlds, 2), np.int32)
    base = np.empty(num_worlds + 1, np.int64)
    total = ctypes.c_int64()
    prims = ctypes.c_int64()
    _check(ctx, _lib.pictura_bins_info(ctx, dims.ctypes.data, base.ctypes.data, ctypes.addressof(total),
                                       ctypes.addressof(prims)))
    return dims, base, int(total.value), int(prims.value)


def pictura_bins_copy(ctx, total_cells: int, num_prims: int):
    start = np.empty(total_cells + 1, np.uint32)
    aabb = np.empty((total_cells, 6), np.float32)
    perm = np.empty(max(num_prims, 1), np.uint32)
    _check(ctx, _lib.pictura_bins_copy(ctx, start.ctypes.data, aabb.ctypes.data, perm.ctypes.data))
    return start, aabb, perm[:num_prims]


def pictura_set_option(ctx, option: int, value: int):
    _check(ctx, _lib.pictura_set_option(ctx, int(option), int(value)))


def pictura_selftest_rcp(ctx, lo_bits: int, count: int) -> int:
    out = ctypes.c_uint64()
    _check(ctx, _lib.pictura_selftest_rcp(ctx, int(lo_bits), int(count), ctypes.addressof(out)))
    return int(out.value)


def pictura_store_probe(ctx, buf, stream=None):
    """Fill the whole uint8 tensor `buf` (a multiple of 16 bytes) with zeros
    using 16-byte non-temporal stores: the HBM write-rate reference."""
    n = buf.numel() if hasattr(buf, "numel") else 0
    ptr = _dev(buf, "buf", "u8", n, ctx)
    _check(ctx, _lib.pictura_store_probe(ctx, ptr, n, _stream(stream)))


def pictura_device_errors(ctx, reset: bool = False) -> int:
    """OR of the device error bits (DEVERR_*) the render kernels set since the
    context was created or last reset; synchronous."""
    out = ctypes.c_uint32()
    _check(ctx, _lib.pictura_device_errors(ctx, ctypes.addressof(out), int(bool(reset))))
    return int(out.value)


def pictura_selftest_rcp_noalloc(ctx, lo_bits: int, count: int) -> int:
    out = ctypes.c_uint64()
    _check(ctx, _lib.pictura_selftest_rcp_noalloc(ctx, int(lo_bits), int(count), ctypes.addressof(out)))
    return int(out.value)


def pictura_stats_copy(ctx, reset: bool = True):
    out = np.zeros(len(STAT_NAMES), np.uint64)
    _check(ctx, _lib.pictura_stats_copy(ctx, out.ctypes.data, len(out), int(bool(reset))))
    return dict(zip(STAT_NAMES, (int(x) for x in out)))


# --- device-resident agents ------------------------------------------------------

@dataclasses.dataclass
class DeviceAgents:
    num_worlds: int
    agents_per_world: int
    x: "object"
    y: "object"
    z0: "object"
    cos_h: "object"
    sin_h: "object"
    length: "object"
    width: "object"
    height: "object"
    cls: "object"
    psi: "object"
    speed: "object"

    @staticmethod
    def from_host(agents, device="cuda"):
        import torch
        f = lambda a, dt=torch.float32: torch.as_tensor(np.ascontiguousarray(a), dtype=dt).to(device)
        return DeviceAgents(int(agents.num_worlds), int(agents.agents_per_world),
                            *[f(getattr(agents, n)) for n in ("x", "y", "z0", "cos_h", "sin_h", "length", "width",
                                                             "height")],
                            f(agents.cls, torch.uint8), f(agents.psi), f(agents.speed))


@dataclasses.dataclass
class DeviceLights:
    num_worlds: int
    lights_per_world: int
    x: "object"
    y: "object"
    z: "object"
    cos_f: "object"
    sin_f: "object"
    radius: "object"
    cls: "object"
    cos_max: float

    @staticmethod
    def from_host(lights, device="cuda"):
        import torch
        f = lambda a, dt=torch.float32: torch.as_tensor(np.ascontiguousarray(a), dtype=dt).to(device)
        return DeviceLights(int(lights.num_worlds), int(lights.lights_per_world),
                            *[f(getattr(lights, n)) for n in ("x", "y", "z", "cos_f", "sin_f", "radius")],
                            f(lights.cls, torch.uint8), float(lights.cos_max))


class Renderer:
    """Owns a library context, its scene and bins."""

    def __init__(self, device: int = 0):
        self.ctx = pictura_create(device)
        self.num_worlds = 0
        self.num_tris = 0
        self.lights = None

    def close(self):
        if self.ctx:
            pictura_destroy(self.ctx)
            self.ctx = None

    def close_checked(self):
        """Close after checking that no render kernel reported a device error."""
        try:
            err = self.device_errors() if self.ctx else 0
        finally:
            self.close()
        if err:
            raise PicturaError(EDEVICE, f"render kernels reported device error bits {err:#x}")

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def upload(self, scene, cell_size: float, stream=None):
        pictura_scene_upload(self.ctx, scene, stream)
        pictura_bin_scene(self.ctx, cell_size, stream)
        self.num_worlds = int(scene.num_worlds)
        self.num_tris = int(scene.tri_offsets[-1])

    def render(self, agents: DeviceAgents, rig, out_cls=None, out_depth=None, stream=None):
        import torch
        V = agents.num_worlds * agents.agents_per_world * int(rig.mount.shape[0])
        shape = (V, int(rig.height), int(rig.width))
        if out_cls is None:
            out_cls = torch.empty(shape, dtype=torch.uint8, device=agents.x.device)
        if out_depth is None:
            out_depth = torch.empty(shape, dtype=torch.float32, device=agents.x.device)
        pictura_render_views(self.ctx, agents, rig, out_cls, out_depth, stream)
        return out_cls, out_depth

    def render_rgb(self, agents: DeviceAgents, rig, stream=None, antialias=False):
        """Returns (cls, depth, rgb) with rgb [V, 3, H, W] uint8 (antialiased when asked)."""
        import torch
        V = agents.num_worlds * agents.agents_per_world * int(rig.mount.shape[0])
        H, W = int(rig.height), int(rig.width)
        dev = agents.x.device
        out_cls = torch.empty((V, H, W), dtype=torch.uint8, device=dev)
        out_depth = torch.empty((V, H, W), dtype=torch.float32, device=dev)
        out_rgb = torch.empty((V, 3, H, W), dtype=torch.uint8, device=dev)
        fn = pictura_render_rgb_aa if antialias else pictura_render_rgb
        fn(self.ctx, agents, rig, out_cls, out_depth, out_rgb, stream)
        return out_cls, out_depth, out_rgb

    def render_instances(self, agents: DeviceAgents, rig, stream=None):
        """Returns (cls, depth, inst, counts): counts [V, A, 2] int32 holding
        (footprint, visible) pixels per agent and view."""
        import torch
        V = agents.num_worlds * agents.agents_per_world * int(rig.mount.shape[0])
        shape = (V, int(rig.height), int(rig.width))
        dev = agents.x.device
        out_cls = torch.empty(shape, dtype=torch.uint8, device=dev)
        out_depth = torch.empty(shape, dtype=torch.float32, device=dev)
        out_inst = torch.empty(shape, dtype=torch.int32, device=dev)
        counts = torch.empty((V, agents.agents_per_world, 2), dtype=torch.int32, device=dev)
        pictura_render_instances(self.ctx, agents, rig, out_cls, out_depth, out_inst, counts, stream)
        return out_cls, out_depth, out_inst, counts

    def agents_step(self, agents: DeviceAgents, steer, accel, dt=0.1, vmax=20.0, stream=None):
        pictura_agents_step(self.ctx, agents, steer, accel, dt, vmax, stream)

    def device_errors(self, reset: bool = False) -> int:
        return pictura_device_errors(self.ctx, reset)

    def set_option(self, option, value):
        pictura_set_option(self.ctx, option, value)

    def set_lights(self, lights: Optional[DeviceLights]):
        pictura_set_lights(self.ctx, lights)
        self.lights = lights   # the context keeps the pointers: hold the tensors

    def bins(self):
        dims, base, total, prims = pictura_bins_info(self.ctx, self.num_worlds)
        start, aabb, perm = pictura_bins_copy(self.ctx, total, prims)
        return dict(dims=dims, cell_base=base, cell_start=start, aabb=aabb, perm=perm)
