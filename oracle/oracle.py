"""ctypes wrapper of the CPU oracle (test infrastructure only).

Only tests, the smoke check and the benchmark's CPU-baseline leg use this
module.  It takes plain NumPy arrays (or objects exposing them as attributes)
and never imports the HIP library or its binding.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "pictura_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

# IEEE fp32 with no contraction and no fast-math: the rules depend on it.
CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-fPIC", "-shared"]


def build(force: bool = False) -> str:
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = LIB + ".tmp"
        subprocess.check_call(["gcc", *CFLAGS, "-o", tmp, SRC, "-lm"])
        os.replace(tmp, LIB)
    return LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(LIB)
        p = ctypes.c_void_p
        L.oracle_render.restype = ctypes.c_int
        L.oracle_render.argtypes = [ctypes.c_int, p, p, p,
                                    ctypes.c_int, p, p, p, p, p, p, p, p, p,
                                    ctypes.c_int, p, p, p, p, p, p, p, ctypes.c_float,
                                    ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                    ctypes.c_float, ctypes.c_float, ctypes.c_float, ctypes.c_float,
                                    ctypes.c_float, ctypes.c_float, p,
                                    ctypes.c_int64, p, p, p, p, p, p, p, p, ctypes.c_int, ctypes.c_int]
        L.oracle_quantize.restype = None
        L.oracle_quantize.argtypes = [p, ctypes.c_int64, ctypes.c_float, ctypes.c_float, p, p]
        L.oracle_bin.restype = ctypes.c_int
        L.oracle_bin.argtypes = [ctypes.c_int, p, p, p, p, ctypes.c_float, p, p, p, p, p, p, p, ctypes.c_int64]
        L.oracle_agents_step.restype = None
        L.oracle_agents_step.argtypes = [ctypes.c_int64, p, p, p, p, p, p, p,
                                         ctypes.c_double, ctypes.c_double, p, p]
        _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def render(scene, agents, rig, view_ids=None, want_flags=True, want_cover=False, num_threads=0, lights=None,
           want_instances=False, want_rgb=False, antialias=False):
    """Render the selected views (default: all).  Returns dict with
    cls [n,H,W] u8, depth [n,H,W] f32, flags [n,H,W] u8 (bit0 EDGE, bit1 TIE),
    and cover [n,H,W] u16 when requested.  lights: object with
    lights_per_world, x, y, z, cos_f, sin_f, radius, cls, cos_max (or None).
    want_instances adds inst [n,H,W] int32 (owning agent or -1) and counts
    [n,A,2] uint32 (footprint, visible pixels per agent); want_rgb switches to
    colour mode (rule R13) and adds rgb [n,3,H,W] uint8; antialias (with
    want_rgb) blends partial-coverage fragments into it (rule R14)."""
    L = lib()
    A = int(agents.agents_per_world)
    C = int(rig.mount.shape[0])
    total = int(scene.num_worlds) * A * C
    if view_ids is None:
        view_ids = np.arange(total, dtype=np.int64)
    view_ids = _c(view_ids, np.int64)
    n = len(view_ids)
    H, W = int(rig.height), int(rig.width)
    out_cls = np.empty((n, H, W), np.uint8)
    out_depth = np.empty((n, H, W), np.float32)
    out_flags = np.empty((n, H, W), np.uint8) if want_flags else None
    out_cover = np.empty((n, H, W), np.uint16) if want_cover else None
    out_inst = np.empty((n, H, W), np.int32) if want_instances else None
    out_counts = np.empty((n, A, 2), np.uint32) if want_instances else None
    out_rgb = np.empty((n, 3, H, W), np.uint8) if want_rgb else None
    keep = [_c(scene.tri_offsets, np.int64), _c(scene.verts, np.float32), _c(scene.cls, np.uint8)]
    af = [_c(getattr(agents, f), np.float32) for f in
          ("x", "y", "z0", "cos_h", "sin_h", "length", "width", "height")]
    acls = _c(agents.cls, np.uint8)
    mount = _c(rig.mount, np.float32)
    NL = int(lights.lights_per_world) if lights is not None else 0
    if NL > 0:
        lf = [_c(getattr(lights, f), np.float32) for f in ("x", "y", "z", "cos_f", "sin_f", "radius")]
        lc = _c(lights.cls, np.uint8)
        cmax = float(lights.cos_max)
    else:
        lf, lc, cmax = [None] * 6, None, 1.0
    rc = L.oracle_render(int(scene.num_worlds), _ptr(keep[0]), _ptr(keep[1]), _ptr(keep[2]),
                         A, *[_ptr(a) for a in af], _ptr(acls),
                         NL, *[_ptr(a) for a in lf], _ptr(lc), cmax,
                         C, W, H, float(rig.fx), float(rig.fy), float(rig.cx), float(rig.cy),
                         float(rig.near), float(rig.far), _ptr(mount),
                         n, _ptr(view_ids), _ptr(out_cls), _ptr(out_depth), _ptr(out_flags),
                         _ptr(out_cover), _ptr(out_inst), _ptr(out_counts), _ptr(out_rgb), int(bool(antialias)),
                         int(num_threads))
    if rc != 0:
        raise ValueError("oracle_render: view id out of range")
    out = dict(cls=out_cls, depth=out_depth)
    if want_flags:
        out["flags"] = out_flags
    if want_cover:
        out["cover"] = out_cover
    if want_rgb:
        out["rgb"] = out_rgb
    if want_instances:
        out["inst"] = out_inst
        out["counts"] = out_counts
    return out


def quantize(iz, near, far):
    """R7/R8: (q24, decoded depth) for an array of inverse depths."""
    L = lib()
    iz = _c(iz, np.float32)
    q = np.empty(iz.shape, np.uint32)
    d = np.empty(iz.shape, np.float32)
    L.oracle_quantize(_ptr(iz), iz.size, float(near), float(far), _ptr(q), _ptr(d))
    return q, d


def bin_scene(scene, cell_size):
    """Uniform-grid binning over primitives (triangles and triangle pairs):
    dims [nw,2], cell_base [nw+1], prims [P] (first triangle | 1 << 31 for a
    pair), home cell per primitive [P], count per cell, member AABB per cell
    [cells,6]."""
    L = lib()
    nw = int(scene.num_worlds)
    b = _c(scene.bounds, np.float32)
    ncell_max = 0
    for w in range(nw):
        nx = max(1, int(np.ceil(np.float32(b[w, 2] - b[w, 0]) / np.float32(cell_size))))
        ny = max(1, int(np.ceil(np.float32(b[w, 3] - b[w, 1]) / np.float32(cell_size))))
        ncell_max += (nx + 1) * (ny + 1)
    dims = np.empty((nw, 2), np.int32)
    base = np.empty(nw + 1, np.int64)
    T = int(scene.tri_offsets[-1])
    prims = np.empty(max(T, 1), np.uint32)
    home = np.empty(max(T, 1), np.int64)
    nprim = np.zeros(1, np.int64)
    count = np.empty(ncell_max, np.int32)
    aabb = np.empty((ncell_max, 6), np.float32)
    offs = _c(scene.tri_offsets, np.int64)
    verts = _c(scene.verts, np.float32)
    cls = _c(scene.cls, np.uint8)
    rc = L.oracle_bin(nw, _ptr(offs), _ptr(verts), _ptr(cls), _ptr(b), float(cell_size), _ptr(dims), _ptr(base),
                      _ptr(prims), _ptr(home), _ptr(nprim), _ptr(count), _ptr(aabb), ncell_max)
    if rc != 0:
        raise RuntimeError("oracle_bin failed")
    nc, npr = int(base[-1]), int(nprim[0])
    return dict(dims=dims, cell_base=base, prims=prims[:npr], home=home[:npr], count=count[:nc], aabb=aabb[:nc])


def agents_step(agents, steer, accel, dt=0.1, vmax=20.0):
    """Kinematic bicycle update in float64; returns dict of float64 arrays."""
    L = lib()
    x = np.array(agents.x, np.float64)
    y = np.array(agents.y, np.float64)
    psi = np.array(agents.psi, np.float64)
    v = np.array(agents.speed, np.float64)
    Ln = _c(agents.length, np.float64)
    st = _c(steer, np.float64)
    ac = _c(accel, np.float64)
    co = np.empty_like(x)
    si = np.empty_like(x)
    L.oracle_agents_step(len(x), _ptr(x), _ptr(y), _ptr(psi), _ptr(v), _ptr(Ln), _ptr(st), _ptr(ac),
                         float(dt), float(vmax), _ptr(co), _ptr(si))
    return dict(x=x, y=y, psi=psi, speed=v, cos_h=co, sin_h=si)
