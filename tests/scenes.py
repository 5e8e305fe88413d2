"""Hand-built test scenes (inputs only) shared by oracle pins and GPU tests."""
import numpy as np

from paper_2607_26005_amd.scenegen import Agents, Rig, Scene


def make_scene(tris, cls, bounds=(-1000.0, -1000.0, 1000.0, 1000.0)):
    """One world from triangles [T,3,3] and classes [T]."""
    tris = np.asarray(tris, np.float32).reshape(-1, 9)
    cls = np.asarray(cls, np.uint8).reshape(-1)
    return Scene(num_worlds=1, verts=np.ascontiguousarray(tris), cls=cls,
                 tri_offsets=np.asarray([0, len(tris)], np.int64),
                 bounds=np.asarray([bounds], np.float32))


def make_agents(rows, num_worlds=1):
    """rows: list of (x, y, z0, cos, sin, L, W, H, cls) for each agent of each world."""
    a = np.asarray([r[:8] for r in rows], np.float64)
    n = len(rows)
    f = lambda k: np.ascontiguousarray(a[:, k].astype(np.float32))
    return Agents(num_worlds=num_worlds, agents_per_world=n // num_worlds,
                  x=f(0), y=f(1), z0=f(2), cos_h=f(3), sin_h=f(4), length=f(5), width=f(6), height=f(7),
                  cls=np.asarray([r[8] for r in rows], np.uint8),
                  psi=np.arctan2(a[:, 4], a[:, 3]).astype(np.float32), speed=np.zeros(n, np.float32))


def make_rig(res=64, near=0.5, far=100.0, mounts=((0.0, 0.0, 0.0, 1.0, 0.0),), f=None, height=None):
    w = res
    h = res if height is None else height
    f = w / 2.0 if f is None else f
    return Rig(width=w, height=h, fx=f, fy=f, cx=w / 2.0, cy=h / 2.0, near=near, far=far,
               mount=np.asarray(mounts, np.float32))


def quad(p0, p1, p2, p3):
    return [[p0, p1, p2], [p0, p2, p3]]


def walled(scene, height=12.0, inset=80.0, reach=95.0, cls=7):
    """The one-world scene with four walls of the given height added around
    its centre (square of half-side `inset`), reaching above any camera."""
    walls = []
    for (a, b) in (((inset, -reach), (inset, reach)), ((-inset, reach), (-inset, -reach)),
                   ((-reach, inset), (reach, inset)), ((reach, -inset), (-reach, -inset))):
        walls += quad((a[0], a[1], 0.0), (b[0], b[1], 0.0), (b[0], b[1], height), (a[0], a[1], height))
    verts = np.concatenate([scene.verts, np.asarray(walls, np.float32).reshape(-1, 9)])
    c = np.concatenate([scene.cls, np.full(len(walls), cls, np.uint8)])
    return Scene(num_worlds=1, verts=np.ascontiguousarray(verts), cls=c,
                 tri_offsets=np.asarray([0, len(verts)], np.int64), bounds=scene.bounds)
