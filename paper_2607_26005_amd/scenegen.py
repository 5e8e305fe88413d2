"""Seeded synthetic driving scenes: the inputs of the batched view rasterizer.

This module only *makes inputs*: static triangle soups (ground, road surface,
lane markings, curbs), agent poses and sizes, the camera rig and per-step
controls.  It holds none of the rasterization arithmetic (camera build, box
triangulation, projection, snapping, coverage, depth); both the HIP path and
the CPU oracle receive the same arrays from here and each does its own maths.

The paper renders CARLA towns and Waymo layouts with a 4-camera rig (Sec. 3.2,
App. A.3, Tab. camera_rig).  Those datasets are not available, so five seeded
workloads of the same kind stand in for them:

  1 tiny       1 world 200x200 m, 2x2 grid of two-lane roads, 8 boxes,
               1 forward camera, 64x64, far 100 m
  2 small      64 worlds 1x1 km, 6+6 straight roads of 2-4 lanes in 2 m
               segments, curbs (43-47k triangles per world), 32 boxes,
               4 cameras, 64x64, far 100 m                     (8,192 views)
  3 dense      256 worlds, same generator, 128 agents (20 % pedestrians),
               no overlap rejection (contact ties)            (131,072 views)
  4 headline   1024 worlds x 64 agents x 4 cameras, far 150 m, agents moved
               every step by the kinematic bicycle update     (262,144 views)
  5 large      128 worlds 4x4 km of cubic-Bezier roads tessellated at 0.5 m
               (~500k triangles per world), 128x128 views, far 200 m
  6 paper rig  64 worlds of the small-batch town seen through the paper's
               four-camera rig at 96x54 (2,048 egos: one render chunk)
  7 town       the paper's other rendering features on the small-batch town:
               building walls along the blocks, parked cars, and traffic
               lights (disks with a limited visibility cone) at every
               intersection, one facing each approach; paper rig, 96x54

Coordinates are metres, world-centred, z up.  Vertical layers are lifted so
that coplanar classes never tie: ground z=0, road top z=0.02, markings
z=0.03, curbs rise 0.15 m from the road top.

Every world w of workload seed s draws from ``np.random.default_rng([s, w])``,
so a workload built with fewer worlds is an exact prefix of the full one.
"""
from __future__ import annotations

import dataclasses
import hashlib
from typing import List, Optional

import numpy as np

# Semantic class IDs.  Sky is never a triangle: it is the background class.
GROUND, ROAD, MARKING, VEHICLE, SKY, CURB, PEDESTRIAN = 0, 1, 2, 3, 4, 5, 6
WALL, LIGHT_RED, LIGHT_AMBER, LIGHT_GREEN = 7, 8, 9, 10
CLASS_NAMES = ["ground", "road", "marking", "vehicle", "sky", "curb", "pedestrian", "wall", "light_red",
               "light_amber", "light_green"]

Z_GROUND = 0.0
Z_ROAD = 0.02
Z_MARK = 0.03
CURB_H = 0.15
LANE_W = 3.5
ROAD_SEG = 2.0      # road surface and curb faces: one quad per 2 m of road (every world >= 40k triangles)
MARK_W = 0.15
DASH_LEN, DASH_GAP = 3.0, 3.0

# Exact (cos, sin) of the four axis headings, so that cameras mounted at
# multiples of 90 degrees get basis vectors with components in {0, +-1}.
_AXIS_CS = {0: (1.0, 0.0), 1: (0.0, 1.0), 2: (-1.0, 0.0), 3: (0.0, -1.0)}


@dataclasses.dataclass
class Scene:
    """Static triangles of all worlds, concatenated world by world."""
    num_worlds: int
    verts: np.ndarray        # float32 [T, 9]: x0 y0 z0 x1 y1 z1 x2 y2 z2
    cls: np.ndarray          # uint8   [T]
    tri_offsets: np.ndarray  # int64   [num_worlds + 1]
    bounds: np.ndarray       # float32 [num_worlds, 4]: xmin ymin xmax ymax

    @property
    def num_tris(self) -> int:
        return int(self.tri_offsets[-1])

    def world(self, w: int):
        a, b = int(self.tri_offsets[w]), int(self.tri_offsets[w + 1])
        return self.verts[a:b], self.cls[a:b]

    def sha256(self) -> str:
        h = hashlib.sha256()
        for arr in (self.verts, self.cls, self.tri_offsets, self.bounds):
            h.update(np.ascontiguousarray(arr).tobytes())
        return h.hexdigest()


@dataclasses.dataclass
class Agents:
    """Structure-of-arrays agent state, index = world * agents_per_world + a."""
    num_worlds: int
    agents_per_world: int
    x: np.ndarray
    y: np.ndarray
    z0: np.ndarray           # height of the box base
    cos_h: np.ndarray
    sin_h: np.ndarray
    length: np.ndarray
    width: np.ndarray
    height: np.ndarray
    cls: np.ndarray          # uint8
    psi: np.ndarray          # heading angle (bicycle state; cos_h/sin_h are its cos/sin)
    speed: np.ndarray        # m/s (bicycle state)

    FIELDS = ("x", "y", "z0", "cos_h", "sin_h", "length", "width", "height")

    @property
    def count(self) -> int:
        return self.num_worlds * self.agents_per_world

    def copy(self) -> "Agents":
        return dataclasses.replace(self, **{f.name: np.array(getattr(self, f.name), copy=True)
                                            for f in dataclasses.fields(self)
                                            if isinstance(getattr(self, f.name), np.ndarray)})


@dataclasses.dataclass
class Lights:
    """Traffic lights, index = world * lights_per_world + l: disks of `radius`
    centred at (x, y, z) with horizontal normal (cos_f, sin_f), seen only from
    within the cone of half-angle acos(cos_max) around that normal."""
    num_worlds: int
    lights_per_world: int
    x: np.ndarray
    y: np.ndarray
    z: np.ndarray
    cos_f: np.ndarray
    sin_f: np.ndarray
    radius: np.ndarray
    cls: np.ndarray          # uint8: the signal state's class
    cos_max: float


@dataclasses.dataclass
class Rig:
    """Pinhole cameras mounted on every agent (yaw-only mounts)."""
    width: int
    height: int
    fx: float
    fy: float
    cx: float
    cy: float
    near: float
    far: float
    mount: np.ndarray        # float32 [num_cams, 5]: x y z cos_yaw sin_yaw (ego frame)

    @property
    def num_cams(self) -> int:
        return int(self.mount.shape[0])


@dataclasses.dataclass
class Workload:
    name: str
    config: int
    seed: int
    scene: Scene
    agents: Agents
    rig: Rig
    cell_size: float
    world_size: float
    lights: Optional[Lights] = None

    @property
    def num_views(self) -> int:
        return self.agents.count * self.rig.num_cams


# ----------------------------------------------------------------------------
# geometry helpers (float64 while building, float32 on output)
# ----------------------------------------------------------------------------

def _quads(p0, p1, p2, p3):
    """Quads [n,3] x4 -> triangles [2n,3,3] as (p0,p1,p2), (p0,p2,p3)."""
    t1 = np.stack([p0, p1, p2], axis=1)
    t2 = np.stack([p0, p2, p3], axis=1)
    return np.stack([t1, t2], axis=1).reshape(-1, 3, 3)


def _xyz(x, y, z):
    x = np.asarray(x, np.float64)
    return np.stack([x, np.broadcast_to(y, x.shape), np.broadcast_to(z, x.shape)], axis=-1)


def ground_tiles(size: float, tile: float) -> np.ndarray:
    n = int(round(size / tile))
    e = -size / 2 + tile * np.arange(n + 1)
    x0, y0 = np.meshgrid(e[:-1], e[:-1], indexing="ij")
    x1, y1 = x0 + tile, y0 + tile
    x0, y0, x1, y1 = (a.ravel() for a in (x0, y0, x1, y1))
    z = Z_GROUND
    return _quads(_xyz(x0, y0, z), _xyz(x1, y0, z), _xyz(x1, y1, z), _xyz(x0, y1, z))


@dataclasses.dataclass
class StraightRoad:
    axis: int          # 0: runs along x (centre at y=c), 1: runs along y (centre at x=c)
    c: float
    lanes: int

    @property
    def width(self):
        return self.lanes * LANE_W


def _map_uv(road: StraightRoad, u, v, z):
    """Road-local (u along, v across) -> world xyz."""
    u = np.asarray(u, np.float64)
    v = np.broadcast_to(np.asarray(v, np.float64), u.shape)
    if road.axis == 0:
        return _xyz(u, road.c + v, z)
    return np.stack([road.c + v, u, np.broadcast_to(z, u.shape)], axis=-1)


def _outside_crossings(u0, u1, crossings):
    keep = np.ones(u0.shape, bool)
    for (uc, wc) in crossings:
        keep &= ~((u1 > uc - wc / 2) & (u0 < uc + wc / 2))
    return keep


def straight_road_tris(road: StraightRoad, size: float, seg: float, crossings,
                       curbs: bool, phase: float):
    """Surface (2 tris per segment), dashed lane dividers, optional curbs."""
    out_t, out_c = [], []
    n = int(round(size / seg))
    u0 = -size / 2 + seg * np.arange(n)
    u1 = u0 + seg
    hw = road.width / 2
    surf = _quads(_map_uv(road, u0, -hw, Z_ROAD), _map_uv(road, u1, -hw, Z_ROAD),
                  _map_uv(road, u1, hw, Z_ROAD), _map_uv(road, u0, hw, Z_ROAD))
    out_t.append(surf)
    out_c.append(np.full(len(surf), ROAD, np.uint8))
    # dashed dividers between lanes
    ds = -size / 2 + phase + (DASH_LEN + DASH_GAP) * np.arange(int(size / (DASH_LEN + DASH_GAP)) + 1)
    ds = ds[ds + DASH_LEN <= size / 2]
    ds = ds[_outside_crossings(ds, ds + DASH_LEN, crossings)]
    for k in range(1, road.lanes):
        v = -hw + k * LANE_W
        m = _quads(_map_uv(road, ds, v - MARK_W / 2, Z_MARK),
                   _map_uv(road, ds + DASH_LEN, v - MARK_W / 2, Z_MARK),
                   _map_uv(road, ds + DASH_LEN, v + MARK_W / 2, Z_MARK),
                   _map_uv(road, ds, v + MARK_W / 2, Z_MARK))
        out_t.append(m)
        out_c.append(np.full(len(m), MARKING, np.uint8))
    if curbs:
        keep = _outside_crossings(u0, u1, crossings)
        a0, a1 = u0[keep], u1[keep]
        for v in (-hw, hw):
            q = _quads(_map_uv(road, a0, v, Z_ROAD), _map_uv(road, a1, v, Z_ROAD),
                       _map_uv(road, a1, v, Z_ROAD + CURB_H), _map_uv(road, a0, v, Z_ROAD + CURB_H))
            out_t.append(q)
            out_c.append(np.full(len(q), CURB, np.uint8))
    return out_t, out_c


def _bezier_road(rng, size: float, step: float):
    """Cubic Bezier centre line resampled at `step` metres of arc length."""
    P = rng.uniform(-size / 2, size / 2, size=(4, 2))
    t = np.linspace(0.0, 1.0, 20001)
    mt = 1.0 - t
    B = (mt ** 3)[:, None] * P[0] + (3 * mt * mt * t)[:, None] * P[1] + \
        (3 * mt * t * t)[:, None] * P[2] + (t ** 3)[:, None] * P[3]
    seglen = np.linalg.norm(np.diff(B, axis=0), axis=1)
    s = np.concatenate([[0.0], np.cumsum(seglen)])
    sk = np.arange(0.0, s[-1], step)
    x = np.interp(sk, s, B[:, 0])
    y = np.interp(sk, s, B[:, 1])
    pts = np.stack([x, y], axis=1)
    tan = np.gradient(pts, axis=0)
    tan /= np.maximum(np.linalg.norm(tan, axis=1, keepdims=True), 1e-12)
    nrm = np.stack([-tan[:, 1], tan[:, 0]], axis=1)
    return sk, pts, tan, nrm


def _strip(pts, nrm, v0, v1, z, mask=None):
    """Quads between consecutive sections, lateral offsets v0..v1 (flat at z)."""
    a, b = pts[:-1], pts[1:]
    na, nb = nrm[:-1], nrm[1:]
    if mask is not None:
        a, b, na, nb = a[mask], b[mask], na[mask], nb[mask]
    def P(p, n, v):
        q = p + v * n
        return _xyz(q[:, 0], q[:, 1], z)
    return _quads(P(a, na, v0), P(b, nb, v0), P(b, nb, v1), P(a, na, v1))


def _curb_strip(pts, nrm, v):
    a, b = pts[:-1] + v * nrm[:-1], pts[1:] + v * nrm[1:]
    return _quads(_xyz(a[:, 0], a[:, 1], Z_ROAD), _xyz(b[:, 0], b[:, 1], Z_ROAD),
                  _xyz(b[:, 0], b[:, 1], Z_ROAD + CURB_H), _xyz(a[:, 0], a[:, 1], Z_ROAD + CURB_H))


# ----------------------------------------------------------------------------
# per-world builders
# ----------------------------------------------------------------------------

@dataclasses.dataclass
class _WorldAgents:
    x: np.ndarray
    y: np.ndarray
    z0: np.ndarray
    c: np.ndarray
    s: np.ndarray
    psi: np.ndarray
    L: np.ndarray
    W: np.ndarray
    H: np.ndarray
    cls: np.ndarray


def _place_on_straight_roads(rng, roads: List[StraightRoad], size, n, min_gap, jitter, ped_frac):
    xs, ys, zs, cs, ss, ps, Ls, Ws, Hs, cl = ([] for _ in range(10))
    n_ped = int(round(n * ped_frac))
    tries = 0
    while len(xs) < n:
        tries += 1
        if tries > 200000:
            raise RuntimeError("agent placement failed")
        is_ped = len(xs) >= n - n_ped
        road = roads[rng.integers(len(roads))]
        u = rng.uniform(-size / 2 + 6.0, size / 2 - 6.0)
        if is_ped:
            side = 1.0 if rng.random() < 0.5 else -1.0
            v = side * (road.width / 2 + rng.uniform(0.5, 3.0))
            ang = rng.uniform(-np.pi, np.pi)
            c, s, psi = np.cos(ang), np.sin(ang), ang
            L, W, H = 0.5, 0.5, 1.7
            z0 = Z_GROUND
            k = PEDESTRIAN
        else:
            lane = rng.integers(road.lanes)
            v = -road.width / 2 + (lane + 0.5) * LANE_W
            if abs(v) < 1e-9:
                fwd = rng.random() < 0.5
            else:
                # right-hand traffic: along +x on the -y side, along +y on the +x side
                fwd = (v < 0) if road.axis == 0 else (v > 0)
            q = (0 if fwd else 2) if road.axis == 0 else (1 if fwd else 3)
            c, s = _AXIS_CS[q]
            psi = q * np.pi / 2
            if psi > np.pi:
                psi -= 2 * np.pi
            j = rng.uniform(1 - jitter, 1 + jitter, size=3) if jitter > 0 else np.ones(3)
            L, W, H = 4.5 * j[0], 1.9 * j[1], 1.5 * j[2]
            z0 = Z_ROAD
            k = VEHICLE
        px, py = (u, road.c + v) if road.axis == 0 else (road.c + v, u)
        if min_gap > 0 and xs:
            d2 = (np.asarray(xs) - px) ** 2 + (np.asarray(ys) - py) ** 2
            if d2.min() < min_gap * min_gap:
                continue
        xs.append(px); ys.append(py); zs.append(z0); cs.append(c); ss.append(s); ps.append(psi)
        Ls.append(L); Ws.append(W); Hs.append(H); cl.append(k)
    return _WorldAgents(*(np.asarray(a, np.float64) for a in (xs, ys, zs, cs, ss, ps, Ls, Ws, Hs)),
                        np.asarray(cl, np.uint8))


def _grid_world(rng, size, tile, n_roads_axis, lane_choices, seg, curbs, n_agents,
                min_gap, jitter, ped_frac, fixed_centres=None, return_roads=False):
    tris, clss = [ground_tiles(size, tile)], []
    clss.append(np.full(len(tris[0]), GROUND, np.uint8))
    roads: List[StraightRoad] = []
    for axis in (0, 1):
        for k in range(n_roads_axis):
            if fixed_centres is not None:
                c = fixed_centres[k]
            else:
                c = (k + 0.5) * size / n_roads_axis - size / 2 + rng.uniform(-0.15, 0.15) * size / n_roads_axis
            lanes = int(lane_choices[rng.integers(len(lane_choices))])
            roads.append(StraightRoad(axis, float(c), lanes))
    for r in roads:
        crossings = [(o.c, o.width) for o in roads if o.axis != r.axis]
        phase = float(rng.uniform(0, DASH_LEN + DASH_GAP))
        t, c = straight_road_tris(r, size, seg, crossings, curbs, phase)
        tris += t
        clss += c
    ag = _place_on_straight_roads(rng, roads, size, n_agents, min_gap, jitter, ped_frac)
    if return_roads:
        return np.concatenate(tris), np.concatenate(clss), ag, roads
    return np.concatenate(tris), np.concatenate(clss), ag


def _aabox_tris(x0, y0, z0, x1, y1, z1):
    """Axis-aligned boxes [n] -> 12 triangles each (scene input: parked cars)."""
    c = [_xyz(np.where(n & 1, x1, x0), np.where(n & 2, y1, y0), np.where(n & 4, z1, z0)) for n in range(8)]
    faces = ((0, 1, 3, 2), (4, 5, 7, 6), (0, 2, 6, 4), (1, 3, 7, 5), (0, 1, 5, 4), (2, 3, 7, 6))
    return np.concatenate([_quads(c[a], c[b], c[d], c[e]) for a, b, d, e in faces])


LIGHT_Z, LIGHT_R, LIGHT_COS_MAX = 5.0, 0.3, 0.5   # head height, disk radius, cone cos(60 deg)
STOP_W, STOP_GAP = 0.4, 1.0                       # stop-line bar width, gap to the crossing road's edge


def light_and_stop_line(cx, cy, dx, dy, hw_cross, hw_own):
    """The signal of one approach and the stop line it governs (Sec. 3.2,
    rendering features: the head is placed apart from its stop line, as at
    junctions whose signal hangs beyond the crossing).  Traffic moving along the
    unit axis (dx, dy) drives on the right-hand half of its road (half width
    hw_own); the crossing road has half width hw_cross.  Returns the head's
    centre (beyond the junction, on the right, facing the approaching traffic)
    and the bar's two triangles (before the junction, across the right-hand
    lanes, at the marking layer)."""
    far = hw_cross + 1.0
    rx, ry = dy, -dx                                   # right-hand side of the travel direction
    head = (cx + dx * far + rx * (hw_own + 1.0), cy + dy * far + ry * (hw_own + 1.0))
    s0, s1 = -(hw_cross + STOP_GAP + STOP_W), -(hw_cross + STOP_GAP)
    corner = lambda s, t: np.array([[cx + dx * s + rx * t, cy + dy * s + ry * t, Z_MARK]])
    # counter-clockwise seen from above: along the travel direction, then across to the left
    bar = _quads(corner(s0, hw_own), corner(s1, hw_own), corner(s1, 0.0), corner(s0, 0.0))
    return head, bar


def _town_world(rng, size, n_agents):
    """Small-batch town plus walls, parked cars and traffic lights."""
    tris, clss, ag, roads = _grid_world(rng, size, 25.0, 6, [2, 3, 4], ROAD_SEG, True, n_agents, 8.0, 0.1, 0.0,
                                        return_roads=True)
    extra_t, extra_c = [], []
    lx, ly, lcf, lsf, lcls = [], [], [], [], []
    for r in roads:
        others = [o for o in roads if o.axis != r.axis]
        hw = r.width / 2
        # blocks between consecutive crossings
        cuts = sorted([-size / 2] + [o.c for o in others] + [size / 2])
        for a, b in zip(cuts[:-1], cuts[1:]):
            wa = a + (0 if a == -size / 2 else max(o.width for o in others if o.c == a) / 2 + 6.0)
            wb = b - (0 if b == size / 2 else max(o.width for o in others if o.c == b) / 2 + 6.0)
            if wb - wa < 20.0:
                continue
            for side in (-1.0, 1.0):
                # building walls 4 m behind the curb: facades of 12..40 m, 6..18 m tall, with gaps
                u = wa
                while u < wb - 8.0:
                    ln = min(rng.uniform(12.0, 40.0), wb - u)
                    h = rng.uniform(6.0, 18.0)
                    v = side * (hw + 4.0)
                    q = _quads(_map_uv(r, np.array([u]), v, Z_GROUND), _map_uv(r, np.array([u + ln]), v, Z_GROUND),
                               _map_uv(r, np.array([u + ln]), v, h), _map_uv(r, np.array([u]), v, h))
                    extra_t.append(q)
                    extra_c.append(np.full(len(q), WALL, np.uint8))
                    u += ln + rng.uniform(2.0, 10.0)
                # parked cars on the strip between curb and wall, 30 % of 7 m slots
                slots = wa + 3.0 + 7.0 * np.arange(int((wb - wa - 6.0) // 7.0))
                slots = slots[rng.random(len(slots)) < 0.3]
                if len(slots):
                    v0, v1 = side * (hw + 0.9), side * (hw + 2.8)
                    p0 = _map_uv(r, slots - 2.25, min(v0, v1), Z_GROUND)
                    p1 = _map_uv(r, slots + 2.25, max(v0, v1), Z_GROUND + 1.5)
                    lo, hi = np.minimum(p0, p1), np.maximum(p0, p1)
                    bx = _aabox_tris(lo[:, 0], lo[:, 1], lo[:, 2], hi[:, 0], hi[:, 1], hi[:, 2])
                    extra_t.append(bx)
                    extra_c.append(np.full(len(bx), VEHICLE, np.uint8))
    # traffic lights: at every crossing one head per approach, on the far side of the
    # junction, facing the traffic that approaches it, and the stop line it governs on
    # the near side; the two axes show opposite states
    xr = [r for r in roads if r.axis == 0]
    yr = [r for r in roads if r.axis == 1]
    for ra in xr:
        for rb in yr:
            cx_, cy_ = rb.c, ra.c
            sx = LIGHT_GREEN if rng.random() < 0.5 else LIGHT_RED
            sy = LIGHT_RED if sx == LIGHT_GREEN else LIGHT_GREEN
            if rng.random() < 0.15:
                sx = LIGHT_AMBER
            # (approach direction (dx, dy), state): traffic driving +x meets a head beyond the crossing at +x
            for (dx, dy, st, hw_cross, hw_own) in ((1, 0, sx, rb.width / 2, ra.width / 2),
                                                   (-1, 0, sx, rb.width / 2, ra.width / 2),
                                                   (0, 1, sy, ra.width / 2, rb.width / 2),
                                                   (0, -1, sy, ra.width / 2, rb.width / 2)):
                (px, py), bar = light_and_stop_line(cx_, cy_, dx, dy, hw_cross, hw_own)
                extra_t.append(bar)
                extra_c.append(np.full(len(bar), MARKING, np.uint8))
                lx.append(px); ly.append(py)
                lcf.append(float(-dx)); lsf.append(float(-dy))
                lcls.append(st)
    if extra_t:
        tris = np.concatenate([tris] + extra_t)
        clss = np.concatenate([clss] + extra_c)
    n = len(lx)
    lights = dict(x=np.asarray(lx), y=np.asarray(ly), z=np.full(n, LIGHT_Z), cos_f=np.asarray(lcf),
                  sin_f=np.asarray(lsf), radius=np.full(n, LIGHT_R), cls=np.asarray(lcls, np.uint8))
    return tris, clss, ag, lights


def _bezier_world(rng, size, tile, target_tris, n_agents, jitter):
    tris, clss = [ground_tiles(size, tile)], []
    clss.append(np.full(len(tris[0]), GROUND, np.uint8))
    total = len(tris[0])
    roads = []
    while total < target_tris:
        lanes = int(rng.integers(2, 5))
        w = lanes * LANE_W
        sk, pts, tan, nrm = _bezier_road(rng, size, 0.5)
        if len(sk) < 8:
            continue
        parts = [(_strip(pts, nrm, -w / 2, w / 2, Z_ROAD), ROAD)]
        phase = rng.uniform(0, DASH_LEN + DASH_GAP)
        mid = 0.5 * (sk[:-1] + sk[1:])
        dash = np.mod(mid - phase, DASH_LEN + DASH_GAP) < DASH_LEN
        for k in range(1, lanes):
            v = -w / 2 + k * LANE_W
            parts.append((_strip(pts, nrm, v - MARK_W / 2, v + MARK_W / 2, Z_MARK, dash), MARKING))
        parts.append((_curb_strip(pts, nrm, -w / 2), CURB))
        parts.append((_curb_strip(pts, nrm, w / 2), CURB))
        for t, k in parts:
            tris.append(t)
            clss.append(np.full(len(t), k, np.uint8))
            total += len(t)
        roads.append((lanes, pts, tan, nrm))
    xs, ys, zs, cs, ss, ps, Ls, Ws, Hs = ([] for _ in range(9))
    for _ in range(n_agents):
        lanes, pts, tan, nrm = roads[rng.integers(len(roads))]
        i = int(rng.integers(len(pts)))
        lane = int(rng.integers(lanes))
        v = -lanes * LANE_W / 2 + (lane + 0.5) * LANE_W
        fwd = v < 0 if abs(v) > 1e-9 else bool(rng.random() < 0.5)
        t = tan[i] if fwd else -tan[i]
        p = pts[i] + v * nrm[i]
        j = rng.uniform(1 - jitter, 1 + jitter, size=3)
        xs.append(p[0]); ys.append(p[1]); zs.append(Z_ROAD)
        cs.append(t[0]); ss.append(t[1]); ps.append(np.arctan2(t[1], t[0]))
        Ls.append(4.5 * j[0]); Ws.append(1.9 * j[1]); Hs.append(1.5 * j[2])
    ag = _WorldAgents(*(np.asarray(a, np.float64) for a in (xs, ys, zs, cs, ss, ps, Ls, Ws, Hs)),
                      np.full(n_agents, VEHICLE, np.uint8))
    return np.concatenate(tris), np.concatenate(clss), ag


# ----------------------------------------------------------------------------
# workloads
# ----------------------------------------------------------------------------

CONFIGS = {
    1: dict(name="tiny", seed=0, worlds=1, size=200.0, agents=8, cams=1, res=64, far=100.0, cell=16.0),
    2: dict(name="small_batch", seed=1, worlds=64, size=1000.0, agents=32, cams=4, res=64, far=100.0, cell=20.0),
    3: dict(name="dense_traffic", seed=2, worlds=256, size=1000.0, agents=128, cams=4, res=64, far=100.0, cell=20.0),
    4: dict(name="throughput_headline", seed=3, worlds=1024, size=1000.0, agents=64, cams=4, res=64, far=150.0, cell=30.0),
    5: dict(name="highres_large_scene", seed=4, worlds=128, size=4000.0, agents=64, cams=4, res=128, far=200.0, cell=16.0),
    # the paper's own rig and batch: 2048 egos x 4 views at 96x54 (App. A.2, Tab. camera_rig; Tab. render_mem)
    6: dict(name="paper_rig", seed=5, worlds=64, size=1000.0, agents=32, cams="paper", res=(96, 54), far=100.0, cell=16.0),
    # the paper's other rendering features (Sec. 3.2, Fig. qualitative): walls, parked cars, traffic lights
    7: dict(name="town_features", seed=6, worlds=64, size=1000.0, agents=32, cams="paper", res=(96, 54), far=100.0, cell=16.0),
}


# The paper's four-camera rig (App. A.2, Tab. camera_rig): a 1920x1080 sensor
# with a 1545 px focal length rendered at 96x54, so the focal length scales by
# 96 / 1920 to 77.25 px; per-camera extrinsics in the ego frame (x forward,
# y left, z up, metres; yaw about z, degrees).
PAPER_SENSOR = (1920, 1080, 1545.0)
PAPER_RENDER = (96, 54)
PAPER_MOUNTS = ((1.66, -0.01, 1.49, 0.0),     # front
                (1.63, 0.12, 1.48, 55.0),     # front-left
                (1.62, -0.16, 1.49, -55.0),   # front-right
                (-0.47, 0.02, 1.43, 180.0))   # back


def make_paper_rig(far: float = 100.0, near: float = 0.5) -> Rig:
    sw, sh, f = PAPER_SENSOR
    w, h = PAPER_RENDER
    fs = f * w / sw
    mounts = []
    for x, y, z, yaw in PAPER_MOUNTS:
        if yaw == 0.0:
            c, s = 1.0, 0.0
        elif yaw == 180.0:
            c, s = -1.0, 0.0
        else:
            c, s = float(np.cos(np.radians(yaw))), float(np.sin(np.radians(yaw)))
        mounts.append([x, y, z, c, s])
    return Rig(width=w, height=h, fx=fs, fy=fs, cx=w / 2.0, cy=h / 2.0, near=near, far=far,
               mount=np.asarray(mounts, np.float32))


def make_rig(num_cams: int, res: int, far: float, near: float = 0.5, cam_height: float = 1.5) -> Rig:
    """Square views with a 90 degree horizontal field of view: fx = fy = res/2."""
    mounts = []
    for k in range(num_cams):
        c, s = _AXIS_CS[k % 4]
        mounts.append([0.0, 0.0, cam_height, c, s])
    f = res / 2.0
    return Rig(width=res, height=res, fx=f, fy=f, cx=res / 2.0, cy=res / 2.0,
               near=near, far=far, mount=np.asarray(mounts, np.float32))


def _build_world(cfg_id: int, cfg: dict, w: int):
    rng = np.random.default_rng([cfg["seed"], w])
    size = cfg["size"]
    if cfg_id == 1:
        return _grid_world(rng, size, 10.0, 2, [2], 2.0, False, cfg["agents"], 8.0, 0.0, 0.0,
                           fixed_centres=[-50.0, 50.0])
    if cfg_id in (2, 4, 6):
        return _grid_world(rng, size, 25.0, 6, [2, 3, 4], ROAD_SEG, True, cfg["agents"], 8.0, 0.1, 0.0)
    if cfg_id == 3:
        return _grid_world(rng, size, 25.0, 6, [2, 3, 4], ROAD_SEG, True, cfg["agents"], 0.0, 0.1, 0.2)
    if cfg_id == 5:
        return _bezier_world(rng, size, 50.0, 500_000, cfg["agents"], 0.1)
    if cfg_id == 7:
        return _town_world(rng, size, cfg["agents"])
    raise ValueError(cfg_id)


def make_config(cfg_id: int, num_worlds: Optional[int] = None, init_speed_seed: bool = True) -> Workload:
    """Build workload `cfg_id` (1..7), optionally only its first `num_worlds` worlds."""
    cfg = CONFIGS[cfg_id]
    nw = cfg["worlds"] if num_worlds is None else int(num_worlds)
    A = cfg["agents"]
    verts, clss, offs = [], [], [0]
    ag_parts, light_parts = [], []
    for w in range(nw):
        built = _build_world(cfg_id, cfg, w)
        t, c, ag = built[:3]
        if len(built) > 3:
            light_parts.append(built[3])
        verts.append(t.reshape(-1, 9))
        clss.append(c)
        offs.append(offs[-1] + len(t))
        ag_parts.append(ag)
    size = cfg["size"]
    scene = Scene(num_worlds=nw,
                  verts=np.ascontiguousarray(np.concatenate(verts).astype(np.float32)),
                  cls=np.ascontiguousarray(np.concatenate(clss)),
                  tri_offsets=np.asarray(offs, np.int64),
                  bounds=np.tile(np.asarray([[-size / 2, -size / 2, size / 2, size / 2]], np.float32), (nw, 1)))

    def cat(f):
        return np.ascontiguousarray(np.concatenate([getattr(a, f) for a in ag_parts]).astype(np.float32))
    speed = np.zeros(nw * A, np.float32)
    if cfg_id == 4:
        srng = np.random.default_rng([cfg["seed"], 1 << 20])
        speed = srng.uniform(0.0, 15.0, size=nw * A).astype(np.float32)
    agents = Agents(num_worlds=nw, agents_per_world=A,
                    x=cat("x"), y=cat("y"), z0=cat("z0"), cos_h=cat("c"), sin_h=cat("s"),
                    length=cat("L"), width=cat("W"), height=cat("H"),
                    cls=np.ascontiguousarray(np.concatenate([a.cls for a in ag_parts])),
                    psi=cat("psi"), speed=speed)
    rig = make_paper_rig(cfg["far"]) if cfg["cams"] == "paper" else make_rig(cfg["cams"], cfg["res"], cfg["far"])
    lights = None
    if light_parts:
        nl = len(light_parts[0]["x"])
        assert all(len(lp["x"]) == nl for lp in light_parts)
        lcat = lambda f, dt=np.float32: np.ascontiguousarray(np.concatenate([lp[f] for lp in light_parts]).astype(dt))
        lights = Lights(num_worlds=nw, lights_per_world=nl, x=lcat("x"), y=lcat("y"), z=lcat("z"),
                        cos_f=lcat("cos_f"), sin_f=lcat("sin_f"), radius=lcat("radius"),
                        cls=lcat("cls", np.uint8), cos_max=LIGHT_COS_MAX)
    return Workload(name=cfg["name"], config=cfg_id, seed=cfg["seed"], scene=scene, agents=agents,
                    rig=rig, cell_size=cfg["cell"], world_size=size, lights=lights)


def controls(num_agents: int, steps: int, seed: int = 3):
    """Per-step random controls of the bicycle update: steer ~ U(-0.3, 0.3) rad,
    accel ~ U(-3, 2) m/s^2.  Returned as float32 [steps, num_agents] each."""
    rng = np.random.default_rng([seed, 1 << 21])
    steer = rng.uniform(-0.3, 0.3, size=(steps, num_agents)).astype(np.float32)
    accel = rng.uniform(-3.0, 2.0, size=(steps, num_agents)).astype(np.float32)
    return steer, accel
