"""Oracle pins for traffic lights: the visibility cone (R10) and the disk (R11).

The paper draws traffic lights as disks visible only within a limited angular
range of the approach they govern (Sec. 3.2, rendering features).  These
tests pin the oracle's reading against closed forms and an independent fp64
ray cast; none of them re-types the oracle's arithmetic.
"""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2607_26005_amd.scenegen import Lights
from tests import raycast as RC
from tests.scenes import make_agents, make_rig, make_scene

RED, GREEN = 8, 10


def lights_of(rows, cos_max=0.5, num_worlds=1):
    """rows: (x, y, z, cos_f, sin_f, radius, cls) per light."""
    a = np.asarray([r[:6] for r in rows], np.float64)
    f = lambda k: np.ascontiguousarray(a[:, k].astype(np.float32))
    return Lights(num_worlds=num_worlds, lights_per_world=len(rows) // num_worlds, x=f(0), y=f(1), z=f(2),
                  cos_f=f(3), sin_f=f(4), radius=f(5), cls=np.asarray([r[6] for r in rows], np.uint8),
                  cos_max=cos_max)


def empty_scene():
    return make_scene(np.zeros((0, 3, 3)), np.zeros(0))


def ego(x=0.0, y=0.0, c=1.0, s=0.0):
    return make_agents([(x, y, 0.0, c, s, 4.5, 1.9, 1.5, 3)])


def polygon_inside(px, py, vx, vy):
    """Strictly inside a convex polygon (vertices counter-clockwise in x-right,
    y-up coordinates) and the distance to its boundary, in fp64."""
    n = len(vx)
    inside = np.ones(px.shape, bool)
    dist = np.full(px.shape, np.inf)
    for k in range(n):
        ax, ay, bx, by = vx[k], vy[k], vx[(k + 1) % n], vy[(k + 1) % n]
        ex, ey = bx - ax, by - ay
        cr = ex * (py - ay) - ey * (px - ax)
        inside &= cr > 0
        dist = np.minimum(dist, np.abs(cr) / np.hypot(ex, ey))
    return inside, dist


@pytest.mark.parametrize("D,r", [(10.0, 2.0), (7.0, 1.3), (25.0, 3.1)])
def test_head_on_disk_is_a_regular_12gon(D, r):
    # camera at the origin looking along +x; the light faces it from distance D on the optical axis
    rig = make_rig()
    L = lights_of([(D, 0.0, 0.0, -1.0, 0.0, r, GREEN)])
    out = O.render(empty_scene(), ego(), rig, lights=L)
    cls, dep = out["cls"][0], out["depth"][0]
    # exact image of the disk: vertex k at angle 30k degrees, radius r f / D pixels around the centre
    R = r * rig.fx / D
    ang = np.radians(30.0 * np.arange(12))
    vx, vy = R * np.cos(ang), R * np.sin(ang)
    jj, ii = np.meshgrid(np.arange(64), np.arange(64), indexing="ij")
    px = ii + 0.5 - rig.cx
    py = rig.cy - (jj + 0.5)
    inside, dist = polygon_inside(px, py, vx, vy)
    sure = dist > 1e-3
    assert sure.sum() > 4000
    assert np.array_equal((cls == GREEN)[sure], inside[sure])
    assert (cls[~inside & sure] == 4).all()
    assert np.all(np.abs(dep[cls == GREEN] / D - 1.0) <= 2.0 ** -20)
    # about the polygon's area, 3 R^2 pixels
    assert abs((cls == GREEN).sum() - 3.0 * R * R) <= 2.0 * 12 * R * np.sin(np.pi / 12) + 4


@pytest.mark.parametrize("theta,seen", [(0, True), (30, True), (55, True), (59, True), (61, False), (75, False),
                                        (90, False), (135, False), (180, False)])
def test_visibility_cone_half_angle(theta, seen):
    # light at the origin facing +x; the camera circles it at 10 m and looks at it
    t = np.radians(theta)
    c, s = np.float32(np.cos(t)), np.float32(np.sin(t))
    L = lights_of([(0.0, 0.0, 0.0, 1.0, 0.0, 1.5, RED)], cos_max=0.5)
    rig = make_rig(f=16.0)   # wide enough to hold the disk at every angle
    out = O.render(empty_scene(), ego(10.0 * float(c), 10.0 * float(s), -float(c), -float(s)), rig, lights=L)
    n = int((out["cls"][0] == RED).sum())
    assert (n > 0) == seen, (theta, n)


def test_cone_is_three_dimensional():
    # from straight above the light's normal the camera is outside a 60 degree cone
    L = lights_of([(0.0, 0.0, 0.0, 1.0, 0.0, 1.5, RED)], cos_max=0.5)
    rig = make_rig(f=16.0, mounts=((0.0, 0.0, 0.0, 1.0, 0.0),))
    near = ego(10.0, 0.0, -1.0, 0.0)
    assert (O.render(empty_scene(), near, rig, lights=L)["cls"][0] == RED).any()
    # same horizontal offset, camera raised so that the elevation exceeds 60 degrees: invisible
    hi = make_agents([(10.0, 0.0, 20.0, -1.0, 0.0, 4.5, 1.9, 1.5, 3)])
    rig_down = make_rig(f=8.0)
    assert not (O.render(empty_scene(), hi, rig_down, lights=L)["cls"][0] == RED).any()
    # raised less (elevation 45 degrees): visible in a wide view
    mid = make_agents([(10.0, 0.0, 10.0, -1.0, 0.0, 4.5, 1.9, 1.5, 3)])
    assert (O.render(empty_scene(), mid, rig_down, lights=L)["cls"][0] == RED).any()


def test_light_occludes_and_is_occluded():
    # a wall quad between camera and light hides it; a light in front of the wall covers it
    wall = [[(8.0, -5.0, -5.0), (8.0, 5.0, -5.0), (8.0, 5.0, 5.0)], [(8.0, -5.0, -5.0), (8.0, 5.0, 5.0), (8.0, -5.0, 5.0)]]
    sc = make_scene(wall, [7, 7])
    rig = make_rig()
    behind = lights_of([(12.0, 0.0, 0.0, -1.0, 0.0, 1.0, RED)])
    assert not (O.render(sc, ego(), rig, lights=behind)["cls"][0] == RED).any()
    front = lights_of([(6.0, 0.0, 0.0, -1.0, 0.0, 1.0, RED)])
    o = O.render(sc, ego(), rig, lights=front)
    assert (o["cls"][0] == RED).sum() > 50
    assert np.all(np.abs(o["depth"][0][o["cls"][0] == RED] / 6.0 - 1.0) <= 2.0 ** -20)


def _disk_tris64(x, y, z, cf, sf, r):
    ang = np.radians(30.0 * np.arange(13))
    a, b = r * np.cos(ang), r * np.sin(ang)
    rim = np.stack([x - a * sf, y + a * cf, z + b], 1)
    c = np.array([x, y, z])
    return np.stack([np.broadcast_to(c, (12, 3)), rim[:12], rim[1:13]], 1)


@pytest.mark.parametrize("seed", range(6))
def test_against_float64_raycast_with_lights(seed):
    rng = np.random.default_rng([77, seed])
    rig = make_rig(res=32, f=16.0, mounts=((0.0, 0.0, 1.5, 1.0, 0.0),))
    ag = ego()
    # a ground plane and a few random lights in front of the camera
    g = [[(-50.0, -50.0, 0.0), (100.0, -50.0, 0.0), (100.0, 50.0, 0.0)],
         [(-50.0, -50.0, 0.0), (100.0, 50.0, 0.0), (-50.0, 50.0, 0.0)]]
    rows = []
    for k in range(5):
        ang = rng.uniform(-np.pi, np.pi)
        rows.append((rng.uniform(4.0, 20.0), rng.uniform(-8.0, 8.0), rng.uniform(0.5, 4.0),
                     float(np.float32(np.cos(ang))), float(np.float32(np.sin(ang))), rng.uniform(0.5, 1.5),
                     8 + k % 3))
    L = lights_of(rows, cos_max=0.3)
    out = O.render(make_scene(g, [0, 0]), ag, rig, lights=L)
    # fp64 reading of R10 and R11 for the ray cast
    C = np.array([0.0, 0.0, 1.5])
    tris, cls = [np.asarray(g, np.float64)], [np.zeros(2, np.int64)]
    for (x, y, z, cf, sf, r, k) in rows:
        x, y, z, r = (float(np.float32(v)) for v in (x, y, z, r))
        d = C - np.array([x, y, z])
        h = cf * d[0] + sf * d[1]
        q = d @ d
        m = np.float32(0.3) ** 2
        if abs(h * h - m * q) <= 1e-6 * q:
            pytest.skip("camera on the cone boundary")
        if h > 0 and h * h >= m * q:
            tris.append(_disk_tris64(x, y, z, cf, sf, r))
            cls.append(np.full(12, k, np.int64))
    T = np.concatenate(tris)
    sc64 = make_scene(T.astype(np.float32), np.concatenate(cls))
    rc, rd, unsure = RC.raycast_view(sc64, make_agents([(0.0, 0.0, 0.0, 1.0, 0.0, 4.5, 1.9, 1.5, 3)]), rig, 0)
    ok = ~unsure
    assert ok.mean() > 0.8
    assert np.array_equal(out["cls"][0][ok], rc[ok])
    fin = ok & np.isfinite(rd)
    assert np.all(np.abs(out["depth"][0][fin] / rd[fin] - 1.0) <= 4e-6)


@pytest.mark.parametrize("dx,dy", [(1, 0), (-1, 0), (0, 1), (0, -1)])
def test_stop_line_before_the_junction_and_head_beyond_it(dx, dy):
    # the scene generator's signal layout: the head hangs beyond the crossing on the
    # right-hand side, the stop line it governs lies across the right-hand lanes before it
    from paper_2607_26005_amd.scenegen import light_and_stop_line, Z_MARK
    cx, cy, hwc, hwo = 10.0, -20.0, 5.25, 3.5
    (hx, hy), bar = light_and_stop_line(cx, cy, dx, dy, hwc, hwo)
    along = lambda x, y: (x - cx) * dx + (y - cy) * dy
    right = lambda x, y: (x - cx) * dy - (y - cy) * dx
    assert along(hx, hy) > hwc and right(hx, hy) > hwo
    assert bar.shape == (2, 3, 3) and np.all(bar[..., 2] == Z_MARK)
    pa, pr = along(bar[..., 0], bar[..., 1]), right(bar[..., 0], bar[..., 1])
    assert np.all(pa < -hwc) and np.all(pa >= -hwc - 1.5)
    assert pr.min() == pytest.approx(0.0) and pr.max() == pytest.approx(hwo)
    # the two triangles tile the bar: their areas add up to its width times the half road
    e1, e2 = bar[:, 1, :2] - bar[:, 0, :2], bar[:, 2, :2] - bar[:, 0, :2]
    area = 0.5 * np.abs(e1[:, 0] * e2[:, 1] - e1[:, 1] * e2[:, 0])
    assert area.sum() == pytest.approx(0.4 * hwo)


def test_approaching_camera_sees_the_stop_line_near_and_its_signal_far():
    # a camera 12 m before a crossing, on the right-hand lane, looking along the road:
    # the stop line is drawn before the crossing road's edge, the red head beyond it
    from paper_2607_26005_amd.scenegen import light_and_stop_line, LIGHT_Z, LIGHT_R
    hwc, hwo = 5.25, 3.5
    (hx, hy), bar = light_and_stop_line(0.0, 0.0, 1, 0, hwc, hwo)
    L = lights_of([(hx, hy, LIGHT_Z, -1.0, 0.0, LIGHT_R, RED)])
    rig = make_rig(res=256, f=256.0, mounts=((0.0, 0.0, 1.5, 1.0, 0.0),))    # camera 1.5 m above the road
    out = O.render(make_scene(bar, [2, 2]), ego(-12.0, -1.75), rig, lights=L)
    cls, dep = out["cls"][0], out["depth"][0]
    mark, red = cls == 2, cls == RED
    assert mark.sum() > 100 and red.sum() > 20
    assert dep[mark].max() < 12.0 - hwc < 12.0 < 12.0 + hx == pytest.approx(dep[red].min())
    rows_m, rows_r = np.nonzero(mark)[0], np.nonzero(red)[0]
    assert rows_r.max() < 128 < rows_m.min()          # the head above the horizon, the bar below it
    assert np.nonzero(red)[1].min() > 128             # the head on the right-hand side
