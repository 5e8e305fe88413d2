"""Pins of the CPU oracle against facts that do not come from the oracle.

Each test checks the oracle against a closed form, an invariant, a special
case that reduces to textbook geometry, or an independent float64 ray
caster, chosen so that a plausible slip (a dropped term, a wrong sign or
index, a transposed operand, a wrong fill-rule case) fails at least one.
"""
import numpy as np
import pytest

from oracle import oracle as O
from tests.raycast import raycast_view
from tests.scenes import make_agents, make_rig, make_scene, quad

SKY = 4


def ego(x=0.0, y=0.0, z0=0.0, c=1.0, s=0.0):
    return (x, y, z0, c, s, 1.0, 1.0, 1.0, 3)


def fronto_quad(D, s, h=0.0, cls=7, axis=0, sign=1.0, centre=(0.0, 0.0)):
    """Square of half-size s facing the camera at distance D along +x (axis 0)
    or +y (axis 1) from `centre`, centred at height h."""
    cx_, cy_ = centre
    pts = []
    for (a, b) in ((-s, -s), (s, -s), (s, s), (-s, s)):
        if axis == 0:
            pts.append((cx_ + sign * D, cy_ + a, h + b))
        else:
            pts.append((cx_ + a, cy_ + sign * D, h + b))
    return quad(*pts)


# ---------------------------------------------------------------------------
# P1: an axis-aligned quad at a known distance covers a known pixel set
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("s,cols", [(1.875, range(24, 39)), (2.0, range(24, 40)), (1.0, range(28, 36)),
                                    (1.87451171875, range(24, 39)), (1.87548828125, range(24, 39))])
def test_fronto_quad_pixel_set_and_depth(s, cols):
    # D = 8, fx = 32: edges project to 32 +- 32*s/8 px.  For s = 1.875 they run
    # exactly through pixel centres 24.5 and 39.5: the left/top edges include
    # them, the right/bottom edges exclude them (top-left rule).
    # The last two sizes put the edges half a subpixel off those centres (256 x
    # = 6272.5 and 10111.5, then 6271.5 and 10112.5): the 8-bit snap rounds the
    # ties to even, onto the centres, which gives the same pixel set; rounding
    # ties upwards (or away from zero) would drop column and row 24 in the first
    # case and add column and row 39 in the second.
    scene = make_scene(fronto_quad(8.0, s), [7, 7])
    r = O.render(scene, make_agents([ego()]), make_rig(), want_cover=True)
    cls, depth, cover = r["cls"][0], r["depth"][0], r["cover"][0]
    want = np.zeros((64, 64), bool)
    want[np.ix_(list(cols), list(cols))] = True
    assert np.array_equal(cls == 7, want)
    assert np.all(cls[~want] == SKY) and np.all(np.isinf(depth[~want]))
    assert np.allclose(depth[want], 8.0, rtol=2 ** -20, atol=0)
    # the shared diagonal passes through pixel centres: each is covered once
    assert np.all(cover[want] == 1) and np.all(cover[~want] == 0)


def test_fronto_quad_rotated_camera_and_mount():
    # Same quad seen by an agent heading +y whose camera sits 1 m ahead of it:
    # exercises the heading rotation and the mount offset of the camera build.
    scene = make_scene(fronto_quad(8.0, 1.875, axis=1, centre=(3.0, 1.0)), [7, 7])
    ag = make_agents([(3.0, 0.0, 0.0, 0.0, 1.0, 1.0, 1.0, 1.0, 3)])
    rig = make_rig(mounts=((1.0, 0.0, 0.0, 1.0, 0.0),))
    r = O.render(scene, ag, rig)
    want = np.zeros((64, 64), bool)
    want[24:39, 24:39] = True
    assert np.array_equal(r["cls"][0] == 7, want)
    assert np.allclose(r["depth"][0][want], 8.0, rtol=2 ** -20)


def test_anisotropic_intrinsics():
    # fx = 32, fy = 16 on a 64x48 image (cx = 32, cy = 24): the square's
    # edges project to 32 -+ 7.5 px across and 24 -+ 3.75 px down, so it
    # covers columns 24..38 and rows 20..27 (centres 20.5 .. 27.5).
    from paper_2607_26005_amd.scenegen import Rig
    scene = make_scene(fronto_quad(8.0, 1.875), [7, 7])
    rig = Rig(width=64, height=48, fx=32.0, fy=16.0, cx=32.0, cy=24.0, near=0.5, far=100.0,
              mount=np.asarray([(0.0, 0.0, 0.0, 1.0, 0.0)], np.float32))
    r = O.render(scene, make_agents([ego()]), rig)
    want = np.zeros((48, 64), bool)
    want[20:28, 24:39] = True
    assert np.array_equal(r["cls"][0] == 7, want)
    assert np.allclose(r["depth"][0][want], 8.0, rtol=2 ** -20)


@pytest.mark.parametrize("heading,yaw,axis,sign", [((1.0, 0.0), (0.0, 1.0), 1, 1.0),    # 0 + 90 deg: faces +y
                                                    ((0.0, 1.0), (0.0, 1.0), 0, -1.0),   # 90 + 90 deg: faces -x
                                                    ((0.0, 1.0), (-1.0, 0.0), 1, -1.0)])  # 90 + 180 deg: faces -y
def test_mount_yaw_composes_with_heading(heading, yaw, axis, sign):
    # Camera heading = agent heading + mount yaw (cosines and sines in {0, +-1},
    # exact in fp32).  The square 8 m along the composed direction, shifted 2 m
    # to that camera's left, covers columns 16..30; straight behind it nothing.
    (c, s_), (cm, sm) = heading, yaw
    fx_, fy_ = c * cm - s_ * sm, s_ * cm + c * sm           # forward of the composed heading
    lx, ly = -fy_, fx_                                      # its left
    centre = (2.0 * lx, 2.0 * ly)
    scene = make_scene(fronto_quad(8.0, 1.875, axis=axis, sign=sign, centre=centre) +
                       fronto_quad(8.0, 1.875, axis=axis, sign=-sign), [7, 7, 5, 5])
    ag = make_agents([(0.0, 0.0, 0.0, c, s_, 1.0, 1.0, 1.0, 3)])
    rig = make_rig(mounts=((0.0, 0.0, 0.0, cm, sm),))
    r = O.render(scene, ag, rig)
    want = np.zeros((64, 64), bool)
    want[24:39, 16:31] = True
    assert np.array_equal(r["cls"][0] == 7, want)
    assert np.all(r["cls"][0][~want] == SKY)


def test_mount_offset_rotates_with_heading():
    # Agent at (5, -3) heading +y (cos 0, sin 1) with its camera mounted 1 m
    # ahead and 2 m to the left: the camera sits at (5 - 2, -3 + 1) and faces
    # +y; a square 8 m ahead of that point fills columns and rows 24..38.
    scene = make_scene(fronto_quad(8.0, 1.875, axis=1, centre=(3.0, -2.0)), [7, 7])
    ag = make_agents([(5.0, -3.0, 0.0, 0.0, 1.0, 1.0, 1.0, 1.0, 3)])
    rig = make_rig(mounts=((1.0, 2.0, 0.0, 1.0, 0.0),))
    r = O.render(scene, ag, rig)
    want = np.zeros((64, 64), bool)
    want[24:39, 24:39] = True
    assert np.array_equal(r["cls"][0] == 7, want)
    assert np.allclose(r["depth"][0][want], 8.0, rtol=2 ** -20)


def test_far_plane_is_inclusive():
    # far = 64: a square exactly 64 m away (half-size 16, so 1/z = 1/64 is
    # exact at every pixel) is drawn, columns and rows 24..39, depth 64; the
    # same square a little farther is not.
    rig = make_rig(far=64.0)
    r = O.render(make_scene(fronto_quad(64.0, 16.0), [7, 7]), make_agents([ego()]), rig)
    want = np.zeros((64, 64), bool)
    want[24:40, 24:40] = True
    assert np.array_equal(r["cls"][0] == 7, want)
    assert np.allclose(r["depth"][0][want], 64.0, rtol=2 ** -20)
    r2 = O.render(make_scene(fronto_quad(64.0625, 16.0), [7, 7]), make_agents([ego()]), rig)
    assert np.all(r2["cls"][0] == SKY)


def test_triangle_wholly_beyond_far_is_not_drawn():
    # far = 110 and a fronto square (half-size 16) one fp32 step beyond it,
    # D = 110 + 2^-17.  Every point of the surface lies beyond the far plane, so
    # it appears in no pixel: the float64 ray cast finds nothing within
    # [near, far].  The per-pixel test alone cannot decide this case: the
    # square's plane gives 1/z = fl(1/D) at every covered centre (its normal
    # has power-of-two length and no x or y term), and fl(1/D) equals
    # fl(1/110), which passes iz >= fl(1/far).  The triangle-level rule of R4
    # (every vertex at zv > far: not drawn) is what keeps the image empty;
    # without it the square shows as a 10 x 10 block at depth 110.
    far = 110.0
    D = float(np.nextafter(np.float32(far), np.float32(np.inf)))
    assert D > far and np.float32(1) / np.float32(D) == np.float32(1) / np.float32(far)
    rig = make_rig(far=far)
    scene = make_scene(fronto_quad(D, 16.0), [7, 7])
    ag = make_agents([ego()])
    r = O.render(scene, ag, rig)
    assert np.all(r["cls"][0] == SKY) and np.all(np.isinf(r["depth"][0]))
    rc, rd, _ = raycast_view(scene, ag, rig, 0)
    assert np.all(rc == SKY) and not np.isfinite(rd).any()
    # the same square on the far plane itself is drawn (inclusive far plane):
    # the 10 x 10 pixel centres within 32 +- 32 * 16 / 110 = 32 +- 4.65 px
    r2 = O.render(make_scene(fronto_quad(far, 16.0), [7, 7]), ag, rig)
    want = np.zeros((64, 64), bool)
    want[27:37, 27:37] = True
    assert np.array_equal(r2["cls"][0] == 7, want)


def _pair_with_unsnappable_vertex():
    """Pair (a, b, c), (a, c, d) at 16 m (f = 64: column 32 - 4 y, row 32 - 4 z)
    whose vertex d sits just past the near plane 40 km to the side: it
    projects 64 * 40000 / 0.5625 ~ 4.6e6 px from the centre, beyond the 2^21
    px (2^29 subpixel) range of R5."""
    a, b, c = (16.0, 6.0, 6.0), (16.0, -2.0, 6.0), (16.0, -2.0, -2.0)   # columns/rows 8 and 40
    d = (0.5625, 40000.0, 0.0)
    assert 64.0 * 40000.0 / 0.5625 > 2.0 ** 21
    return [[a, b, c], [a, c, d]], [a, b, c]


def test_vertex_out_of_snap_range_drops_only_its_triangles():
    # R5 drops the triangles that use the vertex, not the whole pair: the
    # image is that of (a, b, c) alone, which the float64 ray cast confirms
    pair, first = _pair_with_unsnappable_vertex()
    ag = make_agents([ego()])
    rig = make_rig(res=64, f=64.0)
    r = O.render(make_scene(np.asarray(pair, np.float32), [7, 7]), ag, rig, want_rgb=True, antialias=True)
    alone = make_scene(np.asarray([first], np.float32), [7])
    r1 = O.render(alone, ag, rig, want_rgb=True, antialias=True)
    assert (r["cls"][0] == 7).sum() > 400
    assert np.array_equal(r["cls"], r1["cls"]) and np.array_equal(r["depth"], r1["depth"])
    assert np.array_equal(r["rgb"], r1["rgb"])
    rc, _, _ = raycast_view(alone, ag, rig, 0)
    assert ((r["cls"][0] == 7) != (rc == 7)).sum() <= 40   # only on the triangle's edges


def test_vertex_inside_snap_range_is_kept():
    # the same pair with d at 13 km to the side projects 64 * 13000 / 0.5625 ~
    # 1.48e6 px from the centre: past 2^20 px but within R5's 2^21 px (2^29
    # subpixels), so both triangles are drawn, as the float64 ray cast of the
    # whole pair confirms pixel for pixel
    pair, first = _pair_with_unsnappable_vertex()
    d = (0.5625, 13000.0, 0.0)
    assert 2.0 ** 20 < 64.0 * 13000.0 / 0.5625 < 2.0 ** 21
    pair = [pair[0], [pair[1][0], pair[1][1], d]]
    ag = make_agents([ego()])
    rig = make_rig(res=64, f=64.0)
    sc = make_scene(np.asarray(pair, np.float32), [7, 7])
    r = O.render(sc, ag, rig)
    r1 = O.render(make_scene(np.asarray([first], np.float32), [7]), ag, rig)
    rc, _, _ = raycast_view(sc, ag, rig, 0)
    assert (r["cls"][0] == 7).sum() > 2 * (r1["cls"][0] == 7).sum()
    assert ((r["cls"][0] == 7) != (rc == 7)).sum() == 0


def test_depth_error_bound_over_distances():
    # Fronto squares (half-size D/16, 2 px) at 200 seeded distances D in [0.6, 95] m: the decoded depth
    # at the image centre is within 2^-21 (the bucket midpoint) plus a few
    # roundings of the plane (6.5 ulps in all) of the true distance.
    rng = np.random.default_rng(11)
    D = np.sort(rng.uniform(0.6, 95.0, 200)).astype(np.float32)
    tris, cls = [], []
    ags = []
    for k, d in enumerate(D):
        tris += fronto_quad(float(d), float(d) / 16.0, centre=(0.0, 1000.0 * k))
        cls += [7, 7]
        ags.append((0.0, 1000.0 * k, 0.0, 1.0, 0.0, 1.0, 1.0, 1.0, 3))
    # one world per square, so no square sees another
    T = len(tris) // len(D)
    tv = np.asarray(tris, np.float32).reshape(len(D), T, 9)
    from paper_2607_26005_amd.scenegen import Scene
    scene = Scene(num_worlds=len(D), verts=np.ascontiguousarray(tv.reshape(-1, 9)), cls=np.asarray(cls, np.uint8),
                  tri_offsets=np.arange(len(D) + 1, dtype=np.int64) * T,
                  bounds=np.asarray([(-1000.0, 1000.0 * k - 500.0, 1000.0, 1000.0 * k + 500.0) for k in range(len(D))],
                                    np.float32))
    r = O.render(scene, make_agents(ags, num_worlds=len(D)), make_rig())
    z = r["depth"][:, 32, 32].astype(np.float64)
    assert np.all(r["cls"][:, 32, 32] == 7)
    rel = np.abs(z - D.astype(np.float64)) / D
    assert rel.max() <= 6.5 * 2.0 ** -23, rel.max()


def test_offcentre_quad_columns():
    # Quad shifted 2 m to the left (+y): it moves 8 px left on screen.
    scene = make_scene(fronto_quad(8.0, 1.875, centre=(0.0, 2.0)), [7, 7])
    r = O.render(scene, make_agents([ego()]), make_rig())
    want = np.zeros((64, 64), bool)
    want[24:39, 16:31] = True
    assert np.array_equal(r["cls"][0] == 7, want)


def test_quad_raised_rows():
    # Quad raised by 1 m: it moves 4 px up (y grows downwards).
    scene = make_scene(fronto_quad(8.0, 1.875, h=1.0), [7, 7])
    r = O.render(scene, make_agents([ego()]), make_rig())
    want = np.zeros((64, 64), bool)
    want[20:35, 24:39] = True
    assert np.array_equal(r["cls"][0] == 7, want)


# ---------------------------------------------------------------------------
# P2: facing away / beyond far / behind near gives an empty image
# ---------------------------------------------------------------------------

def test_facing_away_is_empty():
    scene = make_scene(fronto_quad(8.0, 2.0), [7, 7])
    r = O.render(scene, make_agents([ego(c=-1.0, s=0.0)]), make_rig())
    assert np.all(r["cls"][0] == SKY) and np.all(np.isinf(r["depth"][0]))


def test_beyond_far_is_empty_and_inside_far_is_not():
    scene = make_scene(fronto_quad(50.0, 20.0), [7, 7])
    r = O.render(scene, make_agents([ego()]), make_rig(far=49.0))
    assert np.all(r["cls"][0] == SKY)
    r = O.render(scene, make_agents([ego()]), make_rig(far=51.0))
    assert np.sum(r["cls"][0] == 7) > 0


def test_closer_than_near_is_clipped():
    scene = make_scene(fronto_quad(0.4, 0.1), [7, 7])
    r = O.render(scene, make_agents([ego()]), make_rig(near=0.5))
    assert np.all(r["cls"][0] == SKY)


# ---------------------------------------------------------------------------
# P3: ground plane closed form (near clip, huge triangles, far test)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("yaw", [0, 1, 2, 3])
@pytest.mark.parametrize("far", [100.0, 90.0])
def test_ground_plane_rows(yaw, far):
    cs = [(1.0, 0.0), (0.0, 1.0), (-1.0, 0.0), (0.0, -1.0)][yaw]
    G = 1000.0
    scene = make_scene(quad((-G, -G, 0.0), (G, -G, 0.0), (G, G, 0.0), (-G, G, 0.0)), [0, 0])
    ag = make_agents([(12.25, -7.5, 0.0, cs[0], cs[1], 1.0, 1.0, 1.0, 3)])
    rig = make_rig(mounts=((0.0, 0.0, 1.5, 1.0, 0.0),), far=far)
    r = O.render(scene, ag, rig, want_cover=True)
    cls, depth, cover = r["cls"][0], r["depth"][0], r["cover"][0]
    j = np.arange(64)
    z = np.where(j + 0.5 - 32 > 0, 1.5 * 32 / np.maximum(j + 0.5 - 32, 1e-9), np.inf)
    ground_rows = (j + 0.5 - 32 > 0) & (z <= far)
    for jj in range(64):
        if ground_rows[jj]:
            assert np.all(cls[jj] == 0), jj
            assert np.allclose(depth[jj], z[jj], rtol=1e-5, atol=0), (jj, depth[jj][:3], z[jj])
            assert np.all(cover[jj] == 1)
        else:
            assert np.all(cls[jj] == SKY), jj
    assert ground_rows.sum() == (32 if far == 100.0 else 31)


def test_ground_mesh_watertight_with_near_clip():
    # P5: a jittered, irregularly split ground mesh whose triangles cross the
    # near plane: every pixel of the ground region is covered exactly once.
    rng = np.random.default_rng(5)
    n = 24
    xs = np.linspace(-30, 60, n + 1)
    ys = np.linspace(-45, 45, n + 1)
    X, Y = np.meshgrid(xs, ys, indexing="ij")
    X = X + rng.uniform(-1.2, 1.2, X.shape)
    Y = Y + rng.uniform(-1.2, 1.2, Y.shape)
    P = np.stack([X, Y, np.zeros_like(X)], -1)
    tris = []
    for i in range(n):
        for k in range(n):
            a, b, c, d = P[i, k], P[i + 1, k], P[i + 1, k + 1], P[i, k + 1]
            if rng.random() < 0.5:
                tris += [[a, b, c], [a, c, d]]
            else:
                tris += [[a, b, d], [b, c, d]]
    scene = make_scene(tris, np.zeros(len(tris)))
    ag = make_agents([(0.3, 0.1, 0.0, 0.8, 0.6, 1.0, 1.0, 1.0, 3)])
    rig = make_rig(mounts=((0.0, 0.0, 1.5, 1.0, 0.0),), far=200.0)
    r = O.render(scene, ag, rig, want_cover=True)
    cover, cls = r["cover"][0], r["cls"][0]
    lower = np.zeros((64, 64), bool)
    lower[40:] = True  # z <= 1.5*32/8.5 < 6 m: well inside the mesh
    assert np.all(cover[lower] == 1)
    assert np.all(cover <= 1)
    assert np.all((cover == 1) == (cls == 0))


def test_vertical_mesh_watertight():
    # P5 on a fronto-parallel mesh with random diagonals and jittered vertices.
    rng = np.random.default_rng(6)
    n = 10
    ys = np.linspace(-12, 12, n + 1)
    zs = np.linspace(-12, 12, n + 1)
    Y, Z = np.meshgrid(ys, zs, indexing="ij")
    Y = Y + rng.uniform(-0.7, 0.7, Y.shape)
    Z = Z + rng.uniform(-0.7, 0.7, Z.shape)
    Xd = 6.0 + rng.uniform(-0.5, 0.5, Y.shape)
    P = np.stack([Xd, Y, Z], -1)
    tris = []
    for i in range(n):
        for k in range(n):
            a, b, c, d = P[i, k], P[i + 1, k], P[i + 1, k + 1], P[i, k + 1]
            tris += [[a, b, c], [a, c, d]] if rng.random() < 0.5 else [[a, b, d], [b, c, d]]
    scene = make_scene(tris, np.full(len(tris), 2))
    r = O.render(scene, make_agents([ego()]), make_rig(), want_cover=True)
    assert np.all(r["cover"][0] == 1)


# ---------------------------------------------------------------------------
# boxes and ego exclusion
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("turn", [0, 1])
def test_box_face_closed_form(turn):
    # A 4 x 2 x 1.5 box whose near face is at x = 10; camera at height 0.75.
    # Near face: y in [-1, 1] -> x_px in (28.8, 35.2) -> columns 29..34;
    # z in [0, 1.5] -> y_px in (29.6, 34.4) -> rows 30..33; depth 10.
    # turn = 1 builds the same box with heading +y and swapped L/W.
    if turn == 0:
        other = (12.0, 0.0, 0.0, 1.0, 0.0, 4.0, 2.0, 1.5, 3)
    else:
        other = (12.0, 0.0, 0.0, 0.0, 1.0, 2.0, 4.0, 1.5, 3)
    ag = make_agents([ego(), other])
    rig = make_rig(mounts=((0.0, 0.0, 0.75, 1.0, 0.0),))
    scene = make_scene(np.zeros((0, 3, 3)), np.zeros(0))
    r = O.render(scene, ag, rig, view_ids=[0])
    want = np.zeros((64, 64), bool)
    want[30:34, 29:35] = True
    assert np.array_equal(r["cls"][0] == 3, want)
    assert np.allclose(r["depth"][0][want], 10.0, rtol=2 ** -20)


def test_ego_box_excluded_other_drawn():
    # Two agents facing each other 20 m apart: each sees the other's box, never its own.
    a0 = (0.0, 0.0, 0.0, 1.0, 0.0, 4.5, 1.9, 1.5, 3)
    a1 = (20.0, 0.0, 0.0, -1.0, 0.0, 4.5, 1.9, 1.5, 6)
    ag = make_agents([a0, a1])
    rig = make_rig(mounts=((0.0, 0.0, 1.0, 1.0, 0.0),))
    scene = make_scene(np.zeros((0, 3, 3)), np.zeros(0))
    r = O.render(scene, ag, rig)
    assert set(np.unique(r["cls"][0])) == {6, SKY}
    assert set(np.unique(r["cls"][1])) == {3, SKY}
    # the visible face is at 20 - 2.25 = 17.75 m
    assert np.allclose(r["depth"][0][r["cls"][0] == 6], 17.75, rtol=2 ** -20)


def test_depth_tie_goes_to_lower_class():
    # Two coincident quads of classes 5 and 2: the lower class wins everywhere,
    # whatever the triangle order, and the oracle flags the pixels as TIE.
    for order in ([5, 5, 2, 2], [2, 2, 5, 5]):
        q = fronto_quad(8.0, 2.0)
        scene = make_scene(q + q, order)
        r = O.render(scene, make_agents([ego()]), make_rig())
        m = r["cls"][0] != SKY
        assert np.all(r["cls"][0][m] == 2)
        assert np.all(r["flags"][0][m] & 2)


def test_permutation_and_duplication_invariance():
    rng = np.random.default_rng(11)
    tris = rng.uniform(-3, 3, size=(40, 3, 3)) + np.array([10.0, 0.0, 0.0])
    cls = rng.integers(0, 7, 40)
    cls[cls == SKY] = 0
    ag = make_agents([ego()])
    base = O.render(make_scene(tris, cls), ag, make_rig())
    perm = rng.permutation(40)
    t2 = np.concatenate([tris[perm], tris[:7]])
    c2 = np.concatenate([cls[perm], cls[:7]])
    other = O.render(make_scene(t2, c2), ag, make_rig())
    assert np.array_equal(base["cls"], other["cls"])
    assert np.array_equal(base["depth"], other["depth"])


# ---------------------------------------------------------------------------
# P4: brute-force float64 ray cast on small random scenes
# ---------------------------------------------------------------------------

def _random_scene(seed):
    rng = np.random.default_rng(seed)
    ang = rng.uniform(-np.pi, np.pi)
    cx_, cy_ = rng.uniform(-50, 50, 2)
    c, s = np.cos(ang), np.sin(ang)
    fwd = np.array([c, s, 0.0])
    left = np.array([-s, c, 0.0])
    tris = []
    n = int(rng.integers(10, 48))
    for _ in range(n):
        d = rng.uniform(0.2, 25.0)
        lat = rng.uniform(-1.2, 1.2) * d
        h = rng.uniform(-1.0, 1.0) * d * 0.8
        centre = np.array([cx_, cy_, 1.0]) + d * fwd + lat * left + np.array([0, 0, h])
        size = rng.uniform(0.2, 8.0)
        tris.append(centre + rng.normal(size=(3, 3)) * size)
    cls = rng.integers(0, 7, n)
    cls[cls == SKY] = 1
    # two other agents ahead
    rows = [(cx_, cy_, 0.0, c, s, 4.5, 1.9, 1.5, 3)]
    for _ in range(2):
        d = rng.uniform(4.0, 20.0)
        p = np.array([cx_, cy_]) + d * fwd[:2] + rng.uniform(-0.6, 0.6) * d * left[:2]
        a2 = rng.uniform(-np.pi, np.pi)
        rows.append((p[0], p[1], 0.0, np.cos(a2), np.sin(a2), 4.0, 1.8, 1.6, 6))
    return make_scene(np.asarray(tris), cls), make_agents(rows)


@pytest.mark.parametrize("seed", range(40))
def test_against_float64_raycast(seed):
    scene, ag = _random_scene(seed)
    rig = make_rig(res=32, near=0.5, far=30.0, mounts=((0.0, 0.0, 1.0, 1.0, 0.0),))
    r = O.render(scene, ag, rig, view_ids=[0])
    cls, depth = r["cls"][0], r["depth"][0]
    rc, rd, unsure = raycast_view(scene, ag, rig, 0)
    sure = ~unsure
    assert sure.mean() > 0.5
    assert np.array_equal(cls[sure], rc[sure]), np.argwhere(sure & (cls != rc))[:5]
    hit = sure & np.isfinite(rd)
    rel = np.abs(depth[hit].astype(np.float64) - rd[hit]) / rd[hit]
    assert rel.max(initial=0.0) <= 1e-5, rel.max()
    assert np.all(np.isinf(depth[sure & ~np.isfinite(rd)]))


# ---------------------------------------------------------------------------
# P6: 24-bit reverse-depth quantizer, exhaustively over fp32
# ---------------------------------------------------------------------------

def test_quantizer_exhaustive():
    near, far = 0.5, 200.0
    lo = np.float32(1.0) / np.float32(far)
    hi = np.float32(2.0)  # smallest power of two >= 1/near
    bits = np.arange(lo.view(np.uint32), hi.view(np.uint32) + 1, dtype=np.uint32)
    iz = bits.view(np.float32)
    q, d = O.quantize(iz, near, far)
    assert q[-1] == 0 and q.max() < (1 << 24) - 1
    assert np.all(q[1:] <= q[:-1])                          # nearer -> smaller key
    z = 1.0 / iz.astype(np.float64)
    rel = np.abs(d.astype(np.float64) - z) / z
    # a code holds 8 consecutive fp32 inverse depths; decoding at the bucket
    # midpoint is within 4 of their ulps (2^-21 relative), the final division
    # adds half an ulp of the depth
    assert rel.max() <= 2.0 ** -21 + 2.0 ** -23
    # outside the range: beyond far is the clear value, nearer than near clamps
    q2, d2 = O.quantize(np.array([lo * 0.999, 3.0, np.nan], np.float32), near, far)
    assert q2[0] == 0xFFFFFF and np.isinf(d2[0]) and q2[1] == 0 and q2[2] == 0xFFFFFF


def test_quantizer_cap_is_the_power_of_two_above_one_over_near():
    # near = 0.3: 1/near = 3.33 and the cap is 4.  Inverse depths up to the cap
    # keep their own codes (3.9 decodes to about 1/3.9, not to the near
    # plane); beyond it they share the cap's code 0, decoded as 1/4.
    q, d = O.quantize(np.array([3.9, 4.0, 5.0, 80.0], np.float32), 0.3, 100.0)
    assert q[0] > 0 and abs(d[0] * 3.9 - 1.0) <= 2.0 ** -20
    assert q[1] == 0 and q[2] == 0 and q[3] == 0
    assert abs(d[2] - 0.25) <= 0.25 * 2.0 ** -20


# ---------------------------------------------------------------------------
# binner: home cell contains the bbox centre; AABBs are tight
# ---------------------------------------------------------------------------

def _pairs_by_rule(sc):
    """The pairing rule written out in numpy: per world, in input order,
    t and t + 1 pair when the classes match and t + 1 = (a, c, d) for
    t = (a, b, c) bit for bit; returns (first triangle, is pair) per primitive."""
    v = sc.verts.reshape(-1, 9).view(np.uint32)
    out = []
    for w in range(sc.num_worlds):
        t, e = int(sc.tri_offsets[w]), int(sc.tri_offsets[w + 1])
        while t < e:
            pair = t + 1 < e and sc.cls[t] == sc.cls[t + 1] and (v[t, 0:3] == v[t + 1, 0:3]).all() and \
                (v[t, 6:9] == v[t + 1, 3:6]).all()
            out.append((t, pair))
            t += 2 if pair else 1
    return out


def test_binner_pairing_rule_cases():
    a, b, c, d, e = (0.0, 0.0, 0.0), (4.0, 0.0, 0.0), (4.0, 3.0, 0.0), (0.0, 3.0, 0.0), (-2.0, 1.0, 0.0)
    tris = [[a, b, c], [a, c, d],          # a quad split along a-c: a pair
            [a, b, c], [a, c, d],          # the same quad, second triangle of another class: no pair
            [a, b, c], [b, c, d],          # shares an edge, but not as (a, c, d): no pair
            [a, b, c], [a, c, d], [a, d, e],   # a fan: the first two pair, the third stands alone
            [a, b, c]]                     # last triangle of the world
    cls = [1, 1, 2, 3, 1, 1, 5, 5, 5, 1]
    from paper_2607_26005_amd.scenegen import Scene
    v = np.asarray(tris, np.float32).reshape(-1, 9)
    sc = Scene(2, v, np.asarray(cls, np.uint8), np.asarray([0, 9, 10], np.int64),
               np.asarray([(-50.0, -50.0, 50.0, 50.0)] * 2, np.float32))
    bn = O.bin_scene(sc, 16.0)
    want = [(0, True), (2, False), (3, False), (4, False), (5, False), (6, True), (8, False), (9, False)]
    got = [(int(p & 0x7FFFFFFF), bool(p >> 31)) for p in bn["prims"]]
    assert got == want == _pairs_by_rule(sc)
    assert bn["count"].sum() == len(want)


def test_binner_home_cells_and_aabbs():
    from paper_2607_26005_amd import scenegen as sg
    wl = sg.make_config(2, num_worlds=2)
    sc = wl.scene
    b = O.bin_scene(sc, 16.0)
    rule = _pairs_by_rule(sc)
    assert [(int(p & 0x7FFFFFFF), bool(p >> 31)) for p in b["prims"]] == rule
    assert all(pr for _, pr in rule)            # the generators emit every quad as such a pair
    assert b["count"].sum() == len(rule) == sc.num_tris // 2
    v = sc.verts.astype(np.float64).reshape(-1, 3, 3)
    # a primitive's vertices: its first triangle's and, for a pair, the next triangle's third vertex
    pv = np.stack([np.concatenate([v[t], v[t + 1][2:3] if pr else v[t][2:3]]) for t, pr in rule])
    lo, hi = pv.min(1), pv.max(1)
    mid = 0.5 * (lo + hi)
    first = np.asarray([t for t, _ in rule])
    for w in range(sc.num_worlds):
        nx, ny = b["dims"][w]
        sel = (first >= sc.tri_offsets[w]) & (first < sc.tri_offsets[w + 1])
        cell = b["home"][sel] - b["cell_base"][w]
        ix, iy = cell % nx, cell // nx
        x0 = sc.bounds[w, 0] + 16.0 * ix
        y0 = sc.bounds[w, 1] + 16.0 * iy
        m = mid[sel]
        inside = (m[:, 0] >= sc.bounds[w, 0]) & (m[:, 0] < sc.bounds[w, 2]) & \
                 (m[:, 1] >= sc.bounds[w, 1]) & (m[:, 1] < sc.bounds[w, 3])
        tol = 1e-3
        ok = (m[:, 0] >= x0 - tol) & (m[:, 0] <= x0 + 16 + tol) & (m[:, 1] >= y0 - tol) & (m[:, 1] <= y0 + 16 + tol)
        assert np.all(ok[inside])
    home = b["home"]
    for c in np.random.default_rng(0).choice(len(b["count"]), 300, replace=False):
        m = home == c
        if not m.any():
            assert b["count"][c] == 0 and np.isinf(b["aabb"][c, 0])
            continue
        assert b["count"][c] == m.sum()
        assert np.array_equal(b["aabb"][c, :3], lo[m].min(0).astype(np.float32))
        assert np.array_equal(b["aabb"][c, 3:], hi[m].max(0).astype(np.float32))


# ---------------------------------------------------------------------------
# kinematic bicycle closed forms
# ---------------------------------------------------------------------------

def _agents_for_bicycle(n, psi, v, L):
    ag = make_agents([(0.0, 0.0, 0.0, np.cos(p), np.sin(p), L, 1.9, 1.5, 3) for p in psi])
    ag.psi = np.asarray(psi, np.float32)
    ag.speed = np.asarray(v, np.float32)
    return ag


def test_bicycle_straight_and_clamps():
    ag = _agents_for_bicycle(3, [0.0, np.pi / 2, 1.0], [10.0, 19.9, 0.1], 4.5)
    out = O.agents_step(ag, np.zeros(3), np.array([1.0, 5.0, -3.0]), dt=0.1)
    assert np.allclose(out["speed"], [10.1, 20.0, 0.0])
    assert np.allclose(out["x"], [1.01, 0.0, 0.0], atol=1e-6)
    assert np.allclose(out["y"], [0.0, 2.0, 0.0], atol=1e-6)
    assert np.allclose(out["psi"], np.float64(np.float32([0.0, np.pi / 2, 1.0])))


def test_bicycle_constant_turn_is_a_circle():
    # Constant speed and steer: heading grows by v/(0.6 L) tan(steer) dt per
    # step and the positions lie on a circle (polygon inscribed in it).
    L, v, st, dt = 4.5, 10.0, 0.2, 0.1
    ag = _agents_for_bicycle(1, [0.0], [v], L)
    omega = v / (0.6 * L) * np.tan(st)
    xs, ys = [0.0], [0.0]
    for k in range(50):
        out = O.agents_step(ag, np.array([st]), np.array([0.0]), dt=dt)
        ag.x, ag.y = out["x"].astype(np.float32), out["y"].astype(np.float32)
        ag.psi, ag.speed = out["psi"].astype(np.float32), out["speed"].astype(np.float32)
        xs.append(float(out["x"][0])); ys.append(float(out["y"][0]))
        assert abs(out["cos_h"][0] - np.cos(out["psi"][0])) < 1e-12
    assert np.isclose(float(ag.psi[0]), ((50 * omega * dt + np.pi) % (2 * np.pi)) - np.pi, atol=1e-4)
    # chord of a step is v dt; all points equidistant from the circle centre
    xs, ys = np.array(xs), np.array(ys)
    chord = np.hypot(np.diff(xs), np.diff(ys))
    assert np.allclose(chord, v * dt, rtol=1e-5)
    A = np.stack([2 * xs, 2 * ys, np.ones_like(xs)], 1)
    sol, *_ = np.linalg.lstsq(A, xs ** 2 + ys ** 2, rcond=None)
    R = np.hypot(xs - sol[0], ys - sol[1])
    assert R.std() < 1e-4 * R.mean()
    assert np.isclose(R.mean(), v * dt / (2 * np.sin(omega * dt / 2)), rtol=1e-3)


def test_bicycle_turns_with_the_updated_speed():
    # Semi-implicit update (speed first, then heading and position with the new
    # speed): from rest with a = 4 m/s^2 and tan(steer) = 1, one 0.1 s step
    # gives v' = 0.4, heading v' / (0.6 L) dt = 0.4 / 3 * 0.1, and moves v' dt
    # along that heading; a heading update with the old speed would not turn.
    L = 5.0
    ag = _agents_for_bicycle(1, [0.0], [0.0], L)
    out = O.agents_step(ag, np.array([np.pi / 4]), np.array([4.0]), dt=0.1)
    psi = 0.4 / (0.6 * L) * 0.1
    assert np.isclose(out["speed"][0], 0.4)
    assert np.isclose(out["psi"][0], psi, rtol=1e-12)
    assert np.isclose(out["x"][0], 0.04 * np.cos(psi), rtol=1e-7)
    assert np.isclose(out["y"][0], 0.04 * np.sin(psi), rtol=1e-7)
