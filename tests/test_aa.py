"""Oracle pins for the antialiased colour mode (rule R14): analytic coverage of
the pixels a surface's edges cross, at one sample per pixel (Sec. 3.2,
rendering features; the appendix on render quality: thin structures such as
lane lines stay visible at low resolution).

The scenes are vertical walls 16 m in front of a camera with f = 64 px on a
64x64 image, placed so that every projected vertex is exact in fp32 and on
the subpixel grid: a world point (16, y, z) lands at x = 32 - 4 y, y_img =
32 - 4 z.  Expected values come from the geometry (pixel areas, strip
widths), not from the rule's arithmetic."""
import numpy as np

from oracle import oracle as O
from tests.scenes import make_agents, make_rig, make_scene, quad

WALL, LANE, SKY = 7, 2, 4
PAL = {WALL: (168, 144, 120), LANE: (232, 232, 224), SKY: (140, 184, 232)}
D = 16.0


def _y(px):   # world y of projected column px at depth D
    return (32.0 - px) / 4.0


def _z(py):   # world z of projected row py at depth D
    return (32.0 - py) / 4.0


def _render(tris, cls, antialias=True, want_flags=False):
    sc = make_scene(np.asarray(tris, np.float32), cls)
    ag = make_agents([(0.0, 0.0, 0.0, 1.0, 0.0, 4.5, 1.9, 1.5, 3)])
    rig = make_rig(res=64, f=64.0, mounts=((0.0, 0.0, 0.0, 1.0, 0.0),))
    return O.render(sc, ag, rig, view_ids=[0], want_rgb=True, antialias=antialias, want_flags=want_flags)


def _blend(fg, bg, a8):
    return tuple((f * a8 + b * (255 - a8) + 127) // 255 for f, b in zip(fg, bg))


def _wall(px_left, x=D, px_right=432.0):
    """A wall whose left edge projects to column px_left (rows far off-screen)."""
    s = D / x
    yl, yr = (32.0 - px_left) / 4.0 / s, (32.0 - px_right) / 4.0 / s
    zt, zb = _z(-200.0) / s, _z(300.0) / s
    return quad((x, yl, zb), (x, yr, zb), (x, yr, zt), (x, yl, zt))


def test_vertical_edge_blends_its_pixel_area():
    # left edge at x = 10.75: pixel 10 ([10, 11]) is a quarter covered and its
    # centre (10.5) is not, so it shows sky with a quarter of the wall over it
    o = _render(_wall(10.75), [WALL, WALL])
    rgb = o["rgb"][0]
    assert (o["cls"][0][:, 10] == SKY).all() and (o["cls"][0][:, 11] == WALL).all()
    want = _blend(PAL[WALL], PAL[SKY], 64)    # rint(255 * 0.25)
    assert all(tuple(rgb[:, j, 10]) == want for j in range(64)), rgb[:, :, 10].T[:4]
    assert (rgb[:, :, 11:] == np.asarray(PAL[WALL], np.uint8)[:, None, None]).all()
    assert (rgb[:, :, :10] == np.asarray(PAL[SKY], np.uint8)[:, None, None]).all()
    # without antialiasing the column is plain sky
    p = _render(_wall(10.75), [WALL, WALL], antialias=False)
    assert (p["rgb"][0][:, :, 10] == np.asarray(PAL[SKY], np.uint8)[:, None]).all()


def test_edge_covering_the_centre_keeps_the_surface_colour():
    # left edge at x = 10.25: pixel 10 is three quarters covered, centre inside;
    # the wall's own fragment does not blend (one sample decides the surface)
    o = _render(_wall(10.25), [WALL, WALL])
    assert (o["rgb"][0][:, :, 10:] == np.asarray(PAL[WALL], np.uint8)[:, None, None]).all()
    assert (o["rgb"][0][:, :, :10] == np.asarray(PAL[SKY], np.uint8)[:, None, None]).all()


def _sliver(xl_top, xr_top, x_bot, x=D):
    """A tall wedge between rows -200 (top, columns xl_top..xr_top) and 300
    (apex at column x_bot)."""
    s = D / x
    return [[(x, _y(xl_top) / s, _z(-200.0) / s), (x, _y(x_bot) / s, _z(300.0) / s),
             (x, _y(xr_top) / s, _z(-200.0) / s)]]


XL, XR, XB = 5274 / 256, 5350 / 256, 20.75   # 20.6015625, 20.8984375


def _sliver_width(j):
    t = (j + 0.5 + 200.0) / 500.0
    return (XR + (XB - XR) * t) - (XL + (XB - XL) * t)


def test_sub_pixel_sliver_shows_with_its_width():
    # the wedge covers no pixel centre (its columns stay within (20.5, 21.5)),
    # yet pixel 20 holds it with coverage equal to its width in that row
    o = _render(_sliver(XL, XR, XB), [LANE])
    assert (o["cls"][0] == SKY).all()
    rgb = o["rgb"][0]
    for j in range(64):
        a = int(np.rint(255.0 * _sliver_width(j)))
        ok = [_blend(PAL[LANE], PAL[SKY], a + d) for d in (-1, 0, 1)]
        assert tuple(rgb[:, j, 20]) in ok, (j, tuple(rgb[:, j, 20]), ok[1])
    assert tuple(rgb[:, 0, 20]) != tuple(rgb[:, 63, 20])   # the width changes down the image
    mask = np.ones((64, 64), bool)
    mask[:, 20] = False
    assert (rgb[:, mask] == np.asarray(PAL[SKY], np.uint8)[:, None]).all()
    # one sample per pixel loses it entirely
    p = _render(_sliver(XL, XR, XB), [LANE], antialias=False)
    assert (p["rgb"][0] == np.asarray(PAL[SKY], np.uint8)[:, None, None]).all()


def test_sliver_in_front_of_a_wall_blends_over_the_wall():
    o = _render(_sliver(XL, XR, XB, x=12.0) + _wall(0.0), [LANE, WALL, WALL])
    rgb = o["rgb"][0]
    for j in (0, 31, 63):
        a = int(np.rint(255.0 * _sliver_width(j)))
        ok = [_blend(PAL[LANE], PAL[WALL], a + d) for d in (-1, 0, 1)]
        assert tuple(rgb[:, j, 20]) in ok, (j, tuple(rgb[:, j, 20]))


def test_sliver_behind_a_wall_is_hidden():
    # a fragment farther than the centre's surface does not blend
    o = _render(_sliver(XL, XR, XB, x=24.0) + _wall(0.0), [LANE, WALL, WALL])
    assert (o["rgb"][0] == np.asarray(PAL[WALL], np.uint8)[:, None, None]).all()


def test_nearest_fragment_wins():
    # two slivers over the same pixel column at 12 m and 14 m, sky behind:
    # the nearer one (wall class) is the one blended
    near = _sliver(XL, XR, XB, x=12.0)
    far_ = _sliver(XL, XR, XB, x=14.0)
    o = _render(far_ + near, [LANE, WALL])
    rgb = o["rgb"][0]
    for j in (0, 63):
        a = int(np.rint(255.0 * _sliver_width(j)))
        ok = [_blend(PAL[WALL], PAL[SKY], a + d) for d in (-1, 0, 1)]
        assert tuple(rgb[:, j, 20]) in ok


def test_classes_and_depth_match_one_sample_mode():
    rng = np.random.default_rng(9)
    tris = rng.uniform([4.0, -12.0, -4.0], [40.0, 12.0, 6.0], size=(60, 3, 3)).astype(np.float32)
    cls = rng.integers(0, 11, size=60)
    sc = make_scene(tris, cls)
    rows = [(0.0, 0.0, 0.0, 1.0, 0.0, 4.5, 1.9, 1.5, 3)]
    for k in range(4):
        rows.append((rng.uniform(6, 30), rng.uniform(-8, 8), 0.0, 1.0, 0.0, 4.5, 1.9, 1.5, 3 if k % 2 else 6))
    ag = make_agents(rows)
    rig = make_rig(res=64, mounts=((0.0, 0.0, 1.5, 1.0, 0.0),))
    a = O.render(sc, ag, rig, view_ids=[0], want_rgb=True, antialias=True)
    b = O.render(sc, ag, rig, view_ids=[0], want_rgb=True, antialias=False)
    assert np.array_equal(a["cls"], b["cls"]) and np.array_equal(a["depth"], b["depth"])
    changed = (a["rgb"][0] != b["rgb"][0]).any(0)
    assert 0 < changed.sum() < 0.5 * changed.size
    # a changed pixel lies within one pixel of a change of shading in the one-sample image
    c = b["rgb"][0].astype(np.int32)
    edge = np.zeros((64, 64), bool)
    for dy in (-1, 0, 1):
        for dx in (-1, 0, 1):
            sh = np.roll(np.roll(c, dy, 1), dx, 2)
            edge |= (sh != c).any(0)
    frac = (changed & edge).sum() / changed.sum()
    assert frac > 0.9, frac


def test_coplanar_neighbours_blend_across_their_shared_edge():
    # two walls in one plane meeting at x = 10.75: pixel 10 is three quarters
    # wall (its centre's surface) and one quarter lane marking
    left = quad((D, _y(-400.0), _z(300.0)), (D, _y(10.75), _z(300.0)), (D, _y(10.75), _z(-200.0)),
                (D, _y(-400.0), _z(-200.0)))
    o = _render(left + _wall(10.75), [WALL, WALL, LANE, LANE])
    rgb = o["rgb"][0]
    assert (o["cls"][0][:, 10] == WALL).all() and (o["cls"][0][:, 11] == LANE).all()
    want = _blend(PAL[LANE], PAL[WALL], 64)
    assert all(tuple(rgb[:, j, 10]) == want for j in range(64))
    assert (rgb[:, :, 11:] == np.asarray(PAL[LANE], np.uint8)[:, None, None]).all()
    assert (rgb[:, :, :10] == np.asarray(PAL[WALL], np.uint8)[:, None, None]).all()


def _strip(xl, xr):
    """A marking 500 rows tall between columns xl and xr, built as one
    triangle pair (a, b, c), (a, c, d) split along its diagonal."""
    return quad((D, _y(xl), _z(300.0)), (D, _y(xr), _z(300.0)), (D, _y(xr), _z(-200.0)), (D, _y(xl), _z(-200.0)))


def test_split_strip_narrower_than_a_pixel_blends_at_full_width():
    # a 76/256 px wide strip inside pixel 20 (no centre covered): the pair is
    # one surface, so every row blends the strip's whole width, 255 * 76/256
    # rounded = 76, wherever the diagonal crosses the row
    o = _render(_strip(XL, XR), [LANE, LANE])
    assert (o["cls"][0] == SKY).all()
    rgb = o["rgb"][0]
    want = _blend(PAL[LANE], PAL[SKY], 76)
    assert all(tuple(rgb[:, j, 20]) == want for j in range(64)), [tuple(rgb[:, j, 20]) for j in (0, 31, 63)]
    mask = np.ones((64, 64), bool)
    mask[:, 20] = False
    assert (rgb[:, mask] == np.asarray(PAL[SKY], np.uint8)[:, None]).all()
    # the same two triangles in the other order are not a pair: each half is
    # then its own surface and only the larger piece of the row shows
    t = _strip(XL, XR)
    p = _render([t[1], t[0]], [LANE, LANE])
    a8 = [int(np.rint((int(p["rgb"][0][0, j, 20]) - PAL[SKY][0]) * 255 / (PAL[LANE][0] - PAL[SKY][0])))
          for j in range(64)]
    assert max(a8) < 76 and min(a8) > 0, a8


def test_split_wide_strip_keeps_its_edge_coverage():
    # 2.25 px wide (columns 20.25 .. 22.5): pixel 20 holds three quarters of
    # its area (centre covered: plain strip), 22 half of it (centre on the
    # right edge, which the top-left rule leaves out: sky under a half blend)
    o = _render(_strip(20.25, 22.5), [LANE, LANE])
    rgb = o["rgb"][0]
    assert (o["cls"][0][:, 20:22] == LANE).all() and (o["cls"][0][:, 22] == SKY).all()
    assert (rgb[:, :, 20:22] == np.asarray(PAL[LANE], np.uint8)[:, None, None]).all()
    want = _blend(PAL[LANE], PAL[SKY], 128)   # rint(255 * 0.5)
    assert all(tuple(rgb[:, j, 22]) == want for j in range(64))


def _dart():
    return (D, _y(18.0), _z(60.0)), (D, _y(30.0), _z(50.0)), (D, _y(21.0), _z(30.0)), (D, _y(30.0), _z(10.0))


def test_pair_that_is_not_convex_keeps_per_triangle_fragments():
    # a dart (reflex vertex at c) is no convex surface: its two triangles
    # leave their own fragments, exactly as the same triangles do when listed
    # in the other order (which does not pair them)
    a, b, c, d = _dart()
    paired = _render([[a, b, c], [a, c, d]], [LANE, LANE])
    apart = _render([[a, c, d], [a, b, c]], [LANE, LANE])
    assert (paired["cls"][0] == LANE).sum() > 0
    assert np.array_equal(paired["rgb"][0], apart["rgb"][0])


def _straight_angle():
    """The triangle (d, b, c) split by the midpoint a of its edge d-b, as the
    pair (a, b, c), (a, c, d)."""
    d, b, c = (D, _y(18.0), _z(10.0)), (D, _y(30.0), _z(50.0)), (D, _y(40.0), _z(16.0))
    return (D, _y(24.0), _z(30.0)), b, c, d


def _folded_before_wall():
    """A convex square (a, b, c), (a, c, d): the first triangle at 16 m facing
    the camera, the second tilting back to d at 48 m; a wall at 30 m behind.
    The left edge (d-a) projects to column 19.75, rows 20 .. 40."""
    a = (D, _y(19.75), _z(20.0))
    b = (D, _y(40.0), _z(20.0))
    c = (D, _y(40.0), _z(40.0))
    d = (48.0, 0.75 * (32.0 - 19.75), 0.75 * (32.0 - 40.0))   # projects to (19.75, 40)
    W = 30.0
    wall = quad((W, 60.0, -60.0), (W, -60.0, -60.0), (W, -60.0, 60.0), (W, 60.0, 60.0))
    return [[a, b, c], [a, c, d]] + wall, [LANE, LANE, WALL, WALL]


def test_pair_with_a_straight_angle_keeps_per_triangle_fragments():
    # the triangle (d, b, c) split by a point a on its edge d-b: the 4-gon
    # (a, b, c, d) turns by zero at a, so it is not strictly convex and no
    # surface; its halves leave their own fragments, as in the unpaired order
    a, bb, c, d = _straight_angle()
    paired = _render([[a, bb, c], [a, c, d]], [LANE, LANE])
    apart = _render([[a, c, d], [a, bb, c]], [LANE, LANE])
    assert (paired["cls"][0] == LANE).sum() > 100
    assert np.array_equal(paired["rgb"][0], apart["rgb"][0])


def test_surface_fragments_take_the_first_triangles_plane():
    # a convex square whose first triangle (a, b, c) faces the camera at 16 m
    # and whose second (a, c, d) tilts back to d at 48 m, in front of a wall at
    # 30 m.  Its left edge (d-a, the second triangle's) lies at column 19.75:
    # pixel 19 is a quarter covered and its centre shows the wall.  The
    # fragment's depth comes from the first triangle's plane (16 m at that
    # centre), nearer than the wall, so every row of the edge blends; the
    # second triangle's plane would put the lower rows behind the wall.
    o = _render(*_folded_before_wall())
    cls = o["cls"][0]
    # column 19's centres show the wall; in column 20 the square's lower rows
    # (its second triangle, past 30 m) are behind the wall as well
    assert (cls[21:40, 19] == WALL).all() and (cls[21:30, 20] == LANE).all() and (cls[36:40, 20] == WALL).all()
    want = _blend(PAL[LANE], PAL[WALL], 64)   # a quarter: a8 = rint(255 / 4) = 64
    got = [tuple(int(v) for v in o["rgb"][0][:, j, 19]) for j in range(21, 40)]
    assert all(g == want for g in got), got


def test_pair_wholly_beyond_far_leaves_nothing():
    # the far-rule pin's square one fp32 step beyond far = 110 (every covered
    # centre's 1/z rounds to fl(1/far) and would pass the per-pixel test),
    # given as a pair: neither half is drawn (R4), so the pair is no surface and
    # leaves no key and no fragment in the antialiased mode either
    from tests.test_oracle_pins import ego, fronto_quad
    far = 110.0
    Dz = float(np.nextafter(np.float32(far), np.float32(np.inf)))
    r = O.render(make_scene(fronto_quad(Dz, 16.0), [WALL, WALL]), make_agents([ego()]), make_rig(far=far),
                 view_ids=[0], want_rgb=True, antialias=True)
    assert (r["cls"][0] == SKY).all()
    assert (r["rgb"][0] == np.asarray(PAL[SKY], np.uint8)[:, None, None]).all()


def _clipped_band():
    """A triangle 2 mm below the camera with v0 behind it, and the points where
    the near plane (0.5 m) cuts its edges v0-v1 and v2-v0 (their midpoints)."""
    z = -0.002
    return ((-0.5, 0.0, z), (1.5, 1.0, z), (1.5, -1.0, z)), ((0.5, 0.5, z), (0.5, -0.5, z))


def test_near_clipped_triangle_is_one_surface():
    # a triangle 2 mm below the camera with one vertex behind it: the near
    # plane (0.5 m) cuts its two edges at their midpoints (t = 1/2, exact), so
    # the clipped 4-gon (c01, v1, v2, c20) is known exactly.  It is a band a
    # tenth to a quarter of a pixel tall across row 32, crossed lengthwise by
    # the fan diagonal.  As one surface (R14) it blends exactly like the same
    # 4-gon given as an unclipped pair (a, b, c), (a, c, d), whose surface the
    # split-strip pin fixes; per-piece fragments would lose the coverage the
    # diagonal splits.
    (v0, v1, v2), (c01, c20) = _clipped_band()
    clipped = _render([[v0, v1, v2]], [LANE])
    pair = _render([[c01, v1, v2], [c01, v2, c20]], [LANE, LANE])
    assert (clipped["cls"][0] == SKY).all()
    band = clipped["rgb"][0][:, 32, :]
    assert (band != np.asarray(PAL[SKY], np.uint8)[:, None]).any(0).sum() > 50
    assert np.array_equal(clipped["rgb"][0], pair["rgb"][0])


def _coverage(poly, px, py):
    """R14 coverage of a positively oriented convex polygon (snapped
    subpixel vertices) at pixel centres (px, py) in subpixels, in float64."""
    n = len(poly)
    s = 0.0
    for k in range(n):
        (ax, ay), (bx, by) = poly[k], poly[(k + 1) % n]
        dx, dy = bx - ax, by - ay
        e = dx * (py - ay) - dy * (px - ax)
        s = s + np.clip(e / (256.0 * np.hypot(dx, dy)) + 0.5, 0.0, 1.0)
    return np.clip(s - (n - 1), 0.0, 1.0)


def test_no_fragment_more_than_half_a_pixel_beyond_the_box():
    # the kernel evaluates R14 only at centres within half a pixel of a
    # surface's snapped box: farther centres must get a = 0 for every
    # triangle and convex 4-gon (slivers and sharp corners included)
    rng = np.random.default_rng(17)
    checked = 0
    for it in range(3000):
        n = 3 if it % 2 else 4
        scale = [64.0, 400.0, 2000.0][it % 3]
        if n == 3:
            pts = rng.integers(-int(scale), int(scale), size=(3, 2)).astype(np.float64)
            if it % 5 == 0:   # a sliver
                pts[2] = np.rint(pts[0] + (pts[1] - pts[0]) * rng.uniform(0.2, 0.8)) + rng.integers(-3, 4, size=2)
        else:
            ang = np.sort(rng.uniform(0, 2 * np.pi, size=4))
            rad = rng.uniform(0.2, 1.0, size=2) * scale
            pts = np.rint(np.stack([rad[0] * np.cos(ang), rad[1] * np.sin(ang)], 1))
        area2 = sum(pts[k, 0] * pts[(k + 1) % n, 1] - pts[(k + 1) % n, 0] * pts[k, 1] for k in range(n))
        if area2 == 0:
            continue
        if area2 < 0:
            pts = pts[::-1]
        if n == 4:   # strictly convex only
            cr = [(pts[(k + 1) % 4, 0] - pts[k, 0]) * (pts[(k + 2) % 4, 1] - pts[(k + 1) % 4, 1]) -
                  (pts[(k + 1) % 4, 1] - pts[k, 1]) * (pts[(k + 2) % 4, 0] - pts[(k + 1) % 4, 0]) for k in range(4)]
            if min(cr) <= 0:
                continue
        lo, hi = pts.min(0), pts.max(0)
        # centres in the band (0.5, 1] px beyond each side, along the whole box
        i = np.arange(np.floor((lo[0] - 512) / 256), np.ceil((hi[0] + 512) / 256) + 1)
        j = np.arange(np.floor((lo[1] - 512) / 256), np.ceil((hi[1] + 512) / 256) + 1)
        cx, cy = np.meshgrid(256 * i + 128, 256 * j + 128)
        band = (((cx < lo[0] - 128) | (cx > hi[0] + 128) | (cy < lo[1] - 128) | (cy > hi[1] + 128)) &
                (cx >= lo[0] - 256) & (cx <= hi[0] + 256) & (cy >= lo[1] - 256) & (cy <= hi[1] + 256))
        a = _coverage([tuple(p) for p in pts], cx[band], cy[band])
        assert (np.rint(255.0 * a) == 0).all(), (pts, a.max())
        checked += int(band.sum())
    assert checked > 20000
