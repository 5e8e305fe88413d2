"""Oracle pins for the shaded colour mode (rule R13): per-face colours of the
agents' boxes with depth-aware brightness, flat colours elsewhere (the paper's
rendering features, Sec. 3.2).  The pins are relations the rule fixes (which
face is seen from where, how brightness falls with depth, what stays flat),
not a retyping of the colour arithmetic."""
import numpy as np
import pytest

from oracle import oracle as O
from tests.scenes import make_agents, make_rig, make_scene, quad

VEH, SKY, GROUND = 3, 4, 0
CAM = 1.0     # camera height above the agent base


def _render(agents, rig, scene=None, views=(0,)):
    sc = scene if scene is not None else make_scene(np.zeros((0, 3, 3)), np.zeros(0))
    return O.render(sc, agents, rig, view_ids=list(views), want_rgb=True)


def _box_view(ego_x, ego_c, box_x, box_c=1.0, far=100.0, mz=CAM, H=1.5, f=None):
    ag = make_agents([(ego_x, 0.0, 0.0, ego_c, 0.0, 4.5, 1.9, 1.5, VEH),
                      (box_x, 0.0, 0.0, box_c, 0.0, 4.5, 1.9, H, VEH)])
    return _render(ag, make_rig(far=far, f=f, mounts=((0.0, 0.0, mz, 1.0, 0.0),)))


def _face_rgb(o):
    sel = o["cls"][0] == VEH
    assert sel.sum() > 20
    return o["rgb"][0][:, sel].astype(np.float64), o["depth"][0][sel]


def test_front_and_back_faces_differ_by_their_factors():
    # box heading +x at x = 12: a camera behind it (at 0, looking +x) sees its back face,
    # a camera ahead of it (at 24, looking -x) its front face, both at 9.75 m
    back, zb = _face_rgb(_box_view(0.0, 1.0, 12.0))
    front, zf = _face_rgb(_box_view(24.0, -1.0, 12.0))
    assert np.allclose(zb, zf)
    ratio = front.mean(1) / back.mean(1)
    assert np.allclose(ratio, 0.85 / 0.55, rtol=0.02), ratio


def test_brightness_falls_with_depth_on_boxes_only():
    near, zn = _face_rgb(_box_view(0.0, 1.0, 12.0, f=96.0))
    far_, zf = _face_rgb(_box_view(0.0, 1.0, 32.0, f=96.0))
    bn = 1 - 0.6 * min(zn.mean() / 100.0, 1)
    bf = 1 - 0.6 * min(zf.mean() / 100.0, 1)
    assert np.allclose(far_.mean(1) / near.mean(1), bf / bn, rtol=0.03)
    # a ground plane keeps one colour at every depth
    g = make_scene(quad((-10.0, -200.0, 0.0), (300.0, -200.0, 0.0), (300.0, 200.0, 0.0), (-10.0, 200.0, 0.0)),
                   [GROUND, GROUND])
    ag = make_agents([(0.0, 0.0, 0.0, 1.0, 0.0, 4.5, 1.9, 1.5, VEH)])
    o = _render(ag, make_rig(far=250.0, mounts=((0.0, 0.0, 1.5, 1.0, 0.0),)), scene=g)
    gp = o["rgb"][0][:, o["cls"][0] == GROUND]
    assert gp.shape[1] > 1000 and (gp == gp[:, :1]).all()
    sky = o["rgb"][0][:, o["cls"][0] == SKY]
    assert sky.shape[1] > 1000 and (sky == sky[:, :1]).all()


def test_top_face_seen_from_above_is_brightest():
    # a low box below the camera: its top face (factor 1) and its back face (0.55) are both seen
    o = _box_view(0.0, 1.0, 8.0, mz=3.0, H=1.0)
    sel = o["cls"][0] == VEH
    lum = o["rgb"][0][2][sel].astype(np.float64)   # blue channel of the vehicle colour
    vals = np.unique(np.round(lum))
    assert len(vals) >= 2
    assert np.isclose(lum.max() / lum.min(), 1.0 / 0.55, rtol=0.12)


def test_side_faces_share_a_factor():
    # box heading +y seen from the origin along +x: its right face (b = -W/2) faces the camera
    ag = make_agents([(0.0, 0.0, 0.0, 1.0, 0.0, 4.5, 1.9, 1.5, VEH), (12.0, 0.0, 0.0, 0.0, 1.0, 4.5, 1.9, 1.5, VEH)])
    side, zs = _face_rgb(_render(ag, make_rig(mounts=((0.0, 0.0, CAM, 1.0, 0.0),))))
    back, zb = _face_rgb(_box_view(0.0, 1.0, 12.0 + (4.5 - 1.9) / 2))
    assert np.allclose(zs.mean(), zb.mean(), rtol=1e-3)
    assert np.allclose(side.mean(1) / back.mean(1), 0.7 / 0.55, rtol=0.02)


def test_colour_mode_classes_match_plain_mode():
    rng = np.random.default_rng(8)
    rows = [(0.0, 0.0, 0.0, 1.0, 0.0, 4.5, 1.9, 1.5, VEH)]
    for k in range(6):
        a = rng.uniform(-np.pi, np.pi)
        rows.append((rng.uniform(5, 30), rng.uniform(-10, 10), 0.0, float(np.float32(np.cos(a))),
                     float(np.float32(np.sin(a))), 4.5, 1.9, 1.5, VEH if k % 2 else 6))
    g = make_scene(quad((-50.0, -50.0, 0.0), (100.0, -50.0, 0.0), (100.0, 50.0, 0.0), (-50.0, 50.0, 0.0)), [0, 0])
    ag = make_agents(rows)
    rig = make_rig(mounts=((0.0, 0.0, 1.5, 1.0, 0.0),))
    plain = O.render(g, ag, rig, view_ids=[0])
    col = O.render(g, ag, rig, view_ids=[0], want_rgb=True)
    unflag = plain["flags"][0] == 0
    assert np.array_equal(plain["cls"][0][unflag], col["cls"][0][unflag])
    assert np.array_equal(plain["depth"][0], col["depth"][0])
