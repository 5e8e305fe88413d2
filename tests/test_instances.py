"""Oracle pins for instance visibility: which agent owns each pixel, and each
agent's footprint (its box drawn alone) and visible pixel count, from which the
occlusion percentage the paper's analysis reads from its renderer follows
(Sec. 5.2)."""
import numpy as np
import pytest

from oracle import oracle as O
from tests import raycast as RC
from tests.scenes import make_agents, make_rig, make_scene, quad

VEH = 3


def _agents(rows):
    return make_agents([(x, y, z0, c, s, L, W, H, VEH) for (x, y, z0, c, s, L, W, H) in rows])


def _empty():
    return make_scene(np.zeros((0, 3, 3)), np.zeros(0))


EGO = (0.0, 0.0, 0.0, 1.0, 0.0, 4.5, 1.9, 1.5)


def test_unoccluded_box_owns_its_pixels():
    ag = _agents([EGO, (9.0, 0.5, -0.75, 1.0, 0.0, 4.5, 1.9, 1.5)])
    o = O.render(_empty(), ag, make_rig(), view_ids=[0], want_instances=True)
    veh = o["cls"][0] == VEH
    assert veh.sum() > 60
    assert np.array_equal(o["inst"][0] == 1, veh) and (o["inst"][0][~veh] == -1).all()
    assert o["counts"][0, 1, 0] == o["counts"][0, 1, 1] == veh.sum()
    assert tuple(o["counts"][0, 0]) == (0, 0)   # the ego's own entry


def test_wall_hides_part_and_then_all_of_a_box():
    ag = _agents([EGO, (9.0, 0.5, -0.75, 1.0, 0.0, 4.5, 1.9, 1.5)])
    rig = make_rig()
    free = O.render(_empty(), ag, rig, view_ids=[0], want_instances=True)
    # a wall at x = 6 covering y >= 0.5 (part of the left half of the view): part of the box hides
    half = make_scene(quad((6.0, 0.5, -5.0), (6.0, 20.0, -5.0), (6.0, 20.0, 5.0), (6.0, 0.5, 5.0)), [7, 7])
    o = O.render(half, ag, rig, view_ids=[0], want_instances=True)
    fp, vis = o["counts"][0, 1]
    assert fp == free["counts"][0, 1, 0]                 # the footprint ignores occluders
    assert vis == (o["cls"][0] == VEH).sum() and 0 < vis < fp
    # a wall across the whole view: fully occluded
    full = make_scene(quad((6.0, -20.0, -5.0), (6.0, 20.0, -5.0), (6.0, 20.0, 5.0), (6.0, -20.0, 5.0)), [7, 7])
    o = O.render(full, ag, rig, view_ids=[0], want_instances=True)
    assert o["counts"][0, 1, 0] == fp and o["counts"][0, 1, 1] == 0
    assert (o["inst"][0] == -1).all()


def test_nearer_box_wins_and_counts_partition_the_vehicle_pixels():
    ag = _agents([EGO, (10.0, 0.8, -0.75, 1.0, 0.0, 4.5, 1.9, 1.5), (18.0, -0.6, -0.75, 1.0, 0.0, 4.5, 1.9, 2.5)])
    o = O.render(_empty(), ag, make_rig(), view_ids=[0], want_instances=True)
    veh = o["cls"][0] == VEH
    c = o["counts"][0]
    assert c[1, 1] + c[2, 1] == veh.sum()
    assert set(np.unique(o["inst"][0][veh])) == {1, 2}
    assert c[1, 0] == c[1, 1]            # nothing in front of the nearer box
    assert 0 < c[2, 1] < c[2, 0]         # the farther one is partly hidden


def test_nearer_box_owns_the_overlap_whatever_its_index():
    # the same two boxes with the farther one listed first: both have the vehicle class, so only the
    # full depth key (not the class alone) tells which one the visible surface belongs to
    ag = _agents([EGO, (18.0, -0.6, -0.75, 1.0, 0.0, 4.5, 1.9, 2.5), (10.0, 0.8, -0.75, 1.0, 0.0, 4.5, 1.9, 1.5)])
    o = O.render(_empty(), ag, make_rig(), view_ids=[0], want_instances=True)
    veh = o["cls"][0] == VEH
    c = o["counts"][0]
    assert c[1, 1] + c[2, 1] == veh.sum()
    assert c[2, 0] == c[2, 1]            # the nearer box, though listed second, keeps all of its pixels
    assert 0 < c[1, 1] < c[1, 0]
    alone = O.render(_empty(), _agents([EGO, (10.0, 0.8, -0.75, 1.0, 0.0, 4.5, 1.9, 1.5)]), make_rig(),
                     view_ids=[0], want_instances=True)
    assert np.array_equal(o["inst"][0] == 2, alone["inst"][0] == 1)


def test_identical_boxes_tie_to_the_lower_index():
    box = (12.0, 0.5, -0.75, 1.0, 0.0, 4.5, 1.9, 1.5)
    o = O.render(_empty(), _agents([EGO, box, box]), make_rig(), view_ids=[0], want_instances=True)
    c = o["counts"][0]
    assert c[1, 0] == c[2, 0] > 0 and c[1, 1] == c[1, 0] and c[2, 1] == 0


@pytest.mark.parametrize("seed", range(4))
def test_footprint_against_float64_raycast(seed):
    # the box drawn alone, as the ray caster sees it, outside the band where snapping may decide either way
    rng = np.random.default_rng([55, seed])
    a = rng.uniform(-np.pi, np.pi)
    box = (rng.uniform(6, 20), rng.uniform(-6, 6), -0.75, float(np.float32(np.cos(a))), float(np.float32(np.sin(a))),
           rng.uniform(3, 5), rng.uniform(1.5, 2.2), rng.uniform(1.2, 2.5))
    ag = _agents([EGO, box])
    rig = make_rig(res=48)
    o = O.render(_empty(), ag, rig, view_ids=[0], want_instances=True)
    rc, rd, unsure = RC.raycast_view(_empty(), ag, rig, 0)
    hit = rc == VEH
    fp = int(o["counts"][0, 1, 0])
    assert int((hit & ~unsure).sum()) <= fp <= int((hit | unsure).sum())
    own = o["inst"][0] == 1
    assert np.array_equal(own[~unsure], hit[~unsure])
