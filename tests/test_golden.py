"""The oracle still reproduces the frozen tiny-workload fixture."""
import json
import os

from tests.golden.make_golden import summary

HERE = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def test_tiny_oracle_fixture():
    with open(os.path.join(HERE, "tiny_oracle.json")) as f:
        want = json.load(f)
    got = summary()
    assert got["scene_sha256"] == want["scene_sha256"], "scene generator changed"
    assert got["views"] == want["views"]
