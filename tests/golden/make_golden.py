"""Writes tests/golden/tiny_oracle.json from the CPU oracle only.

The tiny workload (1 world, seed 0, 8 forward cameras at 64x64) is rendered by
the oracle; per view the file stores the class histogram and SHA-256 digests
of the class and depth images.  The fixture freezes the oracle's behaviour:
any later change to its arithmetic must regenerate it, and the commit that
does so names the passage or reading that justifies the change.

    python tests/golden/make_golden.py
"""
import hashlib
import json
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, os.path.dirname(os.path.dirname(HERE)))

from oracle import oracle as O  # noqa: E402
from paper_2607_26005_amd import scenegen as sg  # noqa: E402


def summary():
    wl = sg.make_config(1)
    r = O.render(wl.scene, wl.agents, wl.rig)
    views = []
    for v in range(wl.num_views):
        views.append(dict(
            view=v,
            class_hist=[int(x) for x in __import__("numpy").bincount(r["cls"][v].ravel(), minlength=7)],
            cls_sha256=hashlib.sha256(r["cls"][v].tobytes()).hexdigest(),
            depth_sha256=hashlib.sha256(r["depth"][v].tobytes()).hexdigest(),
        ))
    return dict(workload="tiny seed 0, 1 world, 8 views, 64x64", scene_sha256=wl.scene.sha256(), views=views)


if __name__ == "__main__":
    with open(os.path.join(HERE, "tiny_oracle.json"), "w") as f:
        json.dump(summary(), f, indent=1)
    print("wrote tiny_oracle.json")
