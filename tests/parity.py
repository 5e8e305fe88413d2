"""Parity criteria between the HIP path and the CPU oracle.

Classes: bit-exact on every pixel the oracle does not flag (EDGE or TIE);
mismatches on flagged pixels are allowed, at most 1e-4 of all pixels.
Depth: within 1e-5 relative where the classes match and the pixel is not
flagged; background (+inf) must match exactly.

Both sides evaluate the same fp32 operations in the same order and exact
integer edge functions, so the expected outcome is stricter than that bar:
no mismatching pixel at all and depth equal bit for bit.  `assert_parity`
checks the stricter outcome too unless asked not to (exact=False).
"""
import numpy as np


def compare(gpu_cls, gpu_depth, ora, rel_tol=1e-5, budget=1e-4):
    oc, od, fl = ora["cls"], ora["depth"], ora["flags"]
    gc = np.asarray(gpu_cls)
    gd = np.asarray(gpu_depth)
    assert gc.shape == oc.shape and gd.shape == od.shape
    total = oc.size
    mism = gc != oc
    flagged = fl != 0
    unflagged_mism = int(np.sum(mism & ~flagged))
    n_mism = int(mism.sum())
    ok = (~mism) & (~flagged)
    fin = ok & np.isfinite(od)
    rel = np.abs(gd[fin].astype(np.float64) - od[fin]) / od[fin]
    inf_bad = int(np.sum(ok & ~np.isfinite(od) & (gd != od)))
    stats = dict(pixels=total, mismatches=n_mism, unflagged_mismatches=unflagged_mism,
                 flagged=int(flagged.sum()), max_rel_depth=float(rel.max(initial=0.0)),
                 depth_bitexact=bool(np.array_equal(gd[ok].view(np.uint32), od[ok].view(np.uint32))),
                 inf_mismatch=inf_bad)
    return stats


def assert_parity(gpu_cls, gpu_depth, ora, label="", exact=True):
    s = compare(gpu_cls, gpu_depth, ora)
    assert s["unflagged_mismatches"] == 0, (label, s)
    assert s["mismatches"] <= 1e-4 * s["pixels"], (label, s)
    assert s["max_rel_depth"] <= 1e-5, (label, s)
    assert s["inf_mismatch"] == 0, (label, s)
    if exact:
        assert s["mismatches"] == 0 and s["depth_bitexact"], (label, s)
    return s
