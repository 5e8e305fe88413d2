"""Brute-force float64 ray caster: an independent check of the oracle.

For every pixel centre it intersects the exact (unsnapped) camera ray with
every triangle (Moller-Trumbore), keeps the nearest hit whose view-space
depth lies in [near, far] (exact depth ties to the lower class), and reports
per pixel the class and depth.  It also reports which pixel centres lie so
close to a projected triangle edge, or to a depth tie, that fixed-point
snapping may legitimately decide them either way.
"""
import numpy as np

SKY = 4


def _cam(agents, rig, g, k):
    m = rig.mount[k].astype(np.float64)
    c, s = float(agents.cos_h[g]), float(agents.sin_h[g])
    C = np.array([agents.x[g] + (m[0] * c - m[1] * s), agents.y[g] + (m[0] * s + m[1] * c),
                  agents.z0[g] + m[2]], np.float64)
    cc, sc = c * m[3] - s * m[4], s * m[3] + c * m[4]
    f = np.array([cc, sc, 0.0])
    r = np.array([sc, -cc, 0.0])
    u = np.array([0.0, 0.0, 1.0])
    return C, f, r, u


def box_tris(x, y, z0, c, s, L, W, H):
    """The 12 triangles of an oriented box (float64, same corner order as R9)."""
    cor = []
    for n in range(8):
        a = L / 2 if n & 1 else -L / 2
        b = W / 2 if n & 2 else -W / 2
        cor.append([x + a * c - b * s, y + a * s + b * c, z0 + H if n & 4 else z0])
    cor = np.asarray(cor)
    idx = [(0, 1, 3), (0, 3, 2), (4, 5, 7), (4, 7, 6), (0, 2, 6), (0, 6, 4),
           (1, 3, 7), (1, 7, 5), (0, 1, 5), (0, 5, 4), (2, 3, 7), (2, 7, 6)]
    return cor[np.asarray(idx)]


def world_tris(scene, agents, w, ego):
    a, b = int(scene.tri_offsets[w]), int(scene.tri_offsets[w + 1])
    tris = [scene.verts[a:b].astype(np.float64).reshape(-1, 3, 3)]
    cls = [scene.cls[a:b].astype(np.int64)]
    A = agents.agents_per_world
    for h in range(w * A, (w + 1) * A):
        if h == ego:
            continue
        tris.append(box_tris(*(float(getattr(agents, f)[h]) for f in
                               ("x", "y", "z0", "cos_h", "sin_h", "length", "width", "height"))))
        cls.append(np.full(12, int(agents.cls[h]), np.int64))
    return np.concatenate(tris), np.concatenate(cls)


def _seg_dist(px, py, ax, ay, bx, by):
    dx, dy = bx - ax, by - ay
    L2 = dx * dx + dy * dy
    t = np.where(L2 > 0, ((px - ax) * dx + (py - ay) * dy) / np.where(L2 > 0, L2, 1.0), 0.0)
    t = np.clip(t, 0.0, 1.0)
    qx, qy = ax + t * dx - px, ay + t * dy - py
    return np.sqrt(qx * qx + qy * qy)


def raycast_view(scene, agents, rig, view, band_px=2.0 / 256, rel_tie=1e-4):
    """Returns (cls[H,W], depth[H,W], unsure[H,W] bool)."""
    A = agents.agents_per_world
    Cn = rig.mount.shape[0]
    w = view // (A * Cn)
    a = (view // Cn) % A
    k = view % Cn
    g = w * A + a
    C, f, r, u = _cam(agents, rig, g, k)
    tris, cls = world_tris(scene, agents, w, g)
    H, W = rig.height, rig.width
    fx, fy, cx, cy = float(rig.fx), float(rig.fy), float(rig.cx), float(rig.cy)
    near, far = float(rig.near), float(rig.far)
    jj, ii = np.meshgrid(np.arange(H), np.arange(W), indexing="ij")
    pxp = (ii + 0.5 - cx) / fx
    pyp = (jj + 0.5 - cy) / fy
    D = f[None, None, :] + pxp[..., None] * r[None, None, :] - pyp[..., None] * u[None, None, :]
    D = D.reshape(-1, 3)
    # Moller-Trumbore, rays x tris
    v0, v1, v2 = tris[:, 0], tris[:, 1], tris[:, 2]
    e1, e2 = v1 - v0, v2 - v0
    pvec = np.cross(D[:, None, :], e2[None, :, :])
    det = np.einsum("tk,rtk->rt", e1, pvec)
    ok = np.abs(det) > 1e-300
    inv = np.where(ok, 1.0 / np.where(ok, det, 1.0), 0.0)
    tvec = C[None, :] - v0
    uu = np.einsum("tk,rtk->rt", tvec, pvec) * inv
    qvec = np.cross(tvec, e1)
    vv = np.einsum("rk,tk->rt", D, qvec) * inv
    tt = np.einsum("tk,tk->t", e2, qvec)[None, :] * inv
    zv = tt * (D @ f)[:, None]
    hit = ok & (uu >= 0) & (vv >= 0) & (uu + vv <= 1) & (zv >= near) & (zv <= far)
    zh = np.where(hit, zv, np.inf)
    # nearest, ties to the lower class
    order_key = zh + 0.0
    best = np.full(D.shape[0], np.inf)
    best_cls = np.full(D.shape[0], SKY, np.int64)
    for t in range(len(tris)):
        z = order_key[:, t]
        better = (z < best) | ((z == best) & np.isfinite(z) & (cls[t] < best_cls))
        best = np.where(better, z, best)
        best_cls = np.where(better, cls[t], best_cls)
    # second best of another class
    second = np.full(D.shape[0], np.inf)
    for t in range(len(tris)):
        z = order_key[:, t]
        diff = cls[t] != best_cls
        second = np.where(diff & (z < second), z, second)
    with np.errstate(invalid="ignore"):
        unsure = np.isfinite(best) & np.isfinite(second) & (second - best <= rel_tie * best)
    unsure |= np.isfinite(best) & ((np.abs(best - far) <= rel_tie * far) | (np.abs(best - near) <= rel_tie * near))
    # band around projected (near-clipped) edges
    band = np.zeros(D.shape[0], bool)
    px = (ii + 0.5).reshape(-1)
    py = (jj + 0.5).reshape(-1)
    for t in range(len(tris)):
        V = [(np.dot(P - C, r), np.dot(P - C, u), np.dot(P - C, f)) for P in tris[t]]
        poly = []
        for e in range(3):
            A_, B_ = V[e], V[(e + 1) % 3]
            ia, ib = A_[2] >= near, B_[2] >= near
            if ia:
                poly.append(A_)
            if ia != ib:
                I, O = (A_, B_) if ia else (B_, A_)
                s_ = (near - I[2]) / (O[2] - I[2])
                poly.append((I[0] + s_ * (O[0] - I[0]), I[1] + s_ * (O[1] - I[1]), near))
        if len(poly) < 3:
            continue
        P2 = [(cx + fx * q[0] / q[2], cy - fy * q[1] / q[2]) for q in poly]
        M = max(max(abs(q[0]), abs(q[1])) for q in P2)
        beta = band_px + 5e-7 * max(1.0, M)
        for e in range(len(P2)):
            (ax, ay), (bx, by) = P2[e], P2[(e + 1) % len(P2)]
            band |= _seg_dist(px, py, ax, ay, bx, by) <= beta
    unsure |= band
    depth = np.where(np.isfinite(best), best, np.inf)
    return (best_cls.reshape(H, W).astype(np.uint8), depth.reshape(H, W), unsure.reshape(H, W))
