// Batched class/depth view rasterizer for gfx950: one 256-thread workgroup
// per view tile (at most 64x64 pixels) whose framebuffer of 32-bit keys lives
// in LDS.
//
// Per tile:
//  1. cells of the world grid around the tile frustum are tested (one lane
//     per cell) against the frustum planes and, when the whole cell is in
//     front of the near plane, against the tile's pixel centres through a
//     conservative projection of the cell's bounding box; visible cells are
//     compacted with a ballot and their triangle counts prefix-summed;
//  2. candidate triangles are mapped to their cell by a max-scan of cell
//     start markers; each wave runs a cheap first pass over 64 at a time
//     (view transform, the near/far rule, a conservative approximate test
//     that the snapped triangle can hold a pixel centre of the tile) and
//     compacts the survivors (ballot + mbcnt) into its own LDS queue;
//  3. each full queue of 64 survivors goes through the exact pass: near
//     clipping, 8-bit subpixel snap, setup, depth plane.  Triangles with a
//     small bounding box are rasterized by their own lane; larger ones are
//     pushed to a block-wide queue that all waves drain, one triangle per
//     wave, the wave tiling the bounding box as (power-of-two columns) x
//     (64 / columns) rows with incremental edge functions;
//  4. leftover survivors of all waves are pooled into full batches at the
//     end;
//  5. visibility is an LDS atomicMin of (24-bit depth | 8-bit class), so the
//     order in which lanes and waves finish does not matter;
//  6. the tile is resolved and written with 16-byte non-temporal stores.
//
// The exact pass evaluates the rasterization rules (camera R1, view
// transform R2, depth plane R3, near clip R4, snap R5, fill R6, key R7,
// resolve R8, boxes R9) in fp32 with no contraction and correctly rounded
// reciprocals and divisions, so every key equals a brute-force evaluation of
// the rules over all triangles of the world.  Everything before it only
// skips triangles that cannot set a key.
#include "pictura_device.h"

#pragma clang fp contract(off)

namespace pictura {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr uint32_t kClearKey = (0xFFFFFFu << 8) | 4u;
constexpr int kWaves = kBlock / 64;
constexpr uint32_t kBoxFlag = 0x80000000u;

struct Cam {
    float x, y, z;     // camera centre (R1)
    float cc, sc;      // camera heading (R1)
};

// View-space frustum of one tile with 0.5 px of margin beyond the outermost
// pixel centres: inside iff every value below is >= 0.
//   left  fx*xv - kl*zv     right  kr*zv - fx*xv
//   top   kt*zv - fy*yv     bottom fy*yv - kb*zv
struct Tile {
    int x0, y0, w, h;
    float kl, kr, kt, kb;
};

// A snapped triangle queued for whole-wave rasterization.
struct BigTri {
    int X0, Y0, X1, Y1, X2, Y2;   // oriented (area2 > 0)
    float pa, pb, pc;             // depth plane (R3)
    uint32_t box;                 // class | i0 << 8 | i1 << 16 | j0 << 24 (tile-local bounding box)
    uint32_t j1;                  // tile-local last row
};

struct alignas(16) Shared {
    uint32_t fb[kTileMaxPx];
    uint32_t cl_start[kBlock];
    uint32_t cl_pre[kBlock + 1];
    union {
        uint16_t mark[kCandCap];       // static phase: cell slot + 1 of each candidate
        uint32_t vis[kAgentBatch];     // box phase: visible agents
    } u;
    uint32_t q[kWaves][kQCap];         // per-wave survivor queues
    BigTri big[kBigCap];               // block-wide queue of large triangles
    uint32_t s_wave[kWaves];
    uint32_t nq_w[kWaves];
    uint32_t n_cells, n_vis, n_big, big_next;
    uint32_t stat[kNumStats];
};

// Optional work counters (P.stats non-null): LDS per block, flushed once.
#define STAT(k, n) do { if (P.stats) atomicAdd(&S.stat[(k)], (uint32_t)(n)); } while (0)
// Phase timers of the stats mode: shader-clock cycles seen by lane 0 of every wave.
#define TSTART(t) long long t = P.stats ? (long long)__builtin_amdgcn_s_memtime() : 0ll
#define TACC(k, t) do { if (P.stats && lane_id() == 0) atomicAdd(&S.stat[(k)], (uint32_t)((long long)__builtin_amdgcn_s_memtime() - (t))); } while (0)

// ---------------------------------------------------------------------------
// arithmetic
// ---------------------------------------------------------------------------

// Correctly rounded 1/x for x in [2^-12, 2^20): hardware reciprocal plus one
// Newton step with fused residual.  Equality with IEEE division over every
// fp32 value of that range is checked on the device (pictura_selftest_rcp).
__device__ __forceinline__ float rcp_rn(float x)
{
    const float r = __builtin_amdgcn_rcpf(x);
    const float e = fmaf(-x, r, 1.0f);
    return fmaf(e, r, r);
}

__device__ __forceinline__ bool rcp_rn_ok(float x) { return x >= 0.000244140625f && x < 1048576.0f; }

// ---------------------------------------------------------------------------
// geometry rules
// ---------------------------------------------------------------------------

__device__ __forceinline__ void view_xform(const Cam& c, float px, float py, float pz,
                                           float& xv, float& yv, float& zv)
{
    const float dx = px - c.x, dy = py - c.y, dz = pz - c.z;
    const float a = dx * c.sc, b = dy * c.cc;
    xv = a - b;
    yv = dz;
    const float e = dx * c.cc, f = dy * c.sc;
    zv = e + f;
}

// R3: depth plane of the unsnapped world-space triangle.
__device__ __forceinline__ bool depth_plane(const RenderParams& P, const Cam& c, const float* t,
                                            float& pa, float& pb, float& pc)
{
    const float e1x = t[3] - t[0], e1y = t[4] - t[1], e1z = t[5] - t[2];
    const float e2x = t[6] - t[0], e2y = t[7] - t[1], e2z = t[8] - t[2];
    const float Nx = e1y * e2z - e1z * e2y;
    const float Ny = e1z * e2x - e1x * e2z;
    const float Nz = e1x * e2y - e1y * e2x;
    const float d0x = t[0] - c.x, d0y = t[1] - c.y, d0z = t[2] - c.z;
    const float nx = Nx * c.sc - Ny * c.cc;
    const float ny = Nz;
    const float nz = Nx * c.cc + Ny * c.sc;
    const float delta = (Nx * d0x + Ny * d0y) + Nz * d0z;
    if (delta == 0.0f || !isfinite(delta)) return false;
    const float rd = 1.0f / delta;
    pa = (nx * rd) * P.rfx;
    pb = -((ny * rd) * P.rfy);
    pc = nz * rd;
    return true;
}

// R5
__device__ __forceinline__ bool snap_vertex(const RenderParams& P, float xv, float yv, float zv, int& X, int& Y)
{
    const float rz = rcp_rn_ok(zv) ? rcp_rn(zv) : 1.0f / zv;
    const float qx = xv * rz, qy = yv * rz;
    const float mx = P.fx256 * qx, my = P.fy256 * qy;
    const float sx = P.cx256 + mx, sy = P.cy256 - my;
    const float rx = rintf(sx), ry = rintf(sy);
    if (!(fabsf(rx) <= 536870912.0f) || !(fabsf(ry) <= 536870912.0f)) return false;
    X = (int)rx;
    Y = (int)ry;
    return true;
}

// R4 crossing point on the edge from inside vertex I to outside vertex O.
__device__ __forceinline__ void near_cross(const RenderParams& P, float ix, float iy, float iz, float ox, float oy,
                                           float oz, float& x, float& y)
{
    const float t = (P.nearp - iz) / (oz - iz);
    x = fmaf(t, ox - ix, ix);
    y = fmaf(t, oy - iy, iy);
}

// R9: triangle `face` of agent h's box.
__device__ __forceinline__ void load_box(const RenderParams& P, int64_t h, int face, float* tri, uint32_t& cls)
{
    const float x = P.ax[h], y = P.ay[h], z0 = P.az0[h], c = P.ac[h], s = P.as[h];
    const float hl = 0.5f * P.al[h], hw = 0.5f * P.aw[h], ztop = z0 + P.ah[h];
    // corner indices (bit 0: +L/2, bit 1: +W/2, bit 2: top) of the 12 triangles
    constexpr uint32_t kBoxTris[12] = {0x310, 0x230, 0x754, 0x674, 0x620, 0x460,
                                       0x731, 0x571, 0x510, 0x450, 0x732, 0x672};
    const uint32_t code = kBoxTris[face];
#pragma unroll
    for (int q = 0; q < 3; ++q) {
        const int n = (code >> (4 * q)) & 15;
        const float aa = (n & 1) ? hl : -hl;
        const float bb = (n & 2) ? hw : -hw;
        const float ac_ = aa * c, bs = bb * s, as_ = aa * s, bc = bb * c;
        const float ox = ac_ - bs, oy = as_ + bc;
        tri[3 * q] = x + ox;
        tri[3 * q + 1] = y + oy;
        tri[3 * q + 2] = (n & 4) ? ztop : z0;
    }
    cls = (uint32_t)P.acls[h];
}

__device__ __forceinline__ void load_static(const RenderParams& P, uint32_t t, float* tri, uint32_t& cls)
{
    const float4 A = P.scene.triA[t];
    const float4 B = P.scene.triB[t];
    const float2 C = P.scene.triC[t];
    tri[0] = A.x; tri[1] = A.y; tri[2] = A.z; tri[3] = A.w;
    tri[4] = B.x; tri[5] = B.y; tri[6] = B.z; tri[7] = B.w; tri[8] = C.x;
    cls = __float_as_uint(C.y);
}

__device__ __forceinline__ void load_entry(const RenderParams& P, uint32_t e, int64_t abase_w, float* tri,
                                           uint32_t& cls)
{
    if (e & kBoxFlag) load_box(P, abase_w + ((e & ~kBoxFlag) >> 4), (int)(e & 15u), tri, cls);
    else load_static(P, e, tri, cls);
}

// Side-plane test of three view-space vertices (conservative, see Tile).
__device__ __forceinline__ bool outside_tile(const RenderParams& P, const Tile& T,
                                             const float* xv, const float* yv, const float* zv)
{
    bool l = true, r = true, t = true, b = true;
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        l = l && (P.fx * xv[k] - T.kl * zv[k] < 0.0f);
        r = r && (T.kr * zv[k] - P.fx * xv[k] < 0.0f);
        t = t && (T.kt * zv[k] - P.fy * yv[k] < 0.0f);
        b = b && (P.fy * yv[k] - T.kb * zv[k] < 0.0f);
    }
    return l || r || t || b;
}

// Can a box of projected x in [xmn, xmx], y in [ymn, ymx] (approximate
// projections whose magnitude is at most mag) hold a pixel centre of the
// tile?  The margin covers half a subpixel of snapping plus the error of the
// hardware reciprocal and of the fp32 arithmetic.
__device__ __forceinline__ bool box_has_centre(const RenderParams& P, const Tile& T, float xmn, float xmx, float ymn,
                                               float ymx, float mag)
{
    const float m = 0.00390625f + (mag + P.cabs) * 3.814697265625e-06f;   // 1/256 + 2^-18 (|p| + |c|)
    const float ilo = fmaxf(ceilf(xmn - m - 0.5f), (float)T.x0);
    const float ihi = fminf(floorf(xmx + m - 0.5f), (float)(T.x0 + T.w - 1));
    const float jlo = fmaxf(ceilf(ymn - m - 0.5f), (float)T.y0);
    const float jhi = fminf(floorf(ymx + m - 0.5f), (float)(T.y0 + T.h - 1));
    return !(ilo > ihi) && !(jlo > jhi);
}

// First pass: false only if the triangle cannot set a key of the tile.  The
// near/far rule uses the exact pass's own arithmetic; for a triangle in front
// of the near plane the approximate projection (hardware reciprocal) is off
// the exact snapped position by less than the margin of box_has_centre.
__device__ __forceinline__ bool first_pass(const RenderParams& P, const Tile& T, const Cam& cam, const float* tri,
                                           bool cull)
{
    float xv[3], yv[3], zv[3];
#pragma unroll
    for (int k = 0; k < 3; ++k) view_xform(cam, tri[3 * k], tri[3 * k + 1], tri[3 * k + 2], xv[k], yv[k], zv[k]);
    const bool in0 = zv[0] >= P.nearp, in1 = zv[1] >= P.nearp, in2 = zv[2] >= P.nearp;
    if (!(in0 || in1 || in2)) return false;
    if (zv[0] > P.farp && zv[1] > P.farp && zv[2] > P.farp) return false;
    if (!cull) return true;
    if (!(in0 && in1 && in2)) return !outside_tile(P, T, xv, yv, zv);
    float xmn = 3.0e38f, xmx = -3.0e38f, ymn = 3.0e38f, ymx = -3.0e38f, mag = 0.0f;
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        const float r = __builtin_amdgcn_rcpf(zv[k]);
        const float px = P.cx + P.fx * (xv[k] * r);
        const float py = P.cy - P.fy * (yv[k] * r);
        xmn = fminf(xmn, px); xmx = fmaxf(xmx, px);
        ymn = fminf(ymn, py); ymx = fmaxf(ymx, py);
        mag = fmaxf(mag, fmaxf(fabsf(px), fabsf(py)));
    }
    return box_has_centre(P, T, xmn, xmx, ymn, ymx, mag);
}

// ---------------------------------------------------------------------------
// raster
// ---------------------------------------------------------------------------

// R7: key of a covered pixel, or 0xFFFFFFFF (no effect on the minimum) when
// the depth test rejects it.  iz >= 1/far > 0 makes the bit patterns of iz
// and IZCAP order like the values, so min() may run on the bits.
__device__ __forceinline__ uint32_t pixel_key(const RenderParams& P, float pxf, float pyf, float pa, float pb,
                                              float pc, uint32_t cls)
{
    const float iz = fmaf(pa, pxf, fmaf(pb, pyf, pc));
    const uint32_t bits = min(__float_as_uint(iz), __float_as_uint(P.izcap));
    const uint32_t key = ((P.qbase - (bits >> 3)) << 8) | cls;
    return iz >= P.izfar ? key : 0xFFFFFFFFu;
}

template <typename I>
__device__ __forceinline__ I imul(int a, int b)
{
    if constexpr (sizeof(I) == 4) return (I)__mul24(a, b);
    else return (I)a * (I)b;
}

// Edge function plus top-left bias, F = E + topleft - 1 (covered iff every
// F >= 0), of edge a->b at the pixel centre (256 i + 128, 256 j + 128).
// I = int is exact when the triangle spans < 2^14 subpixels and the pixel is
// within one bounding-box width of it; long long always is.
template <typename I>
__device__ __forceinline__ I edge_f(int ax, int ay, int bx, int by, int i, int j)
{
    const int dx = bx - ax, dy = by - ay;
    const int tl = (dy < 0) || (dy == 0 && dx > 0);
    return imul<I>(dx, 256 * j + 128 - ay) - imul<I>(dy, 256 * i + 128 - ax) + (I)(tl - 1);
}

// A small triangle rasterized by its own lane over its bounding box.
template <typename I>
__device__ __forceinline__ void raster_lane(const RenderParams& P, Shared& S, const Tile& T, int X0, int Y0, int X1,
                                            int Y1, int X2, int Y2, int i0, int i1, int j0, int j1, float pa,
                                            float pb, float pc, uint32_t cls)
{
    I f0 = edge_f<I>(X1, Y1, X2, Y2, i0, j0);
    I f1 = edge_f<I>(X2, Y2, X0, Y0, i0, j0);
    I f2 = edge_f<I>(X0, Y0, X1, Y1, i0, j0);
    const I sx0 = (I)(Y1 - Y2) * 256, sx1 = (I)(Y2 - Y0) * 256, sx2 = (I)(Y0 - Y1) * 256;
    const I sy0 = (I)(X2 - X1) * 256, sy1 = (I)(X0 - X2) * 256, sy2 = (I)(X1 - X0) * 256;
    for (int j = j0; j <= j1; ++j) {
        I g0 = f0, g1 = f1, g2 = f2;
        const float pyf = ((float)j + 0.5f) - P.cy;
        uint32_t* row = &S.fb[(j - T.y0) * T.w - T.x0];
        for (int i = i0; i <= i1; ++i) {
            if ((g0 | g1 | g2) >= 0) {
                const float pxf = ((float)i + 0.5f) - P.cx;
                atomicMin(&row[i], pixel_key(P, pxf, pyf, pa, pb, pc, cls));
            }
            g0 += sx0; g1 += sx1; g2 += sx2;
        }
        f0 += sy0; f1 += sy1; f2 += sy2;
    }
}

// One queued triangle rasterized by a whole wave: lanes tile its bounding
// box as cw columns (the next power of two >= its width) by 64 / cw rows and
// step down the rows with incremental edge functions.
template <typename I>
__device__ __forceinline__ void raster_wave(const RenderParams& P, Shared& S, const Tile& T, const BigTri& b)
{
    const int lane = lane_id();
    const int i0 = T.x0 + (int)((b.box >> 8) & 255u), i1 = T.x0 + (int)((b.box >> 16) & 255u);
    const int j0 = T.y0 + (int)(b.box >> 24), j1 = T.y0 + (int)b.j1;
    const uint32_t cls = b.box & 255u;
    const int bw = i1 - i0 + 1, bh = j1 - j0 + 1;
    const int lcw = bw > 1 ? 32 - __clz(bw - 1) : 0;   // log2 of the column count
    const int lx = lane & ((1 << lcw) - 1), ly = lane >> lcw;
    const int rows = 64 >> lcw;
    const int i = i0 + lx;
    const bool colok = lx < bw;
    I f0 = edge_f<I>(b.X1, b.Y1, b.X2, b.Y2, i, j0 + ly);
    I f1 = edge_f<I>(b.X2, b.Y2, b.X0, b.Y0, i, j0 + ly);
    I f2 = edge_f<I>(b.X0, b.Y0, b.X1, b.Y1, i, j0 + ly);
    const I st0 = (I)(b.X2 - b.X1) * (I)(256 * rows);
    const I st1 = (I)(b.X0 - b.X2) * (I)(256 * rows);
    const I st2 = (I)(b.X1 - b.X0) * (I)(256 * rows);
    const float pxf = ((float)i + 0.5f) - P.cx;
    uint32_t* col = &S.fb[i - T.x0];
    for (int jr = ly; jr < bh; jr += rows) {
        const int j = j0 + jr;
        if (P.stats && lane == 0) atomicAdd(&S.stat[22], 64u);
        if (colok && (f0 | f1 | f2) >= 0) {
            const float pyf = ((float)j + 0.5f) - P.cy;
            if (P.stats) atomicAdd(&S.stat[13], 1u);
            atomicMin(&col[(j - T.y0) * T.w], pixel_key(P, pxf, pyf, b.pa, b.pb, b.pc, cls));
        }
        f0 += st0; f1 += st1; f2 += st2;
    }
}

// Drain the block-wide queue of large triangles: each wave takes the next
// one until none is left.  Called by the whole block.
__device__ __forceinline__ void drain_big(const RenderParams& P, Shared& S, const Tile& T)
{
    TSTART(tw);
    const uint32_t n = min(S.n_big, (uint32_t)kBigCap);
    for (;;) {
        uint32_t e = 0;
        if (lane_id() == 0) e = atomicAdd(&S.big_next, 1u);
        e = __builtin_amdgcn_readfirstlane(e);
        if (e >= n) break;
        const BigTri b = S.big[e];
        const int minX = min(b.X0, min(b.X1, b.X2)), maxX = max(b.X0, max(b.X1, b.X2));
        const int minY = min(b.Y0, min(b.Y1, b.Y2)), maxY = max(b.Y0, max(b.Y1, b.Y2));
        if ((maxX - minX) < 16384 && (maxY - minY) < 16384) raster_wave<int>(P, S, T, b);
        else raster_wave<long long>(P, S, T, b);
    }
    TACC(21, tw);
}

// ---------------------------------------------------------------------------
// exact pass: one queued survivor per live lane
// ---------------------------------------------------------------------------

__device__ __forceinline__ void exact_pass(const RenderParams& P, Shared& S, const Tile& T, const Cam& cam,
                                           bool live, uint32_t entry, int64_t abase_w)
{
    float tri[9];
    uint32_t cls = 0;
    int np = 0;
    int X0 = 0, Y0 = 0, X1 = 0, Y1 = 0, X2 = 0, Y2 = 0, X3 = 0, Y3 = 0;
    if (live) {
        load_entry(P, entry, abase_w, tri, cls);
        float xv[3], yv[3], zv[3];
#pragma unroll
        for (int k = 0; k < 3; ++k) view_xform(cam, tri[3 * k], tri[3 * k + 1], tri[3 * k + 2], xv[k], yv[k], zv[k]);
        const bool in0 = zv[0] >= P.nearp, in1 = zv[1] >= P.nearp, in2 = zv[2] >= P.nearp;
        bool ok = true;
        if (in0 && in1 && in2) {
            ok = snap_vertex(P, xv[0], yv[0], zv[0], X0, Y0) && snap_vertex(P, xv[1], yv[1], zv[1], X1, Y1) &&
                 snap_vertex(P, xv[2], yv[2], zv[2], X2, Y2);
            np = 3;
        } else {
            // R4: Sutherland-Hodgman output of the six straddling cases, in
            // the order in which v0v1, v1v2, v2v0 visit the edges.
            STAT(8, 1);
            float x01 = 0, y01 = 0, x12 = 0, y12 = 0, x20 = 0, y20 = 0;
            if (in0 != in1) {
                if (in0) near_cross(P, xv[0], yv[0], zv[0], xv[1], yv[1], zv[1], x01, y01);
                else near_cross(P, xv[1], yv[1], zv[1], xv[0], yv[0], zv[0], x01, y01);
            }
            if (in1 != in2) {
                if (in1) near_cross(P, xv[1], yv[1], zv[1], xv[2], yv[2], zv[2], x12, y12);
                else near_cross(P, xv[2], yv[2], zv[2], xv[1], yv[1], zv[1], x12, y12);
            }
            if (in2 != in0) {
                if (in2) near_cross(P, xv[2], yv[2], zv[2], xv[0], yv[0], zv[0], x20, y20);
                else near_cross(P, xv[0], yv[0], zv[0], xv[2], yv[2], zv[2], x20, y20);
            }
            const float nz = P.nearp;
            float px[4], py[4], pz[4];
            const int mcase = (in0 ? 1 : 0) | (in1 ? 2 : 0) | (in2 ? 4 : 0);
            auto setp = [&](int k, float x, float y, float z) { px[k] = x; py[k] = y; pz[k] = z; };
            switch (mcase) {
            case 1: setp(0, xv[0], yv[0], zv[0]); setp(1, x01, y01, nz); setp(2, x20, y20, nz); np = 3; break;
            case 2: setp(0, x01, y01, nz); setp(1, xv[1], yv[1], zv[1]); setp(2, x12, y12, nz); np = 3; break;
            case 4: setp(0, x12, y12, nz); setp(1, xv[2], yv[2], zv[2]); setp(2, x20, y20, nz); np = 3; break;
            case 3: setp(0, xv[0], yv[0], zv[0]); setp(1, xv[1], yv[1], zv[1]); setp(2, x12, y12, nz);
                    setp(3, x20, y20, nz); np = 4; break;
            case 5: setp(0, xv[0], yv[0], zv[0]); setp(1, x01, y01, nz); setp(2, x12, y12, nz);
                    setp(3, xv[2], yv[2], zv[2]); np = 4; break;
            default: setp(0, x01, y01, nz); setp(1, xv[1], yv[1], zv[1]); setp(2, xv[2], yv[2], zv[2]);
                     setp(3, x20, y20, nz); np = 4; break;   // case 6
            }
            if (np == 3) { px[3] = px[2]; py[3] = py[2]; pz[3] = pz[2]; }
            ok = snap_vertex(P, px[0], py[0], pz[0], X0, Y0) && snap_vertex(P, px[1], py[1], pz[1], X1, Y1) &&
                 snap_vertex(P, px[2], py[2], pz[2], X2, Y2) && snap_vertex(P, px[3], py[3], pz[3], X3, Y3);
        }
        if (!ok) np = 0;
    }
    bool have_plane = false, plane_bad = false;
    float pa = 0.0f, pb = 0.0f, pc = 0.0f;
    // fan triangles (p0, p1, p2) and (p0, p2, p3)
#pragma unroll 1
    for (int f = 0; f < 2; ++f) {
        if (!(live && f + 2 < np && !plane_bad)) continue;
        const int ax = X0, ay = Y0;
        int bx = f == 0 ? X1 : X2, by = f == 0 ? Y1 : Y2;
        int cx = f == 0 ? X2 : X3, cy = f == 0 ? Y2 : Y3;
        const int minX = min(ax, min(bx, cx)), maxX = max(ax, max(bx, cx));
        const int minY = min(ay, min(by, cy)), maxY = max(ay, max(by, cy));
        const int i0 = max((minX - 128 + 255) >> 8, T.x0), i1 = min((maxX - 128) >> 8, T.x0 + T.w - 1);
        const int j0 = max((minY - 128 + 255) >> 8, T.y0), j1 = min((maxY - 128) >> 8, T.y0 + T.h - 1);
        if (i0 > i1 || j0 > j1) continue;
        STAT(9, 1);
        const bool small_span = (maxX - minX) < 16384 && (maxY - minY) < 16384;
        long long area2;
        if (small_span) area2 = (long long)(__mul24(bx - ax, cy - ay) - __mul24(by - ay, cx - ax));
        else area2 = (long long)(bx - ax) * (long long)(cy - ay) - (long long)(by - ay) * (long long)(cx - ax);
        if (area2 == 0) continue;
        if (area2 < 0) {
            const int tx = bx, ty = by;
            bx = cx; by = cy; cx = tx; cy = ty;
        }
        if (!have_plane) {
            have_plane = depth_plane(P, cam, tri, pa, pb, pc);
            plane_bad = !have_plane;
            if (plane_bad) continue;
        }
        STAT(10, 1);
        const int npx = (i1 - i0 + 1) * (j1 - j0 + 1);
        if (npx > kSmallPx) {
            const uint32_t slot = atomicAdd(&S.n_big, 1u);
            if (slot < (uint32_t)kBigCap) {
                STAT(11, 1);
                BigTri& q = S.big[slot];
                q.X0 = ax; q.Y0 = ay; q.X1 = bx; q.Y1 = by; q.X2 = cx; q.Y2 = cy;
                q.pa = pa; q.pb = pb; q.pc = pc;
                q.box = cls | (uint32_t)(i0 - T.x0) << 8 | (uint32_t)(i1 - T.x0) << 16 | (uint32_t)(j0 - T.y0) << 24;
                q.j1 = (uint32_t)(j1 - T.y0);
                continue;
            }
            STAT(14, 1);   // queue full: rasterized by this lane instead
        }
        STAT(12, npx);
        if (small_span) raster_lane<int>(P, S, T, ax, ay, bx, by, cx, cy, i0, i1, j0, j1, pa, pb, pc, cls);
        else raster_lane<long long>(P, S, T, ax, ay, bx, by, cx, cy, i0, i1, j0, j1, pa, pb, pc, cls);
    }
}

// Append the lanes with `pred` to this wave's queue (ballot + mbcnt, no
// atomics); returns the new depth, which is uniform across the wave.
__device__ __forceinline__ int queue_push(Shared& S, int wid, int nq, bool pred, uint32_t val)
{
    const uint64_t m = __ballot(pred);
    const uint32_t rank = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
    if (pred) S.q[wid][nq + rank] = val;
    return nq + (int)__popcll(m);
}

// In-place inclusive max-scan of the candidate markers mark[0, kCandCap):
// thread t owns the kMarksPerThread consecutive markers starting at
// t * kMarksPerThread, so the block covers exactly kCandCap of them.
constexpr int kMarksPerThread = kCandCap / kBlock;
static_assert(kMarksPerThread * kBlock == kCandCap, "every marker must belong to one thread");
static_assert(kMarksPerThread % 2 == 0, "markers are cleared two at a time");

__device__ __forceinline__ void max_scan_marks(Shared& S)
{
    const int tid = threadIdx.x, lane = lane_id(), wid = tid >> 6;
    uint16_t* m = S.u.mark + kMarksPerThread * tid;
    uint32_t v[kMarksPerThread];
#pragma unroll
    for (int q = 0; q < kMarksPerThread; ++q) v[q] = m[q];
#pragma unroll
    for (int q = 1; q < kMarksPerThread; ++q) v[q] = max(v[q], v[q - 1]);
    uint32_t x = v[kMarksPerThread - 1];
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        const uint32_t y = __shfl_up(x, o);
        if (lane >= o) x = max(x, y);
    }
    if (lane == 63) S.s_wave[wid] = x;
    __syncthreads();
    uint32_t pre = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w)
        if (w < wid) pre = max(pre, S.s_wave[w]);
    uint32_t xe = __shfl_up(x, 1);
    if (lane == 0) xe = 0;
    const uint32_t base = max(pre, xe);
#pragma unroll
    for (int q = 0; q < kMarksPerThread; ++q) m[q] = (uint16_t)max(v[q], base);
    __syncthreads();
}

// Conservative AABB-vs-plane test: true if the box lies entirely on the
// negative side of n.(P - C) + o.
__device__ __forceinline__ bool box_outside(float cx, float cy, float cz, float hx, float hy, float hz,
                                            float nx, float ny, float nz, float o)
{
    const float v = nx * cx + ny * cy + nz * cz + fabsf(nx) * hx + fabsf(ny) * hy + fabsf(nz) * hz + o;
    const float mag = fabsf(nx) * (fabsf(cx) + hx) + fabsf(ny) * (fabsf(cy) + hy) + fabsf(nz) * (fabsf(cz) + hz)
                      + fabsf(o);
    return v < -1e-4f * mag;
}

struct WorldPlanes {
    float n[6][3];
    float o[6];
};

// Can anything inside the axis-aligned box set a key of the tile?  False if
// the box is outside a frustum plane, or if it lies wholly in front of the
// near plane and its projection holds no pixel centre of the tile.
__device__ __forceinline__ bool aabb_visible(const RenderParams& P, const Tile& T, const WorldPlanes& F,
                                             const Cam& cam, float lox, float loy, float loz, float hix, float hiy,
                                             float hiz)
{
    const float cx = (lox + hix) * 0.5f - cam.x, cy = (loy + hiy) * 0.5f - cam.y, cz = (loz + hiz) * 0.5f - cam.z;
    const float hx = (hix - lox) * 0.5f, hy = (hiy - loy) * 0.5f, hz = (hiz - loz) * 0.5f;
#pragma unroll
    for (int p = 0; p < 6; ++p)
        if (box_outside(cx, cy, cz, hx, hy, hz, F.n[p][0], F.n[p][1], F.n[p][2], F.o[p])) return false;
    // projection of the box: its four vertical edges (yaw-only camera)
    float zmn = 3.0e38f, zmx = -3.0e38f, xmn = 3.0e38f, xmx = -3.0e38f, mag = 0.0f;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const float dx = ((k & 1) ? hix : lox) - cam.x, dy = ((k & 2) ? hiy : loy) - cam.y;
        const float xv = dx * cam.sc - dy * cam.cc, zv = dx * cam.cc + dy * cam.sc;
        zmn = fminf(zmn, zv); zmx = fmaxf(zmx, zv);
        const float px = P.cx + P.fx * (xv * __builtin_amdgcn_rcpf(zv));
        xmn = fminf(xmn, px); xmx = fmaxf(xmx, px);
        mag = fmaxf(mag, fabsf(px));
    }
    if (!(zmn >= P.nearp * 1.00390625f)) return true;   // crosses or nearly touches the near plane
    const float r0 = __builtin_amdgcn_rcpf(zmn), r1 = __builtin_amdgcn_rcpf(zmx);
    const float ylo = loz - cam.z, yhi = hiz - cam.z;
    const float y0 = P.cy - P.fy * (yhi * r0), y1 = P.cy - P.fy * (yhi * r1);
    const float y2 = P.cy - P.fy * (ylo * r0), y3 = P.cy - P.fy * (ylo * r1);
    const float ymn = fminf(fminf(y0, y1), fminf(y2, y3)), ymx = fmaxf(fmaxf(y0, y1), fmaxf(y2, y3));
    mag = fmaxf(mag, fmaxf(fabsf(ymn), fabsf(ymx)));
    // 1e-5 relative slack for the fp32 transform of the box corners
    const float sx = 1e-5f * (fabsf(xmn) + fabsf(xmx) + P.fx), sy = 1e-5f * (fabsf(ymn) + fabsf(ymx) + P.fy);
    return box_has_centre(P, T, xmn - sx, xmx + sx, ymn - sy, ymx + sy, mag);
}

__device__ __forceinline__ int64_t xcd_remap(int64_t b, int64_t nb)
{
    // Workgroups are dispatched round-robin over the 8 XCDs; give each XCD a
    // contiguous range of views so that one world's views share an L2.
    const int64_t q = nb >> 3, r = nb & 7, x = b & 7, k = b >> 3;
    return x * q + (x < r ? x : r) + k;
}

__device__ __forceinline__ float decode_depth(const RenderParams& P, uint32_t key)
{
    const float d = __uint_as_float(((P.qbase - (key >> 8)) << 3) | 4u);
    return P.fast_decode ? rcp_rn(d) : 1.0f / d;
}

__global__ __launch_bounds__(kBlock, 4) void render_views_kernel(const RenderParams P)
{
    __shared__ Shared S;
    const int tid = threadIdx.x, lane = lane_id(), wid = tid >> 6;
    TSTART(t_kernel);
    const int64_t blk = xcd_remap((int64_t)blockIdx.x, P.num_blocks);
    const int tiles = P.tiles_x * P.tiles_y;
    const int64_t v = blk / tiles;
    const int tile = (int)(blk % tiles);

    // R1: camera of view v
    const int64_t per_world = (int64_t)P.A * P.C;
    const int w = (int)(v / per_world);
    const int a = (int)((v / P.C) % P.A);
    const int k = (int)(v % P.C);
    const int64_t g = (int64_t)w * P.A + a;
    Cam cam;
    {
        const float c = P.ac[g], s = P.as[g];
        const float mx = P.mount[k][0], my = P.mount[k][1], mz = P.mount[k][2];
        const float cm = P.mount[k][3], sm = P.mount[k][4];
        const float t1 = mx * c, t2 = my * s, t3 = mx * s, t4 = my * c;
        const float ox = t1 - t2, oy = t3 + t4;
        cam.x = P.ax[g] + ox;
        cam.y = P.ay[g] + oy;
        cam.z = P.az0[g] + mz;
        const float u1 = c * cm, u2 = s * sm, u3 = s * cm, u4 = c * sm;
        cam.cc = u1 - u2;
        cam.sc = u3 + u4;
    }
    Tile T;
    T.x0 = (tile % P.tiles_x) * P.tile_w;
    T.y0 = (tile / P.tiles_x) * P.tile_h;
    T.w = min(P.tile_w, P.W - T.x0);
    T.h = min(P.tile_h, P.H - T.y0);
    T.kl = ((float)T.x0 - 0.5f) - P.cx;
    T.kr = ((float)(T.x0 + T.w) + 0.5f) - P.cx;
    T.kt = P.cy - ((float)T.y0 - 0.5f);
    T.kb = P.cy - ((float)(T.y0 + T.h) + 0.5f);
    const int npx = T.w * T.h;
    const bool cull = P.cull != 0;

    {
        const u32x4 clr = {kClearKey, kClearKey, kClearKey, kClearKey};
        const int n4 = npx & ~3;
        for (int p = 4 * tid; p < n4; p += 4 * kBlock) *(u32x4*)&S.fb[p] = clr;
        if (tid < npx - n4) S.fb[n4 + tid] = kClearKey;
    }
    if (tid == 0) { S.n_cells = 0; S.n_vis = 0; S.n_big = 0; S.big_next = 0; }
    if (P.stats && tid < kNumStats) S.stat[tid] = 0;

    // world-space frustum planes of the tile: four side planes through the
    // camera centre, near and far with margins
    WorldPlanes F;
    {
        const float cc = cam.cc, sc = cam.sc;
        F.n[0][0] = P.fx * sc - T.kl * cc; F.n[0][1] = -P.fx * cc - T.kl * sc; F.n[0][2] = 0.0f; F.o[0] = 0.0f;
        F.n[1][0] = T.kr * cc - P.fx * sc; F.n[1][1] = T.kr * sc + P.fx * cc; F.n[1][2] = 0.0f; F.o[1] = 0.0f;
        F.n[2][0] = T.kt * cc; F.n[2][1] = T.kt * sc; F.n[2][2] = -P.fy; F.o[2] = 0.0f;
        F.n[3][0] = -T.kb * cc; F.n[3][1] = -T.kb * sc; F.n[3][2] = P.fy; F.o[3] = 0.0f;
        F.n[4][0] = cc; F.n[4][1] = sc; F.n[4][2] = 0.0f; F.o[4] = -P.nearp * 0.99609375f;
        F.n[5][0] = -cc; F.n[5][1] = -sc; F.n[5][2] = 0.0f; F.o[5] = P.farp * 1.015625f;
    }

    const WorldGrid grid = P.scene.grids[w];
    const float cs = P.scene.cell_size;
    // rectangle of cells covering the tile frustum's xy footprint up to far
    int ix0 = 0, iy0 = 0, ix1 = grid.nx - 1, iy1 = grid.ny - 1;
    if (cull) {
        const float fz = P.farp * 1.015625f;
        const float tl = T.kl / P.fx, tr = T.kr / P.fx;
        const float ax_ = cam.cc + tl * cam.sc, ay_ = cam.sc - tl * cam.cc;   // f + tl r
        const float bx_ = cam.cc + tr * cam.sc, by_ = cam.sc - tr * cam.cc;   // f + tr r
        const float p1x = cam.x + fz * ax_, p1y = cam.y + fz * ay_;
        const float p2x = cam.x + fz * bx_, p2y = cam.y + fz * by_;
        const float mg = grid.margin + 1.0f;
        const float xlo = fminf(cam.x, fminf(p1x, p2x)) - mg, xhi = fmaxf(cam.x, fmaxf(p1x, p2x)) + mg;
        const float ylo = fminf(cam.y, fminf(p1y, p2y)) - mg, yhi = fmaxf(cam.y, fmaxf(p1y, p2y)) + mg;
        const float fx0 = floorf((xlo - grid.ox) / cs) - 1.0f, fx1 = floorf((xhi - grid.ox) / cs) + 1.0f;
        const float fy0 = floorf((ylo - grid.oy) / cs) - 1.0f, fy1 = floorf((yhi - grid.oy) / cs) + 1.0f;
        ix0 = (int)fmaxf(fx0, 0.0f); iy0 = (int)fmaxf(fy0, 0.0f);
        ix1 = (int)fminf(fx1, (float)(grid.nx - 1)); iy1 = (int)fminf(fy1, (float)(grid.ny - 1));
    }
    const int rw = ix1 - ix0 + 1, rh = iy1 - iy0 + 1;
    const int nrect = (rw > 0 && rh > 0) ? rw * rh : 0;
    const int64_t abase_w = (int64_t)w * P.A;
    int nq = 0;   // depth of this wave's survivor queue (wave-uniform)
    __syncthreads();
    if (tid == 0) { STAT(0, 1); STAT(1, nrect); }
    TACC(16, t_kernel);

    // ---- candidates: static triangles, then agent boxes, then drain ------
    // One phase = one block-wide setup (with barriers) followed by per-wave
    // work without barriers.  A single loop keeps a single inlined copy of
    // the first and exact passes (instruction-cache footprint).
    enum { kStatic = 0, kBoxes = 1, kDrain = 2 };
    int rb = 0, ab = 0;
    uint32_t total = 0, kb = 0, nc = 0;
    bool static_done = nrect == 0;
    for (;;) {
        int kind = kDrain;
        uint32_t nphase = 0;
        TSTART(t_setup);
        if (!static_done) {
            while (kb >= total && rb < nrect) {
                // test one cell per thread, compact the visible ones
                const int r = rb + tid;
                bool vis = false;
                uint32_t start = 0, cnt = 0;
                if (r < nrect) {
                    const int c = grid.cell_base + (iy0 + r / rw) * grid.nx + (ix0 + r % rw);
                    start = P.scene.cell_start[c];
                    cnt = P.scene.cell_start[c + 1] - start;
                    if (cnt > 0) {
                        vis = true;
                        if (cull) {
                            const float4 lo = P.scene.cell_lo[c], hi = P.scene.cell_hi[c];
                            vis = aabb_visible(P, T, F, cam, lo.x, lo.y, lo.z, hi.x, hi.y, hi.z);
                        }
                    }
                }
                const uint32_t slot = wave_append(vis, &S.n_cells);
                if (vis) { S.cl_start[slot] = start; S.cl_pre[slot] = cnt; STAT(2, 1); STAT(3, cnt); }
                __syncthreads();
                nc = S.n_cells;
                {
                    const uint32_t cn = tid < (int)nc ? S.cl_pre[tid] : 0u;
                    uint32_t tot;
                    const uint32_t off = block_excl_scan(cn, S.s_wave, tot);
                    if (tid < (int)nc) S.cl_pre[tid] = off;
                    if (tid == 0) { S.cl_pre[nc] = tot; S.n_cells = 0; }
                }
                __syncthreads();
                total = S.cl_pre[nc];
                kb = 0;
                rb += kBlock;
                __syncthreads();   // the list may be rewritten by the next batch
            }
            if (kb < total) {
                kind = kStatic;
                nphase = min(total - kb, (uint32_t)kCandCap);
                if (tid == 0) STAT(15, 1);
                for (int q = tid; q < kCandCap / 2; q += kBlock) ((uint32_t*)S.u.mark)[q] = 0u;
                __syncthreads();
                if (tid < (int)nc) {
                    const uint32_t ca = S.cl_pre[tid], ce = S.cl_pre[tid + 1];
                    if (ce > kb && ca < kb + nphase) S.u.mark[ca > kb ? ca - kb : 0u] = (uint16_t)(tid + 1);
                }
                __syncthreads();
                max_scan_marks(S);
            } else {
                static_done = true;
            }
        }
        if (static_done) {
            if (ab < P.A) {
                // box cull of one batch of agents, ballot compaction
                kind = kBoxes;
                const int ai = ab + tid;
                bool vis = false;
                if (ai < P.A && ai != a) {
                    vis = true;
                    if (cull) {
                        const int64_t h = abase_w + ai;
                        const float x = P.ax[h], y = P.ay[h], z0 = P.az0[h];
                        const float R = 0.5f * (P.al[h] + P.aw[h]) * 1.0009765625f + 0.0009765625f;
                        vis = aabb_visible(P, T, F, cam, x - R, y - R, z0, x + R, y + R, z0 + P.ah[h]);
                    }
                }
                const uint32_t slot = wave_append(vis, &S.n_vis);
                if (vis) { S.u.vis[slot] = (uint32_t)ai; STAT(4, 1); STAT(5, 12); }
                __syncthreads();
                nphase = S.n_vis * 12u;
                ab += kAgentBatch;
            } else {
                // drain: pool the leftover survivors of all waves
                if (lane == 0) S.nq_w[wid] = (uint32_t)nq;
                __syncthreads();
            }
        }
        TACC(17, t_setup);
        // per-wave work: first pass over 64 candidates at a time and an exact
        // pass on every 64 survivors; when draining, exact passes over the
        // pooled leftovers
        long long t_exact_sum = 0;
        TSTART(t_work);
        uint32_t pw[kWaves + 1];
        uint32_t nbatch = 0;
        pw[0] = 0;
        if (kind == kDrain) {
#pragma unroll
            for (int q = 0; q < kWaves; ++q) pw[q + 1] = pw[q] + S.nq_w[q];
            nbatch = (pw[kWaves] + 63u) / 64u;
        }
        for (uint32_t it = 0;; ++it) {
            bool run = false, live = false;
            uint32_t entry = 0;
            if (kind != kDrain) {
                const uint32_t bb = 64u * (wid + kWaves * it);
                if (bb >= nphase) break;
                const uint32_t kk = bb + lane;
                bool surv = false;
                uint32_t val = 0;
                if (kk < nphase) {
                    float tri[9];
                    uint32_t cls;
                    if (kind == kStatic) {
                        // (the clamp only turns a mapping slip into a parity failure, never an OOB read)
                        const uint32_t j = min((uint32_t)S.u.mark[kk] - 1u, nc - 1u);
                        val = S.cl_start[j] + (kb + kk - S.cl_pre[j]);
                        load_static(P, val, tri, cls);
                    } else {
                        const uint32_t aj = S.u.vis[kk / 12u];
                        const uint32_t face = kk % 12u;
                        load_box(P, abase_w + aj, (int)face, tri, cls);
                        val = kBoxFlag | (aj << 4) | face;
                    }
                    surv = first_pass(P, T, cam, tri, cull);
                }
                if (surv) STAT(6, 1);
                nq = queue_push(S, wid, nq, surv, val);
                if (nq >= 64) {
                    nq -= 64;
                    run = true;
                    live = true;
                    entry = S.q[wid][nq + lane];
                }
            } else {
                const uint32_t batch = wid + kWaves * it;
                if (batch >= nbatch) break;
                const uint32_t e = 64u * batch + lane;
                run = true;
                live = e < pw[kWaves];
                if (live) {
                    int src = 0;
#pragma unroll
                    for (int q = 1; q < kWaves; ++q)
                        if (e >= pw[q]) src = q;
                    entry = S.q[src][e - pw[src]];
                }
            }
            if (run) {
                if (lane == 0) STAT(7, 1);
                TSTART(t_ex);
                exact_pass(P, S, T, cam, live, entry, abase_w);
                if (P.stats) t_exact_sum += (long long)__builtin_amdgcn_s_memtime() - t_ex;
            }
        }
        if (P.stats && lane == 0) {
            atomicAdd(&S.stat[19], (uint32_t)t_exact_sum);
            atomicAdd(&S.stat[18], (uint32_t)((long long)__builtin_amdgcn_s_memtime() - t_work - t_exact_sum));
        }
        TSTART(t_bar);
        __syncthreads();
        TACC(20, t_bar);
        // rasterize the queued large triangles once the queue is half full,
        // and at the end
        if (kind == kDrain || S.n_big >= (uint32_t)(kBigCap / 2)) {
            drain_big(P, S, T);
            __syncthreads();
            if (tid == 0) { S.n_big = 0; S.big_next = 0; }
            __syncthreads();
        }
        if (kind == kDrain) break;
        if (kind == kStatic) {
            kb += kCandCap;
        } else {
            if (tid == 0) S.n_vis = 0;
            __syncthreads();
        }
    }

    // ---- R8 resolve + coalesced write-out of the tile ----
    TSTART(t_out);
    const int64_t view_px = (int64_t)P.W * P.H;
    uint8_t* ocls = P.out_cls + v * view_px;
    float* odep = P.out_depth + v * view_px;
    if (P.vec_out && (P.W % 16) == 0 && (T.w % 16) == 0) {
        const int u16 = T.w / 16, n16 = u16 * T.h;
        for (int u = tid; u < n16; u += kBlock) {
            const int row = u / u16, c16 = u % u16;
            const u32x4* src = (const u32x4*)&S.fb[row * T.w + 16 * c16];
            uint32_t wd[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const u32x4 kq = src[q];
                wd[q] = (kq.x & 255u) | ((kq.y & 255u) << 8) | ((kq.z & 255u) << 16) | ((kq.w & 255u) << 24);
            }
            const u32x4 pk = {wd[0], wd[1], wd[2], wd[3]};
            __builtin_nontemporal_store(pk, (u32x4*)(ocls + (int64_t)(T.y0 + row) * P.W + T.x0 + 16 * c16));
        }
        const int u4 = T.w / 4, n4 = u4 * T.h;
        const float inf = __uint_as_float(0x7F800000u);
        for (int u = tid; u < n4; u += kBlock) {
            const int row = u / u4, c4 = u % u4;
            const u32x4 kq = *(const u32x4*)&S.fb[row * T.w + 4 * c4];
            f32x4 d = {inf, inf, inf, inf};
            if ((kq.x & kq.y & kq.z & kq.w) >> 8 != 0xFFFFFFu) {   // not all background
                d.x = (kq.x >> 8) == 0xFFFFFFu ? inf : decode_depth(P, kq.x);
                d.y = (kq.y >> 8) == 0xFFFFFFu ? inf : decode_depth(P, kq.y);
                d.z = (kq.z >> 8) == 0xFFFFFFu ? inf : decode_depth(P, kq.z);
                d.w = (kq.w >> 8) == 0xFFFFFFu ? inf : decode_depth(P, kq.w);
            }
            __builtin_nontemporal_store(d, (f32x4*)(odep + (int64_t)(T.y0 + row) * P.W + T.x0 + 4 * c4));
        }
    } else {
        for (int p = tid; p < npx; p += kBlock) {
            const int row = p / T.w, col = p % T.w;
            const uint32_t key = S.fb[p];
            const int64_t o = (int64_t)(T.y0 + row) * P.W + T.x0 + col;
            ocls[o] = (uint8_t)(key & 255u);
            odep[o] = (key >> 8) == 0xFFFFFFu ? __uint_as_float(0x7F800000u) : decode_depth(P, key);
        }
    }
    if (P.stats) {
        TACC(23, t_out);
        __syncthreads();
        if (tid < kNumStats) atomicAdd(&P.stats[tid], (unsigned long long)S.stat[tid]);
    }
}

hipError_t launch_render(const RenderParams& p, hipStream_t s)
{
    if (p.num_blocks <= 0) return hipSuccess;
    hipLaunchKernelGGL(render_views_kernel, dim3((unsigned)p.num_blocks), dim3(kBlock), 0, s, p);
    return hipGetLastError();
}

// Device self-check of rcp_rn: counts the fp32 values x in [lo, lo + n)
// (as bit patterns) where rcp_rn(x) differs from 1.0f / x.
__global__ void rcp_check_kernel(uint32_t lo_bits, uint32_t n, unsigned long long* mismatches)
{
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const float x = __uint_as_float(lo_bits + i);
    if (__float_as_uint(rcp_rn(x)) != __float_as_uint(1.0f / x)) atomicAdd(mismatches, 1ull);
}

hipError_t launch_rcp_check(uint32_t lo_bits, uint32_t n, unsigned long long* mismatches, hipStream_t s)
{
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(rcp_check_kernel, dim3((n + 255u) / 256u), dim3(256), 0, s, lo_bits, n, mismatches);
    return hipGetLastError();
}

}  // namespace pictura
