/*
 * Plain CPU oracle of the batched class/depth view rasterizer.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark load this library.  It shares no code,
 * header, table or constant generator with the HIP library: it is written
 * from the rasterization rules below, never from the kernels.
 *
 * What it computes (paper Sec. 3.2, Eq. obs_pv): for every agent i and camera
 * k of its rig, a deterministic image Phi(A_i, W_i, K_ik) of the surrounding
 * agents' boxes and the static map geometry seen through a pinhole camera
 * with the configured intrinsics and extrinsics; the ego's own body is not
 * drawn ("only the surroundings are rendered").  The paper draws flat-shaded
 * RGB; this path draws, per pixel, the semantic class of the visible surface
 * and its view-space depth.  The paper gives no rasterization internals, so
 * the rules are fixed here (and identically, in separate code, on the GPU):
 *
 *  R1 camera   C = agent + Rot(heading) * mount.xy, Cz = z0 + mount.z;
 *              camera heading (cc, sc) = heading (+) mount yaw, as
 *              cc = c*cm - s*sm, sc = s*cm + c*sm (fp32, no contraction).
 *              forward f = (cc, sc, 0), right r = (sc, -cc, 0), up (0, 0, 1)
 *              (ego frame x forward, y left, z up; App. A.2 Tab. camera_rig).
 *  R2 view     d = P - C;  xv = d.x*sc - d.y*cc;  yv = d.z;  zv = d.x*cc + d.y*sc.
 *  R3 depth    plane of the unsnapped triangle: N = (V1-V0) x (V2-V0) in world
 *              space, n_view = (N.x*sc - N.y*cc, N.z, N.x*cc + N.y*sc),
 *              delta = N . (V0 - C); delta == 0 drops the triangle.  With
 *              rd = 1/delta:  pa = (nx*rd)*(1/fx), pb = -(ny*rd)*(1/fy),
 *              pc = nz*rd, and at pixel (i, j):
 *              iz = fma(pa, i+0.5-cx, fma(pb, j+0.5-cy, pc))   (= 1/zv).
 *  R4 near     a triangle with every vertex at zv < near, or every vertex at
 *              zv > far, is not drawn.  Otherwise
 *              Sutherland-Hodgman against zv >= near, edges v0v1, v1v2, v2v0;
 *              each crossing point is computed from the inside vertex I
 *              towards the outside vertex O: t = (near - I.z)/(O.z - I.z),
 *              x = fma(t, O.x - I.x, I.x), y likewise, z = near; the 3- or
 *              4-gon is fanned from its first vertex.  (Parity unpinned: which
 *              end the crossing point is computed from only changes its last
 *              bits, and either choice is watertight; no closed form fixes it,
 *              so only the GPU comparison checks that both sides agree.)
 *  R5 snap     rz = 1/zv;  X = rint(256cx + 256fx*(xv*rz)),
 *              Y = rint(256cy - 256fy*(yv*rz))   (8-bit subpixel, ties to
 *              even); a coordinate with |value| > 2^29 (or NaN) drops the
 *              triangle.
 *  R6 fill     integer edge functions E_ab(p) = (b.x-a.x)(p.y-a.y) -
 *              (b.y-a.y)(p.x-a.x) at pixel centres p = (256i+128, 256j+128);
 *              area2 = E_01(v2): 0 drops, < 0 swaps v1 and v2 (two-sided).
 *              Edge a->b is top-left iff dy < 0 or (dy == 0 and dx > 0)
 *              (y grows downwards).  Covered iff every edge has E > 0, or
 *              E == 0 and the edge is top-left.
 *  R7 key      iz < 1/far (or NaN) rejects the pixel; iz = min(iz, IZCAP)
 *              with IZCAP the smallest power of two >= 1/near;
 *              q = (bits(IZCAP) >> 3) - (bits(iz) >> 3)  (24-bit reverse
 *              depth, monotone in z, relative step 2^-20);
 *              key = (q << 8) | class; the pixel keeps the minimum key, so
 *              the nearest surface wins and an exact depth tie goes to the
 *              lower class ID, whatever the triangle order.
 *  R8 resolve  class = key & 255; depth = +inf when q == 0xFFFFFF (the clear
 *              key carries the sky class 4), else
 *              1 / float_from_bits(((bits(IZCAP) >> 3) - q) << 3 | 4).
 *  R9 boxes    corners (x + (a*c - b*s), y + (a*s + b*c), z0 or z0 + H) with
 *              a = +-L/2, b = +-W/2; 12 triangles (two per face).
 *  R10 lights  (traffic-light disks visible only within a limited angular
 *              range, Sec. 3.2 rendering features) a light with centre L,
 *              horizontal normal (cf, sf) and cone cosine cos_max is drawn
 *              iff, with d = C - L, h = cf*d.x + sf*d.y and
 *              q = (d.x*d.x + d.y*d.y) + d.z*d.z:  h > 0 and
 *              h*h >= (cos_max*cos_max)*q.
 *  R11 disks   12 triangles (L, rim k, rim k+1 mod 12); rim k =
 *              (L.x - a*sf, L.y + a*cf, L.z + b) with a = r*cos(30k deg),
 *              b = r*sin(30k deg), the cosine and sine rounded to fp32.
 *
 * R13 colour (optional output): in colour mode the 12 triangles of a box use
 *              the shading id (class & 15) | (k/2 + 1) << 4 (k the triangle
 *              index of R9: faces bottom, top, back, front, right, left) in
 *              place of the class in the key; the class output is key & 15.
 *              The pixel colour is rint(255 * min(base * (factor * b), 1))
 *              per channel, base = palette[class] / 255, factor by face
 *              (0.45, 1, 0.55, 0.85, 0.7, 0.7; 1 off boxes), b = 1 - 0.6 *
 *              min(z * (1/far), 1) on box faces (z the output depth), else 1.
 * R14 antialiasing (optional, colour mode; the paper smooths edges with
 *              analytic coverage at one sample per pixel, Sec. 3.2 and its
 *              appendix on render quality): every surface leaves, on each
 *              pixel whose centre is within one pixel of its box, a fragment
 *              with coverage a8 = rint(255 a), a = clamp(sum of the edges'
 *              clamp(0.5 + signed centre distance in px) - (edges - 1)), when
 *              0 < a8 < 255 and its R7 key at the centre exists.  A surface
 *              is a strictly convex snapped 4-gon whose two fan pieces are
 *              both drawn (a pair of scene triangles (a, b, c), (a, c, d) in
 *              front of near and not beyond far, or a triangle clipped to
 *              four vertices; its key from the first piece's plane), else a
 *              single snapped fan piece.  The
 *              pixel keeps the least o = (key >> 16) << 16 | (key & 255) << 8
 *              | (255 - a8); a kept fragment not behind the centre's key
 *              (16-bit depth prefix) with another shading id blends over the
 *              centre's colour: (C_o a8 + C (255 - a8) + 127) / 255, C_o the
 *              colour of key ((o >> 16) << 16) | ((o >> 8) & 255).
 *
 * Instances (optional outputs; the road users' occlusion percentages the
 * paper's analysis reads from its renderer, Sec. 5.2): every other agent's box
 * is also drawn alone, with the same rules, into a frame of its own.  Its
 * footprint is the number of pixels that frame covers; a pixel belongs to
 * the lowest-index agent whose own frame holds the pixel's final key there
 * (-1: none); an agent's visible count is the number of pixels it owns.
 *
 * Arithmetic is IEEE fp32 with round-to-nearest and no contraction (this
 * file must be compiled with -ffp-contract=off and without -ffast-math);
 * fmaf() appears only where the rules name fma.  Integer edge functions are
 * exact in int64.
 *
 * Per pixel the oracle also reports parity flags:
 *   bit 0 EDGE  the pixel centre lies within 1e-4 px of an edge of a triangle
 *               whose key there is <= the winning key (a coverage decision
 *               that a one-quantum snap difference could flip);
 *   bit 1 TIE   the best surface of a different class is within 1e-4
 *               relative depth of the winner.
 * and, optionally, how many raster triangles cover the pixel (watertightness).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define SKY_CLASS 4u
#define CLEAR_KEY ((0xFFFFFFu << 8) | SKY_CLASS)

static uint32_t f2u(float f) { uint32_t u; memcpy(&u, &f, 4); return u; }
static float u2f(uint32_t u) { float f; memcpy(&f, &u, 4); return f; }

/* smallest power of two >= x (x > 0, normal) */
static float pow2_ceil(float x)
{
    uint32_t u = f2u(x);
    if ((u & 0x7FFFFFu) == 0) return x;
    return u2f((u & 0x7F800000u) + 0x00800000u);
}

typedef struct {
    float cx_, cy_, cz_;   /* camera position */
    float cc, sc;          /* camera heading */
} Cam;

typedef struct {
    int W, H;
    float fx, fy, cx, cy, nearp, farp;
    float fx256, fy256, cx256, cy256, rfx, rfy;
    float izfar, izcap;
    uint32_t qbase;
} Params;

/* R7: 24-bit reverse-depth code of an inverse depth; 0 when the far rule
 * rejects it (iz < 1/far or NaN), else 1 with *q set.  Depths nearer than the
 * cap (iz > IZCAP) take the cap's code 0. */
static int quantize_iz(const Params* P, float iz, uint32_t* q)
{
    if (!(iz >= P->izfar)) return 0;
    if (iz > P->izcap) iz = P->izcap;
    *q = P->qbase - (f2u(iz) >> 3);
    return 1;
}

/* R8: depth of a code (the midpoint of its bucket of eight fp32 inverse depths). */
static float decode_q(const Params* P, uint32_t q)
{
    return 1.0f / u2f(((P->qbase - q) << 3) | 4u);
}

typedef struct { float x, y, z; } V3;

static V3 to_view(const Cam* c, float px, float py, float pz)
{
    float dx = px - c->cx_, dy = py - c->cy_, dz = pz - c->cz_;
    V3 v;
    float a = dx * c->sc, b = dy * c->cc;
    v.x = a - b;
    v.y = dz;
    float e = dx * c->cc, f = dy * c->sc;
    v.z = e + f;
    return v;
}

/* R3: depth plane from the world-space triangle.  Returns 0 if dropped. */
static int depth_plane(const Cam* c, const Params* P, const float* t /*9*/,
                       float* pa, float* pb, float* pc)
{
    float e1x = t[3] - t[0], e1y = t[4] - t[1], e1z = t[5] - t[2];
    float e2x = t[6] - t[0], e2y = t[7] - t[1], e2z = t[8] - t[2];
    float Nx = e1y * e2z - e1z * e2y;
    float Ny = e1z * e2x - e1x * e2z;
    float Nz = e1x * e2y - e1y * e2x;
    float d0x = t[0] - c->cx_, d0y = t[1] - c->cy_, d0z = t[2] - c->cz_;
    float nx = Nx * c->sc - Ny * c->cc;
    float ny = Nz;
    float nz = Nx * c->cc + Ny * c->sc;
    float delta = (Nx * d0x + Ny * d0y) + Nz * d0z;
    if (delta == 0.0f || !isfinite(delta)) return 0;
    float rd = 1.0f / delta;
    *pa = (nx * rd) * P->rfx;
    *pb = -((ny * rd) * P->rfy);
    *pc = nz * rd;
    return 1;
}

typedef struct {
    uint32_t* key;      /* [H*W] min key */
    uint32_t* edge_key; /* [H*W] min key of fragile coverage decisions */
    uint32_t* k1;       /* best key */
    uint32_t* k2;       /* best key of a class different from k1's */
    uint16_t* cover;    /* optional coverage count */
    uint32_t* frag;     /* R14: [H*W] nearest partial-coverage fragment, or NULL */
} Frame;

static void frame_update_tie(Frame* F, int p, uint32_t k)
{
    uint32_t c = k & 255u;
    uint32_t k1 = F->k1[p], k2 = F->k2[p];
    if (c == (k1 & 255u)) {
        if (k < k1) F->k1[p] = k;
    } else if (k < k1) {
        F->k2[p] = k1;
        F->k1[p] = k;
    } else if (c == (k2 & 255u)) {
        if (k < k2) F->k2[p] = k;
    } else if (k < k2) {
        F->k2[p] = k;
    }
}

static int snap(const Params* P, V3 v, int32_t* X, int32_t* Y)
{
    float rz = 1.0f / v.z;
    float qx = v.x * rz, qy = v.y * rz;
    float mx = P->fx256 * qx, my = P->fy256 * qy;
    float sx = P->cx256 + mx, sy = P->cy256 - my;
    float rx = rintf(sx), ry = rintf(sy);
    if (!(fabsf(rx) <= 536870912.0f) || !(fabsf(ry) <= 536870912.0f)) return 0;
    *X = (int32_t)rx;
    *Y = (int32_t)ry;
    return 1;
}

static int64_t floor_div256(int64_t a) { return a >= 0 ? a / 256 : -((-a + 255) / 256); }

/* R14: analytic coverage of pixel centres near one snapped, positively
 * oriented triangle.  The coverage of a pixel by one edge's half-plane is
 * approximated by 0.5 plus the centre's signed distance to the edge in
 * pixels, clamped to [0, 1]; the triangle's coverage is the sum of its three
 * edges' coverages minus 2, clamped.  Pixels whose centre lies within one
 * pixel of the snapped bounding box are considered. */
static void coverage_fragments(const Params* P, Frame* F, const int32_t* vx, const int32_t* vy, float pa, float pb,
                               float pc, uint32_t cls)
{
    int32_t lo_x = vx[0], hi_x = vx[0], lo_y = vy[0], hi_y = vy[0];
    for (int k = 1; k < 3; ++k) {
        if (vx[k] < lo_x) lo_x = vx[k];
        if (vx[k] > hi_x) hi_x = vx[k];
        if (vy[k] < lo_y) lo_y = vy[k];
        if (vy[k] > hi_y) hi_y = vy[k];
    }
    /* pixel i's centre 256 i + 128 within [lo - 256, hi + 256] */
    int64_t i0 = floor_div256((int64_t)lo_x - 384 + 255), i1 = floor_div256((int64_t)hi_x + 128);
    int64_t j0 = floor_div256((int64_t)lo_y - 384 + 255), j1 = floor_div256((int64_t)hi_y + 128);
    if (i0 < 0) i0 = 0;
    if (j0 < 0) j0 = 0;
    if (i1 > P->W - 1) i1 = P->W - 1;
    if (j1 > P->H - 1) j1 = P->H - 1;
    float inv_len[3];
    for (int e = 0; e < 3; ++e) {
        /* edge e runs from vertex e + 1 to vertex e + 2 (mod 3), as in R6 */
        int64_t dx = (int64_t)vx[(e + 2) % 3] - vx[(e + 1) % 3];
        int64_t dy = (int64_t)vy[(e + 2) % 3] - vy[(e + 1) % 3];
        float len = sqrtf((float)(dx * dx + dy * dy));
        inv_len[e] = 1.0f / (256.0f * len);
    }
    for (int64_t j = j0; j <= j1; ++j) {
        for (int64_t i = i0; i <= i1; ++i) {
            int64_t px = 256 * i + 128, py = 256 * j + 128;
            float sum = 0.0f;
            for (int e = 0; e < 3; ++e) {
                int64_t ax = vx[(e + 1) % 3], ay = vy[(e + 1) % 3];
                int64_t dx = (int64_t)vx[(e + 2) % 3] - ax, dy = (int64_t)vy[(e + 2) % 3] - ay;
                int64_t E = dx * (py - ay) - dy * (px - ax);
                float c = fmaf((float)E, inv_len[e], 0.5f);
                if (c < 0.0f) c = 0.0f;
                if (c > 1.0f) c = 1.0f;
                sum = sum + c;
            }
            float a = sum - 2.0f;
            if (a < 0.0f) a = 0.0f;
            if (a > 1.0f) a = 1.0f;
            uint32_t a8 = (uint32_t)rintf(255.0f * a);
            if (a8 == 0u || a8 == 255u) continue;
            float pxf = ((float)i + 0.5f) - P->cx;
            float pyf = ((float)j + 0.5f) - P->cy;
            float iz = fmaf(pa, pxf, fmaf(pb, pyf, pc));
            uint32_t q;
            if (!quantize_iz(P, iz, &q)) continue;
            uint32_t key = (q << 8) | cls;
            uint32_t o = ((key >> 16) << 16) | ((key & 255u) << 8) | (255u - a8);
            int p = (int)(j * P->W + i);
            if (o < F->frag[p]) F->frag[p] = o;
        }
    }
}

/* R14 for a surface drawn as one convex 4-gon (a triangle pair, or a
 * triangle clipped to four vertices): q[0..3] the snapped vertices in a
 * positive order.  The same estimate over its four edges q_k -> q_(k+1):
 * a = (((c_0 + c_1) + c_2) + c_3) - 3, clamped; the key at the centre is that
 * of the plane given (the first piece's).  A pixel covered partly by each of
 * the two pieces thus gets their summed coverage. */
static void quad_fragments(const Params* P, Frame* F, const int32_t* qx, const int32_t* qy, float pa, float pb,
                           float pc, uint32_t cls)
{
    int32_t lo_x = qx[0], hi_x = qx[0], lo_y = qy[0], hi_y = qy[0];
    for (int k = 1; k < 4; ++k) {
        if (qx[k] < lo_x) lo_x = qx[k];
        if (qx[k] > hi_x) hi_x = qx[k];
        if (qy[k] < lo_y) lo_y = qy[k];
        if (qy[k] > hi_y) hi_y = qy[k];
    }
    int64_t i0 = floor_div256((int64_t)lo_x - 384 + 255), i1 = floor_div256((int64_t)hi_x + 128);
    int64_t j0 = floor_div256((int64_t)lo_y - 384 + 255), j1 = floor_div256((int64_t)hi_y + 128);
    if (i0 < 0) i0 = 0;
    if (j0 < 0) j0 = 0;
    if (i1 > P->W - 1) i1 = P->W - 1;
    if (j1 > P->H - 1) j1 = P->H - 1;
    float inv_len[4];
    for (int e = 0; e < 4; ++e) {
        int64_t dx = (int64_t)qx[(e + 1) % 4] - qx[e], dy = (int64_t)qy[(e + 1) % 4] - qy[e];
        float len = sqrtf((float)(dx * dx + dy * dy));
        inv_len[e] = 1.0f / (256.0f * len);
    }
    for (int64_t j = j0; j <= j1; ++j) {
        for (int64_t i = i0; i <= i1; ++i) {
            int64_t px = 256 * i + 128, py = 256 * j + 128;
            float sum = 0.0f;
            for (int e = 0; e < 4; ++e) {
                int64_t ax = qx[e], ay = qy[e];
                int64_t dx = (int64_t)qx[(e + 1) % 4] - ax, dy = (int64_t)qy[(e + 1) % 4] - ay;
                int64_t E = dx * (py - ay) - dy * (px - ax);
                float c = fmaf((float)E, inv_len[e], 0.5f);
                if (c < 0.0f) c = 0.0f;
                if (c > 1.0f) c = 1.0f;
                sum = sum + c;
            }
            float a = sum - 3.0f;
            if (a < 0.0f) a = 0.0f;
            if (a > 1.0f) a = 1.0f;
            uint32_t a8 = (uint32_t)rintf(255.0f * a);
            if (a8 == 0u || a8 == 255u) continue;
            float pxf = ((float)i + 0.5f) - P->cx;
            float pyf = ((float)j + 0.5f) - P->cy;
            float iz = fmaf(pa, pxf, fmaf(pb, pyf, pc));
            uint32_t q;
            if (!quantize_iz(P, iz, &q)) continue;
            uint32_t key = (q << 8) | cls;
            uint32_t o = ((key >> 16) << 16) | ((key & 255u) << 8) | (255u - a8);
            int p = (int)(j * P->W + i);
            if (o < F->frag[p]) F->frag[p] = o;
        }
    }
}

/* The snapped 4-gon (x[k], y[k]) as one surface for R14: when it is
 * strictly convex (every turn of the same sign, none zero), its vertices in a
 * positive order (reversed when every turn is negative) in qx, qy, and 1;
 * otherwise 0 and each fan piece leaves its own fragments. */
static int convex_quad(const int32_t* x, const int32_t* y, int32_t* qx, int32_t* qy)
{
    int pos = 0, neg = 0;
    for (int k = 0; k < 4; ++k) {
        int64_t ux = (int64_t)x[(k + 1) % 4] - x[k], uy = (int64_t)y[(k + 1) % 4] - y[k];
        int64_t vx = (int64_t)x[(k + 2) % 4] - x[(k + 1) % 4], vy = (int64_t)y[(k + 2) % 4] - y[(k + 1) % 4];
        int64_t cr = ux * vy - uy * vx;
        if (cr > 0) ++pos;
        if (cr < 0) ++neg;
    }
    if (pos != 4 && neg != 4) return 0;
    static const int fwd[4] = {0, 1, 2, 3}, rev[4] = {0, 3, 2, 1};
    const int* o = pos == 4 ? fwd : rev;
    for (int k = 0; k < 4; ++k) { qx[k] = x[o[k]]; qy[k] = y[o[k]]; }
    return 1;
}

/* Rasterize one snapped triangle (R6, R7) into the frame (with its R14
 * fragments unless `frag` is 0: its surface leaves them as a whole). */
static void raster_tri_f(const Params* P, Frame* F, int32_t X0, int32_t Y0, int32_t X1, int32_t Y1,
                         int32_t X2, int32_t Y2, float pa, float pb, float pc, uint32_t cls, int frag)
{
    int64_t area2 = (int64_t)(X1 - X0) * (int64_t)(Y2 - Y0) - (int64_t)(Y1 - Y0) * (int64_t)(X2 - X0);
    if (area2 == 0) return;
    if (area2 < 0) {
        int32_t tx = X1, ty = Y1;
        X1 = X2; Y1 = Y2; X2 = tx; Y2 = ty;
    }
    if (F->frag && frag) {
        const int32_t vx[3] = {X0, X1, X2}, vy[3] = {Y0, Y1, Y2};
        coverage_fragments(P, F, vx, vy, pa, pb, pc, cls);
    }
    int32_t ax[3] = {X1, X2, X0}, ay[3] = {Y1, Y2, Y0};
    int32_t bx[3] = {X2, X0, X1}, by[3] = {Y2, Y0, Y1};
    int tl[3];
    double band[3];
    for (int e = 0; e < 3; ++e) {
        int64_t dx = (int64_t)bx[e] - ax[e], dy = (int64_t)by[e] - ay[e];
        tl[e] = (dy < 0) || (dy == 0 && dx > 0);
        band[e] = 0.0256 * sqrt((double)dx * (double)dx + (double)dy * (double)dy);
    }
    int32_t minX = X0 < X1 ? (X0 < X2 ? X0 : X2) : (X1 < X2 ? X1 : X2);
    int32_t maxX = X0 > X1 ? (X0 > X2 ? X0 : X2) : (X1 > X2 ? X1 : X2);
    int32_t minY = Y0 < Y1 ? (Y0 < Y2 ? Y0 : Y2) : (Y1 < Y2 ? Y1 : Y2);
    int32_t maxY = Y0 > Y1 ? (Y0 > Y2 ? Y0 : Y2) : (Y1 > Y2 ? Y1 : Y2);
    int64_t i0 = floor_div256((int64_t)minX - 128 + 255), i1 = floor_div256((int64_t)maxX - 128);
    int64_t j0 = floor_div256((int64_t)minY - 128 + 255), j1 = floor_div256((int64_t)maxY - 128);
    if (i0 < 0) i0 = 0;
    if (j0 < 0) j0 = 0;
    if (i1 > P->W - 1) i1 = P->W - 1;
    if (j1 > P->H - 1) j1 = P->H - 1;
    for (int64_t j = j0; j <= j1; ++j) {
        int64_t py = 256 * j + 128;
        float pyf = ((float)j + 0.5f) - P->cy;
        for (int64_t i = i0; i <= i1; ++i) {
            int64_t px = 256 * i + 128;
            int covered = 1, near_edge = 0, in_band = 1;
            for (int e = 0; e < 3; ++e) {
                int64_t E = ((int64_t)bx[e] - ax[e]) * (py - ay[e]) - ((int64_t)by[e] - ay[e]) * (px - ax[e]);
                if (!(E > 0 || (E == 0 && tl[e]))) covered = 0;
                double Ed = (double)E;
                if (fabs(Ed) <= band[e]) near_edge = 1;
                if (Ed < -band[e]) in_band = 0;
            }
            if (!covered && !(near_edge && in_band)) continue;
            float pxf = ((float)i + 0.5f) - P->cx;
            float iz = fmaf(pa, pxf, fmaf(pb, pyf, pc));
            uint32_t q;
            if (!quantize_iz(P, iz, &q)) continue;
            uint32_t key = (q << 8) | cls;
            int p = (int)(j * P->W + i);
            if (near_edge && in_band && key < F->edge_key[p] + 0u) {
                if (key < F->edge_key[p]) F->edge_key[p] = key;
            }
            if (covered) {
                if (key < F->key[p]) F->key[p] = key;
                frame_update_tie(F, p, key);
                if (F->cover) F->cover[p]++;
            }
        }
    }
}

/* One world-space triangle through R2..R7. */
static void draw_triangle(const Params* P, const Cam* cam, Frame* F, const float* t, uint32_t cls)
{
    V3 v[3];
    for (int k = 0; k < 3; ++k) v[k] = to_view(cam, t[3 * k], t[3 * k + 1], t[3 * k + 2]);
    int in[3];
    int nin = 0;
    for (int k = 0; k < 3; ++k) { in[k] = v[k].z >= P->nearp; nin += in[k]; }
    if (nin == 0) return;
    if (v[0].z > P->farp && v[1].z > P->farp && v[2].z > P->farp) return;
    float pa, pb, pc;
    if (!depth_plane(cam, P, t, &pa, &pb, &pc)) return;
    V3 poly[4];
    int np = 0;
    if (nin == 3) {
        poly[0] = v[0]; poly[1] = v[1]; poly[2] = v[2]; np = 3;
    } else {
        for (int k = 0; k < 3; ++k) {
            V3 A = v[k], B = v[(k + 1) % 3];
            int ia = in[k], ib = in[(k + 1) % 3];
            if (ia) poly[np++] = A;
            if (ia != ib) {
                V3 I = ia ? A : B, O = ia ? B : A;
                float t_ = (P->nearp - I.z) / (O.z - I.z);
                V3 X;
                X.x = fmaf(t_, O.x - I.x, I.x);
                X.y = fmaf(t_, O.y - I.y, I.y);
                X.z = P->nearp;
                poly[np++] = X;
            }
        }
    }
    int32_t SX[4], SY[4];
    for (int k = 0; k < np; ++k)
        if (!snap(P, poly[k], &SX[k], &SY[k])) return;
    /* R14: a triangle clipped to a convex 4-gon leaves its fragments as one surface */
    int32_t qx[4], qy[4];
    const int whole = F->frag && np == 4 && convex_quad(SX, SY, qx, qy);
    for (int f = 1; f + 1 < np; ++f)
        raster_tri_f(P, F, SX[0], SY[0], SX[f], SY[f], SX[f + 1], SY[f + 1], pa, pb, pc, cls, !whole);
    if (whole) quad_fragments(P, F, qx, qy, pa, pb, pc, cls);
}

/* A triangle pair (a, b, c), (a, c, d) of the scene (see oracle_bin's pairing
 * rule).  Its two triangles are drawn by R2..R7 exactly as two separate
 * triangles; for R14 the pair is one surface when all four vertices lie in
 * front of the near plane, neither triangle lies wholly beyond far, both
 * triangles are drawn (every snap within range, both planes defined) and the
 * snapped 4-gon (a, b, c, d) is strictly convex: its fragments then come from
 * the 4-gon with the first triangle's plane. */
static void draw_pair(const Params* P, const Cam* cam, Frame* F, const float* t1, const float* t2, uint32_t cls)
{
    if (!F->frag) {
        draw_triangle(P, cam, F, t1, cls);
        draw_triangle(P, cam, F, t2, cls);
        return;
    }
    V3 v[4];
    for (int k = 0; k < 3; ++k) v[k] = to_view(cam, t1[3 * k], t1[3 * k + 1], t1[3 * k + 2]);
    v[3] = to_view(cam, t2[6], t2[7], t2[8]);
    int all4 = v[0].z >= P->nearp && v[1].z >= P->nearp && v[2].z >= P->nearp && v[3].z >= P->nearp;
    int far0 = v[0].z > P->farp && v[1].z > P->farp && v[2].z > P->farp;
    int far1 = v[0].z > P->farp && v[2].z > P->farp && v[3].z > P->farp;
    float pa0, pb0, pc0, pa1, pb1, pc1;
    int32_t SX[4], SY[4], qx[4], qy[4];
    int ok = all4 && !far0 && !far1 && depth_plane(cam, P, t1, &pa0, &pb0, &pc0) &&
             depth_plane(cam, P, t2, &pa1, &pb1, &pc1);
    for (int k = 0; k < 4 && ok; ++k) ok = snap(P, v[k], &SX[k], &SY[k]);
    if (!ok || !convex_quad(SX, SY, qx, qy)) {
        draw_triangle(P, cam, F, t1, cls);
        draw_triangle(P, cam, F, t2, cls);
        return;
    }
    raster_tri_f(P, F, SX[0], SY[0], SX[1], SY[1], SX[2], SY[2], pa0, pb0, pc0, cls, 0);
    raster_tri_f(P, F, SX[0], SY[0], SX[2], SY[2], SX[3], SY[3], pa1, pb1, pc1, cls, 0);
    quad_fragments(P, F, qx, qy, pa0, pb0, pc0, cls);
}

static const int BOX_TRIS[12][3] = {
    {0, 1, 3}, {0, 3, 2},   /* bottom */
    {4, 5, 7}, {4, 7, 6},   /* top */
    {0, 2, 6}, {0, 6, 4},   /* back  (a = -L/2) */
    {1, 3, 7}, {1, 7, 5},   /* front (a = +L/2) */
    {0, 1, 5}, {0, 5, 4},   /* right (b = -W/2) */
    {2, 3, 7}, {2, 7, 6},   /* left  (b = +W/2) */
};

static void box_corners(float x, float y, float z0, float c, float s, float L, float Wd, float H, float out[8][3])
{
    float hl = 0.5f * L, hw = 0.5f * Wd;
    for (int n = 0; n < 8; ++n) {
        float a = (n & 1) ? hl : -hl;
        float b = (n & 2) ? hw : -hw;
        float ac = a * c, bs = b * s, as_ = a * s, bc = b * c;
        float ox = ac - bs, oy = as_ + bc;
        out[n][0] = x + ox;
        out[n][1] = y + oy;
        out[n][2] = (n & 4) ? (z0 + H) : z0;
    }
}

/* R13 palette (class -> RGB bytes) and face factors */
static const uint8_t PALETTE[16][3] = {
    {96, 112, 72}, {72, 72, 78}, {232, 232, 224}, {52, 96, 220}, {140, 184, 232}, {160, 160, 152},
    {224, 72, 64}, {168, 144, 120}, {255, 32, 24}, {255, 184, 0}, {32, 224, 96}, {128, 128, 128},
    {128, 128, 128}, {128, 128, 128}, {128, 128, 128}, {128, 128, 128}};
static const float FACE_FACTOR[8] = {1.0f, 0.45f, 1.0f, 0.55f, 0.85f, 0.7f, 0.7f, 1.0f};

static void shade(const Params* P, uint32_t key, uint8_t* c3)
{
    uint32_t cls = key & 15u, face = (key >> 4) & 7u, q = key >> 8;
    float f = FACE_FACTOR[face];
    if (face != 0u && q != 0xFFFFFFu) {
        float z = decode_q(P, q);
        float rfar = 1.0f / P->farp;
        float t = z * rfar;
        if (t > 1.0f) t = 1.0f;
        float b = 1.0f - 0.6f * t;
        f = f * b;
    }
    for (int c = 0; c < 3; ++c) {
        float base = (float)PALETTE[cls][c] / 255.0f;
        float v = base * f;
        if (v > 1.0f) v = 1.0f;
        c3[c] = (uint8_t)rintf(255.0f * v);
    }
}

/* cos and sin of 30k degrees, k = 0..11, rounded to fp32 (R11) */
static void sector_table(float cs[12], float sn[12])
{
    const float h = (float)(sqrt(3.0) / 2.0);
    const float c[12] = {1.0f, h, 0.5f, 0.0f, -0.5f, -h, -1.0f, -h, -0.5f, 0.0f, 0.5f, h};
    for (int k = 0; k < 12; ++k) {
        cs[k] = c[k];
        sn[k] = c[(k + 9) % 12];   /* sin(30k) = cos(30(k - 3)) */
    }
}

/* R10: is the camera centre inside the light's visibility cone? */
static int light_seen(const Cam* cam, float x, float y, float z, float cf, float sf, float cos_max)
{
    float dx = cam->cx_ - x, dy = cam->cy_ - y, dz = cam->cz_ - z;
    float t1 = cf * dx, t2 = sf * dy;
    float h = t1 + t2;
    float xx = dx * dx, yy = dy * dy, zz = dz * dz;
    float q = (xx + yy) + zz;
    float m = cos_max * cos_max;
    return h > 0.0f && h * h >= m * q;
}

static void init_params(Params* P, int W, int H, float fx, float fy, float cx, float cy, float nearp, float farp)
{
    P->W = W; P->H = H; P->fx = fx; P->fy = fy; P->cx = cx; P->cy = cy;
    P->nearp = nearp; P->farp = farp;
    P->fx256 = 256.0f * fx; P->fy256 = 256.0f * fy;
    P->cx256 = 256.0f * cx; P->cy256 = 256.0f * cy;
    P->rfx = 1.0f / fx; P->rfy = 1.0f / fy;
    P->izfar = 1.0f / farp;
    P->izcap = pow2_ceil(1.0f / nearp);
    P->qbase = f2u(P->izcap) >> 3;
}

/* Camera of view v (R1). */
static void make_cam(Cam* cam, int64_t g, const float* mount,
                     const float* ax, const float* ay, const float* az0, const float* ac, const float* as_)
{
    float c = ac[g], s = as_[g];
    float mx = mount[0], my = mount[1], mz = mount[2], cm = mount[3], sm = mount[4];
    float t1 = mx * c, t2 = my * s, t3 = mx * s, t4 = my * c;
    float ox = t1 - t2, oy = t3 + t4;
    cam->cx_ = ax[g] + ox;
    cam->cy_ = ay[g] + oy;
    cam->cz_ = az0[g] + mz;
    float u1 = c * cm, u2 = s * sm, u3 = s * cm, u4 = c * sm;
    cam->cc = u1 - u2;
    cam->sc = u3 + u4;
}

int oracle_render(int num_worlds, const int64_t* tri_offsets, const float* verts, const uint8_t* tcls,
                  int agents_per_world, const float* ax, const float* ay, const float* az0,
                  const float* acos, const float* asin, const float* alen, const float* awid,
                  const float* ahgt, const uint8_t* acls,
                  int lights_per_world, const float* lx, const float* ly, const float* lz,
                  const float* lcf, const float* lsf, const float* lrad, const uint8_t* lcls, float cos_max,
                  int num_cams, int W, int H, float fx, float fy, float cx, float cy,
                  float nearp, float farp, const float* mount,
                  int64_t num_sel, const int64_t* view_ids,
                  uint8_t* out_cls, float* out_depth, uint8_t* out_flags, uint16_t* out_cover,
                  int32_t* out_inst, uint32_t* out_counts, uint8_t* out_rgb, int aa,
                  int num_threads)
{
    Params P;
    init_params(&P, W, H, fx, fy, cx, cy, nearp, farp);
    float sec_c[12], sec_s[12];
    sector_table(sec_c, sec_s);
    const int64_t npx = (int64_t)W * H;
    const int64_t per_world = (int64_t)agents_per_world * num_cams;
    const int64_t total_views = per_world * num_worlds;
    for (int64_t n = 0; n < num_sel; ++n)
        if (view_ids[n] < 0 || view_ids[n] >= total_views) return -1;
#ifdef _OPENMP
    if (num_threads > 0) omp_set_num_threads(num_threads);
#pragma omp parallel
#endif
    {
        Frame F;
        F.key = (uint32_t*)malloc(sizeof(uint32_t) * npx);
        F.edge_key = (uint32_t*)malloc(sizeof(uint32_t) * npx);
        F.k1 = (uint32_t*)malloc(sizeof(uint32_t) * npx);
        F.k2 = (uint32_t*)malloc(sizeof(uint32_t) * npx);
        F.cover = out_cover ? (uint16_t*)malloc(sizeof(uint16_t) * npx) : NULL;
        F.frag = (out_rgb && aa) ? (uint32_t*)malloc(sizeof(uint32_t) * npx) : NULL;
        /* a box drawn alone (instances) */
        Frame G;
        const int want_inst = out_inst != NULL || out_counts != NULL;
        G.key = (uint32_t*)malloc(sizeof(uint32_t) * npx);
        G.edge_key = (uint32_t*)malloc(sizeof(uint32_t) * npx);
        G.k1 = (uint32_t*)malloc(sizeof(uint32_t) * npx);
        G.k2 = (uint32_t*)malloc(sizeof(uint32_t) * npx);
        G.cover = NULL;
        G.frag = NULL;
        int32_t* inst = (int32_t*)malloc(sizeof(int32_t) * npx);
#ifdef _OPENMP
#pragma omp for schedule(dynamic, 1)
#endif
        for (int64_t n = 0; n < num_sel; ++n) {
            int64_t v = view_ids[n];
            int64_t w = v / per_world;
            int64_t a = (v / num_cams) % agents_per_world;
            int64_t k = v % num_cams;
            int64_t g = w * agents_per_world + a;
            Cam cam;
            make_cam(&cam, g, mount + 5 * k, ax, ay, az0, acos, asin);
            for (int64_t p = 0; p < npx; ++p) {
                F.key[p] = CLEAR_KEY;
                F.edge_key[p] = 0xFFFFFFFFu;
                F.k1[p] = CLEAR_KEY;
                F.k2[p] = 0xFFFFFFFFu;
                if (F.cover) F.cover[p] = 0;
                if (F.frag) F.frag[p] = 0xFFFFFFFFu;
            }
            for (int64_t t = tri_offsets[w]; t < tri_offsets[w + 1];) {
                const float* a = verts + 9 * t;
                int pair = t + 1 < tri_offsets[w + 1] && tcls[t] == tcls[t + 1] && memcmp(a, a + 9, 12) == 0 &&
                           memcmp(a + 6, a + 12, 12) == 0;
                if (pair) draw_pair(&P, &cam, &F, a, a + 9, tcls[t]);
                else draw_triangle(&P, &cam, &F, a, tcls[t]);
                t += pair ? 2 : 1;
            }
            for (int64_t b = 0; b < agents_per_world; ++b) {
                int64_t h = w * agents_per_world + b;
                if (h == g) continue; /* the ego's own body is not drawn */
                float cor[8][3];
                box_corners(ax[h], ay[h], az0[h], acos[h], asin[h], alen[h], awid[h], ahgt[h], cor);
                for (int f = 0; f < 12; ++f) {
                    float tri[9];
                    for (int q = 0; q < 3; ++q) {
                        tri[3 * q] = cor[BOX_TRIS[f][q]][0];
                        tri[3 * q + 1] = cor[BOX_TRIS[f][q]][1];
                        tri[3 * q + 2] = cor[BOX_TRIS[f][q]][2];
                    }
                    uint32_t sid = acls[h];
                    if (out_rgb) sid = (sid & 15u) | (uint32_t)(f / 2 + 1) << 4;
                    draw_triangle(&P, &cam, &F, tri, sid);
                }
            }
            for (int64_t l = 0; l < lights_per_world; ++l) {
                int64_t h = w * lights_per_world + l;
                if (!light_seen(&cam, lx[h], ly[h], lz[h], lcf[h], lsf[h], cos_max)) continue;
                float rim[12][3];
                for (int k = 0; k < 12; ++k) {
                    float a = lrad[h] * sec_c[k], b = lrad[h] * sec_s[k];
                    float as_ = a * lsf[h], ac = a * lcf[h];
                    rim[k][0] = lx[h] - as_;
                    rim[k][1] = ly[h] + ac;
                    rim[k][2] = lz[h] + b;
                }
                for (int k = 0; k < 12; ++k) {
                    int k1 = (k + 1) % 12;
                    float tri[9] = {lx[h], ly[h], lz[h], rim[k][0], rim[k][1], rim[k][2],
                                    rim[k1][0], rim[k1][1], rim[k1][2]};
                    draw_triangle(&P, &cam, &F, tri, lcls[h]);
                }
            }
            if (want_inst) {
                for (int64_t p = 0; p < npx; ++p) inst[p] = -1;
                for (int64_t b = 0; b < agents_per_world; ++b) {
                    int64_t h = w * agents_per_world + b;
                    uint32_t footprint = 0;
                    if (h != g) {
                        for (int64_t p = 0; p < npx; ++p) {
                            G.key[p] = CLEAR_KEY;
                            G.edge_key[p] = 0xFFFFFFFFu;
                            G.k1[p] = CLEAR_KEY;
                            G.k2[p] = 0xFFFFFFFFu;
                        }
                        float cor[8][3];
                        box_corners(ax[h], ay[h], az0[h], acos[h], asin[h], alen[h], awid[h], ahgt[h], cor);
                        for (int f = 0; f < 12; ++f) {
                            float tri[9];
                            for (int q = 0; q < 3; ++q) {
                                tri[3 * q] = cor[BOX_TRIS[f][q]][0];
                                tri[3 * q + 1] = cor[BOX_TRIS[f][q]][1];
                                tri[3 * q + 2] = cor[BOX_TRIS[f][q]][2];
                            }
                            draw_triangle(&P, &cam, &G, tri, acls[h]);
                        }
                        for (int64_t p = 0; p < npx; ++p) {
                            if (G.key[p] == CLEAR_KEY) continue;
                            ++footprint;
                            if (G.key[p] == F.key[p] && inst[p] < 0) inst[p] = (int32_t)b;
                        }
                    }
                    if (out_counts) out_counts[(n * agents_per_world + b) * 2] = footprint;
                }
                if (out_counts) {
                    for (int64_t b = 0; b < agents_per_world; ++b) out_counts[(n * agents_per_world + b) * 2 + 1] = 0;
                    for (int64_t p = 0; p < npx; ++p)
                        if (inst[p] >= 0) out_counts[(n * agents_per_world + inst[p]) * 2 + 1]++;
                }
                if (out_inst)
                    for (int64_t p = 0; p < npx; ++p) out_inst[n * npx + p] = inst[p];
            }
            for (int64_t p = 0; p < npx; ++p) {
                uint32_t key = F.key[p];
                uint32_t q = key >> 8;
                out_cls[n * npx + p] = (uint8_t)(key & (out_rgb ? 15u : 255u));
                if (out_rgb) {
                    uint8_t c3[3];
                    shade(&P, key, c3);
                    uint32_t o = F.frag ? F.frag[p] : 0xFFFFFFFFu;
                    /* R14: a fragment not behind the centre's surface, of another
                     * shading id, is blended over it with its coverage */
                    if (o != 0xFFFFFFFFu && (o >> 16) <= (key >> 16) && ((o >> 8) & 255u) != (key & 255u)) {
                        uint8_t f3[3];
                        shade(&P, ((o >> 16) << 16) | ((o >> 8) & 255u), f3);
                        uint32_t a8 = 255u - (o & 255u);
                        for (int c = 0; c < 3; ++c)
                            c3[c] = (uint8_t)(((uint32_t)f3[c] * a8 + (uint32_t)c3[c] * (255u - a8) + 127u) / 255u);
                    }
                    for (int c = 0; c < 3; ++c) out_rgb[(n * 3 + c) * npx + p] = c3[c];
                }
                if (q == 0xFFFFFFu) {
                    out_depth[n * npx + p] = INFINITY;
                } else {
                    out_depth[n * npx + p] = decode_q(&P, q);
                }
                if (out_flags) {
                    uint8_t fl = 0;
                    if (F.edge_key[p] <= key) fl |= 1;
                    uint32_t k2 = F.k2[p];
                    if (k2 != 0xFFFFFFFFu && (k2 >> 8) != 0xFFFFFFu && q != 0xFFFFFFu) {
                        double z1 = 1.0 / (double)u2f(((P.qbase - q) << 3) | 4u);
                        double z2 = 1.0 / (double)u2f(((P.qbase - (k2 >> 8)) << 3) | 4u);
                        if (fabs(z2 - z1) <= 1e-4 * z1) fl |= 2;
                    }
                    out_flags[n * npx + p] = fl;
                }
                if (out_cover) out_cover[n * npx + p] = F.cover[p];
            }
        }
        free(F.key); free(F.edge_key); free(F.k1); free(F.k2); free(F.cover); free(F.frag);
        free(G.key); free(G.edge_key); free(G.k1); free(G.k2); free(inst);
    }
    return 0;
}

/* R7/R8 quantizer exposed for exhaustive checks: the same quantize_iz and
 * decode_q that the renderer applies to every pixel. */
void oracle_quantize(const float* iz, int64_t n, float nearp, float farp, uint32_t* q_out, float* depth_out)
{
    Params P;
    init_params(&P, 1, 1, 1.0f, 1.0f, 0.5f, 0.5f, nearp, farp);
    for (int64_t k = 0; k < n; ++k) {
        uint32_t q;
        if (!quantize_iz(&P, iz[k], &q)) { q_out[k] = 0xFFFFFFu; depth_out[k] = INFINITY; continue; }
        q_out[k] = q;
        depth_out[k] = decode_q(&P, q);
    }
}

/*
 * Uniform-grid binning of one scene, over primitives.  Walking each world's
 * triangles in order, triangle t and t + 1 form a pair when they have the same
 * class and t + 1 is (a, c, d) for t = (a, b, c), the shared a and c equal bit
 * for bit (a quad split along its diagonal); any other triangle is a
 * primitive on its own.  prim_out[p] = first triangle | (1 << 31 for a pair).
 * Each primitive belongs to the cell that holds the centre of the xy
 * bounding box of its vertices (clamped into the grid); a cell records its
 * primitive count and the 3-D bounding box of its members' vertices.
 * Grid of world w: origin (bounds[w].xmin, bounds[w].ymin), square cells of
 * `cell` metres, nx = max(1, ceil(width / cell)) columns, ny rows, cells
 * numbered row-major (iy * nx + ix) after those of the previous worlds.
 */
int oracle_bin(int num_worlds, const int64_t* tri_offsets, const float* verts, const uint8_t* cls,
               const float* bounds, float cell, int32_t* dims_out /*[nw][2]*/, int64_t* cell_base_out /*[nw+1]*/,
               uint32_t* prim_out /*[<= T]*/, int64_t* home_out /*[<= T]*/, int64_t* nprim_out,
               int32_t* count_out, float* aabb_out /*[cells][6]*/, int64_t max_cells)
{
    int64_t base = 0;
    for (int w = 0; w < num_worlds; ++w) {
        float wx = bounds[4 * w + 2] - bounds[4 * w + 0];
        float wy = bounds[4 * w + 3] - bounds[4 * w + 1];
        float fnx = ceilf(wx / cell), fny = ceilf(wy / cell);
        int32_t nx = fnx < 1.0f ? 1 : (int32_t)fnx;
        int32_t ny = fny < 1.0f ? 1 : (int32_t)fny;
        dims_out[2 * w] = nx;
        dims_out[2 * w + 1] = ny;
        cell_base_out[w] = base;
        base += (int64_t)nx * ny;
    }
    cell_base_out[num_worlds] = base;
    if (base > max_cells) return -1;
    for (int64_t c = 0; c < base; ++c) {
        count_out[c] = 0;
        aabb_out[6 * c + 0] = aabb_out[6 * c + 1] = aabb_out[6 * c + 2] = INFINITY;
        aabb_out[6 * c + 3] = aabb_out[6 * c + 4] = aabb_out[6 * c + 5] = -INFINITY;
    }
    int64_t np_ = 0;
    for (int w = 0; w < num_worlds; ++w) {
        int32_t nx = dims_out[2 * w], ny = dims_out[2 * w + 1];
        for (int64_t t = tri_offsets[w]; t < tri_offsets[w + 1];) {
            const float* v = verts + 9 * t;
            int pair = t + 1 < tri_offsets[w + 1] && cls[t] == cls[t + 1] && memcmp(v, v + 9, 12) == 0 &&
                       memcmp(v + 6, v + 12, 12) == 0;
            float lo[3], hi[3];
            for (int d = 0; d < 3; ++d) {
                lo[d] = fminf(fminf(v[d], v[3 + d]), v[6 + d]);
                hi[d] = fmaxf(fmaxf(v[d], v[3 + d]), v[6 + d]);
                if (pair) {   /* the second triangle's third vertex */
                    lo[d] = fminf(lo[d], v[15 + d]);
                    hi[d] = fmaxf(hi[d], v[15 + d]);
                }
            }
            float mx = (lo[0] + hi[0]) * 0.5f, my = (lo[1] + hi[1]) * 0.5f;
            float fx = floorf((mx - bounds[4 * w + 0]) / cell);
            float fy = floorf((my - bounds[4 * w + 1]) / cell);
            int32_t ix = !(fx >= 0.0f) ? 0 : (fx >= (float)(nx - 1) ? nx - 1 : (int32_t)fx);
            int32_t iy = !(fy >= 0.0f) ? 0 : (fy >= (float)(ny - 1) ? ny - 1 : (int32_t)fy);
            int64_t c = cell_base_out[w] + (int64_t)iy * nx + ix;
            prim_out[np_] = (uint32_t)t | (pair ? 0x80000000u : 0u);
            home_out[np_] = c;
            ++np_;
            count_out[c]++;
            for (int d = 0; d < 3; ++d) {
                if (lo[d] < aabb_out[6 * c + d]) aabb_out[6 * c + d] = lo[d];
                if (hi[d] > aabb_out[6 * c + 3 + d]) aabb_out[6 * c + 3 + d] = hi[d];
            }
            t += pair ? 2 : 1;
        }
    }
    *nprim_out = np_;
    return 0;
}

/*
 * Kinematic bicycle update (the per-step agent motion of the headline
 * workload), in double precision:  v' = clamp(v + accel*dt, 0, vmax);
 * psi' = psi + (v' / (0.6 L)) tan(steer) dt, wrapped into (-pi, pi];
 * x' = x + v' cos(psi') dt, y' = y + v' sin(psi') dt.
 */
void oracle_agents_step(int64_t n, double* x, double* y, double* psi, double* v,
                        const double* L, const double* steer, const double* accel,
                        double dt, double vmax, double* cos_out, double* sin_out)
{
    const double PI = 3.14159265358979323846;
    for (int64_t k = 0; k < n; ++k) {
        double vn = v[k] + accel[k] * dt;
        if (vn < 0.0) vn = 0.0;
        if (vn > vmax) vn = vmax;
        double p = psi[k] + vn / (0.6 * L[k]) * tan(steer[k]) * dt;
        if (p > PI) p -= 2.0 * PI;
        if (p <= -PI) p += 2.0 * PI;
        x[k] += vn * cos(p) * dt;
        y[k] += vn * sin(p) * dt;
        psi[k] = p;
        v[k] = vn;
        cos_out[k] = cos(p);
        sin_out[k] = sin(p);
    }
}
