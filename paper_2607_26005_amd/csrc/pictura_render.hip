// Batched class/depth view rasterizer for gfx950.  One workgroup renders one
// view tile (at most 64x64 pixels) into a framebuffer of 32-bit keys in LDS;
// the workgroup has kViewWaves waves that share the framebuffer and split the
// tile's cells and agents between them, each running the whole pipeline on
// its share with no barrier until the write-out:
//
//  1. cells of the world grid in the rectangle around the tile frustum are
//     taken 64 at a time (one lane per cell): a cheap test of the cell
//     rectangle (widened by the world's margin) against the side, near and
//     far planes, then the cell's triangle range and bounding box are loaded
//     and tested against all six planes and, when the box lies in front of the
//     near plane, against the tile's pixel centres through a conservative
//     projection.  Visible cells are compacted with a ballot and their
//     triangle counts prefix-summed across the wave;
//  2. candidate triangles (then the twelve triangles of every visible agent
//     box) go through a first pass 64 at a time: view transform, the near/far
//     rule and a conservative test that the snapped triangle can hold a pixel
//     centre of the tile; survivors are appended to the wave's LDS queue;
//  3. every 64 survivors go through the exact pass, one lane per primitive (a
//     triangle, or a pair of triangles sharing a diagonal, set up once and
//     drawn as two fan pieces): near clipping, 8-bit subpixel snap,
//     orientation, depth planes.  The bounding-box pixels of all pieces with
//     at most kSmallPx of them are numbered across the lanes and handed out
//     64 per step (the packed raster).  For a larger piece the lane computes a
//     raster record (exact edge functions at the tile origin, box, depth
//     plane) and hands it to the view's record ring, which both waves drain:
//     every lane tests one 8x8 pixel block of the record's bounding box
//     against its three edges, and the passing blocks are rasterized one per
//     step, lane l handling pixel (l & 7, l >> 3) of the block;
//  4. visibility is an LDS atomicMin of (24-bit depth | 8-bit class), so the
//     order in which lanes and waves finish does not matter;
//  5. the tile is resolved and written with 16-byte non-temporal stores.
//
// The exact pass evaluates the rasterization rules (camera R1, view
// transform R2, depth plane R3, near clip R4, snap R5, fill R6, key R7,
// resolve R8, boxes R9) in fp32 with no contraction and correctly rounded
// reciprocals and divisions.  Edge functions are exact: int32 (24-bit
// multiplies) when every value over the tile fits, otherwise fp64 fused
// multiply-adds whose sign is exact for every pixel of the tile.  So every
// key equals a brute-force evaluation of the rules over all triangles of the
// world; everything before the exact pass only skips triangles that cannot
// set a key.
#include <mutex>
#include <type_traits>

#include "pictura_device.h"

#pragma clang fp contract(off)

#ifndef PICTURA_VIEW_WAVES
#define PICTURA_VIEW_WAVES 2
#endif
#ifndef PICTURA_SMALL_PX
#define PICTURA_SMALL_PX 128
#endif

namespace pictura {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr uint32_t kClearKey = (0xFFFFFFu << 8) | 4u;
// Queue entries.  Static primitive p: (p << 2) | kind (p < 2^29), kind 0 a
// lone triangle, 1 and 2 the first (a, b, c) and second (a, c, d) half of a
// pair taken alone, 3 the whole pair with all four vertices in front of the
// near plane.  Boxes and lights set bit 31 (and lights bit 30 too).
constexpr uint32_t kBoxFlag = 0x80000000u;     // queue entry: kBoxFlag | (agent << 4) | face of a box
constexpr uint32_t kLightFlag = 0xC0000000u;   // queue entry: kLightFlag | (light << 4) | sector of a traffic light
enum { kTri = 0, kHalf0 = 1, kHalf1 = 2, kPair = 3 };
constexpr int kViewWaves = PICTURA_VIEW_WAVES;   // waves per view tile
constexpr int kThreads = 64 * kViewWaves;
constexpr int kWavesPerSimd = 4;  // register budget: four waves per SIMD (as many as the LDS admits)
constexpr int kSmallPx = PICTURA_SMALL_PX;   // pieces with at most this many bounding-box pixels take the packed raster
constexpr int kQueue = 192;       // per-wave queue of first-pass survivors
// Framebuffer rows are padded to a pitch of 4 mod 32 words, so the 64 lanes
// of an 8x8 block hit every LDS bank exactly twice.
constexpr int kFbCap = 64 * 68;
static_assert(kViewWaves == 1 || kViewWaves == 2 || kViewWaves == 4, "1, 2 or 4 waves per view tile");

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
    int pitch;         // framebuffer words per row
    float kl, kr, kt, kb;
    float cm;          // base margin (px) of the projected-box centre test
};

// Raster record of a snapped, oriented triangle with more than kSmallPx
// pixels in its tile bounding box.  Edge k (v1->v2, v2->v0, v0->v1) at tile
// pixel (i, j) is
//   E_k = c_k + a_k i + b_k j,   a_k = -256 dy_k,  b_k = 256 dx_k,
// with c_k its value at the tile's pixel (0, 0) plus the top-left bias;
// covered iff every E_k >= 0.  Since a_k and b_k are multiples of 256,
//   floor(E_k / 256) = floor(c_k / 256) - dy_k i + dx_k j
// exactly, and it has the sign of E_k: the int32 path tests that instead.
// The exact pass leaves a record in the lane of its triangle as twelve
// words: the int32 path (every value over the tile fits) holds -dy_k, dx_k,
// floor(c_k / 256) in words 0..8; the fp64 path holds c_k as doubles (words
// 0..5) and dx_k, dy_k (words 6..11).  c_k is an integer below 2^61: as a
// double it is exact below 2^53, and beyond that its rounding keeps the sign,
// which no pixel of the tile can change.

// Per-wave LDS: the visible-cell (or agent) list of a refill and the queue
// of first-pass survivors.
struct alignas(16) WaveLds {
    union {
        struct {
            uint32_t start[64];
            uint32_t count[64];
        } cells;
        uint32_t agents[64];
        uint32_t bits[128];   // instance mode, after the static pass: coverage of one box, 2 words per tile row
    } u;
    uint32_t q[kQueue];
};

struct alignas(16) Shared {
    uint32_t fb[kFbCap];
    WaveLds wv[kViewWaves];
    uint32_t stat[kNumStats];
    uint32_t ctl[4];   // record ring: reserved, claimed; wave 0 and wave 1 finished producing
};

enum { kRecTail = 0, kRecHead = 1, kDone0 = 2 };
constexpr uint32_t kRecReady = 0x5EC0DE01u;   // differs from the clear key the padding starts with

enum Stat {
    kStTiles = 0, kStCellsRect, kStCellsPre, kStCellsVis, kStCand, kStBoxesVis, kStBoxTris, kStSurv,
    kStExact, kStClipped, kStRasterTris, kStLaneTris, kStLanePx, kStRecTris, kStRecWide, kStBlocksTested,
    kStBlocksPassed, kStChunks, kCycPrologue, kCycSource, kCycFirst, kCycExact, kCycRecords, kCycWriteout,
    kStAaPacked, kStAaPackedPx, kStAaPackedSteps, kStAaSwept, kStAaBlocks, kStAaFrags
};
static_assert(kStAaFrags + 1 == kNumStats, "stat count");

// Optional work counters (P.stats non-null): LDS per block, flushed once.
#define STAT(k, n) do { if (P.stats) atomicAdd(&S.stat[(k)], (uint32_t)(n)); } while (0)
#define STAT1(k, n) do { if (P.stats && lane_id() == 0) atomicAdd(&S.stat[(k)], (uint32_t)(n)); } while (0)
// Phase timers of the stats mode: shader-clock cycles seen by lane 0 of every wave.
#define TSTART(t) long long t = P.stats ? (long long)__builtin_amdgcn_s_memtime() : 0ll
#define TACC(k, t) do { if (P.stats && lane_id() == 0) atomicAdd(&S.stat[(k)], (uint32_t)((long long)__builtin_amdgcn_s_memtime() - (t))); } while (0)

// ---------------------------------------------------------------------------
// arithmetic
// ---------------------------------------------------------------------------

// Correctly rounded 1/x for |x| in [2^-12, 2^20): hardware reciprocal plus
// one Newton step with fused residual.  Equality with IEEE division over
// every fp32 value of that range, of either sign, is checked on the device
// (pictura_selftest_rcp).
__device__ __forceinline__ float rcp_rn(float x)
{
    const float r = __builtin_amdgcn_rcpf(x);
    const float e = fmaf(-x, r, 1.0f);
    return fmaf(e, r, r);
}

__device__ __forceinline__ bool rcp_rn_ok(float x) { return x >= 0.000244140625f && x < 1048576.0f; }

// Correctly rounded 1/x for any x: the division runs only when a lane of the
// wave needs it.
__device__ __forceinline__ float recip_rn(float x)
{
    const bool ok = rcp_rn_ok(fabsf(x));
    if (__ballot(!ok) == 0) return rcp_rn(x);
    return ok ? rcp_rn(x) : 1.0f / x;
}

__device__ __forceinline__ uint32_t mbcnt(uint64_t m)
{
    return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

__device__ __forceinline__ uint32_t readfirst(uint32_t v) { return (uint32_t)__builtin_amdgcn_readfirstlane((int)v); }

__device__ __forceinline__ uint32_t lds_load_acquire(const uint32_t* p)
{
    return __hip_atomic_load(p, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP);
}

__device__ __forceinline__ void lds_store_release(uint32_t* p, uint32_t v)
{
    __hip_atomic_store(p, v, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
}

__device__ __forceinline__ uint32_t readlane(uint32_t v, int l)
{
    return (uint32_t)__builtin_amdgcn_readlane((int)v, l);
}

__device__ __forceinline__ float readlane_f(float v, int l) { return __uint_as_float(readlane(__float_as_uint(v), l)); }

__device__ __forceinline__ double readlane_d(double v, int l)
{
    const unsigned long long b = (unsigned long long)__double_as_longlong(v);
    const unsigned long long lo = readlane((uint32_t)b, l), hi = readlane((uint32_t)(b >> 32), l);
    return __longlong_as_double((long long)((hi << 32) | lo));
}

// Inclusive scans over the wave with DPP row shifts and row broadcasts (no
// LDS round trip): shifts by 1, 2, 4, 8 within each row of 16 lanes (lanes
// shifted in read 0), then the last lane of row 0 (and of row 2) into rows 1
// and 3, then the last lane of row 1 into rows 2 and 3.
template <int Ctrl, int RowMask, bool BoundZero>
__device__ __forceinline__ uint32_t dpp_mov(uint32_t x)
{
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, Ctrl, RowMask, 0xf, BoundZero);
}

__device__ __forceinline__ uint32_t wave_incl_max(uint32_t x)
{
    x = max(x, dpp_mov<0x111, 0xf, true>(x));
    x = max(x, dpp_mov<0x112, 0xf, true>(x));
    x = max(x, dpp_mov<0x114, 0xf, true>(x));
    x = max(x, dpp_mov<0x118, 0xf, true>(x));
    x = max(x, dpp_mov<0x142, 0xa, false>(x));
    x = max(x, dpp_mov<0x143, 0xc, false>(x));
    return x;
}

__device__ __forceinline__ uint32_t wave_incl_sum(uint32_t x)
{
    x += dpp_mov<0x111, 0xf, true>(x);
    x += dpp_mov<0x112, 0xf, true>(x);
    x += dpp_mov<0x114, 0xf, true>(x);
    x += dpp_mov<0x118, 0xf, true>(x);
    x += dpp_mov<0x142, 0xa, false>(x);
    x += dpp_mov<0x143, 0xc, false>(x);
    return x;
}

// Exclusive prefix sum over the wave; `total` receives the sum of all lanes.
__device__ __forceinline__ uint32_t wave_excl_scan(uint32_t v, uint32_t& total)
{
    const uint32_t x = wave_incl_sum(v);
    total = readlane(x, 63);
    return x - v;
}

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
    const float rd = recip_rn(delta);
    pa = (nx * rd) * P.rfx;
    pb = -((ny * rd) * P.rfy);
    pc = nz * rd;
    return true;
}

// R5
__device__ __forceinline__ bool snap_vertex(const RenderParams& P, float xv, float yv, float zv, int& X, int& Y)
{
    const float rz = recip_rn(zv);
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
    const float4 r0 = P.apk[3 * h], r1 = P.apk[3 * h + 1];
    const float x = r0.x, y = r0.y, z0 = r0.z, c = r1.x, s = r1.y;
    const float hl = 0.5f * r1.z, hw = 0.5f * r1.w, ztop = z0 + r0.w;
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
    cls = __float_as_uint(P.apk[3 * h + 2].x);
    // R13: in RGB mode the shading id adds the face (1 bottom, 2 top, 3 back, 4 front, 5 right, 6 left)
    if (P.out_rgb) cls = (cls & 15u) | ((uint32_t)(face >> 1) + 1u) << 4;
}

// R11: sector k of light h, the triangle (centre, rim k, rim k + 1).  Rim
// vertex k is centre + r cos(30k deg) u + r sin(30k deg) up, with
// u = (-sin_f, cos_f, 0) and the cosines and sines rounded to fp32.
__device__ __forceinline__ void light_rim(float r, float cf, float sf, int k, float x, float y, float z, float* o)
{
    constexpr float kS3 = 0.866025403784438646763723f;   // sqrt(3) / 2
    constexpr float kCos12[12] = {1.0f, kS3, 0.5f, 0.0f, -0.5f, -kS3, -1.0f, -kS3, -0.5f, 0.0f, 0.5f, kS3};
    constexpr float kSin12[12] = {0.0f, 0.5f, kS3, 1.0f, kS3, 0.5f, 0.0f, -0.5f, -kS3, -1.0f, -kS3, -0.5f};
    const float a = r * kCos12[k], b = r * kSin12[k];
    const float as_ = a * sf, ac = a * cf;
    o[0] = x - as_;
    o[1] = y + ac;
    o[2] = z + b;
}

__device__ __forceinline__ void load_light(const RenderParams& P, int64_t h, int k, float* tri, uint32_t& cls)
{
    const float x = P.lx[h], y = P.ly[h], z = P.lz[h], cf = P.lcf[h], sf = P.lsf[h], r = P.lr[h];
    tri[0] = x;
    tri[1] = y;
    tri[2] = z;
    light_rim(r, cf, sf, k, x, y, z, tri + 3);
    light_rim(r, cf, sf, k == 11 ? 0 : k + 1, x, y, z, tri + 6);
    cls = (uint32_t)P.lcls[h];
}

// R10: does the camera centre lie in light h's visibility cone?
//   d = C - centre;  h = cf d.x + sf d.y;  visible iff h > 0 and h^2 >= cos_max^2 |d|^2
__device__ __forceinline__ bool light_visible(const RenderParams& P, const Cam& cam, int64_t h)
{
    const float dx = cam.x - P.lx[h], dy = cam.y - P.ly[h], dz = cam.z - P.lz[h];
    const float t1 = P.lcf[h] * dx, t2 = P.lsf[h] * dy;
    const float hh = t1 + t2;
    const float q = (dx * dx + dy * dy) + dz * dz;
    return hh > 0.0f && hh * hh >= P.lcos2 * q;
}

// Static primitive p: vertices a, b, c, d in v[0..11] (d = 0 for a lone
// triangle), the class and whether it is a pair.
__device__ __forceinline__ void load_prim(const RenderParams& P, uint32_t p, float* v, uint32_t& cls, bool& pair)
{
    const float4 A = P.scene.primA[p];
    const float4 B = P.scene.primB[p];
    const float4 C = P.scene.primC[p];
    v[0] = A.x; v[1] = A.y; v[2] = A.z; v[3] = A.w;
    v[4] = B.x; v[5] = B.y; v[6] = B.z; v[7] = B.w; v[8] = C.x;
    v[9] = C.z; v[10] = C.w; v[11] = P.scene.primD[p];
    const uint32_t cw = __float_as_uint(C.y);
    cls = cw & 255u;
    pair = (cw & kPrimPair) != 0u;
}

// The world-space polygon of a queue entry: a triangle in tri[0..8], or for a
// whole pair the 4-gon (a, b, c, d) in tri[0..11] (returns true).
template <bool kHasLights>
__device__ __forceinline__ bool load_entry(const RenderParams& P, uint32_t e, int64_t abase_w, int64_t lbase_w,
                                           float* tri, uint32_t& cls)
{
    if (kHasLights && (e & kLightFlag) == kLightFlag) {
        load_light(P, lbase_w + ((e & ~kLightFlag) >> 4), (int)(e & 15u), tri, cls);
        return false;
    }
    if (e & kBoxFlag) {
        load_box(P, abase_w + ((e & ~kBoxFlag) >> 4), (int)(e & 15u), tri, cls);
        return false;
    }
    bool pair;
    load_prim(P, e >> 2, tri, cls, pair);
    const uint32_t kind = e & 3u;
    if (kind == kHalf1) {   // (a, c, d)
        tri[3] = tri[6]; tri[4] = tri[7]; tri[5] = tri[8];
        tri[6] = tri[9]; tri[7] = tri[10]; tri[8] = tri[11];
    }
    return kind == kPair;
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
// tile (with antialiasing: come within half a pixel of one)?  The margin covers
// half a subpixel of snapping plus the error of the hardware reciprocal and of
// the fp32 arithmetic.
__device__ __forceinline__ bool box_has_centre(const RenderParams& P, const Tile& T, float xmn, float xmx, float ymn,
                                               float ymx, float mag)
{
    const float m = T.cm + (mag + P.cabs) * 3.814697265625e-06f;   // base + 2^-18 (|p| + |c|)
    // compared as integers against the tile's (scalar) bounds, after clamping
    // to +-2^30 (a NaN bound clamps to -2^30, which may cull a triangle with a
    // non-finite vertex: one that the snap's range rule drops anyway)
    auto toi = [](float x) { return (int)fminf(fmaxf(x, -1073741824.0f), 1073741824.0f); };
    const int ilo = max(toi(ceilf(xmn - m - 0.5f)), T.x0);
    const int ihi = min(toi(floorf(xmx + m - 0.5f)), T.x0 + T.w - 1);
    const int jlo = max(toi(ceilf(ymn - m - 0.5f)), T.y0);
    const int jhi = min(toi(floorf(ymx + m - 0.5f)), T.y0 + T.h - 1);
    return ilo <= ihi && jlo <= jhi;
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

// First pass of a static primitive (lane-wise).  r0, r1 for the halves (a, b,
// c) and (a, c, d) (a lone triangle has only the first): 0 the half cannot
// set a key of the tile, 1 it can and its vertices all lie in front of the near
// plane, 2 it can and it reaches behind the near plane.  A pair whose four
// vertices lie in front of the near plane and neither of whose halves lies
// wholly beyond far is tested once, by the projected box of all four vertices
// (conservative for each half); any other primitive tests each half with
// first_pass.
__device__ __forceinline__ void first_pass_prim(const RenderParams& P, const Tile& T, const Cam& cam, const float* v,
                                                bool pair, bool cull, int& r0, int& r1)
{
    float xv[4], yv[4], zv[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) view_xform(cam, v[3 * k], v[3 * k + 1], v[3 * k + 2], xv[k], yv[k], zv[k]);
    const bool all4 = zv[0] >= P.nearp && zv[1] >= P.nearp && zv[2] >= P.nearp && zv[3] >= P.nearp;
    const bool far0 = zv[0] > P.farp && zv[1] > P.farp && zv[2] > P.farp;
    const bool far1 = zv[0] > P.farp && zv[2] > P.farp && zv[3] > P.farp;
    if (pair && all4 && !far0 && !far1) {
        bool pass = true;
        if (cull) {
            float xmn = 3.0e38f, xmx = -3.0e38f, ymn = 3.0e38f, ymx = -3.0e38f, mag = 0.0f;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const float r = __builtin_amdgcn_rcpf(zv[k]);
                const float px = P.cx + P.fx * (xv[k] * r);
                const float py = P.cy - P.fy * (yv[k] * r);
                xmn = fminf(xmn, px); xmx = fmaxf(xmx, px);
                ymn = fminf(ymn, py); ymx = fmaxf(ymx, py);
                mag = fmaxf(mag, fmaxf(fabsf(px), fabsf(py)));
            }
            pass = box_has_centre(P, T, xmn, xmx, ymn, ymx, mag);
        }
        r0 = r1 = pass ? 1 : 0;
        return;
    }
    const float h0[9] = {v[0], v[1], v[2], v[3], v[4], v[5], v[6], v[7], v[8]};
    r0 = first_pass(P, T, cam, h0, cull) ? (zv[0] >= P.nearp && zv[1] >= P.nearp && zv[2] >= P.nearp ? 1 : 2) : 0;
    r1 = 0;
    if (pair) {
        const float h1[9] = {v[0], v[1], v[2], v[6], v[7], v[8], v[9], v[10], v[11]};
        r1 = first_pass(P, T, cam, h1, cull) ? (zv[0] >= P.nearp && zv[2] >= P.nearp && zv[3] >= P.nearp ? 1 : 2) : 0;
    }
}

// ---------------------------------------------------------------------------
// raster
// ---------------------------------------------------------------------------

// R7 key (Q24 << 8) | cls for 1/z = iz >= 1/far > 0, Q24 = (bits(IZCAP) >> 3) -
// (bits(min(iz, IZCAP)) >> 3).  Positive floats order like their bit patterns,
// and IZCAP is a power of two (low bits zero), so min(bits, bits(IZCAP)) >> 3 =
// min(bits >> 3, qbase): the clamp is a saturating subtract, one instruction.
// The class/depth kernel keeps the explicit minimum (the same key), with which
// its schedule ran faster.
__device__ __forceinline__ uint32_t depth_key(const RenderParams& P, float iz, uint32_t cls)
{
#ifdef PICTURA_RENDER_PLAIN
    const uint32_t bits = min(__float_as_uint(iz), __float_as_uint(P.izcap));
    return ((P.qbase - (bits >> 3)) << 8) | cls;
#else
    return (__builtin_elementwise_sub_sat(P.qbase, __float_as_uint(iz) >> 3) << 8) | cls;
#endif
}

// R7: key of a covered pixel, or 0xFFFFFFFF (no effect on the minimum) when
// the depth test rejects it.
__device__ __forceinline__ uint32_t pixel_key(const RenderParams& P, float pxf, float pyf, float pa, float pb,
                                              float pc, uint32_t cls)
{
    const float iz = fmaf(pa, pxf, fmaf(pb, pyf, pc));
    const uint32_t key = depth_key(P, iz, cls);
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

// A small triangle rasterized by its own lane over its bounding box.  With
// Exact (P.pix_exact) the pixel-centre offset of the next column is the
// previous one plus 1, exactly.
template <typename I, bool Exact>
__device__ __forceinline__ void raster_lane(const RenderParams& P, Shared& S, const Tile& T, int X0, int Y0, int X1,
                                            int Y1, int X2, int Y2, int i0, int i1, int j0, int j1, float pa,
                                            float pb, float pc, uint32_t cls)
{
    I f0 = edge_f<I>(X1, Y1, X2, Y2, i0, j0);
    I f1 = edge_f<I>(X2, Y2, X0, Y0, i0, j0);
    I f2 = edge_f<I>(X0, Y0, X1, Y1, i0, j0);
    const I sx0 = (I)(Y1 - Y2) * 256, sx1 = (I)(Y2 - Y0) * 256, sx2 = (I)(Y0 - Y1) * 256;
    const I sy0 = (I)(X2 - X1) * 256, sy1 = (I)(X0 - X2) * 256, sy2 = (I)(X1 - X0) * 256;
    const uint32_t kcls = cls;
    const float px0 = ((float)i0 + 0.5f) - P.cx;
    for (int j = j0; j <= j1; ++j) {
        I g0 = f0, g1 = f1, g2 = f2;
        const float pyf = ((float)j + 0.5f) - P.cy;
        const float inner = fmaf(pb, pyf, pc);
        uint32_t* row = &S.fb[(j - T.y0) * T.pitch - T.x0];
        float pxf = px0;
        for (int i = i0; i <= i1; ++i) {
            if constexpr (!Exact) pxf = ((float)i + 0.5f) - P.cx;
            const float iz = fmaf(pa, pxf, inner);
            const uint32_t key = depth_key(P, iz, kcls);
            if (((g0 | g1 | g2) >= 0) & (iz >= P.izfar)) atomicMin(&row[i], key);
            g0 += sx0; g1 += sx1; g2 += sx2;
            if constexpr (Exact) pxf += 1.0f;
        }
        f0 += sy0; f1 += sy1; f2 += sy2;
    }
}

// Rasterize the small triangles of the wave's lanes together: the pixels of
// their bounding boxes are numbered consecutively (exclusive prefix over the
// lanes) and every step hands 64 of them to the 64 lanes.  The lane owning
// slot k is found by marking where each triangle's range starts and taking
// a running maximum over the wave; its setup (the int32 record words, see
// above) is fetched from that lane with ds_bpermute.
__device__ __forceinline__ uint32_t bperm(int owner, uint32_t v)
{
    return (uint32_t)__builtin_amdgcn_ds_bpermute(owner * 4, (int)v);
}

__device__ __forceinline__ void raster_packed(const RenderParams& P, Shared& S, WaveLds& L, const Tile& T, bool on,
                                              const uint32_t* rv, int i0, int i1, int j0, int j1, float pa,
                                              float pb, float pc, uint32_t cls)
{
    const int lane = lane_id();
    const int w = i1 - i0 + 1;
    const uint32_t npx = on ? (uint32_t)(w * (j1 - j0 + 1)) : 0u;
    const uint32_t incl = wave_incl_sum(npx);
    const uint32_t n = readlane(incl, 63), pre = incl - npx;
    const uint32_t geo = (uint32_t)(i0 - T.x0) | (uint32_t)(j0 - T.y0) << 8 | (uint32_t)w << 16 | cls << 24;
    const float rw = __builtin_amdgcn_rcpf((float)w);   // row = floor((p + 0.5) / w) for p < 2^12
    uint32_t carry = 0;
    uint32_t* mark = L.u.cells.start;
    for (uint32_t s0 = 0; s0 < n; s0 += 64) {
        mark[lane] = 0u;
        __builtin_amdgcn_wave_barrier();
        if (npx != 0 && pre >= s0 && pre < s0 + 64u) mark[pre - s0] = (uint32_t)lane + 1u;
        __builtin_amdgcn_wave_barrier();
        const uint32_t o = wave_incl_max(max(mark[lane], carry));
        carry = readlane(o, 63);
        const int t = (int)o - 1;
        const uint32_t slot = s0 + (uint32_t)lane;
        const int p = (int)(slot - bperm(t, pre));
        const uint32_t g = bperm(t, geo);
        const int tw = (int)((g >> 16) & 255u);
        const int tn = (int)bperm(t, npx);
        const int jj = (int)(((float)p + 0.5f) * __uint_as_float(bperm(t, __float_as_uint(rw))));
        const int ii = p - jj * tw;
        const int x = (int)(g & 255u) + ii, y = (int)((g >> 8) & 255u) + jj;
        // scaled edge values floor(E / 256) at the tile-local pixel (x, y)
        const int e0 = (int)bperm(t, rv[6]) + __mul24((int)bperm(t, rv[0]), x) + __mul24((int)bperm(t, rv[3]), y);
        const int e1 = (int)bperm(t, rv[7]) + __mul24((int)bperm(t, rv[1]), x) + __mul24((int)bperm(t, rv[4]), y);
        const int e2 = (int)bperm(t, rv[8]) + __mul24((int)bperm(t, rv[2]), x) + __mul24((int)bperm(t, rv[5]), y);
        const float pxf = ((float)(T.x0 + x) + 0.5f) - P.cx;
        const float pyf = ((float)(T.y0 + y) + 0.5f) - P.cy;
        const float tpa = __uint_as_float(bperm(t, __float_as_uint(pa)));
        const float tpb = __uint_as_float(bperm(t, __float_as_uint(pb)));
        const float tpc = __uint_as_float(bperm(t, __float_as_uint(pc)));
        const float iz = fmaf(tpa, pxf, fmaf(tpb, pyf, tpc));
        const uint32_t key = depth_key(P, iz, (g >> 24));
        // p in range keeps the address inside the tile whatever the owner
        // search found; other lanes take word `lane` (distinct banks) and the
        // key 0xFFFFFFFF, which changes nothing, so the LDS minimum needs no
        // branch
        const bool inr = (slot < n) & (p >= 0) & (p < tn);
        const bool hit = inr & ((e0 | e1 | e2) >= 0) & (iz >= P.izfar);
        atomicMin(&S.fb[inr ? y * T.pitch + x : lane], hit ? key : 0xFFFFFFFFu);
        __builtin_amdgcn_wave_barrier();
    }
}

// Rasterize one record with the whole wave.  Lane b tests 8x8 block b of
// the bounding box (a tile has at most 8 x 8 blocks): the edge value at the
// block corner that maximises it must be >= 0 for all three edges.  The
// passing blocks are then rasterized one per step, lane l handling pixel
// (l & 7, l >> 3): its edge values at that pixel of block (0, 0) plus the
// block's offsets, which the lane that tested the block computed.
//
// int32 path (I32): the scaled edge floor(E / 256) with |dx|, |dy| < 2^22 and
// |floor(c / 256)| < 2^30, so dx, dy fit a 24-bit multiply and the value stays
// below 2^30 + 2 * 63 * 2^22 < 2^31 anywhere in the tile.
// fp64 path: |a_k|, |b_k| <= 2^38, so with tile coordinates below 64 every
// product and partial sum is an exact integer when |c| < 2^52; otherwise |c|
// exceeds the sum of all other terms by 2^9 and fixes the sign of every sum.
// Fast: the tile is a whole number of blocks and pixel-centre offsets are
// exact sums (P.pix_exact), so no lane leaves the tile and the offset of a
// pixel centre is the lane's own plus the block's.
template <bool I32, bool Fast>
__device__ __forceinline__ void raster_blocks(const RenderParams& P, Shared& S, const Tile& T, const uint32_t* u,
                                              float pa, float pb, float pc, uint32_t box, uint32_t j1w,
                                              float pxl, float pyl, int loff4)
{
    typedef typename std::conditional<I32, int, double>::type E;
    const int lane = lane_id(), lx = lane & 7, ly = lane >> 3;
    const uint32_t cls = box & 255u;
    const int i0 = (int)((box >> 8) & 255u), i1 = (int)((box >> 16) & 255u);
    const int j0 = (int)(box >> 24), j1 = (int)(j1w & 255u);
    const int bx0 = i0 >> 3, by0 = j0 >> 3;
    const int nbx = (i1 >> 3) - bx0 + 1, nb = nbx * ((j1 >> 3) - by0 + 1);
    // b / nbx == (b * rinv) >> 16 for b < 64 and nbx <= 8
    const uint32_t rinv = nbx == 1 ? 65536u : nbx == 2 ? 32768u : nbx == 3 ? 21846u : nbx == 4 ? 16384u
                        : nbx == 5 ? 13108u : nbx == 6 ? 10923u : nbx == 7 ? 9363u : 8192u;
    E A[3], B[3], Cc[3], Eb[3], off[3];
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        if constexpr (I32) {
            A[k] = (int)u[k];
            B[k] = (int)u[3 + k];
            Cc[k] = (int)u[6 + k];
            Eb[k] = __mul24(A[k], lx) + (__mul24(B[k], ly) + Cc[k]);
        } else {
            A[k] = -(double)(int)u[9 + k] * 256.0;
            B[k] = (double)(int)u[6 + k] * 256.0;
            Cc[k] = __longlong_as_double((long long)(((unsigned long long)u[2 * k + 1] << 32) | u[2 * k]));
            Eb[k] = fma(A[k], (double)lx, fma(B[k], (double)ly, Cc[k]));
        }
    }
    // lane b: block b of the box
    const int eby = (int)(((uint32_t)lane * rinv) >> 16), ebx = lane - eby * nbx;
    // (lanes past the box hold no block; the masks keep X and Y below 64, so the
    // products below stay 24-bit multiplies)
    const int X = ((bx0 + ebx) & 7) * 8, Y = ((by0 + eby) & 7) * 8;
    bool pass = lane < nb;
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        if constexpr (I32) {
            off[k] = __mul24(A[k], X) + __mul24(B[k], Y);
            const int d = 7 * (max(A[k], 0) + max(B[k], 0));
            pass = pass & ((Cc[k] + d) + off[k] >= 0);
        } else {
            off[k] = fma(A[k], (double)X, B[k] * (double)Y);
            const double d = 7.0 * (fmax(A[k], 0.0) + fmax(B[k], 0.0));
            pass = pass & ((Cc[k] + d) + off[k] >= 0.0);
        }
    }
    const float pxu = (float)(T.x0 + X), pyu = (float)(T.y0 + Y);
    const uint32_t xy = (uint32_t)X | ((uint32_t)Y << 8);
    const uint32_t boff = (uint32_t)((Y * T.pitch + X) * 4);   // byte offset of the block in the framebuffer
    uint64_t m = __ballot(pass);
    if (P.stats && lane == 0) {
        atomicAdd(&S.stat[kStBlocksTested], (uint32_t)nb);
        atomicAdd(&S.stat[kStBlocksPassed], (uint32_t)__popcll(m));
    }
    // Lanes that miss the piece take the key 0xFFFFFFFF, which changes
    // nothing, so the LDS minimum needs no branch (every address lies inside
    // the framebuffer: rows below 64, columns below the pitch).
    auto key_at = [&](int b, uint32_t& addr) -> uint32_t {
        if constexpr (I32 && Fast) {
            // the block's offsets, as the lane that tested it computed them
            // (broadcast through the LDS crossbar: no vector ALU instruction)
            // (all six fetched before any is used: one LDS round trip per block)
            const uint32_t ga = bperm(b, boff);
            const uint32_t g0 = bperm(b, (uint32_t)off[0]), g1 = bperm(b, (uint32_t)off[1]);
            const uint32_t g2 = bperm(b, (uint32_t)off[2]);
            const uint32_t gx = bperm(b, __float_as_uint(pxu)), gy = bperm(b, __float_as_uint(pyu));
            const int e0 = Eb[0] + (int)g0;
            const int e1 = Eb[1] + (int)g1;
            const int e2 = Eb[2] + (int)g2;
            const float pxf = pxl + __uint_as_float(gx);
            const float pyf = pyl + __uint_as_float(gy);
            const float iz = fmaf(pa, pxf, fmaf(pb, pyf, pc));
            const uint32_t key = depth_key(P, iz, cls);
            addr = ga + (uint32_t)loff4;
            return (((e0 | e1 | e2) >= 0) && iz >= P.izfar) ? key : 0xFFFFFFFFu;
        }
        const uint32_t q = readlane(xy, b);
        const int bX = (int)(q & 255u), bY = (int)(q >> 8);
        bool cov;
        if constexpr (I32) {
            const int e0 = Eb[0] + (A[0] * bX + B[0] * bY);
            const int e1 = Eb[1] + (A[1] * bX + B[1] * bY);
            const int e2 = Eb[2] + (A[2] * bX + B[2] * bY);
            cov = (e0 | e1 | e2) >= 0;
        } else {
            const double e0 = Eb[0] + readlane_d(off[0], b);
            const double e1 = Eb[1] + readlane_d(off[1], b);
            const double e2 = Eb[2] + readlane_d(off[2], b);
            cov = (e0 >= 0.0) & (e1 >= 0.0) & (e2 >= 0.0);
        }
        float pxf, pyf;
        if constexpr (Fast) {
            pxf = pxl + readlane_f(pxu, b);
            pyf = pyl + readlane_f(pyu, b);
        } else {
            cov = cov & (lx < T.w - bX) & (ly < T.h - bY);
            pxf = ((float)(T.x0 + bX + lx) + 0.5f) - P.cx;
            pyf = ((float)(T.y0 + bY + ly) + 0.5f) - P.cy;
        }
        const float iz = fmaf(pa, pxf, fmaf(pb, pyf, pc));
        const uint32_t key = depth_key(P, iz, cls);
        addr = (uint32_t)((bY * T.pitch + bX) * 4 + loff4);
        return (cov && iz >= P.izfar) ? key : 0xFFFFFFFFu;
    };
    while (m) {
        const int b0 = __builtin_ctzll(m);
        m &= m - 1;
        uint32_t a0;
        const uint32_t k0 = key_at(b0, a0);
        atomicMin((uint32_t*)((char*)S.fb + a0), k0);
    }
}

// ---------------------------------------------------------------------------
// exact pass: one queued survivor per live lane
// ---------------------------------------------------------------------------

// R2, R4 and R5 for one world-space triangle: view transform, near clip
// (Sutherland-Hodgman, explicit cases), snap.  Returns 0 (not drawn), 3, or 4
// (a quad drawn as the fan pieces (p0, p1, p2) and (p0, p2, p3)).
__device__ __forceinline__ int setup_triangle(const RenderParams& P, Shared& S, const Cam& cam, const float* tri,
                                              int& X0, int& Y0, int& X1, int& Y1, int& X2, int& Y2, int& X3,
                                              int& Y3)
{
    int np = 0;
    float xv[3], yv[3], zv[3];
#pragma unroll
    for (int k = 0; k < 3; ++k) view_xform(cam, tri[3 * k], tri[3 * k + 1], tri[3 * k + 2], xv[k], yv[k], zv[k]);
    const bool in0 = zv[0] >= P.nearp, in1 = zv[1] >= P.nearp, in2 = zv[2] >= P.nearp;
    // R4: nothing of the triangle inside near .. far
    if (!(in0 || in1 || in2)) return 0;
    if (zv[0] > P.farp && zv[1] > P.farp && zv[2] > P.farp) return 0;
    bool ok = true;
    if (in0 && in1 && in2) {
        ok = snap_vertex(P, xv[0], yv[0], zv[0], X0, Y0) && snap_vertex(P, xv[1], yv[1], zv[1], X1, Y1) &&
             snap_vertex(P, xv[2], yv[2], zv[2], X2, Y2);
        np = 3;
    } else {
        // R4: Sutherland-Hodgman output of the six straddling cases, in
        // the order in which v0v1, v1v2, v2v0 visit the edges.
        STAT(kStClipped, 1);
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
                 setp(3, x20, y20, nz); np = 4; break;   // case 6 (cases 0 and 7 returned above)
        }
        if (np == 3) { px[3] = px[2]; py[3] = py[2]; pz[3] = pz[2]; }
        ok = snap_vertex(P, px[0], py[0], pz[0], X0, Y0) && snap_vertex(P, px[1], py[1], pz[1], X1, Y1) &&
             snap_vertex(P, px[2], py[2], pz[2], X2, Y2) && snap_vertex(P, px[3], py[3], pz[3], X3, Y3);
    }
    return ok ? np : 0;
}

// R14 (colour antialiasing): the fragments a surface leaves on the pixels its
// edges cross.  A surface is a fan piece, or a whole convex 4-gon: a pair
// whose two halves are both drawn, or a triangle clipped to four vertices,
// when the snapped 4-gon is strictly convex (its pieces then leave no
// fragments of their own, so the diagonal does not cut the coverage of a
// surface narrower than a pixel).  For every tile pixel whose centre lies
// within one pixel of the surface's snapped bounding box: with E_k the exact
// edge function of R6 at the centre (no top-left bias) and L_k the edge's
// length in subpixels, E_k / (256 L_k) is the centre's distance to the edge in
// pixels (positive inside); c_k = min(max(fma(fl(E_k), fl(1 / (256 L_k)),
// 0.5), 0), 1), coverage a = min(max(((c_0 + c_1) + c_2) - 2, 0), 1) for a
// triangle (edges b->c, c->a, a->b) and min(max((((c_0 + c_1) + c_2) + c_3) -
// 3, 0), 1) for a 4-gon (edges p_k -> p_k+1), a8 = rint(255 a).  A pixel with
// 0 < a8 < 255 whose key (R7, the first piece's plane at the centre) exists
// takes the minimum of (key >> 16) << 16 | (key & 255) << 8 | (255 - a8) in
// the edge buffer.  fl(E_k) is the same value whichever exact integer type
// carries E_k.
__device__ __forceinline__ float aa_cover(double e, float r)
{
    return fminf(fmaxf(fmaf((float)e, r, 0.5f), 0.0f), 1.0f);
}

__device__ __forceinline__ float aa_cover(int e, float r)
{
    return fminf(fmaxf(fmaf((float)e, r, 0.5f), 0.0f), 1.0f);
}

// Coverage fragment of one pixel (c the edge coverages, c3 used by a 4-gon
// only): the edge buffer word, or 0xFFFFFFFF when the pixel takes none.
__device__ __forceinline__ uint32_t aa_fragment(const RenderParams& P, bool q4, float c0, float c1, float c2, float c3,
                                                float pxf, float pyf, float pa, float pb, float pc, uint32_t cls)
{
    const float s = (c0 + c1) + c2;
    const float a = fminf(fmaxf(q4 ? (s + c3) - 3.0f : s - 2.0f, 0.0f), 1.0f);
    const uint32_t a8 = (uint32_t)rintf(255.0f * a);
    const uint32_t key = pixel_key(P, pxf, pyf, pa, pb, pc, cls);
    const bool frag = a8 != 0u && a8 != 255u && key != 0xFFFFFFFFu;
    return frag ? ((key >> 16) << 16) | ((key & 255u) << 8) | (255u - a8) : 0xFFFFFFFFu;
}

// Pieces with small windows, all lanes together: the window pixels are
// numbered consecutively over the lanes and every step hands 64 of them to the
// 64 lanes (as the packed raster does).  With spans below 2^14 subpixels the
// edge function at any window pixel is below 2^30 in magnitude, so it is an
// int32 value plus int32 steps from the window's first pixel.
constexpr int kAaSmall = 128;   // most window pixels of a packed piece

__device__ __forceinline__ void aa_packed(const RenderParams& P, Shared& S, WaveLds& L, uint32_t* fbo, const Tile& T, bool on,
                                          bool q4, bool any4, int i0, int j0, int w, int npx_, const int* e,
                                          const int* sa, const int* sb, const float* r, float pa, float pb, float pc,
                                          uint32_t cls)
{
    const int lane = lane_id();
    const uint32_t npx = on ? (uint32_t)npx_ : 0u;
    const uint32_t incl = wave_incl_sum(npx);
    const uint32_t n = readlane(incl, 63), pre = incl - npx;
    const uint32_t geo = (uint32_t)i0 | (q4 ? 128u : 0u) | (uint32_t)j0 << 8 | (uint32_t)w << 16 | cls << 24;
    const float rw = __builtin_amdgcn_rcpf((float)w);   // row = floor((p + 0.5) / w) for p < 2^12
    STAT1(kStAaPackedPx, n);
    STAT1(kStAaPackedSteps, (n + 63u) >> 6);
    uint32_t carry = 0;
    uint32_t* mark = L.u.cells.start;
    for (uint32_t s0 = 0; s0 < n; s0 += 64) {
        mark[lane] = 0u;
        __builtin_amdgcn_wave_barrier();
        if (npx != 0 && pre >= s0 && pre < s0 + 64u) mark[pre - s0] = (uint32_t)lane + 1u;
        __builtin_amdgcn_wave_barrier();
        const uint32_t o = wave_incl_max(max(mark[lane], carry));
        carry = readlane(o, 63);
        const int t = (int)o - 1;
        const uint32_t slot = s0 + (uint32_t)lane;
        const int p = (int)(slot - bperm(t, pre));
        const uint32_t g = bperm(t, geo);
        const int tw = (int)((g >> 16) & 255u);
        const int tn = (int)bperm(t, npx);
        const int jj = (int)(((float)p + 0.5f) * __uint_as_float(bperm(t, __float_as_uint(rw))));
        const int ii = p - jj * tw;
        const int x = (int)(g & 127u) + ii, y = (int)((g >> 8) & 255u) + jj;   // tile pixel
        float c[4] = {0.0f, 0.0f, 0.0f, 1.0f};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if (k == 3 && !any4) break;
            const int ek = (int)bperm(t, (uint32_t)e[k]) + __mul24((int)bperm(t, (uint32_t)sa[k]), ii) +
                           __mul24((int)bperm(t, (uint32_t)sb[k]), jj);
            c[k] = aa_cover(ek, __uint_as_float(bperm(t, __float_as_uint(r[k]))));
        }
        const float pxf = ((float)(T.x0 + x) + 0.5f) - P.cx;
        const float pyf = ((float)(T.y0 + y) + 0.5f) - P.cy;
        const uint32_t f = aa_fragment(P, (g & 128u) != 0u, c[0], c[1], c[2], c[3], pxf, pyf,
                                       __uint_as_float(bperm(t, __float_as_uint(pa))),
                                       __uint_as_float(bperm(t, __float_as_uint(pb))),
                                       __uint_as_float(bperm(t, __float_as_uint(pc))), g >> 24);
        // p in range keeps the address inside the window, hence the tile
        const bool inr = (slot < n) & (p >= 0) & (p < tn);
        STAT(kStAaFrags, inr && f != 0xFFFFFFFFu ? 1 : 0);
        if (inr && f != 0xFFFFFFFFu) atomicMin(&fbo[y * P.W + x], f);
        __builtin_amdgcn_wave_barrier();
    }
}

// Window of a surface: the tile pixels whose centre lies within half a pixel
// of its snapped bounding box, 256 i + 128 in [minX - 128, maxX + 128].  The
// rule considers centres within one pixel, but one more than half a pixel
// beyond the box (say left of the leftmost vertex v) takes no fragment: the
// two edges at v leave from v rightwards, at angles phi_1 < phi_2 within
// [-pi/2, pi/2] of the x axis; with d_k the centre's inside distance to edge
// k, d_1 + d_2 = 2 sin(theta/2) (dy sin psi - g cos psi) for the centre at
// (-g, dy) from v, psi the bisector's angle and theta = phi_2 - phi_1, and
// d_1 + d_2 > 0 together with d_2 > -1/2 would need g cos(theta/2) <
// sin(psi) / 2 <= cos(theta/2) / 2 (as phi_2 <= pi/2), which g > 1/2 rules
// out (likewise d_1 > -1/2 for psi < 0).  So c_1 + c_2 <= 1 and the sum of
// all coverages is at most 2 (a triangle) or 3 (a 4-gon): a = 0, and the
// fp32 rounding (below 1e-6) keeps rint(255 a) at 0.
// Surfaces whose window has at most kAaSmall pixels and whose box spans below
// 2^14 subpixels take the packed path; the others are swept by the whole wave
// one at a time in 8x8 blocks (lane = pixel), E_k evaluated in fp64 from its
// exact integer value at the tile origin plus exact integer steps: exact while
// |E_k| < 2^53, and beyond that c_k is 0 or 1 whatever the rounding
// (|E_k| / (256 L_k) > 2^14 with L_k < 2^31).  c_k grows with E_k, so a block
// whose largest E_k gives c_k = 0 for some edge, or whose smallest E_k give
// c_k = 1 for every edge, has no fragment and is skipped.  The surface is the
// triangle (a, b, c) in either orientation, or with q4 the 4-gon (a, b, c, d)
// in positive orientation; a triangle's fourth edge is a constant c_3 = 1
// that its coverage does not use.
__device__ void aa_pieces(const RenderParams& P, Shared& S, WaveLds& L, uint32_t* fbo, const Tile& T, bool ok, bool q4, int ax,
                          int ay, int bx, int by, int cx, int cy, int dx4, int dy4, float pa, float pb, float pc,
                          uint32_t cls)
{
    const int lane = lane_id(), lx = lane & 7, ly = lane >> 3;
    int i0 = 0, i1 = -1, j0 = 0, j1 = -1;
    int dxs[4] = {0, 0, 0, 0}, dys[4] = {0, 0, 0, 0};
    long long e0[4] = {0, 0, 0, 1ll << 30};
    float rden[4] = {0.0f, 0.0f, 0.0f, 1.0f};
    bool small = false;
    if (ok) {
        int vx[4], vy[4];   // edge k runs from v_k to v_k+1 (cyclically over 3 or 4)
        if (q4) {
            vx[0] = ax; vx[1] = bx; vx[2] = cx; vx[3] = dx4;
            vy[0] = ay; vy[1] = by; vy[2] = cy; vy[3] = dy4;
        } else {
            const long long area2 =
                (long long)(bx - ax) * (long long)(cy - ay) - (long long)(by - ay) * (long long)(cx - ax);
            if (area2 < 0) {
                const int tx = bx, ty = by;
                bx = cx; by = cy; cx = tx; cy = ty;
            }
            ok = area2 != 0;
            vx[0] = bx; vx[1] = cx; vx[2] = ax; vx[3] = ax;
            vy[0] = by; vy[1] = cy; vy[2] = ay; vy[3] = ay;
        }
        const int minX = min(min(vx[0], vx[1]), min(vx[2], vx[3])), maxX = max(max(vx[0], vx[1]), max(vx[2], vx[3]));
        const int minY = min(min(vy[0], vy[1]), min(vy[2], vy[3])), maxY = max(max(vy[0], vy[1]), max(vy[2], vy[3]));
        i0 = max((minX - 1) >> 8, T.x0) - T.x0; i1 = min(maxX >> 8, T.x0 + T.w - 1) - T.x0;
        j0 = max((minY - 1) >> 8, T.y0) - T.y0; j1 = min(maxY >> 8, T.y0 + T.h - 1) - T.y0;
        ok = ok && i0 <= i1 && j0 <= j1;
        small = ok && (maxX - minX) < 16384 && (maxY - minY) < 16384 && (i1 - i0 + 1) * (j1 - j0 + 1) <= kAaSmall;
        // edge functions at the window's first pixel (small) or at the tile's
        const int px0 = 256 * (T.x0 + (small ? i0 : 0)) + 128, py0 = 256 * (T.y0 + (small ? j0 : 0)) + 128;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            if (k == 3 && !q4) break;
            const int nk = k == 3 || (k == 2 && !q4) ? 0 : k + 1;
            const int dx = vx[nk] - vx[k], dy = vy[nk] - vy[k];
            e0[k] = (long long)dx * (long long)(py0 - vy[k]) - (long long)dy * (long long)(px0 - vx[k]);
            dxs[k] = dx;
            dys[k] = dy;
            const float len = sqrtf((float)((long long)dx * dx + (long long)dy * dy));
            rden[k] = 1.0f / (256.0f * len);
        }
    }
    const bool any4 = __ballot(ok && q4) != 0;
    STAT(kStAaPacked, small ? 1 : 0);
    STAT(kStAaSwept, ok && !small ? 1 : 0);
    if (__ballot(small) != 0) {
        const int e[4] = {(int)e0[0], (int)e0[1], (int)e0[2], (int)e0[3]};
        const int sa[4] = {-256 * dys[0], -256 * dys[1], -256 * dys[2], -256 * dys[3]};
        const int sb[4] = {256 * dxs[0], 256 * dxs[1], 256 * dxs[2], 256 * dxs[3]};
        aa_packed(P, S, L, fbo, T, small, q4, any4, i0, j0, i1 - i0 + 1, (i1 - i0 + 1) * (j1 - j0 + 1), e, sa, sb, rden,
                  pa, pb, pc, cls);
    }
    uint64_t m = __ballot(ok && !small);
    while (m) {
        const int l = __builtin_ctzll(m);
        m &= m - 1;
        const int ri0 = (int)readlane((uint32_t)i0, l), ri1 = (int)readlane((uint32_t)i1, l);
        const int rj0 = (int)readlane((uint32_t)j0, l), rj1 = (int)readlane((uint32_t)j1, l);
        const bool rq4 = readlane(q4 ? 1u : 0u, l) != 0u;
        double re[4], rsx[4], rsy[4];
        float rr[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            const unsigned long long u = (unsigned long long)e0[k];
            re[k] = (double)(long long)(((unsigned long long)readlane((uint32_t)(u >> 32), l) << 32) |
                                        readlane((uint32_t)u, l));
            rsx[k] = -256.0 * (double)(int)readlane((uint32_t)dys[k], l);
            rsy[k] = 256.0 * (double)(int)readlane((uint32_t)dxs[k], l);
            rr[k] = readlane_f(rden[k], l);
        }
        const float rpa = readlane_f(pa, l), rpb = readlane_f(pb, l), rpc = readlane_f(pc, l);
        const uint32_t rcls = readlane(cls, l);
        const int nbx = (ri1 - ri0 + 8) >> 3, nby = (rj1 - rj0 + 8) >> 3;   // at most 8 x 8 blocks
        uint64_t bm = 1;
        if (nbx * nby > 1) {
            // lane = block (lx, ly) of the window: does it hold a fragment?
            bool need = false;
            if (lx < nbx && ly < nby) {
                const int bi0 = ri0 + 8 * lx, bi1 = min(bi0 + 7, ri1);
                const int bj0 = rj0 + 8 * ly, bj1 = min(bj0 + 7, rj1);
                bool out = false, in = true;
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const double emax = fma(rsy[k], (double)(rsy[k] > 0.0 ? bj1 : bj0),
                                            fma(rsx[k], (double)(rsx[k] > 0.0 ? bi1 : bi0), re[k]));
                    const double emin = fma(rsy[k], (double)(rsy[k] > 0.0 ? bj0 : bj1),
                                            fma(rsx[k], (double)(rsx[k] > 0.0 ? bi0 : bi1), re[k]));
                    out = out || aa_cover(emax, rr[k]) == 0.0f;
                    in = in && aa_cover(emin, rr[k]) == 1.0f;
                }
                need = !out && !in;
            }
            bm = __ballot(need);
        }
        STAT1(kStAaBlocks, __popcll(bm));
        while (bm) {
            const int b = __builtin_ctzll(bm);
            bm &= bm - 1;
            const int i = ri0 + 8 * (b & 7) + lx, j = rj0 + 8 * (b >> 3) + ly;   // tile pixel
            if (i > ri1 || j > rj1) continue;
            const double di = (double)i, dj = (double)j;
            const uint32_t f = aa_fragment(P, rq4, aa_cover(fma(rsy[0], dj, fma(rsx[0], di, re[0])), rr[0]),
                                           aa_cover(fma(rsy[1], dj, fma(rsx[1], di, re[1])), rr[1]),
                                           aa_cover(fma(rsy[2], dj, fma(rsx[2], di, re[2])), rr[2]),
                                           aa_cover(fma(rsy[3], dj, fma(rsx[3], di, re[3])), rr[3]),
                                           ((float)(T.x0 + i) + 0.5f) - P.cx, ((float)(T.y0 + j) + 0.5f) - P.cy, rpa,
                                           rpb, rpc, rcls);
            STAT(kStAaFrags, f != 0xFFFFFFFFu ? 1 : 0);
            if (f != 0xFFFFFFFFu) atomicMin(&fbo[j * P.W + i], f);
        }
    }
}

template <bool kAA, bool kHasLights>
__device__ __forceinline__ void exact_pass(const RenderParams& P, Shared& S, WaveLds& L, const Tile& T, const Cam& cam,
                                           bool live, uint32_t entry, int64_t abase_w, int64_t lbase_w, float pxl,
                                           float pyl, int loff4, uint32_t* fbo)
{
    float tri[12] = {};
    uint32_t cls = 0;
    int np = 0;
    bool quad = false;   // a whole pair: the 4-gon (a, b, c, d), every vertex in front of the near plane
    bool snap0 = true, snap1 = true;   // a whole pair's halves: every vertex snapped
    int X0 = 0, Y0 = 0, X1 = 0, Y1 = 0, X2 = 0, Y2 = 0, X3 = 0, Y3 = 0;
    if (live) {
        quad = load_entry<kHasLights>(P, entry, abase_w, lbase_w, tri, cls);
        float xv[3], yv[3], zv[3];
#pragma unroll
        for (int k = 0; k < 3; ++k) view_xform(cam, tri[3 * k], tri[3 * k + 1], tri[3 * k + 2], xv[k], yv[k], zv[k]);
        const bool in0 = zv[0] >= P.nearp, in1 = zv[1] >= P.nearp, in2 = zv[2] >= P.nearp;
        bool ok = true;
        if (quad) {
            // the pair's halves (a, b, c) and (a, c, d) are the fan pieces of (a, b, c, d)
            float x3, y3, z3;
            view_xform(cam, tri[9], tri[10], tri[11], x3, y3, z3);
            const bool s0 = snap_vertex(P, xv[0], yv[0], zv[0], X0, Y0);
            const bool s1 = snap_vertex(P, xv[1], yv[1], zv[1], X1, Y1);
            const bool s2 = snap_vertex(P, xv[2], yv[2], zv[2], X2, Y2);
            const bool s3 = snap_vertex(P, x3, y3, z3, X3, Y3);
            // R5: a vertex out of range drops only the halves that use it
            snap0 = s0 && s1 && s2;
            snap1 = s0 && s2 && s3;
            ok = snap0 || snap1;
            np = 4;
        } else if (in0 && in1 && in2) {
            ok = snap_vertex(P, xv[0], yv[0], zv[0], X0, Y0) && snap_vertex(P, xv[1], yv[1], zv[1], X1, Y1) &&
                 snap_vertex(P, xv[2], yv[2], zv[2], X2, Y2);
            np = 3;
        } else {
            // R4: Sutherland-Hodgman output of the six straddling cases, in
            // the order in which v0v1, v1v2, v2v0 visit the edges.
            STAT(kStClipped, 1);
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
    const int nfan = __ballot(np == 4) != 0 ? 2 : 1;
    // R3 depth planes: the unclipped triangle's, shared by the fan pieces of a
    // clipped triangle; each half of a pair has its own
    float pa0 = 0.0f, pb0 = 0.0f, pc0 = 0.0f;
    const bool okp0 = np != 0 && depth_plane(P, cam, tri, pa0, pb0, pc0);
    bool ok0 = okp0 && snap0;
    float pa1 = pa0, pb1 = pb0, pc1 = pc0;
    bool ok1 = ok0;
    if (__ballot(quad) != 0) {
        const float t2[9] = {tri[0], tri[1], tri[2], tri[6], tri[7], tri[8], tri[9], tri[10], tri[11]};
        float qa = 0.0f, qb = 0.0f, qc = 0.0f;
        const bool okq = depth_plane(P, cam, t2, qa, qb, qc);
        if (quad) {
            pa1 = qa; pb1 = qb; pc1 = qc;
            ok1 = np != 0 && okq && snap1;
        }
    }
    // R14: a 4-gon (whole pair or clipped triangle) with both pieces drawn
    // is one surface when strictly convex; (q_k) its positive order
    bool aaq = false;
    int qx[4] = {X0, X1, X2, X3}, qy[4] = {Y0, Y1, Y2, Y3};
    if constexpr (kAA) {
        if (np == 4 && ok0 && ok1) {
            int pos = 0, neg = 0;
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int k1 = (k + 1) & 3, k2 = (k + 2) & 3;
                const long long cr = (long long)(qx[k1] - qx[k]) * (long long)(qy[k2] - qy[k1]) -
                                     (long long)(qy[k1] - qy[k]) * (long long)(qx[k2] - qx[k1]);
                pos += cr > 0;
                neg += cr < 0;
            }
            aaq = pos == 4 || neg == 4;
            if (neg == 4) {   // (q0, q3, q2, q1)
                qx[1] = X3; qy[1] = Y3;
                qx[3] = X1; qy[3] = Y1;
            }
        }
    }
    const int px0 = 256 * T.x0 + 128, py0 = 256 * T.y0 + 128;
    // fan triangles (p0, p1, p2) and (p0, p2, p3)
#pragma unroll 1
    for (int f = 0; f < nfan; ++f) {
        const float pa = f ? pa1 : pa0, pb = f ? pb1 : pb0, pc = f ? pc1 : pc0;
        const bool piece = f + 2 < np && (f ? ok1 : ok0);
        bool valid = false;
        const int ax = X0, ay = Y0;
        int bx = f == 0 ? X1 : X2, by = f == 0 ? Y1 : Y2;
        int cx = f == 0 ? X2 : X3, cy = f == 0 ? Y2 : Y3;
        int i0 = 0, i1 = -1, j0 = 0, j1 = -1;
        if (piece) {
            const int minX = min(ax, min(bx, cx)), maxX = max(ax, max(bx, cx));
            const int minY = min(ay, min(by, cy)), maxY = max(ay, max(by, cy));
            i0 = max((minX - 128 + 255) >> 8, T.x0); i1 = min((maxX - 128) >> 8, T.x0 + T.w - 1);
            j0 = max((minY - 128 + 255) >> 8, T.y0); j1 = min((maxY - 128) >> 8, T.y0 + T.h - 1);
            if (i0 <= i1 && j0 <= j1) {
                STAT(kStRasterTris, 1);
                const bool small_span = (maxX - minX) < 16384 && (maxY - minY) < 16384;
                long long area2;
                if (small_span) area2 = (long long)(__mul24(bx - ax, cy - ay) - __mul24(by - ay, cx - ax));
                else area2 = (long long)(bx - ax) * (long long)(cy - ay) - (long long)(by - ay) * (long long)(cx - ax);
                if (area2 != 0) {
                    if (area2 < 0) {
                        const int tx = bx, ty = by;
                        bx = cx; by = cy; cx = tx; cy = ty;
                    }
                    valid = true;
                }
            }
        }
        // edge setup: edges v1->v2, v2->v0, v0->v1 at the tile's pixel (0, 0),
        // in the int32 form (floor(c / 256), -dy, dx) when every value fits
        uint32_t rv[12] = {0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0};
        bool e32 = true;
        if (valid) {
            const int ex[3] = {bx, cx, ax}, ey[3] = {by, cy, ay};
            const int fx[3] = {cx, ax, bx}, fy[3] = {cy, ay, by};
            long long cv[3];
            int dxs[3], dys[3];
#pragma unroll
            for (int k = 0; k < 3; ++k) {
                const int dx = fx[k] - ex[k], dy = fy[k] - ey[k];
                const int tl = (dy < 0) || (dy == 0 && dx > 0);
                cv[k] = (long long)dx * (long long)(py0 - ey[k]) - (long long)dy * (long long)(px0 - ex[k]) +
                        (long long)(tl - 1);
                const long long c8 = cv[k] >> 8;   // floor(c / 256)
                e32 = e32 && dx > -4194304 && dx < 4194304 && dy > -4194304 && dy < 4194304 &&
                      c8 > -1073741824ll && c8 < 1073741824ll;
                dxs[k] = dx;
                dys[k] = dy;
            }
#pragma unroll
            for (int k = 0; k < 3; ++k) {
                if (e32) {
                    rv[k] = (uint32_t)(-dys[k]);
                    rv[3 + k] = (uint32_t)dxs[k];
                    rv[6 + k] = (uint32_t)(int)(cv[k] >> 8);
                } else {
                    const unsigned long long cb = (unsigned long long)__double_as_longlong((double)cv[k]);
                    rv[2 * k] = (uint32_t)cb;
                    rv[2 * k + 1] = (uint32_t)(cb >> 32);
                    rv[6 + k] = (uint32_t)dxs[k];
                    rv[9 + k] = (uint32_t)dys[k];
                }
            }
        }
        const int npx = (i1 - i0 + 1) * (j1 - j0 + 1);
        const bool big = valid && npx > kSmallPx;
        const bool packed = valid && npx <= kSmallPx && e32;
        if (valid && npx <= kSmallPx) {
            STAT(kStLaneTris, 1);
            STAT(kStLanePx, npx);
            if (!e32)
                raster_lane<long long, false>(P, S, T, ax, ay, bx, by, cx, cy, i0, i1, j0, j1, pa, pb, pc, cls);
        }
        if (__ballot(packed) != 0) raster_packed(P, S, L, T, packed, rv, i0, i1, j0, j1, pa, pb, pc, cls);
        uint64_t m = __ballot(big);
        if (m == 0) continue;
        uint32_t rbox = 0, rj1 = 0;
        if (big) {
            rbox = cls | (uint32_t)(i0 - T.x0) << 8 | (uint32_t)(i1 - T.x0) << 16 | (uint32_t)(j0 - T.y0) << 24;
            rj1 = (uint32_t)(j1 - T.y0) | (e32 ? 256u : 0u);
            STAT(kStRecTris, 1);
            if (!e32) STAT(kStRecWide, 1);
        }
        const bool fast = P.pix_exact && (T.w & 7) == 0 && (T.h & 7) == 0;
        // hand int32-form records to the view's record ring (both waves drain it at the end)
        const uint64_t md = __ballot(big && e32);
        const uint32_t cap = (uint32_t)T.h >> 2;
        if (md != 0 && cap != 0) {
            const int l0 = __builtin_ctzll(md);
            uint32_t base = 0;
            if (lane_id() == l0) base = atomicAdd(&S.ctl[kRecTail], (uint32_t)__popcll(md));
            base = readlane(base, l0);
            const uint32_t slot = base + mbcnt(md);
            const bool put = big && e32 && slot < cap;
            if (put) {
                u32x4* g = (u32x4*)&S.fb[4 * (int)slot * T.pitch + T.pitch - 4];
                const int rs = T.pitch >> 2;   // 16-byte units per framebuffer row
                g[0] = u32x4{rv[0], rv[1], rv[2], rv[3]};
                g[rs] = u32x4{rv[4], rv[5], rv[6], rv[7]};
                g[2 * rs] = u32x4{rv[8], __float_as_uint(pa), __float_as_uint(pb), __float_as_uint(pc)};
                uint32_t* w3 = &S.fb[(4 * (int)slot + 3) * T.pitch + T.pitch - 4];
                w3[0] = rbox;
                w3[1] = rj1;
                lds_store_release(&w3[2], kRecReady);
            }
            m &= ~__ballot(put);
        }
        TSTART(t_rec);
        while (m) {
            const int l = __builtin_ctzll(m);
            m &= m - 1;
            const float rpa = readlane_f(pa, l), rpb = readlane_f(pb, l), rpc = readlane_f(pc, l);
            const uint32_t rb = readlane(rbox, l), rj = readlane(rj1, l);
            uint32_t uw[12];
            if (rj & 256u) {
#pragma unroll
                for (int q = 0; q < 9; ++q) uw[q] = readlane(rv[q], l);
                if (fast) raster_blocks<true, true>(P, S, T, uw, rpa, rpb, rpc, rb, rj, pxl, pyl, loff4);
                else raster_blocks<true, false>(P, S, T, uw, rpa, rpb, rpc, rb, rj, pxl, pyl, loff4);
            } else {
#pragma unroll
                for (int q = 0; q < 12; ++q) uw[q] = readlane(rv[q], l);
                if (fast) raster_blocks<false, true>(P, S, T, uw, rpa, rpb, rpc, rb, rj, pxl, pyl, loff4);
                else raster_blocks<false, false>(P, S, T, uw, rpa, rpb, rpc, rb, rj, pxl, pyl, loff4);
            }
        }
        TACC(kCycRecords, t_rec);
    }
    // R14 fragments after both pieces' keys (the two buffers take minima, so
    // the order does not matter; here fewer values are live)
    if constexpr (kAA) {
#pragma unroll 1
        for (int f = 0; f < nfan; ++f) {
            const bool piece = f + 2 < np && (f ? ok1 : ok0);
            const bool sq = aaq && f == 0;   // the whole surface, with the first piece's plane
            const int bx = f == 0 ? X1 : X2, by = f == 0 ? Y1 : Y2;
            const int cx = f == 0 ? X2 : X3, cy = f == 0 ? Y2 : Y3;
            aa_pieces(P, S, L, fbo, T, sq || (piece && !aaq), sq, sq ? qx[0] : X0, sq ? qy[0] : Y0, sq ? qx[1] : bx,
                      sq ? qy[1] : by, sq ? qx[2] : cx, sq ? qy[2] : cy, qx[3], qy[3], f ? pa1 : pa0, f ? pb1 : pb0,
                      f ? pc1 : pc0, cls);
        }
    }
}

// Append the lanes with `pred` to this wave's queue (ballot + mbcnt, no
// atomics); returns the new depth, which is uniform across the wave.
__device__ __forceinline__ int queue_push(WaveLds& L, int nq, bool pred, uint32_t val)
{
    const uint64_t m = __ballot(pred);
    if (pred) L.q[nq + mbcnt(m)] = val;
    return nq + (int)__popcll(m);
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

// The same test for a rectangle in the xy plane against a plane with nz = 0.
__device__ __forceinline__ bool rect_outside(float cx, float cy, float h, float nx, float ny, float o)
{
    const float v = nx * cx + ny * cy + (fabsf(nx) + fabsf(ny)) * h + o;
    const float mag = fabsf(nx) * (fabsf(cx) + h) + fabsf(ny) * (fabsf(cy) + h) + fabsf(o);
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
    if (!(zmn >= P.near_cull)) return true;   // crosses or nearly touches the near plane
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

__device__ __forceinline__ uint32_t xcd_remap(uint32_t b, uint32_t nb)
{
    // Workgroups are dispatched round-robin over the 8 XCDs; give each XCD a
    // contiguous range of views so that one world's views share an L2.
    const uint32_t q = nb >> 3, r = nb & 7u, x = b & 7u, k = b >> 3;
    return x * q + (x < r ? x : r) + k;
}

// n / d for n < 2^31 (see Div31)
__device__ __forceinline__ uint32_t div31(uint32_t n, Div31 d) { return d.m ? (__umulhi(n, d.m) >> d.s) : n; }

// R13: colour of a resolved key.  Shading id sid = key & 255: class = sid & 15,
// face = sid >> 4 (0: not a box face).  v = base[class] * (face factor * b),
// b = 1 - 0.6 min(z / far, 1) on box faces (depth-aware brightness, z the
// decoded depth of R8), 1 elsewhere; byte = rint(255 min(v, 1)).
__device__ __forceinline__ float decode_depth(const RenderParams& P, uint32_t key)
{
    const float d = __uint_as_float(((P.qbase - (key >> 8)) << 3) | 4u);
    return P.fast_decode ? rcp_rn(d) : 1.0f / d;
}

constexpr uint8_t kPal[16][3] = {{96, 112, 72},   {72, 72, 78},    {232, 232, 224}, {52, 96, 220},
                                 {140, 184, 232}, {160, 160, 152}, {224, 72, 64},   {168, 144, 120},
                                 {255, 32, 24},   {255, 184, 0},   {32, 224, 96},   {128, 128, 128},
                                 {128, 128, 128}, {128, 128, 128}, {128, 128, 128}, {128, 128, 128}};
// base = palette / 255 as the correctly rounded fp32 quotient, folded at
// compile time (the same bits a run-time IEEE division gives)
struct PalBase {
    float v[16][3];
};
constexpr PalBase make_pal_base()
{
    PalBase b{};
    for (int k = 0; k < 16; ++k)
        for (int c = 0; c < 3; ++c) b.v[k][c] = (float)kPal[k][c] / 255.0f;
    return b;
}
constexpr PalBase kPalBase = make_pal_base();

__device__ __forceinline__ void shade_rgb(const RenderParams& P, uint32_t key, uint32_t* c3)
{
    constexpr float kFace[8] = {1.0f, 0.45f, 1.0f, 0.55f, 0.85f, 0.7f, 0.7f, 1.0f};
    const uint32_t cls = key & 15u, face = (key >> 4) & 7u;
    float f = kFace[face];
    if (face != 0u && (key >> 8) != 0xFFFFFFu) {
        const float z = decode_depth(P, key);
        const float t = fminf(z * P.rfar, 1.0f);
        const float b = 1.0f - 0.6f * t;
        f = f * b;
    }
#pragma unroll
    for (int c = 0; c < 3; ++c) {
        const float val = fminf(kPalBase.v[cls][c] * f, 1.0f);
        c3[c] = (uint32_t)rintf(255.0f * val);
    }
}

// ---------------------------------------------------------------------------
// instance pass (render_instances): which agent's box owns each pixel's
// visible surface, and how many pixels each box covers when drawn alone
// ---------------------------------------------------------------------------


// Draw agent `agent`'s box (world index h) alone with the rules R2-R7 and the
// same arithmetic as the raster: every covered pixel sets its coverage bit,
// and a pixel whose key equals the final key of the view and that no box has
// claimed yet is claimed by this agent, which is written to the instance image.
// The caller draws the boxes in ascending agent order, so each pixel goes to
// the lowest agent whose own frame holds its final key (one triangle of the
// box with that key there is the same as the box's own minimum being it, as
// the final key is the minimum over every triangle).  The claim bits sit in
// the framebuffer's padding columns (words pitch - 4 and pitch - 3 of each row,
// idle once the record ring has drained).  Adds the covered pixels to the
// agent's footprint and the claimed ones to its visible count.  One wave;
// simple lane-per-pixel sweeps with exact int64 edge values.
__device__ void draw_box_instances(const RenderParams& P, Shared& S, const Tile& T, const Cam& cam,
                                   int64_t h, uint32_t agent, int64_t v)
{
    const int lane = lane_id(), wid = threadIdx.x >> 6;
    uint32_t* bits = S.wv[wid].u.bits;
    bits[lane] = 0u;
    bits[lane + 64] = 0u;
    uint32_t nclaim = 0;   // pixels this lane claimed
    __builtin_amdgcn_wave_barrier();
    const bool live = lane < 12;
    float tri[9] = {};
    uint32_t cls = 0;
    int X0 = 0, Y0 = 0, X1 = 0, Y1 = 0, X2 = 0, Y2 = 0, X3 = 0, Y3 = 0;
    int np = 0;
    if (live) {
        load_box(P, h, lane, tri, cls);
        np = setup_triangle(P, S, cam, tri, X0, Y0, X1, Y1, X2, Y2, X3, Y3);
    }
    float pa = 0.0f, pb = 0.0f, pc = 0.0f;
    if (np != 0 && !depth_plane(P, cam, tri, pa, pb, pc)) np = 0;
    const int px0 = 256 * T.x0 + 128, py0 = 256 * T.y0 + 128;
#pragma unroll 1
    for (int f = 0; f < 2; ++f) {
        // fan piece f, oriented, with its edge values at the tile's pixel (0, 0) (R6)
        int ax = X0, ay = Y0, bx = f == 0 ? X1 : X2, by = f == 0 ? Y1 : Y2, cx = f == 0 ? X2 : X3,
            cy = f == 0 ? Y2 : Y3;
        bool valid = f + 2 < np;
        int i0 = 0, i1 = -1, j0 = 0, j1 = -1;
        long long cv[3] = {0, 0, 0};
        int dxs[3] = {0, 0, 0}, dys[3] = {0, 0, 0};
        if (valid) {
            const int minX = min(ax, min(bx, cx)), maxX = max(ax, max(bx, cx));
            const int minY = min(ay, min(by, cy)), maxY = max(ay, max(by, cy));
            i0 = max((minX - 128 + 255) >> 8, T.x0) - T.x0; i1 = min((maxX - 128) >> 8, T.x0 + T.w - 1) - T.x0;
            j0 = max((minY - 128 + 255) >> 8, T.y0) - T.y0; j1 = min((maxY - 128) >> 8, T.y0 + T.h - 1) - T.y0;
            const long long area2 = (long long)(bx - ax) * (long long)(cy - ay) - (long long)(by - ay) * (long long)(cx - ax);
            valid = i0 <= i1 && j0 <= j1 && area2 != 0;
            if (area2 < 0) {
                const int tx = bx, ty = by;
                bx = cx; by = cy; cx = tx; cy = ty;
            }
            const int ex[3] = {bx, cx, ax}, ey[3] = {by, cy, ay};
            const int fx[3] = {cx, ax, bx}, fy[3] = {cy, ay, by};
#pragma unroll
            for (int k = 0; k < 3; ++k) {
                const int dx = fx[k] - ex[k], dy = fy[k] - ey[k];
                const int tl = (dy < 0) || (dy == 0 && dx > 0);
                cv[k] = (long long)dx * (long long)(py0 - ey[k]) - (long long)dy * (long long)(px0 - ex[k]) +
                        (long long)(tl - 1);
                dxs[k] = dx;
                dys[k] = dy;
            }
        }
        uint64_t m = __ballot(valid);
        while (m) {
            const int l = __builtin_ctzll(m);
            m &= m - 1;
            const int ri0 = (int)readlane((uint32_t)i0, l), ri1 = (int)readlane((uint32_t)i1, l);
            const int rj0 = (int)readlane((uint32_t)j0, l), rj1 = (int)readlane((uint32_t)j1, l);
            long long rc[3];
            int rdx[3], rdy[3];
#pragma unroll
            for (int k = 0; k < 3; ++k) {
                const unsigned long long u = (unsigned long long)cv[k];
                rc[k] = (long long)(((unsigned long long)readlane((uint32_t)(u >> 32), l) << 32) |
                                    readlane((uint32_t)u, l));
                rdx[k] = (int)readlane((uint32_t)dxs[k], l);
                rdy[k] = (int)readlane((uint32_t)dys[k], l);
            }
            const float rpa = readlane_f(pa, l), rpb = readlane_f(pb, l), rpc = readlane_f(pc, l);
            const uint32_t rcls = readlane(cls, l);
            const int bw = ri1 - ri0 + 1, n = bw * (rj1 - rj0 + 1);
            for (int s0 = 0; s0 < n; s0 += 64) {
                const int p = s0 + lane;
                if (p < n) {
                    const int jj = p / bw, i = ri0 + (p - jj * bw), j = rj0 + jj;   // tile pixel
                    bool cov = true;
#pragma unroll
                    for (int k = 0; k < 3; ++k)
                        cov = cov && rc[k] - 256ll * rdy[k] * i + 256ll * rdx[k] * j >= 0;
                    const float pxf = ((float)(T.x0 + i) + 0.5f) - P.cx;
                    const float pyf = ((float)(T.y0 + j) + 0.5f) - P.cy;
                    const uint32_t key = pixel_key(P, pxf, pyf, rpa, rpb, rpc, rcls);
                    if (cov && key != 0xFFFFFFFFu) {
                        atomicOr(&bits[2 * j + (i >> 5)], 1u << (i & 31));
                        if (key == S.fb[j * T.pitch + i]) {
                            const uint32_t b = 1u << (i & 31);
                            if (!(atomicOr(&S.fb[j * T.pitch + T.pitch - 4 + (i >> 5)], b) & b)) {
                                ++nclaim;
                                P.out_inst[v * (int64_t)P.W * P.H + (int64_t)(T.y0 + j) * P.W + T.x0 + i] =
                                    (int32_t)agent;
                            }
                        }
                    }
                }
            }
        }
    }
    __builtin_amdgcn_wave_barrier();
    const uint32_t cnt = (uint32_t)(__popc(bits[lane]) + __popc(bits[lane + 64]));
    const uint32_t tot = readlane(wave_incl_sum(cnt), 63);
    const uint32_t vis = readlane(wave_incl_sum(nclaim), 63);
    if (lane == 0 && tot != 0) atomicAdd(&P.out_counts[2 * (v * P.A + agent)], tot);
    if (lane == 0 && vis != 0) atomicAdd(&P.out_counts[2 * (v * P.A + agent) + 1], vis);
    __builtin_amdgcn_wave_barrier();
}

// Edge buffer of the antialiased mode: the nearest partial-coverage fragment of
// each pixel (0xFFFFFFFF none), a global minimum kept in the words of the
// caller's depth image, row pitch W.  The view tile's workgroup fills its words
// before the static pass, takes the fragments with atomic minima, reads them
// back in the colour resolve (loads that bypass the CU's L1) and only then
// writes the depths over them, so the mode needs no LDS beyond the class/depth
// kernel's and draws 64 x 64 tiles.

// Every mode runs four waves per SIMD (the LDS of eight view tiles per CU).
// kMode: 0 class and depth, 1 with instance visibility, 2 with antialiased
// colour, 3 with colour.  kDebug: the work counters and the option to turn
// culling off are read at run time; otherwise the counter pointer is a
// constant null and culling constantly on, so every counting site and the
// unculled paths fold away (and so does the colour code outside modes 2 and 3).
// kShape (the launcher checks every condition): 0 any view; 1 every tile is
// 64x64 (the view's width and height are multiples of 64), with exact
// pixel-centre offsets, 16-byte aligned outputs and depths the fast
// reciprocal decodes, and no traffic lights; 2 as 1, and the view is one
// tile.  The tile's size (and with 2 its origin) is then known at compile
// time, and the paths of other tile shapes, of the IEEE decode and of the
// lights fold away.
template <int kMode, bool kDebug, int kShape = 0>
__global__ __launch_bounds__(kThreads, kWavesPerSimd)
void render_views_kernel(const RenderParams P_)
{
    constexpr bool kInst = kMode == 1, kAA = kMode == 2;
    constexpr bool kTile64 = kShape >= 1;
    constexpr bool kHasLights = !kTile64;
    RenderParams P = P_;
    if constexpr (!kDebug) {
        P.stats = nullptr;
        P.cull = 1;
    }
    if constexpr (kTile64) {
        P.tile_w = 64; P.tile_h = 64;
        P.pix_exact = 1;
        P.vec_out = 1;
        P.fast_decode = 1;
        P.L = 0;
    }
    if constexpr (kShape == 2) {
        P.W = 64; P.H = 64;
        P.tiles_x = 1; P.tiles_y = 1;
        P.div_tiles = Div31{0u, 0u};
    }
    if constexpr (kMode == 0 || kMode == 1) P.out_rgb = nullptr;
    __shared__ Shared S;
    const int tid = threadIdx.x, lane = lane_id(), wid = tid >> 6;
    WaveLds& L = S.wv[wid];
    TSTART(t_kernel);
    // block -> (view, tile) -> (agent g = w * A + a, camera k), in 32 bits
    // (fewer than 2^31 view tiles per launch)
    const uint32_t blk = xcd_remap(blockIdx.x, (uint32_t)P.num_blocks);
    const uint32_t v32 = div31(blk, P.div_tiles);
    const int tile = (int)(blk - v32 * (uint32_t)(P.tiles_x * P.tiles_y));
    const uint32_t g32 = div31(v32, P.div_cams);
    const int k = (int)(v32 - g32 * (uint32_t)P.C);
    const int w = (int)div31(g32, P.div_agents);
    const int a = (int)(g32 - (uint32_t)w * (uint32_t)P.A);
    const int64_t v = (int64_t)v32, g = (int64_t)g32;
    Cam cam;
    {
        const float4 q0 = P.apk[3 * g], q1 = P.apk[3 * g + 1];
        const float c = q1.x, s = q1.y;
        const float mx = P_.mount[k][0], my = P_.mount[k][1], mz = P_.mount[k][2];
        const float cm = P_.mount[k][3], sm = P_.mount[k][4];
        const float t1 = mx * c, t2 = my * s, t3 = mx * s, t4 = my * c;
        const float ox = t1 - t2, oy = t3 + t4;
        cam.x = q0.x + ox;
        cam.y = q0.y + oy;
        cam.z = q0.z + mz;
        const float u1 = c * cm, u2 = s * sm, u3 = s * cm, u4 = c * sm;
        cam.cc = u1 - u2;
        cam.sc = u3 + u4;
    }
    Tile T;
    T.x0 = (tile % P.tiles_x) * P.tile_w;
    T.y0 = (tile / P.tiles_x) * P.tile_h;
    T.w = min(P.tile_w, P.W - T.x0);
    T.h = min(P.tile_h, P.H - T.y0);
    if constexpr (kTile64) {   // the view is a whole number of tiles
        T.w = 64;
        T.h = 64;
    }
    T.pitch = ((T.w + 31) & ~31) + 4;
    // culling reaches the pixel centres of the tile, and with antialiasing the
    // centres within half a pixel more, where a surface's edge fragments land
    constexpr float tpad = kAA ? 1.0f : 0.5f;
    T.kl = ((float)T.x0 - tpad) - P.cx;
    T.kr = ((float)(T.x0 + T.w) + tpad) - P.cx;
    T.kt = P.cy - ((float)T.y0 - tpad);
    T.kb = P.cy - ((float)(T.y0 + T.h) + tpad);
    T.cm = kAA ? 0.50390625f : 0.00390625f;
    const int npx = T.w * T.h;
    static_assert(sizeof(Shared) <= 65536, "LDS");
    const bool cull = P.cull != 0;

    {
        // whole padded rows (the pitch is a multiple of 4)
        const u32x4 clr = {kClearKey, kClearKey, kClearKey, kClearKey};
        const int n4 = T.h * T.pitch;
        for (int p = 4 * tid; p < n4; p += 4 * kThreads) *(u32x4*)&S.fb[p] = clr;
    }
    // per-lane constants of the 8x8 block raster: pixel (lane & 7, lane >> 3)
    const float pxl = (float)(lane & 7) + P.hx, pyl = (float)(lane >> 3) + P.hy;
    const int loff4 = ((lane >> 3) * T.pitch + (lane & 7)) * 4;
    if (P.stats && tid < kNumStats) S.stat[tid] = 0;
    if (tid < 4) S.ctl[tid] = 0;
    // antialiased mode: the edge buffer (in the depth image's words) starts empty
    uint32_t* const ebuf = kAA ? (uint32_t*)P.out_depth + v * (int64_t)P.W * P.H + (int64_t)T.y0 * P.W + T.x0 : nullptr;
    if constexpr (kAA) {
        for (int row = wid; row < T.h; row += kViewWaves)
            if (lane < T.w) ebuf[(int64_t)row * P.W + lane] = 0xFFFFFFFFu;
    }

    // world-space frustum planes of the tile: four side planes through the
    // camera centre, near and far with margins
    WorldPlanes F;
    {
        const float cc = cam.cc, sc = cam.sc;
        F.n[0][0] = P.fx * sc - T.kl * cc; F.n[0][1] = -P.fx * cc - T.kl * sc; F.n[0][2] = 0.0f; F.o[0] = 0.0f;
        F.n[1][0] = T.kr * cc - P.fx * sc; F.n[1][1] = T.kr * sc + P.fx * cc; F.n[1][2] = 0.0f; F.o[1] = 0.0f;
        F.n[2][0] = T.kt * cc; F.n[2][1] = T.kt * sc; F.n[2][2] = -P.fy; F.o[2] = 0.0f;
        F.n[3][0] = -T.kb * cc; F.n[3][1] = -T.kb * sc; F.n[3][2] = P.fy; F.o[3] = 0.0f;
        F.n[4][0] = cc; F.n[4][1] = sc; F.n[4][2] = 0.0f; F.o[4] = P.near_off;
        F.n[5][0] = -cc; F.n[5][1] = -sc; F.n[5][2] = 0.0f; F.o[5] = P.far_off;
    }

    const WorldGrid grid = P.scene.grids[w];
    const float cs = P.scene.cell_size;
    // rectangle of cells covering the tile frustum's xy footprint up to far
    int ix0 = 0, iy0 = 0, ix1 = grid.nx - 1, iy1 = grid.ny - 1;
    if (cull) {
        const float fz = P.far_off;
        const float tl = T.kl * P.rfx, tr = T.kr * P.rfx;
        const float ax_ = cam.cc + tl * cam.sc, ay_ = cam.sc - tl * cam.cc;   // f + tl r
        const float bx_ = cam.cc + tr * cam.sc, by_ = cam.sc - tr * cam.cc;   // f + tr r
        const float p1x = cam.x + fz * ax_, p1y = cam.y + fz * ay_;
        const float p2x = cam.x + fz * bx_, p2y = cam.y + fz * by_;
        const float mg = grid.margin + 1.0f;
        const float xlo = fminf(cam.x, fminf(p1x, p2x)) - mg, xhi = fmaxf(cam.x, fmaxf(p1x, p2x)) + mg;
        const float ylo = fminf(cam.y, fminf(p1y, p2y)) - mg, yhi = fmaxf(cam.y, fmaxf(p1y, p2y)) + mg;
        // (a product by the rounded reciprocal may floor one cell off: the margin cell covers it)
        const float fx0 = floorf((xlo - grid.ox) * P.rcs) - 1.0f, fx1 = floorf((xhi - grid.ox) * P.rcs) + 1.0f;
        const float fy0 = floorf((ylo - grid.oy) * P.rcs) - 1.0f, fy1 = floorf((yhi - grid.oy) * P.rcs) + 1.0f;
        ix0 = (int)fmaxf(fx0, 0.0f); iy0 = (int)fmaxf(fy0, 0.0f);
        ix1 = (int)fminf(fx1, (float)(grid.nx - 1)); iy1 = (int)fminf(fy1, (float)(grid.ny - 1));
    }
    const int rw = ix1 - ix0 + 1, rh = iy1 - iy0 + 1;
    const int nrect = (rw > 0 && rh > 0) ? rw * rh : 0;
    // (approximate: the cell index below corrects a row off by one)
    const float rrw = rw > 0 ? __builtin_amdgcn_rcpf((float)rw) : 0.0f;
    const float hc = 0.5f * cs + grid.margin;   // half extent of a cell rectangle widened by the margin
    const int64_t abase_w = (int64_t)w * P.A;
    const int64_t lbase_w = (int64_t)w * P.L;
    if (tid == 0) { STAT(kStTiles, 1); STAT(kStCellsRect, nrect); }
    // antialiased mode: every wave's fills of the edge buffer have completed
    // (vmcnt 0) before any wave passes the barrier and adds fragments
    if constexpr (kAA) __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    TACC(kCycPrologue, t_kernel);

    // ---- per-wave pipeline: sources -> first pass -> queue -> exact pass ----
    // One loop with one inlined copy of the first and exact passes keeps the
    // whole kernel in the instruction cache.
    enum { kStatic = 0, kBoxes = 1, kLights = 2, kDone = 3 };
    int phase = kStatic;
    // wave w of the view takes the cells (and agents) whose index is w mod
    // kViewWaves; each wave exact-passes its own survivors
    int chunk = 0;                   // next 64-cell chunk of this wave
    int achunk = 0;                  // next 64-agent (then 64-light) chunk of this wave
    uint32_t total = 0, s0 = 0;      // candidate slots of the current chunk, next slot
    uint32_t my_start = 0, my_pre = 0;   // lane i: visible cell i (first triangle, exclusive prefix) or agent i
    int nvis = 0, cfirst = 0;
    int nq = 0;                      // depth of this wave's survivor queue (wave-uniform)
    for (;;) {
        TSTART(t_src);
        // refill: the next chunk of cells (then of agents) with a visible member
        while (phase == kStatic && s0 >= total) {
            if (chunk * 64 * kViewWaves >= nrect) { phase = kBoxes; total = 0; s0 = 0; break; }
            const int r = (chunk * 64 + lane) * kViewWaves + wid;
            ++chunk;
            bool vis = false;
            uint32_t start = 0, cnt = 0;
            if (r < nrect) {
                int iy = (int)(((float)r + 0.5f) * rrw);
                int ix = r - iy * rw;
                if (ix < 0) { --iy; ix += rw; }
                if (ix >= rw) { ++iy; ix -= rw; }
                // an even row width would give each wave whole columns: alternate per row instead
                if ((rw & 1) == 0) ix ^= (iy & 1);
                bool pre = true;
                if (cull) {
                    const float ccx = (grid.ox + ((float)(ix0 + ix) + 0.5f) * cs) - cam.x;
                    const float ccy = (grid.oy + ((float)(iy0 + iy) + 0.5f) * cs) - cam.y;
                    pre = !rect_outside(ccx, ccy, hc, F.n[0][0], F.n[0][1], F.o[0]) &&
                          !rect_outside(ccx, ccy, hc, F.n[1][0], F.n[1][1], F.o[1]) &&
                          !rect_outside(ccx, ccy, hc, F.n[4][0], F.n[4][1], F.o[4]) &&
                          !rect_outside(ccx, ccy, hc, F.n[5][0], F.n[5][1], F.o[5]);
                }
                if (pre) {
                    STAT(kStCellsPre, 1);
                    const int c = grid.cell_base + (iy0 + iy) * grid.nx + (ix0 + ix);
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
            }
            const uint64_t m = __ballot(vis);
            nvis = __popcll(m);
            if (nvis == 0) continue;
            if (vis) {
                const uint32_t slot = mbcnt(m);
                L.u.cells.start[slot] = start;
                L.u.cells.count[slot] = cnt;
                STAT(kStCellsVis, 1);
                STAT(kStCand, cnt);
            }
            __builtin_amdgcn_wave_barrier();
            const uint32_t cn = lane < nvis ? L.u.cells.count[lane] : 0u;
            my_start = lane < nvis ? L.u.cells.start[lane] : 0u;
            my_pre = wave_excl_scan(cn, total);
            s0 = 0;
            cfirst = 0;
            __builtin_amdgcn_wave_barrier();
        }
        while (phase == kBoxes && s0 >= total) {
            if (achunk * 64 * kViewWaves >= P.A) { phase = kLights; achunk = 0; break; }
            const int ai = (achunk * 64 + lane) * kViewWaves + wid;
            ++achunk;
            bool vis = false;
            if (ai < P.A && ai != a) {
                vis = true;
                if (cull) {
                    const int64_t h = abase_w + ai;
                    const float4 r0 = P.apk[3 * h], r1 = P.apk[3 * h + 1];
                    const float R = 0.5f * (r1.z + r1.w) * 1.0009765625f + 0.0009765625f;
                    vis = aabb_visible(P, T, F, cam, r0.x - R, r0.y - R, r0.z, r0.x + R, r0.y + R, r0.z + r0.w);
                }
            }
            const uint64_t m = __ballot(vis);
            nvis = __popcll(m);
            if (nvis == 0) continue;
            if (vis) {
                L.u.agents[mbcnt(m)] = (uint32_t)ai;
                STAT(kStBoxesVis, 1);
                STAT(kStBoxTris, 12);
            }
            __builtin_amdgcn_wave_barrier();
            my_start = lane < nvis ? L.u.agents[lane] : 0u;
            total = 12u * (uint32_t)nvis;
            s0 = 0;
            __builtin_amdgcn_wave_barrier();
        }
        if (!kHasLights && phase == kLights) phase = kDone;
        while (kHasLights && phase == kLights && s0 >= total) {
            // traffic lights whose visibility cone holds the camera (R10)
            if (achunk * 64 * kViewWaves >= P.L) { phase = kDone; break; }
            const int li = (achunk * 64 + lane) * kViewWaves + wid;
            ++achunk;
            bool vis = false;
            if (li < P.L) {
                const int64_t h = lbase_w + li;
                vis = light_visible(P, cam, h);
                if (vis && cull) {
                    // the disk lies within r of its centre; the margin covers the rounding of the rim vertices
                    const float x = P.lx[h], y = P.ly[h], z = P.lz[h];
                    const float R = P.lr[h] * 1.0009765625f + (fabsf(x) + fabsf(y) + fabsf(z)) * 9.5367431640625e-07f
                                    + 0.0009765625f;
                    vis = aabb_visible(P, T, F, cam, x - R, y - R, z - R, x + R, y + R, z + R);
                }
            }
            const uint64_t m = __ballot(vis);
            nvis = __popcll(m);
            if (nvis == 0) continue;
            if (vis) L.u.agents[mbcnt(m)] = (uint32_t)li;
            __builtin_amdgcn_wave_barrier();
            my_start = lane < nvis ? L.u.agents[lane] : 0u;
            total = 12u * (uint32_t)nvis;
            s0 = 0;
            __builtin_amdgcn_wave_barrier();
        }
        TACC(kCycSource, t_src);
        if (phase == kStatic) {
            // first pass over candidate primitives s0 .. s0 + 63 (a pair may queue
            // two entries, so one chunk per step keeps the queue within kQueue:
            // fewer than 64 entries wait before a step, at most 128 join)
            TSTART(t_first);
            const uint32_t slot = s0 + (uint32_t)lane;
            // the cell holding each slot (every visible cell holds a primitive)
            uint32_t bs = 0, bp = 0;
            int c = cfirst;
            for (; c < nvis; ++c) {
                const uint32_t pc = readlane(my_pre, c);
                if (pc >= s0 + 64u) break;
                const uint32_t sc = readlane(my_start, c);
                if (slot >= pc) { bs = sc; bp = pc; }
            }
            // the cell holding slot s0 + 64: the one that ended the loop if it starts there, else the last visited
            cfirst = (c < nvis && readlane(my_pre, c) == s0 + 64u) ? c : max(c - 1, 0);
            const uint32_t e = bs + (slot - bp);
            float v[12] = {};
            uint32_t vcls = 0;
            bool pair = false;
            int r0 = 0, r1 = 0;
            if (slot < total) {
                load_prim(P, e, v, vcls, pair);
                first_pass_prim(P, T, cam, v, pair, cull, r0, r1);
            }
            // the whole pair when both halves pass with every vertex in front of
            // the near plane; otherwise each passing half (or the lone triangle)
            const bool whole = r0 == 1 && r1 == 1;
            const uint32_t k0 = whole ? (uint32_t)kPair : pair ? (uint32_t)kHalf0 : (uint32_t)kTri;
            if (r0 != 0) STAT(kStSurv, 1);
            if (r1 != 0) STAT(kStSurv, 1);
            STAT1(kStChunks, 1);
            nq = queue_push(L, nq, r0 != 0, (e << 2) | k0);
            nq = queue_push(L, nq, r1 != 0 && !whole, (e << 2) | (uint32_t)kHalf1);
            s0 += 64;
            TACC(kCycFirst, t_first);
        } else if (phase != kDone) {
            // first pass over box (or light) slots s0 .. s0 + 63
            TSTART(t_first);
            const uint32_t slot = s0 + (uint32_t)lane;
            float tri[9] = {};
            uint32_t cls = 0;
            // slot = 12 * (visible box or light) + triangle; the multiply-shift divides exactly for slot < 831
            const uint32_t vi = (slot * 43691u) >> 19;
            const uint32_t face = slot - 12u * vi;
            const uint32_t ai = (uint32_t)__shfl((int)my_start, (int)min(vi, 63u));
            const bool boxes = !kHasLights || phase == kBoxes;
            const uint32_t entry = (boxes ? kBoxFlag : kLightFlag) | (ai << 4) | face;
            if (slot < total) {
                if (boxes) load_box(P, abase_w + ai, (int)face, tri, cls);
                else load_light(P, lbase_w + ai, (int)face, tri, cls);
            }
            const bool surv = slot < total && first_pass(P, T, cam, tri, cull);
            if (surv) STAT(kStSurv, 1);
            STAT1(kStChunks, 1);
            nq = queue_push(L, nq, surv, entry);
            s0 += 64;
            TACC(kCycFirst, t_first);
        }
        while (nq >= 64 || (phase == kDone && nq > 0)) {
            // exact pass over the newest 64 survivors (or all that are left)
            const int n = min(nq, 64);
            const bool live = lane < n;
            const uint32_t entry = live ? L.q[nq - n + lane] : 0u;
            nq -= n;
            __builtin_amdgcn_wave_barrier();
            STAT1(kStExact, 1);
            TSTART(t_ex);
            exact_pass<kAA, kHasLights>(P, S, L, T, cam, live, entry, abase_w, lbase_w, pxl, pyl, loff4, ebuf);
            TACC(kCycExact, t_ex);
        }
        if (phase == kDone && nq == 0) break;
    }

    // ---- record ring: this wave produces no more records; rasterize the ring's
    // records, the other wave's too, until both waves are done and it is empty
    {
        static_assert(kViewWaves == 2, "two done flags");
        if (lane == 0) lds_store_release(&S.ctl[kDone0 + wid], 1u);
        const uint32_t cap = (uint32_t)T.h >> 2;
        const bool fast = P.pix_exact && (T.w & 7) == 0 && (T.h & 7) == 0;
        TSTART(t_ring);
        // Every wait below ends: a claimed slot was reserved by a wave that
        // publishes it right after reserving it, and each wave sets its done
        // flag after its last reservation.  The sleep counts are bounded all
        // the same (about a second), so a broken invariant never hangs a wave:
        // it leaves the record undrawn and sets kDevErrRingWait in the
        // context's error word, which pictura_device_errors reports.
        uint32_t naps = 0;
        for (; naps < (1u << 22); ) {
            // the done flags first: once both are set, the reserved count is final
            const bool fin = readfirst(lds_load_acquire(&S.ctl[kDone0])) != 0 &&
                             readfirst(lds_load_acquire(&S.ctl[kDone0 + 1])) != 0;
            const uint32_t t = min(readfirst(lds_load_acquire(&S.ctl[kRecTail])), cap);
            const uint32_t h = readfirst(lds_load_acquire(&S.ctl[kRecHead]));
            if (h < t) {
                uint32_t got = 0;
                if (lane == 0) got = atomicCAS(&S.ctl[kRecHead], h, h + 1u);
                if (readlane(got, 0) != h) continue;
                // slot h is reserved; wait until its producer has published it
                const uint32_t* w3 = &S.fb[(4 * (int)h + 3) * T.pitch + T.pitch - 4];
                while (readfirst(lds_load_acquire(&w3[2])) != kRecReady && ++naps < (1u << 22))
                    __builtin_amdgcn_s_sleep(1);
                if (naps >= (1u << 22)) {
                    // never published (cannot happen): skip it, do not read it, and say so
                    if (lane == 0) atomicOr(P.dev_err, kDevErrRingWait);
                    break;
                }
                const u32x4* g = (const u32x4*)&S.fb[4 * (int)h * T.pitch + T.pitch - 4];
                const int rs = T.pitch >> 2;
                const u32x4 g0 = g[0], g1 = g[rs], g2 = g[2 * rs];
                uint32_t uw[9] = {readfirst(g0.x), readfirst(g0.y), readfirst(g0.z), readfirst(g0.w),
                                  readfirst(g1.x), readfirst(g1.y), readfirst(g1.z), readfirst(g1.w),
                                  readfirst(g2.x)};
                const float rpa = __uint_as_float(readfirst(g2.y)), rpb = __uint_as_float(readfirst(g2.z));
                const float rpc = __uint_as_float(readfirst(g2.w));
                const uint32_t rb = readfirst(w3[0]), rj = readfirst(w3[1]);
                if (fast) raster_blocks<true, true>(P, S, T, uw, rpa, rpb, rpc, rb, rj, pxl, pyl, loff4);
                else raster_blocks<true, false>(P, S, T, uw, rpa, rpb, rpc, rb, rj, pxl, pyl, loff4);
                continue;
            }
            if (fin) break;
            ++naps;
            __builtin_amdgcn_s_sleep(2);
        }
        TACC(kCycRecords, t_ring);
    }
    __syncthreads();

    if constexpr (kInst) {
        // claim bits of the tile's pixels: two padding words per framebuffer row
        for (int r = tid; r < T.h; r += kThreads) {
            S.fb[r * T.pitch + T.pitch - 4] = 0u;
            S.fb[r * T.pitch + T.pitch - 3] = 0u;
        }
        __syncthreads();
        // every non-ego box that can reach the tile, in ascending agent order, by one wave
        if (wid == 0) {
            for (int ac = 0; ac * 64 < P.A; ++ac) {
                const int ai = ac * 64 + lane;
                bool vis = ai < P.A && ai != a;
                if (vis && cull) {
                    const int64_t h = abase_w + ai;
                    const float4 r0 = P.apk[3 * h], r1 = P.apk[3 * h + 1];
                    const float R = 0.5f * (r1.z + r1.w) * 1.0009765625f + 0.0009765625f;
                    vis = aabb_visible(P, T, F, cam, r0.x - R, r0.y - R, r0.z, r0.x + R, r0.y + R, r0.z + r0.w);
                }
                uint64_t m = __ballot(vis);
                while (m) {
                    const int l = __builtin_ctzll(m);
                    m &= m - 1;
                    const uint32_t agent = readlane((uint32_t)ai, l);
                    draw_box_instances(P, S, T, cam, abase_w + agent, agent, v);
                }
            }
        }
        __syncthreads();
        // pixels no box claimed own nothing (a wave per row, a lane per column: tiles are at most 64 wide)
        int32_t* const ibase = P.out_inst + v * (int64_t)P.W * P.H + (int64_t)T.y0 * P.W + T.x0;
        for (int row = wid; row < T.h; row += kViewWaves) {
            const uint32_t cw = S.fb[row * T.pitch + T.pitch - 4 + (lane >> 5)];
            if (lane < T.w && !((cw >> (lane & 31)) & 1u)) ibase[(int64_t)row * P.W + lane] = -1;
        }
    }

    // ---- R8 resolve + coalesced write-out of the tile ----
    TSTART(t_out);
    const int64_t view_px = (int64_t)P.W * P.H;
    uint8_t* ocls = P.out_cls + v * view_px;
    float* odep = P.out_depth + v * view_px;
    auto colour_resolve = [&]() {
        // R13: shaded colour of each pixel, planar [3][H][W] per view.  Off box
        // faces (face bits 0) the colour depends on the class alone: a table of
        // the 16 such colours, computed by shade_rgb itself, in the wave's list
        // area (idle after the static pass)
        uint32_t* const pal0 = S.wv[wid].u.bits;
        if (lane < 16) {
            uint32_t t3[3];
            shade_rgb(P, (uint32_t)lane, t3);
            pal0[lane] = t3[0] | t3[1] << 8 | t3[2] << 16;
        }
        __builtin_amdgcn_wave_barrier();
        // colour of a key, packed r | g << 8 | b << 16
        auto shade = [&](uint32_t key) -> uint32_t {
            if (((key >> 4) & 7u) == 0u) return pal0[key & 15u];
            uint32_t c3[3];
            shade_rgb(P, key, c3);
            return c3[0] | c3[1] << 8 | c3[2] << 16;
        };
        // colour of tile pixel (row, col) with key `key`, packed
        auto pixel = [&](int row, int col, uint32_t key) -> uint32_t {
            uint32_t q = shade(key);
            if constexpr (kAA) {
                // R14: a partial-coverage fragment not behind the centre's surface and
                // of another shading id blends over it
                const uint32_t ko = __hip_atomic_load(&ebuf[(int64_t)row * P.W + col], __ATOMIC_RELAXED,
                                                      __HIP_MEMORY_SCOPE_AGENT);
                if (ko != 0xFFFFFFFFu && (ko >> 16) <= (key >> 16) && ((ko >> 8) & 255u) != (key & 255u)) {
                    const uint32_t o = shade(((ko >> 16) << 16) | ((ko >> 8) & 255u));
                    const uint32_t a8 = 255u - (ko & 255u);
                    uint32_t b = 0;
#pragma unroll
                    for (int c = 0; c < 3; ++c) {
                        const uint32_t oc = (o >> (8 * c)) & 255u, cc = (q >> (8 * c)) & 255u;
                        b |= ((oc * a8 + cc * (255u - a8) + 127u) / 255u) << (8 * c);
                    }
                    q = b;
                }
            }
            return q;
        };
        uint8_t* const rgb = P.out_rgb + v * 3 * view_px;
        if ((reinterpret_cast<uintptr_t>(P.out_rgb) & 3u) == 0 && (P.W % 4) == 0 && (T.w % 4) == 0 && (T.x0 % 4) == 0) {
            // four pixels of a row per thread, one 32-bit store per channel plane
            // (u / u4 = (u * ceil(2^16 / u4)) >> 16 exactly for u * u4 < 2^16: u < 1024, u4 <= 16)
            const int u4 = T.w >> 2, n4 = u4 * T.h;
            const uint32_t r4 = (65535u + (uint32_t)u4) / (uint32_t)u4;
            for (int u = tid; u < n4; u += kThreads) {
                const int row = (int)(((uint32_t)u * r4) >> 16), c4 = u - row * u4;
                const u32x4 kq = *(const u32x4*)&S.fb[row * T.pitch + 4 * c4];
                const uint32_t q0 = pixel(row, 4 * c4, kq.x), q1 = pixel(row, 4 * c4 + 1, kq.y);
                const uint32_t q2 = pixel(row, 4 * c4 + 2, kq.z), q3 = pixel(row, 4 * c4 + 3, kq.w);
                const int64_t o = (int64_t)(T.y0 + row) * P.W + T.x0 + 4 * c4;
#pragma unroll
                for (int c = 0; c < 3; ++c) {
                    const uint32_t sh = 8u * (uint32_t)c;
                    const uint32_t w = ((q0 >> sh) & 255u) | ((q1 >> sh) & 255u) << 8 | ((q2 >> sh) & 255u) << 16 |
                                       ((q3 >> sh) & 255u) << 24;
                    *(uint32_t*)(rgb + c * view_px + o) = w;
                }
            }
        } else {
            for (int p = tid; p < npx; p += kThreads) {
                const int row = p / T.w, col = p % T.w;
                const uint32_t q = pixel(row, col, S.fb[row * T.pitch + col]);
                const int64_t o = (int64_t)(T.y0 + row) * P.W + T.x0 + col;
                rgb[o] = (uint8_t)q;
                rgb[view_px + o] = (uint8_t)(q >> 8);
                rgb[2 * view_px + o] = (uint8_t)(q >> 16);
            }
        }
    };
    if constexpr (kAA) {
        // every wave's fragment minima have completed (vmcnt 0) before any is read,
        // and every one is read before the depths overwrite the edge buffer
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        colour_resolve();
        __syncthreads();
    }
    if (P.vec_out && (P.W % 16) == 0 && (T.w % 16) == 0) {
        // tile origin in the view's images; the offsets below stay 32-bit
        uint8_t* const cbase = ocls + ((int64_t)T.y0 * P.W + T.x0);
        float* const dbase = odep + ((int64_t)T.y0 * P.W + T.x0);
        // u / n = (u * ceil(2^16 / n)) >> 16 exactly for u * n < 2^16 (here u < 1024, n <= 16)
        const int u16 = T.w >> 4, n16 = u16 * T.h;
        const uint32_t r16 = (65535u + (uint32_t)u16) / (uint32_t)u16;
        const uint32_t cm = P.out_rgb ? 15u : 255u;   // class byte (R13: the face bits are not part of the class)
        for (int u = tid; u < n16; u += kThreads) {
            const int row = (int)(((uint32_t)u * r16) >> 16), c16 = u - row * u16;
            const u32x4* src = (const u32x4*)&S.fb[row * T.pitch + 16 * c16];
            uint32_t wd[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const u32x4 kq = src[q];
                wd[q] = (kq.x & cm) | ((kq.y & cm) << 8) | ((kq.z & cm) << 16) | ((kq.w & cm) << 24);
            }
            const u32x4 pk = {wd[0], wd[1], wd[2], wd[3]};
            __builtin_nontemporal_store(pk, (u32x4*)(cbase + (uint32_t)(row * P.W + 16 * c16)));
        }
        const int u4 = T.w >> 2, n4 = u4 * T.h;
        const uint32_t r4 = (65535u + (uint32_t)u4) / (uint32_t)u4;
        const float inf = __uint_as_float(0x7F800000u);
        auto depth_quad = [&](int u, auto decode) {
            const int row = (int)(((uint32_t)u * r4) >> 16), c4 = u - row * u4;
            const u32x4 kq = *(const u32x4*)&S.fb[row * T.pitch + 4 * c4];
            f32x4 d = {inf, inf, inf, inf};
            if ((kq.x & kq.y & kq.z & kq.w) >> 8 != 0xFFFFFFu) {   // not all background
                d.x = (kq.x >> 8) == 0xFFFFFFu ? inf : decode(kq.x);
                d.y = (kq.y >> 8) == 0xFFFFFFu ? inf : decode(kq.y);
                d.z = (kq.z >> 8) == 0xFFFFFFu ? inf : decode(kq.z);
                d.w = (kq.w >> 8) == 0xFFFFFFu ? inf : decode(kq.w);
            }
            __builtin_nontemporal_store(d, (f32x4*)((char*)dbase + (uint32_t)((row * P.W + 4 * c4) * 4)));
        };
        if (P.fast_decode) {
            const auto dec = [&](uint32_t key) { return rcp_rn(__uint_as_float(((P.qbase - (key >> 8)) << 3) | 4u)); };
            for (int u = tid; u < n4; u += kThreads) depth_quad(u, dec);
        } else {
            const auto dec = [&](uint32_t key) { return 1.0f / __uint_as_float(((P.qbase - (key >> 8)) << 3) | 4u); };
            for (int u = tid; u < n4; u += kThreads) depth_quad(u, dec);
        }
    } else {
        for (int p = tid; p < npx; p += kThreads) {
            const int row = p / T.w, col = p % T.w;
            const uint32_t key = S.fb[row * T.pitch + col];
            const int64_t o = (int64_t)(T.y0 + row) * P.W + T.x0 + col;
            ocls[o] = (uint8_t)(key & (P.out_rgb ? 15u : 255u));
            odep[o] = (key >> 8) == 0xFFFFFFu ? __uint_as_float(0x7F800000u) : decode_depth(P, key);
        }
    }
    if constexpr (kMode == 3) colour_resolve();
    if (P.stats) {
        TACC(kCycWriteout, t_out);
        __syncthreads();
        if (tid < kNumStats) atomicAdd(&P.stats[tid], (unsigned long long)S.stat[tid]);
    }
}

// The most specialised kShape whose assumptions the launch meets.
static int shape_of(const RenderParams& p)
{
    if (!(p.tile_w == 64 && p.tile_h == 64 && p.W % 64 == 0 && p.H % 64 == 0 && p.pix_exact && p.vec_out &&
          p.fast_decode && p.L == 0))
        return 0;
    return p.W == 64 && p.H == 64 ? 2 : 1;
}

#if defined(PICTURA_RENDER_PLAIN)
// This object (the source compiled once more, with its own scheduler setting)
// holds only the production class/depth kernels.
hipError_t launch_render_plain(const RenderParams& p, hipStream_t s)
{
    const dim3 grid((unsigned)p.num_blocks), block(kThreads);
    switch (shape_of(p)) {
    case 2: hipLaunchKernelGGL((render_views_kernel<0, false, 2>), grid, block, 0, s, p); break;
    case 1: hipLaunchKernelGGL((render_views_kernel<0, false, 1>), grid, block, 0, s, p); break;
    default: hipLaunchKernelGGL((render_views_kernel<0, false>), grid, block, 0, s, p); break;
    }
    return hipGetLastError();
}
#elif defined(PICTURA_RENDER_SIDE)
// Likewise for the production instance (mode 1) and one-sample colour (mode 3) kernels.
hipError_t launch_render_side(const RenderParams& p, int mode, hipStream_t s)
{
    const dim3 grid((unsigned)p.num_blocks), block(kThreads);
    const int shape = shape_of(p);
    if (mode == 1) {
        if (shape == 2) hipLaunchKernelGGL((render_views_kernel<1, false, 2>), grid, block, 0, s, p);
        else if (shape == 1) hipLaunchKernelGGL((render_views_kernel<1, false, 1>), grid, block, 0, s, p);
        else hipLaunchKernelGGL((render_views_kernel<1, false>), grid, block, 0, s, p);
    } else {
        if (shape == 2) hipLaunchKernelGGL((render_views_kernel<3, false, 2>), grid, block, 0, s, p);
        else if (shape == 1) hipLaunchKernelGGL((render_views_kernel<3, false, 1>), grid, block, 0, s, p);
        else hipLaunchKernelGGL((render_views_kernel<3, false>), grid, block, 0, s, p);
    }
    return hipGetLastError();
}
#else
hipError_t launch_render(const RenderParams& p, hipStream_t s)
{
    if (p.num_blocks <= 0) return hipSuccess;
    const dim3 grid((unsigned)p.num_blocks), block(kThreads);
    const int mode = p.out_inst ? 1 : p.out_rgb ? (p.aa ? 2 : 3) : 0;
    if (p.stats || !p.cull) {
        if (mode == 1) hipLaunchKernelGGL((render_views_kernel<1, true>), grid, block, 0, s, p);
        else if (mode == 2) hipLaunchKernelGGL((render_views_kernel<2, true>), grid, block, 0, s, p);
        else if (mode == 3) hipLaunchKernelGGL((render_views_kernel<3, true>), grid, block, 0, s, p);
        else hipLaunchKernelGGL((render_views_kernel<0, true>), grid, block, 0, s, p);
    } else {
        if (mode == 2) {
            const int shape = shape_of(p);
            if (shape == 2) hipLaunchKernelGGL((render_views_kernel<2, false, 2>), grid, block, 0, s, p);
            else if (shape == 1) hipLaunchKernelGGL((render_views_kernel<2, false, 1>), grid, block, 0, s, p);
            else hipLaunchKernelGGL((render_views_kernel<2, false>), grid, block, 0, s, p);
        } else if (mode != 0) return launch_render_side(p, mode, s);
        else return launch_render_plain(p, s);
    }
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

// ---------------------------------------------------------------------------
// allocation-free self-check: the mismatch counter lives in a file-scope
// device array instead of a per-call allocation
// ---------------------------------------------------------------------------

// Every GPU the library runs on holds its own copy until the process ends.
// Word 0 is the mismatch counter of pictura_selftest_rcp_noalloc; the rest is
// reserved.  Host code never passes `scratch` itself to a kernel (in host code
// the name is a stand-in, not a device address): it uses the address
// hipGetSymbolAddress returned for the device.
static __device__ __align__(256) unsigned long long scratch[kNoAllocScratchWords];

namespace {
std::mutex g_scratch_mu;
void* g_scratch_ptr[kNoAllocMaxDevices] = {};
}  // namespace

hipError_t noalloc_scratch_init(int device)
{
    if (device < 0 || device >= kNoAllocMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[device]) return hipSuccess;
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));   // the current device's copy
    if (e != hipSuccess) return e;
    g_scratch_ptr[device] = p;
    return hipSuccess;
}

void* noalloc_scratch(int device)
{
    if (device < 0 || device >= kNoAllocMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    return g_scratch_ptr[device];
}

__global__ void fill_u32_kernel(uint32_t* p, size_t n, uint32_t value)
{
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = value;
}

hipError_t launch_fill_u32(uint32_t* p, size_t n, uint32_t value, hipStream_t s)
{
    if (n == 0) return hipSuccess;
    const size_t blocks = (n + 255) / 256;
    hipLaunchKernelGGL(fill_u32_kernel, dim3((unsigned)(blocks < 4096 ? blocks : 4096)), dim3(256), 0, s, p, n, value);
    return hipGetLastError();
}

__global__ void clear_words_kernel(unsigned long long* p, int n)
{
    const int i = (int)(blockIdx.x * blockDim.x + threadIdx.x);
    if (i < n) p[i] = 0ull;
}

hipError_t launch_rcp_check_noalloc(uint32_t lo_bits, uint32_t n, unsigned long long* counter, hipStream_t s)
{
    // a fill kernel, not a memset, so the sequence can also be captured in a graph
    hipLaunchKernelGGL(clear_words_kernel, dim3(1), dim3(64), 0, s, counter, 1);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_rcp_check(lo_bits, n, counter, s);
}

#endif  // PICTURA_RENDER_PLAIN, PICTURA_RENDER_SIDE

}  // namespace pictura
