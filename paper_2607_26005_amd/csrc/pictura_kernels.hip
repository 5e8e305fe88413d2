// HIP kernels for gfx950: uniform-grid scene binner, batched class/depth view
// rasterizer, kinematic bicycle step.
//
// The rasterization rules (camera R1, view transform R2, depth plane R3, near
// clip R4, 8-bit subpixel snap R5, top-left fill R6, 24|8-bit visibility key
// R7, resolve R8, boxes R9) are implemented here in fp32 with no contraction
// and correctly rounded division, so each pixel's key is the same as a plain
// brute-force evaluation of the rules over every triangle of the world.
// Binning, culling, compaction and tiling are optimisations: they never drop
// a triangle that could set a pixel's key, and min() is order-independent.
#include "pictura_internal.h"

#pragma clang fp contract(off)

namespace pictura {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr uint32_t kClearKey = (0xFFFFFFu << 8) | 4u;

// ---------------------------------------------------------------------------
// small helpers
// ---------------------------------------------------------------------------

__device__ __forceinline__ uint32_t ord_bits(float f)
{
    uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ float ord_float(uint32_t o)
{
    uint32_t u = (o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o;
    return __uint_as_float(u);
}

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

// Append the calling lanes whose `pred` is set to an LDS list: one ballot, an
// mbcnt prefix inside the wave and a single LDS atomic per wave.  Must be
// reached by every active lane of the wave.  Returns the slot (or ~0u).
__device__ __forceinline__ uint32_t wave_append(bool pred, uint32_t* counter)
{
    const uint64_t m = __ballot(pred);
    if (m == 0) return ~0u;
    const uint32_t rank = __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                    __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
    const int leader = __ffsll((unsigned long long)m) - 1;
    uint32_t base = 0;
    if (lane_id() == leader) base = atomicAdd(counter, (uint32_t)__popcll(m));
    base = __shfl(base, leader);
    return pred ? base + rank : ~0u;
}

// Exclusive scan of one value per thread over the 256-thread block.
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* s_wave, uint32_t& total)
{
    const int lane = lane_id(), wid = threadIdx.x >> 6;
    uint32_t x = v;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
        uint32_t y = __shfl_up(x, o);
        if (lane >= o) x += y;
    }
    if (lane == 63) s_wave[wid] = x;
    __syncthreads();
    uint32_t off = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < kBlock / 64; ++w) {
        uint32_t s = s_wave[w];
        if (w < wid) off += s;
        tot += s;
    }
    __syncthreads();
    total = tot;
    return off + x - v;
}

// ---------------------------------------------------------------------------
// binner
// ---------------------------------------------------------------------------

__global__ void bin_init_kernel(uint32_t* count, uint32_t* aabb_bits, int64_t cells, uint32_t* margin_bits, int nw)
{
    int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (c <= cells) count[c] = 0;
    if (c < cells) {
        uint32_t* a = aabb_bits + 8 * c;
        const uint32_t pinf = 0xFF800000u, ninf = 0x007FFFFFu; // ord(+inf), ord(-inf)
        a[0] = pinf; a[1] = pinf; a[2] = pinf;
        a[3] = ninf; a[4] = ninf; a[5] = ninf;
    }
    if (c < nw) margin_bits[c] = 0;
}

__device__ __forceinline__ int world_of(const int64_t* offs, int nw, int64_t t)
{
    int lo = 0, hi = nw - 1;   // largest w with offs[w] <= t
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if (offs[mid] <= t) lo = mid; else hi = mid - 1;
    }
    return lo;
}

__global__ void bin_count_kernel(BinWork W)
{
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= W.T) return;
    const int w = world_of(W.tri_offsets, W.num_worlds, t);
    const WorldGrid g = W.grids[w];
    const float* v = W.verts + 9 * t;
    float lo[3], hi[3];
#pragma unroll
    for (int d = 0; d < 3; ++d) {
        lo[d] = fminf(fminf(v[d], v[3 + d]), v[6 + d]);
        hi[d] = fmaxf(fmaxf(v[d], v[3 + d]), v[6 + d]);
    }
    const float mx = (lo[0] + hi[0]) * 0.5f, my = (lo[1] + hi[1]) * 0.5f;
    const float fx = floorf((mx - g.ox) / W.cell_size);
    const float fy = floorf((my - g.oy) / W.cell_size);
    const int ix = !(fx >= 0.0f) ? 0 : (fx >= (float)(g.nx - 1) ? g.nx - 1 : (int)fx);
    const int iy = !(fy >= 0.0f) ? 0 : (fy >= (float)(g.ny - 1) ? g.ny - 1 : (int)fy);
    const uint32_t c = (uint32_t)(g.cell_base + iy * g.nx + ix);
    W.home[t] = c;
    W.rank[t] = atomicAdd(&W.count[c], 1u);
    uint32_t* a = W.aabb_bits + 8 * (int64_t)c;
#pragma unroll
    for (int d = 0; d < 3; ++d) {
        atomicMin(&a[d], ord_bits(lo[d]));
        atomicMax(&a[3 + d], ord_bits(hi[d]));
    }
}

// Three-phase exclusive scan over n = cells + 1 counters (in place).
constexpr int kScanItems = 4;
constexpr int kScanTile = kBlock * kScanItems;

int64_t scan_tmp_needed(int64_t n) { return (n + kScanTile - 1) / kScanTile + 1; }

__global__ __launch_bounds__(kBlock) void scan_tiles_kernel(uint32_t* data, int64_t n, uint32_t* tile_sums)
{
    __shared__ uint32_t s_wave[kBlock / 64];
    const int64_t base = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kScanItems;
    uint32_t v[kScanItems], sum = 0;
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
        v[k] = (base + k < n) ? data[base + k] : 0u;
        sum += v[k];
    }
    uint32_t total;
    uint32_t off = block_excl_scan(sum, s_wave, total);
#pragma unroll
    for (int k = 0; k < kScanItems; ++k) {
        if (base + k < n) data[base + k] = off;
        off += v[k];
    }
    if (threadIdx.x == 0) tile_sums[blockIdx.x] = total;
}

__global__ __launch_bounds__(kBlock) void scan_sums_kernel(uint32_t* sums, int64_t n)
{
    __shared__ uint32_t s_wave[kBlock / 64];
    uint32_t carry = 0;
    for (int64_t b = 0; b < n; b += kBlock) {
        const int64_t i = b + threadIdx.x;
        const uint32_t v = i < n ? sums[i] : 0u;
        uint32_t total;
        const uint32_t off = block_excl_scan(v, s_wave, total);
        if (i < n) sums[i] = carry + off;
        carry += total;
    }
}

__global__ void scan_add_kernel(uint32_t* data, int64_t n, const uint32_t* tile_sums)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) data[i] += tile_sums[i / kScanTile];
}

__global__ void bin_scatter_kernel(BinWork W)
{
    const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (t >= W.T) return;
    const uint32_t dst = W.count[W.home[t]] + W.rank[t];   // count[] now holds cell starts
    const float* v = W.verts + 9 * t;
    W.triA[dst] = make_float4(v[0], v[1], v[2], v[3]);
    W.triB[dst] = make_float4(v[4], v[5], v[6], v[7]);
    W.triC[dst] = make_float2(v[8], __uint_as_float((uint32_t)W.cls[t]));
    W.perm[dst] = (uint32_t)t;
}

__device__ __forceinline__ int world_of_cell(const WorldGrid* g, int nw, int64_t c)
{
    int lo = 0, hi = nw - 1;
    while (lo < hi) {
        int mid = (lo + hi + 1) >> 1;
        if ((int64_t)g[mid].cell_base <= c) lo = mid; else hi = mid - 1;
    }
    return lo;
}

__global__ void bin_finalize_kernel(BinWork W)
{
    const int64_t c = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= W.total_cells) return;
    const uint32_t* a = W.aabb_bits + 8 * c;
    const float4 lo = make_float4(ord_float(a[0]), ord_float(a[1]), ord_float(a[2]), 0.0f);
    const float4 hi = make_float4(ord_float(a[3]), ord_float(a[4]), ord_float(a[5]), 0.0f);
    W.cell_lo[c] = lo;
    W.cell_hi[c] = hi;
    if (W.count[c + 1] == W.count[c]) return;   // empty cell
    const int w = world_of_cell(W.grids, W.num_worlds, c);
    const WorldGrid g = W.grids[w];
    const int64_t local = c - g.cell_base;
    const int ix = (int)(local % g.nx), iy = (int)(local / g.nx);
    const float x0 = g.ox + (float)ix * W.cell_size, x1 = g.ox + (float)(ix + 1) * W.cell_size;
    const float y0 = g.oy + (float)iy * W.cell_size, y1 = g.oy + (float)(iy + 1) * W.cell_size;
    float ext = fmaxf(fmaxf(x0 - lo.x, hi.x - x1), fmaxf(y0 - lo.y, hi.y - y1));
    ext = fmaxf(ext, 0.0f);
    atomicMax(&W.margin_bits[w], __float_as_uint(ext));
}

__global__ void bin_margin_kernel(BinWork W)
{
    const int w = blockIdx.x * blockDim.x + threadIdx.x;
    if (w >= W.num_worlds) return;
    const float m = __uint_as_float(W.margin_bits[w]);
    W.grids[w].margin = m * 1.0009765625f + 0.0009765625f;   // (1 + 2^-10) m + 2^-10
}

hipError_t launch_bin(const BinWork& W, hipStream_t s)
{
    const int64_t cells = W.total_cells;
    const int64_t n = cells + 1;
    auto blocks = [](int64_t m) { return (unsigned)((m + kBlock - 1) / kBlock); };
    const int64_t init_n = (n > W.num_worlds ? n : W.num_worlds);
    hipLaunchKernelGGL(bin_init_kernel, dim3(blocks(init_n)), dim3(kBlock), 0, s,
                       W.count, W.aabb_bits, cells, W.margin_bits, W.num_worlds);
    if (W.T > 0)
        hipLaunchKernelGGL(bin_count_kernel, dim3(blocks(W.T)), dim3(kBlock), 0, s, W);
    const int64_t tiles = (n + kScanTile - 1) / kScanTile;
    hipLaunchKernelGGL(scan_tiles_kernel, dim3((unsigned)tiles), dim3(kBlock), 0, s, W.count, n, W.scan_tmp);
    hipLaunchKernelGGL(scan_sums_kernel, dim3(1), dim3(kBlock), 0, s, W.scan_tmp, tiles);
    hipLaunchKernelGGL(scan_add_kernel, dim3(blocks(n)), dim3(kBlock), 0, s, W.count, n, W.scan_tmp);
    if (W.T > 0)
        hipLaunchKernelGGL(bin_scatter_kernel, dim3(blocks(W.T)), dim3(kBlock), 0, s, W);
    if (cells > 0)
        hipLaunchKernelGGL(bin_finalize_kernel, dim3(blocks(cells)), dim3(kBlock), 0, s, W);
    hipLaunchKernelGGL(bin_margin_kernel, dim3(blocks(W.num_worlds)), dim3(kBlock), 0, s, W);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// renderer
// ---------------------------------------------------------------------------

struct Cam {
    float x, y, z;     // camera centre (R1)
    float cc, sc;      // camera heading (R1)
};

// View-space frustum of one tile, with 0.5 px of margin beyond the outermost
// pixel centres: inside iff every value below is >= 0.
//   left  fx*xv - kl*zv     right  kr*zv - fx*xv
//   top   kt*zv - fy*yv     bottom fy*yv - kb*zv
struct Tile {
    int x0, y0, w, h;  // pixel rectangle
    float kl, kr, kt, kb;
};

struct BigTri {
    int X0, Y0, X1, Y1, X2, Y2;
    float pa, pb, pc;
    uint32_t cls;
    int16_t i0, i1, j0, j1;
};

struct Shared {
    uint32_t fb[kTileMaxPx];
    uint32_t cl_start[kCellCap];
    uint32_t cl_cnt[kCellCap];
    uint32_t cl_pre[kCellCap + 1];
    BigTri big[kBigCap];
    uint32_t vis[kAgentBatch];
    uint32_t s_wave[kBlock / 64];
    uint32_t n_cells, n_big, n_vis, pad;
};

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
    const float rz = 1.0f / zv;
    const float qx = xv * rz, qy = yv * rz;
    const float mx = P.fx256 * qx, my = P.fy256 * qy;
    const float sx = P.cx256 + mx, sy = P.cy256 - my;
    const float rx = rintf(sx), ry = rintf(sy);
    if (!(fabsf(rx) <= 536870912.0f) || !(fabsf(ry) <= 536870912.0f)) return false;
    X = (int)rx;
    Y = (int)ry;
    return true;
}

// R7: depth test + key + LDS min for one covered pixel.
__device__ __forceinline__ void write_key(const RenderParams& P, Shared& S, const Tile& T, int i, int j,
                                          float pyf, float pa, float pb, float pc, uint32_t cls)
{
    const float pxf = ((float)i + 0.5f) - P.cx;
    float iz = fmaf(pa, pxf, fmaf(pb, pyf, pc));
    if (!(iz >= P.izfar)) return;
    iz = fminf(iz, P.izcap);
    const uint32_t q = P.qbase - (__float_as_uint(iz) >> 3);
    const uint32_t key = (q << 8) | cls;
    atomicMin(&S.fb[(j - T.y0) * T.w + (i - T.x0)], key);
}

// Edge-function coverage over a rectangle of pixel centres, evaluated
// incrementally.  F = E + topleft - 1, so a pixel is covered iff every F >= 0.
// I is int (exact when the triangle spans < 2^15 subpixels) or long long.
template <typename I>
struct Edges {
    I f0, f1, f2;      // at the current pixel
    I sx0, sx1, sx2;   // step +1 column
    I sy0, sy1, sy2;   // step +1 row
};

template <typename I>
__device__ __forceinline__ I edge_mul(int a, int b)
{
    if constexpr (sizeof(I) == 4) return (I)__mul24(a, b);
    else return (I)a * (I)b;
}

template <typename I>
__device__ __forceinline__ void edges_at(Edges<I>& E, int X0, int Y0, int X1, int Y1, int X2, int Y2, int px, int py)
{
    // edges a->b: (v1, v2), (v2, v0), (v0, v1)
    const int ax[3] = {X1, X2, X0}, ay[3] = {Y1, Y2, Y0};
    const int bx[3] = {X2, X0, X1}, by[3] = {Y2, Y0, Y1};
    I f[3], sx[3], sy[3];
#pragma unroll
    for (int e = 0; e < 3; ++e) {
        const int dx = bx[e] - ax[e], dy = by[e] - ay[e];
        const int tl = (dy < 0) || (dy == 0 && dx > 0);
        f[e] = edge_mul<I>(dx, py - ay[e]) - edge_mul<I>(dy, px - ax[e]) + (I)(tl - 1);
        sx[e] = -(I)dy * (I)256;
        sy[e] = (I)dx * (I)256;
    }
    E.f0 = f[0]; E.f1 = f[1]; E.f2 = f[2];
    E.sx0 = sx[0]; E.sx1 = sx[1]; E.sx2 = sx[2];
    E.sy0 = sy[0]; E.sy1 = sy[1]; E.sy2 = sy[2];
}

template <typename I>
__device__ void raster_rect_lane(const RenderParams& P, Shared& S, const Tile& T,
                                 int X0, int Y0, int X1, int Y1, int X2, int Y2,
                                 int i0, int i1, int j0, int j1, float pa, float pb, float pc, uint32_t cls)
{
    Edges<I> E;
    edges_at<I>(E, X0, Y0, X1, Y1, X2, Y2, 256 * i0 + 128, 256 * j0 + 128);
    for (int j = j0; j <= j1; ++j) {
        I g0 = E.f0, g1 = E.f1, g2 = E.f2;
        const float pyf = ((float)j + 0.5f) - P.cy;
        for (int i = i0; i <= i1; ++i) {
            if ((g0 | g1 | g2) >= 0) write_key(P, S, T, i, j, pyf, pa, pb, pc, cls);
            g0 += E.sx0; g1 += E.sx1; g2 += E.sx2;
        }
        E.f0 += E.sy0; E.f1 += E.sy1; E.f2 += E.sy2;
    }
}

// One wave rasterizes a large triangle: lanes tile the bounding box as
// cw columns x (64 / cw) rows and walk down the rows incrementally.
template <typename I>
__device__ void raster_big_wave(const RenderParams& P, Shared& S, const Tile& T, const BigTri& b)
{
    const int lane = lane_id();
    const int bw = b.i1 - b.i0 + 1, bh = b.j1 - b.j0 + 1;
    int cw = 1;
    while (cw < bw && cw < 64) cw <<= 1;
    const int rows = 64 / cw;
    const int lx = lane % cw, ly = lane / cw;
    for (int cb = 0; cb < bw; cb += cw) {
        const int i = b.i0 + cb + lx;
        if (i > b.i1) continue;
        Edges<I> E;
        edges_at<I>(E, b.X0, b.Y0, b.X1, b.Y1, b.X2, b.Y2, 256 * i + 128, 256 * (b.j0 + ly) + 128);
        const I st0 = E.sy0 * (I)rows, st1 = E.sy1 * (I)rows, st2 = E.sy2 * (I)rows;
        for (int jr = ly; jr < bh; jr += rows) {
            const int j = b.j0 + jr;
            if ((E.f0 | E.f1 | E.f2) >= 0) {
                const float pyf = ((float)j + 0.5f) - P.cy;
                write_key(P, S, T, i, j, pyf, b.pa, b.pb, b.pc, b.cls);
            }
            E.f0 += st0; E.f1 += st1; E.f2 += st2;
        }
    }
}

__device__ __forceinline__ int floor_div256(int a) { return a >> 8; }   // arithmetic shift

// R6 setup of one snapped triangle, then rasterize it in this lane when its
// clipped bounding box is small, else queue it for a whole wave.
__device__ void setup_and_raster(const RenderParams& P, Shared& S, const Tile& T,
                                 int X0, int Y0, int X1, int Y1, int X2, int Y2,
                                 const float* tri, const Cam& cam, bool& have_plane,
                                 float& pa, float& pb, float& pc, uint32_t cls)
{
    const int minX = min(X0, min(X1, X2)), maxX = max(X0, max(X1, X2));
    const int minY = min(Y0, min(Y1, Y2)), maxY = max(Y0, max(Y1, Y2));
    int i0 = floor_div256(minX - 128 + 255), i1 = floor_div256(maxX - 128);
    int j0 = floor_div256(minY - 128 + 255), j1 = floor_div256(maxY - 128);
    i0 = max(i0, T.x0); j0 = max(j0, T.y0);
    i1 = min(i1, T.x0 + T.w - 1); j1 = min(j1, T.y0 + T.h - 1);
    if (i0 > i1 || j0 > j1) return;
    const bool small_span = (maxX - minX) < 32768 && (maxY - minY) < 32768;
    long long area2;
    if (small_span) area2 = (long long)(__mul24(X1 - X0, Y2 - Y0) - __mul24(Y1 - Y0, X2 - X0));
    else area2 = (long long)(X1 - X0) * (long long)(Y2 - Y0) - (long long)(Y1 - Y0) * (long long)(X2 - X0);
    if (area2 == 0) return;
    if (area2 < 0) {
        int tx = X1, ty = Y1;
        X1 = X2; Y1 = Y2; X2 = tx; Y2 = ty;
    }
    if (!have_plane) {
        if (!depth_plane(P, cam, tri, pa, pb, pc)) return;   // delta == 0: dropped
        have_plane = true;
    }
    const int npx = (i1 - i0 + 1) * (j1 - j0 + 1);
    if (npx > kSmallPx) {
        const uint32_t slot = atomicAdd(&S.n_big, 1u);
        if (slot < (uint32_t)kBigCap) {
            BigTri& b = S.big[slot];
            b.X0 = X0; b.Y0 = Y0; b.X1 = X1; b.Y1 = Y1; b.X2 = X2; b.Y2 = Y2;
            b.pa = pa; b.pb = pb; b.pc = pc; b.cls = cls;
            b.i0 = (int16_t)i0; b.i1 = (int16_t)i1; b.j0 = (int16_t)j0; b.j1 = (int16_t)j1;
            return;
        }
    }
    if (small_span) raster_rect_lane<int>(P, S, T, X0, Y0, X1, Y1, X2, Y2, i0, i1, j0, j1, pa, pb, pc, cls);
    else raster_rect_lane<long long>(P, S, T, X0, Y0, X1, Y1, X2, Y2, i0, i1, j0, j1, pa, pb, pc, cls);
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

// R2..R7 for one world-space triangle.
__device__ void draw_triangle(const RenderParams& P, Shared& S, const Tile& T, const Cam& cam,
                              const float* tri, uint32_t cls, bool cull)
{
    float xv[3], yv[3], zv[3];
#pragma unroll
    for (int k = 0; k < 3; ++k) view_xform(cam, tri[3 * k], tri[3 * k + 1], tri[3 * k + 2], xv[k], yv[k], zv[k]);
    const bool in0 = zv[0] >= P.nearp, in1 = zv[1] >= P.nearp, in2 = zv[2] >= P.nearp;
    if (!(in0 || in1 || in2)) return;
    if (zv[0] > P.farp && zv[1] > P.farp && zv[2] > P.farp) return;
    if (cull && outside_tile(P, T, xv, yv, zv)) return;
    bool have_plane = false;
    float pa = 0.0f, pb = 0.0f, pc = 0.0f;
    if (in0 && in1 && in2) {
        int X0, Y0, X1, Y1, X2, Y2;
        if (!snap_vertex(P, xv[0], yv[0], zv[0], X0, Y0)) return;
        if (!snap_vertex(P, xv[1], yv[1], zv[1], X1, Y1)) return;
        if (!snap_vertex(P, xv[2], yv[2], zv[2], X2, Y2)) return;
        setup_and_raster(P, S, T, X0, Y0, X1, Y1, X2, Y2, tri, cam, have_plane, pa, pb, pc, cls);
        return;
    }
    // R4: Sutherland-Hodgman against zv >= near, crossing points computed
    // from the inside vertex towards the outside one.
    const bool in[3] = {in0, in1, in2};
    float px[4], py[4], pz[4];
    int np = 0;
#pragma unroll
    for (int k = 0; k < 3; ++k) {
        const int k1 = (k + 1) % 3;
        if (in[k]) { px[np] = xv[k]; py[np] = yv[k]; pz[np] = zv[k]; ++np; }
        if (in[k] != in[k1]) {
            const int ii = in[k] ? k : k1, oo = in[k] ? k1 : k;
            const float t = (P.nearp - zv[ii]) / (zv[oo] - zv[ii]);
            px[np] = fmaf(t, xv[oo] - xv[ii], xv[ii]);
            py[np] = fmaf(t, yv[oo] - yv[ii], yv[ii]);
            pz[np] = P.nearp;
            ++np;
        }
    }
    int SX[4], SY[4];
    for (int k = 0; k < np; ++k)
        if (!snap_vertex(P, px[k], py[k], pz[k], SX[k], SY[k])) return;
    for (int f = 1; f + 1 < np; ++f)
        setup_and_raster(P, S, T, SX[0], SY[0], SX[f], SY[f], SX[f + 1], SY[f + 1], tri, cam, have_plane,
                         pa, pb, pc, cls);
}

// Rasterize the queued large triangles (one wave per triangle) and empty
// the queue.  Called by the whole block.
__device__ void flush_big(const RenderParams& P, Shared& S, const Tile& T)
{
    __syncthreads();
    const uint32_t n = min(S.n_big, (uint32_t)kBigCap);
    if (n > 0) {
        for (uint32_t e = threadIdx.x >> 6; e < n; e += kBlock / 64) {
            const BigTri b = S.big[e];
            const int minX = min(b.X0, min(b.X1, b.X2)), maxX = max(b.X0, max(b.X1, b.X2));
            const int minY = min(b.Y0, min(b.Y1, b.Y2)), maxY = max(b.Y0, max(b.Y1, b.Y2));
            if ((maxX - minX) < 32768 && (maxY - minY) < 32768) raster_big_wave<int>(P, S, T, b);
            else raster_big_wave<long long>(P, S, T, b);
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) S.n_big = 0;
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

__device__ __forceinline__ bool aabb_culled(const WorldPlanes& F, const Cam& cam,
                                            float lox, float loy, float loz, float hix, float hiy, float hiz)
{
    const float cx = (lox + hix) * 0.5f - cam.x, cy = (loy + hiy) * 0.5f - cam.y, cz = (loz + hiz) * 0.5f - cam.z;
    const float hx = (hix - lox) * 0.5f, hy = (hiy - loy) * 0.5f, hz = (hiz - loz) * 0.5f;
#pragma unroll
    for (int p = 0; p < 6; ++p)
        if (box_outside(cx, cy, cz, hx, hy, hz, F.n[p][0], F.n[p][1], F.n[p][2], F.o[p])) return true;
    return false;
}

__device__ __forceinline__ int64_t xcd_remap(int64_t b, int64_t nb)
{
    // Blocks are dispatched round-robin over the 8 XCDs; give each XCD a
    // contiguous range of views so that one world's views share an L2.
    const int64_t q = nb >> 3, r = nb & 7, x = b & 7, k = b >> 3;
    return x * q + (x < r ? x : r) + k;
}

__global__ __launch_bounds__(kBlock) void render_views_kernel(const RenderParams P)
{
    __shared__ Shared S;
    const int tid = threadIdx.x;
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

    for (int p = tid; p < npx; p += kBlock) S.fb[p] = kClearKey;
    if (tid == 0) { S.n_cells = 0; S.n_big = 0; S.n_vis = 0; }

    // world-space frustum planes of the tile (side planes through the camera,
    // near and far with margins)
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
    // cell rectangle covering the tile frustum's xy footprint up to far
    int ix0 = 0, iy0 = 0, ix1 = grid.nx - 1, iy1 = grid.ny - 1;
    if (cull) {
        const float fz = P.farp * 1.015625f;
        const float tl = T.kl / P.fx, tr = T.kr / P.fx;
        const float ax_ = cam.cc + tl * cam.sc, ay_ = cam.sc - tl * cam.cc;   // f + tl*r
        const float bx_ = cam.cc + tr * cam.sc, by_ = cam.sc - tr * cam.cc;   // f + tr*r
        const float p1x = cam.x + fz * ax_, p1y = cam.y + fz * ay_;
        const float p2x = cam.x + fz * bx_, p2y = cam.y + fz * by_;
        const float m = grid.margin + 1.0f;
        const float xlo = fminf(cam.x, fminf(p1x, p2x)) - m, xhi = fmaxf(cam.x, fmaxf(p1x, p2x)) + m;
        const float ylo = fminf(cam.y, fminf(p1y, p2y)) - m, yhi = fmaxf(cam.y, fmaxf(p1y, p2y)) + m;
        const float fx0 = floorf((xlo - grid.ox) / cs) - 1.0f, fx1 = floorf((xhi - grid.ox) / cs) + 1.0f;
        const float fy0 = floorf((ylo - grid.oy) / cs) - 1.0f, fy1 = floorf((yhi - grid.oy) / cs) + 1.0f;
        ix0 = (int)fmaxf(fx0, 0.0f); iy0 = (int)fmaxf(fy0, 0.0f);
        ix1 = (int)fminf(fx1, (float)(grid.nx - 1)); iy1 = (int)fminf(fy1, (float)(grid.ny - 1));
    }
    const int rw = ix1 - ix0 + 1, rh = iy1 - iy0 + 1;
    const int nrect = (rw > 0 && rh > 0) ? rw * rh : 0;
    __syncthreads();

    // ---- static triangles: cell gather, cull, ballot compaction, raster ----
    for (int rbase = 0; rbase < nrect; rbase += kCellCap) {
#pragma unroll
        for (int q = 0; q < kCellCap / kBlock; ++q) {
            const int r = rbase + q * kBlock + tid;
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
                        vis = !aabb_culled(F, cam, lo.x, lo.y, lo.z, hi.x, hi.y, hi.z);
                    }
                }
            }
            const uint32_t slot = wave_append(vis, &S.n_cells);
            if (vis) { S.cl_start[slot] = start; S.cl_cnt[slot] = cnt; }
        }
        __syncthreads();
        const uint32_t nc = S.n_cells;
        // prefix of the gathered cells' triangle counts (two entries per thread)
        {
            const uint32_t e0 = 2 * tid, e1 = 2 * tid + 1;
            const uint32_t c0 = e0 < nc ? S.cl_cnt[e0] : 0u, c1 = e1 < nc ? S.cl_cnt[e1] : 0u;
            uint32_t total;
            const uint32_t off = block_excl_scan(c0 + c1, S.s_wave, total);
            if (e0 < nc) S.cl_pre[e0] = off;
            if (e1 < nc) S.cl_pre[e1] = off + c0;
            if (tid == 0) { S.cl_pre[nc] = total; S.n_cells = 0; }
        }
        __syncthreads();
        const uint32_t total = S.cl_pre[nc];
        for (uint32_t kb = 0; kb < total; kb += kBlock) {
            const uint32_t kk = kb + tid;
            if (kk < total) {
                uint32_t lo = 0, hi = nc - 1;   // last cell with pre <= kk
                while (lo < hi) {
                    const uint32_t mid = (lo + hi + 1) >> 1;
                    if (S.cl_pre[mid] <= kk) lo = mid; else hi = mid - 1;
                }
                const uint32_t t = S.cl_start[lo] + (kk - S.cl_pre[lo]);
                const float4 A4 = P.scene.triA[t];
                const float4 B4 = P.scene.triB[t];
                const float2 C2 = P.scene.triC[t];
                const float tri[9] = {A4.x, A4.y, A4.z, A4.w, B4.x, B4.y, B4.z, B4.w, C2.x};
                draw_triangle(P, S, T, cam, tri, __float_as_uint(C2.y), cull);
            }
            flush_big(P, S, T);
        }
    }

    // ---- agent boxes: box cull, ballot compaction, 12 triangles each ----
    const int64_t abase_w = (int64_t)w * P.A;
    for (int ab = 0; ab < P.A; ab += kAgentBatch) {
        const int ai = ab + tid;
        bool vis = false;
        if (ai < P.A && ai != a) {
            vis = true;
            if (cull) {
                const int64_t h = abase_w + ai;
                const float x = P.ax[h], y = P.ay[h], z0 = P.az0[h];
                const float R = 0.5f * (P.al[h] + P.aw[h]) * 1.0009765625f + 0.0009765625f;
                const float H = P.ah[h];
                vis = !aabb_culled(F, cam, x - R, y - R, z0, x + R, y + R, z0 + H);
            }
        }
        const uint32_t slot = wave_append(vis, &S.n_vis);
        if (vis) S.vis[slot] = (uint32_t)ai;
        __syncthreads();
        const uint32_t ntri = S.n_vis * 12u;
        for (uint32_t kb = 0; kb < ntri; kb += kBlock) {
            const uint32_t kk = kb + tid;
            if (kk < ntri) {
                const int64_t h = abase_w + S.vis[kk / 12u];
                const int face = (int)(kk % 12u);
                // R9: the three corners of this face triangle
                const float x = P.ax[h], y = P.ay[h], z0 = P.az0[h], c = P.ac[h], s = P.as[h];
                const float hl = 0.5f * P.al[h], hw = 0.5f * P.aw[h], ztop = z0 + P.ah[h];
                // corner indices of the 12 triangles, packed 4 bits per corner
                const uint32_t kBoxTris[12] = {0x310, 0x230, 0x754, 0x674, 0x620, 0x460,
                                               0x731, 0x571, 0x510, 0x450, 0x732, 0x672};
                const uint32_t code = kBoxTris[face];
                float tri[9];
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
                draw_triangle(P, S, T, cam, tri, (uint32_t)P.acls[h], cull);
            }
            flush_big(P, S, T);
        }
        if (tid == 0) S.n_vis = 0;
        __syncthreads();
    }

    // ---- R8 resolve + coalesced write-out of the tile ----
    __syncthreads();
    const int64_t view_px = (int64_t)P.W * P.H;
    uint8_t* ocls = P.out_cls + v * view_px;
    float* odep = P.out_depth + v * view_px;
    const uint32_t qbase = P.qbase;
    auto decode = [qbase](uint32_t key) -> float {
        const uint32_t q = key >> 8;
        if (q == 0xFFFFFFu) return __uint_as_float(0x7F800000u);
        return 1.0f / __uint_as_float(((qbase - q) << 3) | 4u);
    };
    if (P.vec_out && (P.W % 16) == 0 && (T.w % 16) == 0) {
        const int u16 = T.w / 16, n16 = u16 * T.h;
        for (int u = tid; u < n16; u += kBlock) {
            const int row = u / u16, c16 = u % u16;
            const uint32_t* src = &S.fb[row * T.w + 16 * c16];
            uint32_t wd[4];
#pragma unroll
            for (int q = 0; q < 4; ++q)
                wd[q] = (src[4 * q] & 255u) | ((src[4 * q + 1] & 255u) << 8) | ((src[4 * q + 2] & 255u) << 16) |
                        ((src[4 * q + 3] & 255u) << 24);
            u32x4 pk = {wd[0], wd[1], wd[2], wd[3]};
            __builtin_nontemporal_store(pk, (u32x4*)(ocls + (int64_t)(T.y0 + row) * P.W + T.x0 + 16 * c16));
        }
        const int u4 = T.w / 4, n4 = u4 * T.h;
        for (int u = tid; u < n4; u += kBlock) {
            const int row = u / u4, c4 = u % u4;
            const uint32_t* src = &S.fb[row * T.w + 4 * c4];
            f32x4 d = {decode(src[0]), decode(src[1]), decode(src[2]), decode(src[3])};
            __builtin_nontemporal_store(d, (f32x4*)(odep + (int64_t)(T.y0 + row) * P.W + T.x0 + 4 * c4));
        }
    } else {
        for (int p = tid; p < npx; p += kBlock) {
            const int row = p / T.w, col = p % T.w;
            const uint32_t key = S.fb[p];
            const int64_t o = (int64_t)(T.y0 + row) * P.W + T.x0 + col;
            ocls[o] = (uint8_t)(key & 255u);
            odep[o] = decode(key);
        }
    }
}

hipError_t launch_render(const RenderParams& p, hipStream_t s)
{
    if (p.num_blocks <= 0) return hipSuccess;
    hipLaunchKernelGGL(render_views_kernel, dim3((unsigned)p.num_blocks), dim3(kBlock), 0, s, p);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// kinematic bicycle step
// ---------------------------------------------------------------------------

__global__ void agents_step_kernel(const AgentStepParams p)
{
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= p.count) return;
    const float kPi = 3.14159265358979323846f;
    float v = p.speed[i] + p.accel[i] * p.dt;
    v = fminf(fmaxf(v, 0.0f), p.vmax);
    float psi = p.psi[i] + v / (0.6f * p.length[i]) * tanf(p.steer[i]) * p.dt;
    if (psi > kPi) psi -= 2.0f * kPi;
    if (psi <= -kPi) psi += 2.0f * kPi;
    float sn, cs;
    sincosf(psi, &sn, &cs);
    p.x[i] += v * cs * p.dt;
    p.y[i] += v * sn * p.dt;
    p.psi[i] = psi;
    p.speed[i] = v;
    p.cos_h[i] = cs;
    p.sin_h[i] = sn;
}

hipError_t launch_agents_step(const AgentStepParams& p, hipStream_t s)
{
    if (p.count <= 0) return hipSuccess;
    hipLaunchKernelGGL(agents_step_kernel, dim3((unsigned)((p.count + 255) / 256)), dim3(256), 0, s, p);
    return hipGetLastError();
}

}  // namespace pictura
