// HIP kernels for gfx950: uniform-grid scene binner over primitives
// (triangles and triangle pairs: count, exclusive scan, scatter into cell
// order, per-cell bounding boxes) and the kinematic bicycle step of the
// agents.
#include "pictura_device.h"

#pragma clang fp contract(off)

namespace pictura {

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

// The vertices of primitive p: a, b, c of its first triangle and, for a pair,
// d (the third vertex of the second triangle (a, c, d)).  Returns 3 or 4.
__device__ __forceinline__ int prim_verts(const BinWork& W, int64_t p, float* v)
{
    const uint32_t e = W.prims[p];
    const float* a = W.verts + 9 * (int64_t)(e & ~kPrimFlagPair);
#pragma unroll
    for (int k = 0; k < 9; ++k) v[k] = a[k];
    v[9] = v[10] = v[11] = 0.0f;
    if (!(e & kPrimFlagPair)) return 3;
    v[9] = a[15]; v[10] = a[16]; v[11] = a[17];
    return 4;
}

__global__ void bin_count_kernel(BinWork W)
{
    const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (p >= W.P) return;
    const int w = world_of(W.prim_offsets, W.num_worlds, p);
    const WorldGrid g = W.grids[w];
    float v[12];
    const int nv = prim_verts(W, p, v);
    float lo[3], hi[3];
#pragma unroll
    for (int d = 0; d < 3; ++d) {
        lo[d] = fminf(fminf(v[d], v[3 + d]), v[6 + d]);
        hi[d] = fmaxf(fmaxf(v[d], v[3 + d]), v[6 + d]);
        if (nv == 4) { lo[d] = fminf(lo[d], v[9 + d]); hi[d] = fmaxf(hi[d], v[9 + d]); }
    }
    const float mx = (lo[0] + hi[0]) * 0.5f, my = (lo[1] + hi[1]) * 0.5f;
    const float fx = floorf((mx - g.ox) / W.cell_size);
    const float fy = floorf((my - g.oy) / W.cell_size);
    const int ix = !(fx >= 0.0f) ? 0 : (fx >= (float)(g.nx - 1) ? g.nx - 1 : (int)fx);
    const int iy = !(fy >= 0.0f) ? 0 : (fy >= (float)(g.ny - 1) ? g.ny - 1 : (int)fy);
    const uint32_t c = (uint32_t)(g.cell_base + iy * g.nx + ix);
    W.home[p] = c;
    W.rank[p] = atomicAdd(&W.count[c], 1u);
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
    const int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (p >= W.P) return;
    const uint32_t dst = W.count[W.home[p]] + W.rank[p];   // count[] now holds cell starts
    float v[12];
    const int nv = prim_verts(W, p, v);
    const uint32_t e = W.prims[p];
    const uint32_t cw = (uint32_t)W.cls[e & ~kPrimFlagPair] | (nv == 4 ? kPrimPair : 0u);
    W.primA[dst] = make_float4(v[0], v[1], v[2], v[3]);
    W.primB[dst] = make_float4(v[4], v[5], v[6], v[7]);
    W.primC[dst] = make_float4(v[8], __uint_as_float(cw), v[9], v[10]);
    W.primD[dst] = v[11];
    W.perm[dst] = e;
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
    if (W.P > 0)
        hipLaunchKernelGGL(bin_count_kernel, dim3(blocks(W.P)), dim3(kBlock), 0, s, W);
    const int64_t tiles = (n + kScanTile - 1) / kScanTile;
    hipLaunchKernelGGL(scan_tiles_kernel, dim3((unsigned)tiles), dim3(kBlock), 0, s, W.count, n, W.scan_tmp);
    hipLaunchKernelGGL(scan_sums_kernel, dim3(1), dim3(kBlock), 0, s, W.scan_tmp, tiles);
    hipLaunchKernelGGL(scan_add_kernel, dim3(blocks(n)), dim3(kBlock), 0, s, W.count, n, W.scan_tmp);
    if (W.P > 0)
        hipLaunchKernelGGL(bin_scatter_kernel, dim3(blocks(W.P)), dim3(kBlock), 0, s, W);
    if (cells > 0)
        hipLaunchKernelGGL(bin_finalize_kernel, dim3(blocks(cells)), dim3(kBlock), 0, s, W);
    hipLaunchKernelGGL(bin_margin_kernel, dim3(blocks(W.num_worlds)), dim3(kBlock), 0, s, W);
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

// The agents of a render call in the render kernels' layout (RenderParams::apk).
__global__ void pack_agents_kernel(const RenderParams p, int64_t count)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= count) return;
    p.apk[3 * i] = make_float4(p.ax[i], p.ay[i], p.az0[i], p.ah[i]);
    p.apk[3 * i + 1] = make_float4(p.ac[i], p.as[i], p.al[i], p.aw[i]);
    p.apk[3 * i + 2] = make_float4(__uint_as_float((uint32_t)p.acls[i]), 0.0f, 0.0f, 0.0f);
}

hipError_t launch_pack_agents(const RenderParams& p, int64_t count, hipStream_t s)
{
    if (count <= 0) return hipSuccess;
    hipLaunchKernelGGL(pack_agents_kernel, dim3((unsigned)((count + 255) / 256)), dim3(256), 0, s, p, count);
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// streaming-store reference: zeros written with 16-byte non-temporal stores,
// the store pattern of the render's write-out, at whatever rate HBM accepts
// ---------------------------------------------------------------------------

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

__global__ void store_probe_kernel(u32x4_t* dst, uint64_t n16)
{
    const u32x4_t z = {0u, 0u, 0u, 0u};
    const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
    for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride)
        __builtin_nontemporal_store(z, dst + i);
}

hipError_t launch_store_probe(void* dst, uint64_t bytes, hipStream_t s)
{
    const uint64_t n16 = bytes / 16u;
    if (n16 == 0) return hipSuccess;
    // 8 workgroups of 256 threads per CU slot pair, each thread a strided run of 16-byte stores
    const uint64_t want = (n16 + 255u) / 256u;
    const unsigned blocks = (unsigned)(want < 16384u ? want : 16384u);
    hipLaunchKernelGGL(store_probe_kernel, dim3(blocks), dim3(256), 0, s, (u32x4_t*)dst, n16);
    return hipGetLastError();
}

}  // namespace pictura
