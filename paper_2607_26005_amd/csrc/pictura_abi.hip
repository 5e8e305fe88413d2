// C ABI of the batched class/depth view rasterizer: context, argument
// validation, device memory of the scene and its bins, kernel launches.
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "pictura.h"
#include "pictura_internal.h"

using namespace pictura;

struct pictura_ctx_s {
    int device = 0;
    std::string err;
    // scene (original order)
    int32_t num_worlds = 0;
    int64_t T = 0;
    std::vector<int64_t> offsets_h;
    std::vector<float> bounds_h;
    float* verts = nullptr;
    uint8_t* cls = nullptr;
    int64_t* offsets_d = nullptr;
    // primitives: triangles and triangle pairs (see SceneDev)
    int64_t P = 0;
    uint32_t* prims = nullptr;        // [P] first triangle | kPrimFlagPair
    int64_t* prim_offsets_d = nullptr;   // [nw + 1]
    bool have_scene = false;
    uint8_t max_cls = 0;   // largest class ID of the static triangles
    // bins
    bool binned = false;
    float cell_size = 0.0f;
    int64_t total_cells = 0;
    std::vector<WorldGrid> grids_h;
    WorldGrid* grids = nullptr;
    uint32_t* home = nullptr;
    uint32_t* rank = nullptr;
    uint32_t* cell_start = nullptr;
    uint32_t* aabb_bits = nullptr;
    uint32_t* margin_bits = nullptr;
    uint32_t* scan_tmp = nullptr;
    float4* primA = nullptr;
    float4* primB = nullptr;
    float4* primC = nullptr;
    float* primD = nullptr;
    uint32_t* perm = nullptr;
    float4* cell_lo = nullptr;
    float4* cell_hi = nullptr;
    // options
    int cull = 1;
    int tile = 0;
    int stats_on = 0;
    unsigned long long* stats = nullptr;   // [kNumStats] device counters
    // traffic lights (caller-owned device arrays; lights.lights_per_world == 0: none)
    pictura_lights lights{};
    uint32_t* dev_err = nullptr;   // device error word (pictura_device_errors), allocated by pictura_create
    // the agents of the latest render call, packed for the kernels (RenderParams::apk), grown on demand
    float4* apk = nullptr;
    size_t apk_cap = 0;   // bytes
    // render calls share apk: each records apk_event after its kernels, and one
    // on another stream than the last waits for that event first
    hipEvent_t apk_event = nullptr;
    hipStream_t apk_stream = nullptr;
    bool apk_used = false;
};

namespace {

pictura_status fail(pictura_ctx c, pictura_status st, const char* fmt, ...)
{
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    if (c) c->err = buf;
    return st;
}

Div31 make_div31(uint32_t d)
{
    if (d <= 1) return Div31{0u, 0u};
    uint32_t l = 0;
    while ((1ull << l) < d) ++l;
    const uint64_t m = ((1ull << (31 + l)) / d) + 1ull;   // < 2^32 for d >= 2
    return Div31{(uint32_t)m, l - 1};
}

pictura_status hip_fail(pictura_ctx c, hipError_t e, const char* what)
{
    if (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation)
        return fail(c, PICTURA_ENOMEM, "%s: %s", what, hipGetErrorString(e));
    return fail(c, PICTURA_EDEVICE, "%s: %s", what, hipGetErrorString(e));
}

template <typename T>
void dfree(T*& p)
{
    if (p) (void)hipFree((void*)p);
    p = nullptr;
}

template <typename T>
hipError_t dalloc(T*& p, size_t count)
{
    dfree(p);
    if (count == 0) count = 1;
    return hipMalloc((void**)&p, count * sizeof(T));
}

void free_bins(pictura_ctx c)
{
    dfree(c->grids); dfree(c->home); dfree(c->rank); dfree(c->cell_start); dfree(c->aabb_bits);
    dfree(c->margin_bits); dfree(c->scan_tmp); dfree(c->primA); dfree(c->primB); dfree(c->primC);
    dfree(c->primD); dfree(c->perm); dfree(c->cell_lo); dfree(c->cell_hi);
    c->binned = false;
    c->total_cells = 0;
    c->grids_h.clear();
}

void free_scene(pictura_ctx c)
{
    free_bins(c);
    dfree(c->verts); dfree(c->cls); dfree(c->offsets_d); dfree(c->stats);
    dfree(c->prims); dfree(c->prim_offsets_d);
    c->have_scene = false;
    c->T = 0;
    c->P = 0;
    c->num_worlds = 0;
}

struct DeviceGuard {
    int prev = -1;
    explicit DeviceGuard(int d) { if (hipGetDevice(&prev) != hipSuccess) prev = -1; (void)hipSetDevice(d); }
    ~DeviceGuard() { if (prev >= 0) (void)hipSetDevice(prev); }
};

// Primitives of one upload: walking each world's triangles in order, triangle
// t and t + 1 form a pair when they have the same class and t + 1 = (a, c, d)
// for t = (a, b, c) (the same a and c, bit for bit); a triangle that starts no
// pair and is not the second half of one is a primitive of its own.
void make_prims(int nw, const int64_t* offs, const float* verts, const uint8_t* cls, std::vector<uint32_t>& prims,
                std::vector<int64_t>& prim_offs)
{
    prims.clear();
    prim_offs.assign(1, 0);
    for (int w = 0; w < nw; ++w) {
        for (int64_t t = offs[w]; t < offs[w + 1];) {
            const float* a = verts + 9 * t;
            const bool pair = t + 1 < offs[w + 1] && cls[t] == cls[t + 1] && std::memcmp(a, a + 9, 12) == 0 &&
                              std::memcmp(a + 6, a + 12, 12) == 0;
            prims.push_back((uint32_t)t | (pair ? kPrimFlagPair : 0u));
            t += pair ? 2 : 1;
        }
        prim_offs.push_back((int64_t)prims.size());
    }
}

uint32_t f2u(float f) { uint32_t u; std::memcpy(&u, &f, 4); return u; }
float u2f(uint32_t u) { float f; std::memcpy(&f, &u, 4); return f; }

float pow2_ceil(float x)
{
    uint32_t u = f2u(x);
    if ((u & 0x7FFFFFu) == 0) return x;
    return u2f((u & 0x7F800000u) + 0x00800000u);
}

}  // namespace

extern "C" {

pictura_status pictura_create(int32_t device, pictura_ctx* out)
{
    if (!out) return PICTURA_EINVAL;
    *out = nullptr;
    int n = 0;
    if (hipGetDeviceCount(&n) != hipSuccess || n <= 0) return PICTURA_EDEVICE;
    if (device < 0 || device >= n) return PICTURA_EDEVICE;
    auto* c = new (std::nothrow) pictura_ctx_s();
    if (!c) return PICTURA_ENOMEM;
    c->device = device;
    {
        DeviceGuard g(device);
        if (hipMalloc((void**)&c->dev_err, sizeof(uint32_t)) != hipSuccess) {
            delete c;
            return PICTURA_ENOMEM;
        }
        if (hipMemset(c->dev_err, 0, sizeof(uint32_t)) != hipSuccess || noalloc_scratch_init(device) != hipSuccess) {
            (void)hipFree(c->dev_err);
            delete c;
            return PICTURA_EDEVICE;
        }
    }
    *out = c;
    return PICTURA_OK;
}

void pictura_destroy(pictura_ctx c)
{
    if (!c) return;
    {
        DeviceGuard g(c->device);
        (void)hipDeviceSynchronize();
        free_scene(c);
        dfree(c->dev_err);
        dfree(c->apk);
        if (c->apk_event) (void)hipEventDestroy(c->apk_event);
    }
    delete c;
}

const char* pictura_last_error(pictura_ctx c) { return c ? c->err.c_str() : "null context"; }

pictura_status pictura_scene_upload(pictura_ctx c, const pictura_scene* s, void* stream)
{
    if (!c) return PICTURA_EINVAL;
    c->err.clear();
    if (!s || !s->tri_offsets || !s->bounds) return fail(c, PICTURA_EINVAL, "scene_upload: null scene pointer");
    if (s->num_worlds < 1) return fail(c, PICTURA_EINVAL, "scene_upload: num_worlds must be >= 1");
    const int nw = s->num_worlds;
    if (s->tri_offsets[0] != 0) return fail(c, PICTURA_EINVAL, "scene_upload: tri_offsets[0] must be 0");
    for (int w = 0; w < nw; ++w)
        if (s->tri_offsets[w + 1] < s->tri_offsets[w])
            return fail(c, PICTURA_EINVAL, "scene_upload: tri_offsets must be non-decreasing");
    const int64_t T = s->tri_offsets[nw];
    if (T > 0x7FFFFFFFll) return fail(c, PICTURA_ERANGE, "scene_upload: more than 2^31-1 triangles");
    if (T > 0 && (!s->verts || !s->cls)) return fail(c, PICTURA_EINVAL, "scene_upload: null verts/cls");
    uint8_t max_cls = 0;
    for (int64_t t = 0; t < T; ++t) {
        if (s->cls[t] == 255) return fail(c, PICTURA_EINVAL, "scene_upload: class ID 255 is reserved");
        max_cls = s->cls[t] > max_cls ? s->cls[t] : max_cls;
    }
    for (int w = 0; w < nw; ++w) {
        const float* b = s->bounds + 4 * w;
        if (!(std::isfinite(b[0]) && std::isfinite(b[1]) && std::isfinite(b[2]) && std::isfinite(b[3])) ||
            !(b[2] > b[0]) || !(b[3] > b[1]))
            return fail(c, PICTURA_EINVAL, "scene_upload: bounds of world %d are not a finite rectangle", w);
    }
    std::vector<uint32_t> prims;
    std::vector<int64_t> prim_offs;
    make_prims(nw, s->tri_offsets, s->verts, s->cls, prims, prim_offs);
    const int64_t P = (int64_t)prims.size();
    if (P >= (1ll << 29)) return fail(c, PICTURA_ERANGE, "scene_upload: 2^29 or more primitives (triangles and pairs)");
    DeviceGuard g(c->device);
    hipStream_t st = (hipStream_t)stream;
    free_scene(c);
    hipError_t e;
    if ((e = dalloc(c->prims, (size_t)P)) != hipSuccess || (e = dalloc(c->prim_offsets_d, (size_t)nw + 1)) != hipSuccess) {
        free_scene(c);
        return hip_fail(c, e, "scene_upload alloc");
    }
    if ((e = dalloc(c->verts, (size_t)T * 9)) != hipSuccess) { free_scene(c); return hip_fail(c, e, "scene_upload alloc"); }
    if ((e = dalloc(c->cls, (size_t)T)) != hipSuccess) { free_scene(c); return hip_fail(c, e, "scene_upload alloc"); }
    if ((e = dalloc(c->offsets_d, (size_t)nw + 1)) != hipSuccess) { free_scene(c); return hip_fail(c, e, "scene_upload alloc"); }
    // Synchronous-from-the-caller's-view copies: pageable host memory is staged
    // by the runtime before hipMemcpyAsync returns, so the caller may reuse it.
    if (T > 0) {
        if ((e = hipMemcpyAsync(c->verts, s->verts, (size_t)T * 9 * sizeof(float), hipMemcpyHostToDevice, st)) != hipSuccess ||
            (e = hipMemcpyAsync(c->cls, s->cls, (size_t)T, hipMemcpyHostToDevice, st)) != hipSuccess) {
            free_scene(c);
            return hip_fail(c, e, "scene_upload copy");
        }
    }
    if ((e = hipMemcpyAsync(c->offsets_d, s->tri_offsets, (size_t)(nw + 1) * sizeof(int64_t), hipMemcpyHostToDevice, st)) != hipSuccess ||
        (e = hipMemcpyAsync(c->prim_offsets_d, prim_offs.data(), (size_t)(nw + 1) * sizeof(int64_t), hipMemcpyHostToDevice, st)) != hipSuccess ||
        (P > 0 && (e = hipMemcpyAsync(c->prims, prims.data(), (size_t)P * sizeof(uint32_t), hipMemcpyHostToDevice, st)) != hipSuccess)) {
        free_scene(c);
        return hip_fail(c, e, "scene_upload copy");
    }
    if ((e = hipStreamSynchronize(st)) != hipSuccess) { free_scene(c); return hip_fail(c, e, "scene_upload sync"); }
    c->offsets_h.assign(s->tri_offsets, s->tri_offsets + nw + 1);
    c->bounds_h.assign(s->bounds, s->bounds + 4 * nw);
    c->num_worlds = nw;
    c->T = T;
    c->P = P;
    c->have_scene = true;
    c->max_cls = max_cls;
    return PICTURA_OK;
}

pictura_status pictura_bin_scene(pictura_ctx c, float cell, void* stream)
{
    if (!c) return PICTURA_EINVAL;
    c->err.clear();
    if (!c->have_scene) return fail(c, PICTURA_ESTATE, "bin_scene: no scene uploaded");
    if (!(cell > 0.0f) || !std::isfinite(cell)) return fail(c, PICTURA_EINVAL, "bin_scene: cell size must be > 0");
    const int nw = c->num_worlds;
    std::vector<WorldGrid> grids(nw);
    int64_t total = 0;
    for (int w = 0; w < nw; ++w) {
        const float* b = &c->bounds_h[4 * w];
        const float wx = b[2] - b[0], wy = b[3] - b[1];
        const float fnx = std::ceil(wx / cell), fny = std::ceil(wy / cell);
        if (!(fnx < 1.0e9f) || !(fny < 1.0e9f)) return fail(c, PICTURA_ERANGE, "bin_scene: grid too large");
        WorldGrid& g = grids[w];
        g.ox = b[0]; g.oy = b[1];
        g.nx = fnx < 1.0f ? 1 : (int32_t)fnx;
        g.ny = fny < 1.0f ? 1 : (int32_t)fny;
        g.cell_base = (int32_t)total;
        g.margin = 0.0f;
        g.pad0 = g.pad1 = 0;
        total += (int64_t)g.nx * g.ny;
        if (total >= 0x7FFFFFFFll) return fail(c, PICTURA_ERANGE, "bin_scene: more than 2^31-1 cells");
    }
    DeviceGuard dg(c->device);
    hipStream_t st = (hipStream_t)stream;
    free_bins(c);
    const int64_t P = c->P;
    hipError_t e = hipSuccess;
    const int64_t ntmp = scan_tmp_needed(total + 1);
    if ((e = dalloc(c->grids, (size_t)nw)) != hipSuccess || (e = dalloc(c->home, (size_t)P)) != hipSuccess ||
        (e = dalloc(c->rank, (size_t)P)) != hipSuccess || (e = dalloc(c->cell_start, (size_t)total + 1)) != hipSuccess ||
        (e = dalloc(c->aabb_bits, (size_t)total * 8)) != hipSuccess || (e = dalloc(c->margin_bits, (size_t)nw)) != hipSuccess ||
        (e = dalloc(c->scan_tmp, (size_t)ntmp)) != hipSuccess || (e = dalloc(c->primA, (size_t)P)) != hipSuccess ||
        (e = dalloc(c->primB, (size_t)P)) != hipSuccess || (e = dalloc(c->primC, (size_t)P)) != hipSuccess ||
        (e = dalloc(c->primD, (size_t)P)) != hipSuccess ||
        (e = dalloc(c->perm, (size_t)P)) != hipSuccess || (e = dalloc(c->cell_lo, (size_t)total)) != hipSuccess ||
        (e = dalloc(c->cell_hi, (size_t)total)) != hipSuccess) {
        free_bins(c);
        return hip_fail(c, e, "bin_scene alloc");
    }
    if ((e = hipMemcpyAsync(c->grids, grids.data(), sizeof(WorldGrid) * nw, hipMemcpyHostToDevice, st)) != hipSuccess) {
        free_bins(c);
        return hip_fail(c, e, "bin_scene copy");
    }
    BinWork W{};
    W.verts = c->verts; W.cls = c->cls; W.prims = c->prims; W.prim_offsets = c->prim_offsets_d; W.P = P;
    W.num_worlds = nw;
    W.grids = c->grids; W.total_cells = total; W.cell_size = cell;
    W.home = c->home; W.rank = c->rank; W.count = c->cell_start; W.aabb_bits = c->aabb_bits;
    W.margin_bits = c->margin_bits; W.scan_tmp = c->scan_tmp; W.scan_tmp_len = ntmp;
    W.primA = c->primA; W.primB = c->primB; W.primC = c->primC; W.primD = c->primD; W.perm = c->perm;
    W.cell_lo = c->cell_lo; W.cell_hi = c->cell_hi;
    if ((e = launch_bin(W, st)) != hipSuccess) { free_bins(c); return hip_fail(c, e, "bin_scene launch"); }
    // the host copy of the grids is needed again for render's argument checks
    if ((e = hipStreamSynchronize(st)) != hipSuccess) { free_bins(c); return hip_fail(c, e, "bin_scene sync"); }
    c->grids_h = grids;
    c->cell_size = cell;
    c->total_cells = total;
    c->binned = true;
    return PICTURA_OK;
}

// Argument checks and the parameter block of one render call; the launch is the caller's.
// Returns PICTURA_OK with *empty set when there is nothing to render.
static pictura_status render_setup(pictura_ctx c, const pictura_agents* ag, const pictura_rig* rig,
                                   uint8_t* out_cls, float* out_depth, RenderParams& P, bool* empty)
{
    *empty = false;
    if (!ag || !rig || !out_cls || !out_depth) return fail(c, PICTURA_EINVAL, "render_views: null argument");
    if (!c->binned) return fail(c, PICTURA_ESTATE, "render_views: scene not binned");
    if (ag->num_worlds != c->num_worlds)
        return fail(c, PICTURA_EINVAL, "render_views: agents.num_worlds %d != scene num_worlds %d", ag->num_worlds, c->num_worlds);
    if (ag->agents_per_world < 1 || ag->agents_per_world > (1 << 26))
        return fail(c, PICTURA_EINVAL, "render_views: agents_per_world must be 1..2^26");
    if (!ag->x || !ag->y || !ag->z0 || !ag->cos_h || !ag->sin_h || !ag->length || !ag->width || !ag->height || !ag->cls)
        return fail(c, PICTURA_EINVAL, "render_views: null agent array");
    if (rig->num_cams < 1 || rig->num_cams > PICTURA_MAX_CAMS) return fail(c, PICTURA_EINVAL, "render_views: num_cams must be 1..8");
    if (rig->width < 1 || rig->height < 1 || rig->width > 4096 || rig->height > 4096)
        return fail(c, PICTURA_EINVAL, "render_views: width/height must be 1..4096");
    if (!(rig->fx > 0.0f) || !(rig->fy > 0.0f) || !std::isfinite(rig->fx) || !std::isfinite(rig->fy) ||
        !std::isfinite(rig->cx) || !std::isfinite(rig->cy))
        return fail(c, PICTURA_EINVAL, "render_views: intrinsics must be finite with fx, fy > 0");
    if (!(rig->near_m > 0.0f) || !(rig->far_m > rig->near_m) || !std::isfinite(rig->far_m))
        return fail(c, PICTURA_EINVAL, "render_views: need 0 < near < far < inf");
    for (int k = 0; k < rig->num_cams; ++k)
        for (int q = 0; q < 5; ++q)
            if (!std::isfinite(rig->mount[k][q])) return fail(c, PICTURA_EINVAL, "render_views: mount %d not finite", k);
    const float izfar = 1.0f / rig->far_m;
    const float izcap = pow2_ceil(1.0f / rig->near_m);
    if (!(izfar > 0.0f) || !std::isfinite(izcap) || ((f2u(izcap) >> 3) - (f2u(izfar) >> 3)) >= 0xFFFFFFu)
        return fail(c, PICTURA_EINVAL, "render_views: far/near ratio too large for the 24-bit depth key");
    const int64_t V = (int64_t)c->num_worlds * ag->agents_per_world * rig->num_cams;
    if (V == 0) { *empty = true; return PICTURA_OK; }

    P = RenderParams{};
    P.scene.primA = c->primA; P.scene.primB = c->primB; P.scene.primC = c->primC; P.scene.primD = c->primD;
    P.scene.cell_start = c->cell_start; P.scene.cell_lo = c->cell_lo; P.scene.cell_hi = c->cell_hi;
    P.scene.grids = c->grids; P.scene.cell_size = c->cell_size; P.scene.num_worlds = c->num_worlds;
    P.ax = ag->x; P.ay = ag->y; P.az0 = ag->z0; P.ac = ag->cos_h; P.as = ag->sin_h;
    P.al = ag->length; P.aw = ag->width; P.ah = ag->height; P.acls = ag->cls;
    P.A = ag->agents_per_world; P.C = rig->num_cams;
    P.W = rig->width; P.H = rig->height;
    P.fx = rig->fx; P.fy = rig->fy; P.cx = rig->cx; P.cy = rig->cy; P.nearp = rig->near_m; P.farp = rig->far_m;
    for (int k = 0; k < PICTURA_MAX_CAMS; ++k)
        for (int q = 0; q < 5; ++q) P.mount[k][q] = k < rig->num_cams ? rig->mount[k][q] : 0.0f;
    P.fx256 = 256.0f * P.fx; P.fy256 = 256.0f * P.fy; P.cx256 = 256.0f * P.cx; P.cy256 = 256.0f * P.cy;
    P.rfx = 1.0f / P.fx; P.rfy = 1.0f / P.fy;
    P.izfar = izfar; P.izcap = izcap; P.qbase = f2u(izcap) >> 3;
    P.cabs = std::fabs(P.cx) > std::fabs(P.cy) ? std::fabs(P.cx) : std::fabs(P.cy);
    P.near_cull = P.nearp * 1.00390625f;
    P.near_off = -P.nearp * 0.99609375f;
    P.far_off = P.farp * 1.015625f;
    // pixel-centre offsets: with c a multiple of 2^-8 below 2^14 in magnitude,
    // 0.5 - c and i + (0.5 - c) (i < 4096) are exact in fp32
    P.hx = 0.5f - P.cx;
    P.hy = 0.5f - P.cy;
    auto eighth_bit = [](float c) { const double s = (double)c * 256.0; return std::fabs(c) < 16384.0f && s == std::rint(s); };
    P.pix_exact = (eighth_bit(P.cx) && eighth_bit(P.cy)) ? 1 : 0;
    // decoded inverse depths lie in [1/far (1 - 2^-20), IZCAP]
    P.fast_decode = (izfar >= 0.000244140625f * 1.0000038f && izcap < 1048576.0f) ? 1 : 0;
    int tw = 64, th = 64;
    if (c->tile > 0) {
        tw = c->tile;
        th = c->tile;
    } else {
        // as few 64-wide columns and rows of tiles as the view needs, split
        // evenly (96 wide: two tiles of 48 rather than 64 and 32); for a view
        // whose width is a multiple of 16 (the vector write-out's unit) the tile
        // width is one too, as long as that keeps the count
        const int nx = (P.W + 63) / 64, ny = (P.H + 63) / 64;
        const int ex = (P.W + nx - 1) / nx, ey = (P.H + ny - 1) / ny;
        const int ex16 = (ex + 15) & ~15;
        tw = (P.W % 16) == 0 && ex16 <= 64 && (P.W + ex16 - 1) / ex16 == nx ? ex16 : ex;
        th = ey;
    }
    tw = tw < P.W ? tw : P.W;
    th = th < P.H ? th : P.H;
    P.tile_w = tw; P.tile_h = th;
    P.tiles_x = (P.W + tw - 1) / tw;
    P.tiles_y = (P.H + th - 1) / th;
    P.num_views = V;
    P.num_blocks = V * P.tiles_x * P.tiles_y;
    if (P.num_blocks > 0x7FFFFFFFll) return fail(c, PICTURA_ERANGE, "render_views: too many view tiles in one call");
    P.div_tiles = make_div31((uint32_t)(P.tiles_x * P.tiles_y));
    P.div_cams = make_div31((uint32_t)P.C);
    P.div_agents = make_div31((uint32_t)P.A);
    P.rcs = 1.0f / c->cell_size;
    P.out_cls = out_cls; P.out_depth = out_depth;
    P.dev_err = c->dev_err;
    P.cull = c->cull;
    P.vec_out = ((reinterpret_cast<uintptr_t>(out_cls) | reinterpret_cast<uintptr_t>(out_depth)) & 15u) == 0 ? 1 : 0;
    if (c->lights.lights_per_world > 0) {
        const pictura_lights& l = c->lights;
        if (l.num_worlds != c->num_worlds)
            return fail(c, PICTURA_EINVAL, "render_views: lights.num_worlds %d != scene num_worlds %d", l.num_worlds,
                        c->num_worlds);
        P.lx = l.x; P.ly = l.y; P.lz = l.z; P.lcf = l.cos_f; P.lsf = l.sin_f; P.lr = l.radius; P.lcls = l.cls;
        P.L = l.lights_per_world;
        P.lcos2 = l.cos_max * l.cos_max;
    }
    {
        // the packed agents (written by every render call before its kernels)
        const size_t need = (size_t)c->num_worlds * (size_t)P.A * 3u * sizeof(float4);
        hipError_t ae = hipSuccess;
        if (need > c->apk_cap) {
            if (c->apk && (ae = hipDeviceSynchronize()) != hipSuccess)   // a render may still read the old one
                return hip_fail(c, ae, "render_views sync");
            dfree(c->apk);
            c->apk_cap = 0;
            if ((ae = hipMalloc((void**)&c->apk, need)) != hipSuccess) {
                c->apk = nullptr;
                return hip_fail(c, ae, "render_views agents alloc");
            }
            c->apk_cap = need;
        }
        if (!c->apk_event && (ae = hipEventCreateWithFlags(&c->apk_event, hipEventDisableTiming)) != hipSuccess) {
            c->apk_event = nullptr;
            return hip_fail(c, ae, "render_views event");
        }
        P.apk = c->apk;
    }
    if (c->stats_on) {
        hipError_t se = hipSuccess;
        if (!c->stats) {
            if ((se = dalloc(c->stats, (size_t)kNumStats)) != hipSuccess) return hip_fail(c, se, "render_views stats alloc");
            if ((se = hipMemset(c->stats, 0, sizeof(unsigned long long) * kNumStats)) != hipSuccess)
                return hip_fail(c, se, "render_views stats clear");
        }
        P.stats = c->stats;
    }
    return PICTURA_OK;
}

// Launch a render set up by render_setup on stream s: pack the agents, then
// the render kernel.  A call on another stream than the previous render call
// first waits for that call's kernels, which read the same packed agents.
static hipError_t render_launch(pictura_ctx c, const RenderParams& P, hipStream_t s)
{
    hipError_t e = hipSuccess;
    if (c->apk_used && c->apk_stream != s && (e = hipStreamWaitEvent(s, c->apk_event, 0)) != hipSuccess) return e;
    if ((e = launch_pack_agents(P, (int64_t)c->num_worlds * P.A, s)) != hipSuccess) return e;
    if ((e = launch_render(P, s)) != hipSuccess) return e;
    if ((e = hipEventRecord(c->apk_event, s)) != hipSuccess) return e;
    c->apk_stream = s;
    c->apk_used = true;
    return hipSuccess;
}

pictura_status pictura_render_views(pictura_ctx c, const pictura_agents* ag, const pictura_rig* rig,
                                    uint8_t* out_cls, float* out_depth, void* stream)
{
    if (!c) return PICTURA_EINVAL;
    c->err.clear();
    DeviceGuard dg(c->device);
    RenderParams P;
    bool empty = false;
    const pictura_status st = render_setup(c, ag, rig, out_cls, out_depth, P, &empty);
    if (st != PICTURA_OK || empty) return st;
    hipError_t e = render_launch(c, P, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(c, e, "render_views launch");
    return PICTURA_OK;
}

static pictura_status render_rgb(pictura_ctx c, const pictura_agents* ag, const pictura_rig* rig, uint8_t* out_cls,
                                 float* out_depth, uint8_t* out_rgb, void* stream, bool aa)
{
    if (!c) return PICTURA_EINVAL;
    c->err.clear();
    if (!out_rgb) return fail(c, PICTURA_EINVAL, "render_rgb: null argument");
    if (c->have_scene && c->max_cls > 15) return fail(c, PICTURA_EINVAL, "render_rgb: scene class IDs must be below 16");
    DeviceGuard dg(c->device);
    RenderParams P;
    bool empty = false;
    const pictura_status st = render_setup(c, ag, rig, out_cls, out_depth, P, &empty);
    if (st != PICTURA_OK || empty) return st;
    P.out_rgb = out_rgb;
    P.rfar = 1.0f / P.farp;
    P.aa = aa ? 1 : 0;
    hipError_t e = render_launch(c, P, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(c, e, "render_rgb launch");
    return PICTURA_OK;
}

pictura_status pictura_render_rgb(pictura_ctx c, const pictura_agents* ag, const pictura_rig* rig, uint8_t* out_cls,
                                  float* out_depth, uint8_t* out_rgb, void* stream)
{
    return render_rgb(c, ag, rig, out_cls, out_depth, out_rgb, stream, false);
}

pictura_status pictura_render_rgb_aa(pictura_ctx c, const pictura_agents* ag, const pictura_rig* rig, uint8_t* out_cls,
                                     float* out_depth, uint8_t* out_rgb, void* stream)
{
    return render_rgb(c, ag, rig, out_cls, out_depth, out_rgb, stream, true);
}

pictura_status pictura_render_instances(pictura_ctx c, const pictura_agents* ag, const pictura_rig* rig,
                                        uint8_t* out_cls, float* out_depth, int32_t* out_inst,
                                        uint32_t* out_counts, void* stream)
{
    if (!c) return PICTURA_EINVAL;
    c->err.clear();
    if (!out_inst || !out_counts) return fail(c, PICTURA_EINVAL, "render_instances: null argument");
    DeviceGuard dg(c->device);
    RenderParams P;
    bool empty = false;
    const pictura_status st = render_setup(c, ag, rig, out_cls, out_depth, P, &empty);
    if (st != PICTURA_OK || empty) return st;
    P.out_inst = out_inst;
    P.out_counts = out_counts;
    hipError_t e = launch_fill_u32(out_counts, (size_t)P.num_views * (size_t)P.A * 2u, 0u, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(c, e, "render_instances clear");
    e = render_launch(c, P, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(c, e, "render_instances launch");
    return PICTURA_OK;
}

pictura_status pictura_agents_step(pictura_ctx c, const pictura_agent_state* s, const float* steer,
                                   const float* accel, float dt, float vmax, void* stream)
{
    if (!c) return PICTURA_EINVAL;
    c->err.clear();
    if (!s || !steer || !accel) return fail(c, PICTURA_EINVAL, "agents_step: null argument");
    if (s->count < 0) return fail(c, PICTURA_EINVAL, "agents_step: count < 0");
    if (s->count > 0 && (!s->x || !s->y || !s->psi || !s->speed || !s->cos_h || !s->sin_h || !s->length))
        return fail(c, PICTURA_EINVAL, "agents_step: null state array");
    if (!std::isfinite(dt) || !std::isfinite(vmax)) return fail(c, PICTURA_EINVAL, "agents_step: dt/vmax not finite");
    AgentStepParams p{};
    p.x = s->x; p.y = s->y; p.psi = s->psi; p.speed = s->speed; p.cos_h = s->cos_h; p.sin_h = s->sin_h;
    p.length = s->length; p.steer = steer; p.accel = accel; p.dt = dt; p.vmax = vmax; p.count = s->count;
    DeviceGuard dg(c->device);
    hipError_t e = launch_agents_step(p, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(c, e, "agents_step launch");
    return PICTURA_OK;
}

pictura_status pictura_store_probe(pictura_ctx c, void* dst, uint64_t bytes, void* stream)
{
    if (!c) return PICTURA_EINVAL;
    c->err.clear();
    if (!dst) return fail(c, PICTURA_EINVAL, "store_probe: null buffer");
    if ((reinterpret_cast<uintptr_t>(dst) & 15u) != 0 || (bytes & 15u) != 0)
        return fail(c, PICTURA_EINVAL, "store_probe: buffer and size must be multiples of 16 bytes");
    DeviceGuard dg(c->device);
    const hipError_t e = launch_store_probe(dst, bytes, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(c, e, "store_probe launch");
    return PICTURA_OK;
}

pictura_status pictura_bins_info(pictura_ctx c, int32_t* dims, int64_t* cell_base, int64_t* total_cells,
                                 int64_t* total_prims)
{
    if (!c) return PICTURA_EINVAL;
    c->err.clear();
    if (!c->binned) return fail(c, PICTURA_ESTATE, "bins_info: scene not binned");
    for (int w = 0; w < c->num_worlds; ++w) {
        if (dims) { dims[2 * w] = c->grids_h[w].nx; dims[2 * w + 1] = c->grids_h[w].ny; }
        if (cell_base) cell_base[w] = c->grids_h[w].cell_base;
    }
    if (cell_base) cell_base[c->num_worlds] = c->total_cells;
    if (total_cells) *total_cells = c->total_cells;
    if (total_prims) *total_prims = c->P;
    return PICTURA_OK;
}

pictura_status pictura_bins_copy(pictura_ctx c, uint32_t* cell_start, float* cell_aabb, uint32_t* perm)
{
    if (!c) return PICTURA_EINVAL;
    c->err.clear();
    if (!c->binned) return fail(c, PICTURA_ESTATE, "bins_copy: scene not binned");
    DeviceGuard dg(c->device);
    hipError_t e;
    if ((e = hipDeviceSynchronize()) != hipSuccess) return hip_fail(c, e, "bins_copy sync");
    const int64_t n = c->total_cells;
    if (cell_start && (e = hipMemcpy(cell_start, c->cell_start, sizeof(uint32_t) * (n + 1), hipMemcpyDeviceToHost)) != hipSuccess)
        return hip_fail(c, e, "bins_copy");
    if (cell_aabb) {
        std::vector<float4> lo(n), hi(n);
        if ((e = hipMemcpy(lo.data(), c->cell_lo, sizeof(float4) * n, hipMemcpyDeviceToHost)) != hipSuccess ||
            (e = hipMemcpy(hi.data(), c->cell_hi, sizeof(float4) * n, hipMemcpyDeviceToHost)) != hipSuccess)
            return hip_fail(c, e, "bins_copy");
        for (int64_t k = 0; k < n; ++k) {
            float* o = cell_aabb + 6 * k;
            o[0] = lo[k].x; o[1] = lo[k].y; o[2] = lo[k].z; o[3] = hi[k].x; o[4] = hi[k].y; o[5] = hi[k].z;
        }
    }
    if (perm && c->P > 0 && (e = hipMemcpy(perm, c->perm, sizeof(uint32_t) * c->P, hipMemcpyDeviceToHost)) != hipSuccess)
        return hip_fail(c, e, "bins_copy");
    return PICTURA_OK;
}

pictura_status pictura_set_lights(pictura_ctx c, const pictura_lights* l)
{
    if (!c) return PICTURA_EINVAL;
    c->err.clear();
    if (!l || l->lights_per_world == 0) {
        c->lights = pictura_lights{};
        return PICTURA_OK;
    }
    if (l->num_worlds < 1) return fail(c, PICTURA_EINVAL, "set_lights: num_worlds must be >= 1");
    if (l->lights_per_world < 0 || l->lights_per_world > (1 << 20))
        return fail(c, PICTURA_EINVAL, "set_lights: lights_per_world must be 0..2^20");
    if (!l->x || !l->y || !l->z || !l->cos_f || !l->sin_f || !l->radius || !l->cls)
        return fail(c, PICTURA_EINVAL, "set_lights: null array");
    if (!(l->cos_max >= 0.0f && l->cos_max <= 1.0f)) return fail(c, PICTURA_EINVAL, "set_lights: cos_max must lie in [0, 1]");
    if ((int64_t)l->num_worlds * l->lights_per_world > 0x7FFFFFFFll)
        return fail(c, PICTURA_ERANGE, "set_lights: more than 2^31 - 1 lights");
    c->lights = *l;
    return PICTURA_OK;
}

pictura_status pictura_set_option(pictura_ctx c, int32_t option, int32_t value)
{
    if (!c) return PICTURA_EINVAL;
    c->err.clear();
    if (option == PICTURA_OPT_CULL) {
        if (value != 0 && value != 1) return fail(c, PICTURA_EINVAL, "set_option: CULL must be 0 or 1");
        c->cull = value;
        return PICTURA_OK;
    }
    if (option == PICTURA_OPT_STATS) {
        if (value != 0 && value != 1) return fail(c, PICTURA_EINVAL, "set_option: STATS must be 0 or 1");
        c->stats_on = value;
        return PICTURA_OK;
    }
    if (option == PICTURA_OPT_TILE) {
        if (value != 0 && (value < 8 || value > 64)) return fail(c, PICTURA_EINVAL, "set_option: TILE must be 0 or 8..64");
        c->tile = value;
        return PICTURA_OK;
    }
    return fail(c, PICTURA_EINVAL, "set_option: unknown option %d", option);
}

pictura_status pictura_selftest_rcp(pictura_ctx c, uint32_t lo_bits, uint32_t count, uint64_t* mismatches)
{
    if (!c) return PICTURA_EINVAL;
    c->err.clear();
    if (!mismatches) return fail(c, PICTURA_EINVAL, "selftest_rcp: null output");
    if ((uint64_t)(lo_bits & 0x7FFFFFFFu) + count > 0x7F800000ull)
        return fail(c, PICTURA_EINVAL, "selftest_rcp: range leaves the finite floats of one sign");
    DeviceGuard dg(c->device);
    unsigned long long* d = nullptr;
    hipError_t e;
    if ((e = hipMalloc((void**)&d, sizeof(unsigned long long))) != hipSuccess) return hip_fail(c, e, "selftest_rcp alloc");
    unsigned long long h = 0;
    if ((e = hipMemcpy(d, &h, sizeof h, hipMemcpyHostToDevice)) != hipSuccess ||
        (e = launch_rcp_check(lo_bits, count, d, nullptr)) != hipSuccess ||
        (e = hipMemcpy(&h, d, sizeof h, hipMemcpyDeviceToHost)) != hipSuccess) {
        (void)hipFree(d);
        return hip_fail(c, e, "selftest_rcp");
    }
    (void)hipFree(d);
    *mismatches = (uint64_t)h;
    return PICTURA_OK;
}

pictura_status pictura_selftest_rcp_noalloc(pictura_ctx c, uint32_t lo_bits, uint32_t count, uint64_t* mismatches)
{
    if (!c) return PICTURA_EINVAL;
    c->err.clear();
    if (!mismatches) return fail(c, PICTURA_EINVAL, "selftest_rcp_noalloc: null output");
    if ((uint64_t)(lo_bits & 0x7FFFFFFFu) + count > 0x7F800000ull)
        return fail(c, PICTURA_EINVAL, "selftest_rcp_noalloc: range leaves the finite floats of one sign");
    DeviceGuard dg(c->device);
    auto* counter = (unsigned long long*)noalloc_scratch(c->device);
    if (!counter) return fail(c, PICTURA_ESTATE, "selftest_rcp_noalloc: no scratch address for device %d", c->device);
    hipError_t e;
    unsigned long long h = 0;
    if ((e = launch_rcp_check_noalloc(lo_bits, count, counter, nullptr)) != hipSuccess ||
        (e = hipMemcpy(&h, counter, sizeof h, hipMemcpyDeviceToHost)) != hipSuccess)
        return hip_fail(c, e, "selftest_rcp_noalloc");
    *mismatches = (uint64_t)h;
    return PICTURA_OK;
}

pictura_status pictura_device_errors(pictura_ctx c, uint32_t* out, int32_t reset)
{
    if (!c) return PICTURA_EINVAL;
    c->err.clear();
    if (!out) return fail(c, PICTURA_EINVAL, "device_errors: null output");
    DeviceGuard dg(c->device);
    hipError_t e;
    if ((e = hipDeviceSynchronize()) != hipSuccess) return hip_fail(c, e, "device_errors sync");
    uint32_t h = 0;
    if ((e = hipMemcpy(&h, c->dev_err, sizeof h, hipMemcpyDeviceToHost)) != hipSuccess)
        return hip_fail(c, e, "device_errors copy");
    *out = h;
    if (reset && h != 0 && (e = hipMemset(c->dev_err, 0, sizeof h)) != hipSuccess)
        return hip_fail(c, e, "device_errors reset");
    return PICTURA_OK;
}

pictura_status pictura_stats_copy(pictura_ctx c, uint64_t* out, int32_t n, int32_t reset)
{
    if (!c) return PICTURA_EINVAL;
    c->err.clear();
    if (!out || n < 0) return fail(c, PICTURA_EINVAL, "stats_copy: bad output");
    DeviceGuard dg(c->device);
    hipError_t e;
    if ((e = hipDeviceSynchronize()) != hipSuccess) return hip_fail(c, e, "stats_copy sync");
    unsigned long long tmp[kNumStats] = {0};
    if (c->stats && (e = hipMemcpy(tmp, c->stats, sizeof tmp, hipMemcpyDeviceToHost)) != hipSuccess)
        return hip_fail(c, e, "stats_copy");
    for (int k = 0; k < n; ++k) out[k] = k < kNumStats ? (uint64_t)tmp[k] : 0;
    if (reset && c->stats && (e = hipMemset(c->stats, 0, sizeof tmp)) != hipSuccess) return hip_fail(c, e, "stats_copy reset");
    return PICTURA_OK;
}

}  // extern "C"
