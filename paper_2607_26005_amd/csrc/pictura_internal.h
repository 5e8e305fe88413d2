// Internal structures of the HIP library: device scene layout, kernel
// parameter blocks and launcher declarations.  Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pictura {

constexpr int kBlock = 256;          // threads per workgroup of the binning kernels
constexpr int kNumStats = 30;        // optional work counters of the render kernel

// Grid of one world.  Cells are numbered row-major from cell_base.
struct WorldGrid {
    float ox, oy;        // grid origin (bounds xmin, ymin)
    int32_t nx, ny;
    int32_t cell_base;
    float margin;        // how far any cell's triangle AABB reaches beyond its cell rectangle
    int32_t pad0, pad1;
};

// The binned unit is a primitive: one triangle (a, b, c), or a pair of input
// triangles (a, b, c), (a, c, d) that share the edge a-c and the class (a quad
// split along a diagonal: the generators' ground tiles, road segments,
// markings and curbs are all such pairs).  A pair is culled, loaded and set up
// once; its two halves are still separate triangles with their own depth
// planes.  Re-laid-out primitive p (cell order) is split over four arrays, so
// that a wave reading 64 consecutive primitives issues coalesced loads:
//   A[p] = (ax, ay, az, bx), B[p] = (by, bz, cx, cy),
//   C[p] = (cz, bits(class | pair << 8), dx, dy), D[p] = dz   (d = 0 for a triangle).
constexpr uint32_t kPrimPair = 256u;   // in the class word of C: the primitive is a pair

struct SceneDev {
    const float4* primA;
    const float4* primB;
    const float4* primC;
    const float* primD;
    const uint32_t* cell_start;   // [cells + 1]
    const float4* cell_lo;        // [cells] xmin ymin zmin -
    const float4* cell_hi;        // [cells] xmax ymax zmax -
    const WorldGrid* grids;       // [num_worlds]
    float cell_size;
    int32_t num_worlds;
};

// n / d for 0 <= n < 2^31 without a division: with l = ceil(log2 d) and
// m = floor(2^(31 + l) / d) + 1 (which fits 32 bits), n / d equals
// umulhi(n, m) >> (l - 1) (Granlund and Montgomery, "Division by invariant
// integers using multiplication", 1994).  m == 0 encodes d == 1.
struct Div31 {
    uint32_t m;
    uint32_t s;
};

struct RenderParams {
    SceneDev scene;
    // agents (SoA)
    const float* ax; const float* ay; const float* az0;
    const float* ac; const float* as; const float* al; const float* aw; const float* ah;
    const uint8_t* acls;
    int32_t A;          // agents per world
    int32_t C;          // cameras per agent
    // rig
    int32_t W, H;
    float fx, fy, cx, cy, nearp, farp;
    float mount[8][5];
    // derived constants
    float fx256, fy256, cx256, cy256, rfx, rfy, izfar, izcap;
    float cabs;         // max(|cx|, |cy|)
    float near_cull;    // near * (1 + 2^-8): boxes at least this far in front skip the near-plane case
    float near_off;     // -near * (1 - 2^-8): offset of the near frustum plane (with margin)
    float far_off;      // far * (1 + 2^-6): offset of the far frustum plane (with margin)
    float hx, hy;       // 0.5 - cx, 0.5 - cy
    int32_t pix_exact;  // 1: (i + 0.5) - cx equals i + hx exactly for every pixel index (same for y)
    uint32_t qbase;
    // tiling
    int32_t tile_w, tile_h, tiles_x, tiles_y;
    int64_t num_views;
    int64_t num_blocks;
    Div31 div_tiles, div_cams, div_agents;   // by tiles_x * tiles_y, C and A
    float rcs;          // 1 / cell size (rounded; used only with a one-cell margin)
    // outputs
    uint8_t* out_cls;
    float* out_depth;
    int32_t cull;       // 1: cell + triangle + box frustum culling
    int32_t vec_out;    // 1: output pointers are 16-byte aligned
    int32_t fast_decode; // 1: every decoded 1/z lies where the fast reciprocal is exact
    unsigned long long* stats;  // optional [kNumStats] work counters (null: off)
    // instance outputs (both null: off): [V][H][W] agent index within the world
    // of the visible surface or -1, and [V][A][2] footprint / visible pixels (zeroed before the launch)
    int32_t* out_inst;
    uint32_t* out_counts;
    // shaded RGB output (null: off), planar [V][3][H][W] uint8 (rule R13); when set,
    // box triangles carry their face in bits 4..6 of the class byte
    uint8_t* out_rgb;
    float rfar;         // 1 / far (rounded)
    int32_t aa;         // 1: colour antialiasing (R14; with out_rgb)
    // traffic lights (R10, R11), SoA [num_worlds * L]; L == 0: none
    const float* lx; const float* ly; const float* lz;
    const float* lcf; const float* lsf; const float* lr;
    const uint8_t* lcls;
    int32_t L;
    float lcos2;        // cos_max * cos_max (fp32)
    uint32_t* dev_err;  // context-owned device word: bits of kDevErr* OR-ed in by the kernels
    // the agents as the render kernels read them (pack_agents_kernel, run by
    // every render call first): agent g = w * A + a is apk[3g] = (x, y, z0,
    // height), apk[3g + 1] = (cos h, sin h, length, width), apk[3g + 2].x =
    // the class as bits; one pointer instead of nine keeps scalar registers free
    float4* apk;
};

// Device error bits (pictura_device_errors)
constexpr uint32_t kDevErrRingWait = 1u;   // a raster record reserved in the ring was never published


struct AgentStepParams {
    float* x; float* y; float* psi; float* speed; float* cos_h; float* sin_h;
    const float* length;
    const float* steer; const float* accel;
    float dt, vmax;
    int32_t count;
};

// Binning workspace (owned by the context).
struct BinWork {
    const float* verts;          // [T][9] original order
    const uint8_t* cls;          // [T]
    const uint32_t* prims;       // [P] first triangle of each primitive | kPrimFlagPair
    const int64_t* prim_offsets; // [nw + 1] (device): world w owns primitives [prim_offsets[w], prim_offsets[w+1])
    int64_t P;
    int32_t num_worlds;
    WorldGrid* grids;            // [nw]
    int64_t total_cells;
    float cell_size;
    uint32_t* home;              // [P]
    uint32_t* rank;              // [P]
    uint32_t* count;             // [cells + 1] -> exclusive scan -> cell_start
    uint32_t* aabb_bits;         // [cells][8] order-preserving bits (6 used)
    uint32_t* margin_bits;       // [nw]
    uint32_t* scan_tmp;          // block sums
    int64_t scan_tmp_len;
    float4* primA; float4* primB; float4* primC; float* primD;
    uint32_t* perm;              // [P] the primitive's entry of prims, in cell order
    float4* cell_lo; float4* cell_hi;
};

// prims[p]: index of the primitive's first input triangle, with this bit set
// when the primitive is the pair (that triangle, the next one)
constexpr uint32_t kPrimFlagPair = 0x80000000u;

hipError_t launch_render(const RenderParams& p, hipStream_t s);
// the production class/depth kernel alone, and the production instance (1) and
// one-sample colour (3) kernels: objects of their own, each built with its own
// scheduler setting
hipError_t launch_render_plain(const RenderParams& p, hipStream_t s);
hipError_t launch_render_side(const RenderParams& p, int mode, hipStream_t s);
hipError_t launch_bin(const BinWork& w, hipStream_t s);
hipError_t launch_agents_step(const AgentStepParams& p, hipStream_t s);
// Pack the num_worlds * A agents of p's SoA arrays into p.apk.
hipError_t launch_pack_agents(const RenderParams& p, int64_t count, hipStream_t s);
hipError_t launch_store_probe(void* dst, uint64_t bytes, hipStream_t s);
int64_t scan_tmp_needed(int64_t n);
hipError_t launch_rcp_check(uint32_t lo_bits, uint32_t n, unsigned long long* mismatches, hipStream_t s);

// Allocation-free variant: a file-scope device array of kNoAllocScratchWords
// 64-bit words per GPU (256 bytes); its address on `device` is taken once, by
// noalloc_scratch_init with that device current (pictura_create calls it).
constexpr int kNoAllocScratchWords = 32;
constexpr int kNoAllocMaxDevices = 64;
hipError_t noalloc_scratch_init(int device);
void* noalloc_scratch(int device);   // null before noalloc_scratch_init(device)
hipError_t launch_rcp_check_noalloc(uint32_t lo_bits, uint32_t n, unsigned long long* counter, hipStream_t s);

// Fill n 32-bit words at p with `value` on stream s (a kernel, so a caller
// may capture it in a graph).
hipError_t launch_fill_u32(uint32_t* p, size_t n, uint32_t value, hipStream_t s);

}  // namespace pictura
