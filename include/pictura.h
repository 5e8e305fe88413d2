/*
 * pictura.h -- C ABI of the MI355X (gfx950) batched class/depth view rasterizer.
 *
 * The library renders, for every agent of every world and every camera of
 * the agent's rig, a perspective image of the surrounding agents' boxes and
 * the static map triangles (paper Sec. 3.2, Eq. obs_pv: I_ik = Phi(A_i, W_i,
 * K_ik); "only the surroundings are rendered", so a view never draws its own
 * agent).  Each pixel receives the class ID of the nearest surface (uint8)
 * and its view-space depth in metres (fp32, +inf for background).  Fixed
 * rules make the result independent of triangle order and of how the work is
 * split (all fp32 arithmetic without contraction, correctly rounded
 * divisions): R1 camera = agent pose composed with the mount (yaw only);
 * R2 view transform; R3 1/z plane of the unsnapped triangle; R4 Sutherland-
 * Hodgman clip against z = near, fanned from the first vertex, and a
 * triangle whose three vertices all lie beyond far (or all nearer than near)
 * is not drawn, since no point of it lies inside the view volume; R5 snap to
 * 1/256 pixel, ties to even; R6 exact integer edge functions at pixel
 * centres, top-left fill rule, two-sided; R7 key = (24-bit reverse depth from
 * the fp32 bits of 1/z, capped at the power of two above 1/near) << 8 | class,
 * the minimum key wins, 1/z below 1/far is rejected; R8 depth = 1 / the code's
 * bucket midpoint; R9 agent boxes of 12 triangles, the ego's own box skipped.
 *
 * Conventions
 *  - Plain C99; no HIP/CUDA or C++ types.  A `void* stream` is a hipStream_t
 *    (NULL = the device's null stream).  Device pointers are HIP device
 *    allocations on the context's device; host pointers are ordinary memory.
 *  - Every call returns a pictura_status.  Argument errors are detected on the
 *    host and returned synchronously without launching anything; the context
 *    stays usable after any error.  pictura_last_error() gives a message.
 *  - Work is enqueued on `stream` and the calls return without synchronising,
 *    except where a call says it copies to host memory.
 *  - A context is not thread-safe: use one context per host thread.
 *  - Every render call first copies the agents into a context-owned device
 *    buffer in the layout its kernels read (48 bytes per agent), so a render
 *    call on another stream than the previous render call of the context is
 *    ordered after that call's kernels (an event wait on the device, not a
 *    host synchronisation).  A call with more agents than any before it grows
 *    the buffer, which synchronises the device once.
 */
#ifndef PICTURA_H
#define PICTURA_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t pictura_status;
#define PICTURA_OK        0
#define PICTURA_EINVAL   (-1) /* bad argument (null pointer, size, rig value) */
#define PICTURA_ENOMEM   (-2) /* device allocation failed */
#define PICTURA_EDEVICE  (-3) /* no usable HIP device, or a HIP call failed */
#define PICTURA_ESTATE   (-4) /* call order violated (e.g. render before binning) */
#define PICTURA_ERANGE   (-5) /* a size exceeds a supported limit */

#define PICTURA_MAX_CAMS 8

typedef struct pictura_ctx_s* pictura_ctx;

/* Static scene of all worlds (host memory; the library copies it).
 * Triangles are concatenated world by world: world w owns triangles
 * [tri_offsets[w], tri_offsets[w+1]).  verts[t] = x0 y0 z0 x1 y1 z1 x2 y2 z2 in
 * world metres (z up).  cls[t] is the class ID (0..254).  bounds[w] =
 * xmin ymin xmax ymax is the rectangle the world's binning grid covers;
 * triangles outside it are still drawn (they are binned into edge cells). */
typedef struct {
    int32_t num_worlds;
    const int64_t* tri_offsets; /* host, [num_worlds + 1], non-decreasing, [0] == 0 */
    const float* verts;         /* host, [T][9] */
    const uint8_t* cls;         /* host, [T] */
    const float* bounds;        /* host, [num_worlds][4] */
} pictura_scene;

/* Agents (device memory, caller-owned, structure of arrays).  Agent
 * g = w * agents_per_world + a; (cos_h, sin_h) is its heading; the box spans
 * length x width around (x, y) and z0 .. z0 + height. */
typedef struct {
    int32_t num_worlds;
    int32_t agents_per_world;
    const float* x;
    const float* y;
    const float* z0;
    const float* cos_h;
    const float* sin_h;
    const float* length;
    const float* width;
    const float* height;
    const uint8_t* cls;
} pictura_agents;

/* Camera rig shared by all agents (host, by value).  Pinhole intrinsics in
 * pixels (x right, y down, pixel (i, j) centre at (i + 0.5, j + 0.5)); mount k
 * = x y z cos_yaw sin_yaw in the ego frame (x forward, y left, z up; paper
 * App. A.2, Tab. camera_rig).  near_m > 0, far_m > near_m. */
typedef struct {
    int32_t num_cams;
    int32_t width;
    int32_t height;
    float fx, fy, cx, cy;
    float near_m, far_m;
    float mount[PICTURA_MAX_CAMS][5];
} pictura_rig;

/* Mutable kinematic-bicycle state (device memory, caller-owned). */
typedef struct {
    int32_t count;
    float* x;
    float* y;
    float* psi;      /* heading angle, kept in (-pi, pi] */
    float* speed;    /* m/s */
    float* cos_h;    /* written: cos(psi) */
    float* sin_h;    /* written: sin(psi) */
    const float* length; /* wheelbase is 0.6 * length */
} pictura_agent_state;

/* Traffic lights (paper Sec. 3.2, rendering features: disks visible only
 * within a limited angular range, drawn for the approach they govern and
 * culled once the camera faces away).  Device memory, caller-owned, structure
 * of arrays; light l of world w has index w * lights_per_world + l.  A light
 * is a disk of radius `radius` centred at (x, y, z) whose normal is the
 * horizontal unit vector (cos_f, sin_f).  Rule R10: with d = C - centre (C
 * the camera centre of rule R1), h = cos_f * d.x + sin_f * d.y and
 * q = (d.x^2 + d.y^2) + d.z^2 (fp32, in this order), a view draws the light
 * iff h > 0 and h * h >= (cos_max * cos_max) * q.  Rule R11: the disk is 12
 * triangles (centre, rim k, rim k+1 mod 12), rim k = centre +
 * radius * (cos 30k deg * u + sin 30k deg * up) with u = (-sin_f, cos_f, 0),
 * up = (0, 0, 1), the cosines and sines rounded to fp32 and each coordinate
 * computed as x - (r cos) * sin_f, y + (r cos) * cos_f, z + r sin.  Its
 * pixels take class cls[l] (e.g. the signal state). */
typedef struct {
    int32_t num_worlds;
    int32_t lights_per_world;
    const float* x;
    const float* y;
    const float* z;
    const float* cos_f;
    const float* sin_f;
    const float* radius;
    const uint8_t* cls;
    float cos_max;   /* cosine of the visibility cone's half-angle, in [0, 1] */
} pictura_lights;

/* Create a context on HIP device `device`.  Returns PICTURA_EDEVICE when no
 * such device exists.  *out is set to NULL on failure. */
pictura_status pictura_create(int32_t device, pictura_ctx* out);

/* Release all device memory owned by the context.  NULL is ignored. */
void pictura_destroy(pictura_ctx ctx);

/* Message of the last error on this context ("" if none).  Owned by ctx. */
const char* pictura_last_error(pictura_ctx ctx);

/* Copy the static scene to device memory owned by the context (replacing any
 * previous scene and invalidating its bins).  Enqueued on `stream`; the host
 * arrays may be reused as soon as the call returns (the copy is staged).
 * EINVAL: null pointers, num_worlds < 1, offsets not non-decreasing, a class
 * ID of 255.  ERANGE: more than 2^31 - 1 triangles.  ENOMEM: allocation. */
pictura_status pictura_scene_upload(pictura_ctx ctx, const pictura_scene* scene, void* stream);

/* Build the uniform grid of every world: square cells of `cell_size_m`
 * metres covering the world's bounds (ceil(extent / cell) cells per axis);
 * each triangle belongs to the cell holding the centre of its xy bounding
 * box (clamped into the grid); each cell records its triangle range and the
 * 3-D bounding box of its triangles.  The library re-lays the triangles out
 * in cell order.  ESTATE: no scene.  EINVAL: cell_size_m not > 0.
 * ERANGE: more than 2^31 - 1 cells.  Enqueued on `stream`. */
pictura_status pictura_bin_scene(pictura_ctx ctx, float cell_size_m, void* stream);

/* Render all V = num_worlds * agents_per_world * num_cams views (paper
 * Sec. 3.2, Eq. obs_pv), with the traffic lights attached by
 * pictura_set_lights, if any.  View v = (w * agents_per_world + a) * num_cams + k
 * writes out_cls[v][y][x] (uint8 class; 4 = sky for background) and
 * out_depth[v][y][x] (fp32 view-space depth in metres, +inf for background),
 * row-major, y down.  Both outputs are caller-owned device buffers of
 * V * height * width elements.  ESTATE: scene not binned.  EINVAL: null
 * pointers, num_worlds different from the scene's, rig values out of range
 * (num_cams 1..8, width/height 1..4096, fx, fy > 0, 0 < near < far, far/near
 * small enough for the 24-bit depth key).  Asynchronous on `stream`. */
pictura_status pictura_render_views(pictura_ctx ctx, const pictura_agents* agents, const pictura_rig* rig,
                                    uint8_t* out_cls, float* out_depth, void* stream);

/* Render like pictura_render_views and also a shaded colour image (rule R13;
 * the paper's observations are RGB images, Sec. 3.2, rendering features: agents
 * are cuboids coloured per face with depth-aware brightness).  In this mode a
 * box triangle's visibility key carries a shading id, class | (face + 1) << 4
 * with face 0 bottom, 1 top, 2 back, 3 front, 4 right, 5 left (the order of
 * rule R9's triangles, two per face), in place of its class; every other
 * triangle keeps its class.  out_cls receives key & 15.  out_rgb[v][c][y][x]
 * (uint8, planar, c = red, green, blue): with base = palette[class] / 255
 * (class: R G B -- 0 ground 96 112 72, 1 road 72 72 78, 2 marking 232 232 224,
 * 3 vehicle 52 96 220, 4 sky 140 184 232, 5 curb 160 160 152, 6 pedestrian
 * 224 72 64, 7 wall 168 144 120, 8 red light 255 32 24, 9 amber 255 184 0,
 * 10 green 32 224 96, 11..15 128 128 128), factor = 0.45, 1, 0.55, 0.85, 0.7,
 * 0.7 for the faces bottom .. left and 1 for other surfaces, b = 1 - 0.6 *
 * min(z / far, 1) on box faces (z the output depth) and 1 elsewhere:
 * rint(255 * min(base * (factor * b), 1)), fp32 in this order.  One sample
 * per pixel (pictura_render_rgb_aa antialiases).  Device buffers, caller-owned:
 * out_rgb V*3*H*W bytes.  EINVAL as pictura_render_views, a null out_rgb, or a
 * scene class ID above 15 (agent and light classes are taken modulo 16).
 * Asynchronous on `stream`. */
pictura_status pictura_render_rgb(pictura_ctx ctx, const pictura_agents* agents, const pictura_rig* rig,
                                  uint8_t* out_cls, float* out_depth, uint8_t* out_rgb, void* stream);

/* pictura_render_rgb with analytic-coverage antialiasing at one sample per
 * pixel (rule R14; the paper's production renders smooth edges this way so
 * that thin structures such as lane lines stay visible at low resolution,
 * Sec. 3.2, rendering features, and App. on render quality).  out_cls and
 * out_depth are those of pictura_render_views (the pixel centre's surface).
 * A surface is a snapped 4-gon whose two fan pieces are both drawn and whose
 * turns all have one sign, none zero: a pair of scene triangles (a, b, c),
 * (a, c, d) of one class (see pictura_scene_upload) with all four vertices in
 * front of the near plane and neither triangle wholly beyond far, or a
 * triangle that the near clip turns into a 4-gon; otherwise each fan piece of
 * rule R6 is a surface of its own.  A surface leaves a fragment on every pixel
 * whose centre is within one pixel of its snapped bounding box and that it
 * covers in part: with E_k the edge function of R6 at the centre (no top-left
 * bias) and L_k the edge's length, both in subpixels, c_k = min(max(
 * fma(fl(E_k), fl(1 / (256 L_k)), 0.5), 0), 1), coverage a = min(max(((c_0 +
 * c_1) + c_2) - 2, 0), 1) for a triangle (edges v1->v2, v2->v0, v0->v1) and
 * min(max((((c_0 + c_1) + c_2) + c_3) - 3, 0), 1) for a 4-gon in positive
 * order (edges p_k->p_k+1), a8 = rint(255 a), fp32; the fragment exists when
 * 0 < a8 < 255 and the depth plane of the surface's first piece passes R7's
 * test at the centre.  A pixel keeps its nearest fragment, ordered by o =
 * (key >> 16) << 16 | (key & 255) << 8 | (255 - a8) with key the fragment's R7
 * key.  With key_c the pixel's final key, when o >> 16 <= key_c >> 16 (the
 * fragment is not behind the centre's surface) and (o >> 8) & 255 != key_c &
 * 255 (another shading id), the pixel's colour is (C_o * a8 + C_c * (255 -
 * a8) + 127) / 255 per channel in integers, C_o the R13 colour of the key
 * ((o >> 16) << 16) | ((o >> 8) & 255) and C_c that of key_c; otherwise C_c.
 * During the call the kernel keeps each pixel's nearest fragment in the words
 * of out_depth and writes the depths over them at the end, so out_depth must
 * not overlap out_cls or out_rgb.  Buffers, errors and ordering as
 * pictura_render_rgb. */
pictura_status pictura_render_rgb_aa(pictura_ctx ctx, const pictura_agents* agents, const pictura_rig* rig,
                                     uint8_t* out_cls, float* out_depth, uint8_t* out_rgb, void* stream);

/* Render like pictura_render_views (same out_cls, out_depth) and also the
 * instance visibility the paper's analysis reads from its renderer, each road
 * user's occlusion percentage (Sec. 5.2, "Grounding in What the Cameras
 * See": probes of the trained policy):
 *  - out_inst[v][y][x] (int32): the agent index a (0 .. agents_per_world - 1,
 *    within the view's world) whose box owns the pixel's visible surface: among
 *    the boxes with a fragment whose visibility key (rule R7) equals the pixel's
 *    final key, the lowest index; -1 where no box does (map geometry, traffic
 *    lights, sky).
 *  - out_counts[v][a][2] (uint32): footprint, the pixels agent a's box covers in
 *    view v when drawn alone (rules R2-R7, far plane included), and visible, the
 *    pixels of out_inst equal to a.  The ego's own entry is 0.  Occlusion
 *    fraction = 1 - visible / footprint.
 * Device buffers, caller-owned: out_inst V*H*W int32, out_counts
 * V*agents_per_world*2 uint32 (the library clears it on `stream` first).
 * After the class/depth pass the kernel draws the visible boxes in ascending
 * agent order; a pixel is claimed through one bit in the framebuffer's
 * padding and its owner stored straight into out_inst.  Errors as
 * pictura_render_views, and EINVAL for a null out_inst or out_counts.
 * Asynchronous on `stream`. */
pictura_status pictura_render_instances(pictura_ctx ctx, const pictura_agents* agents, const pictura_rig* rig,
                                        uint8_t* out_cls, float* out_depth, int32_t* out_inst,
                                        uint32_t* out_counts, void* stream);

/* Attach traffic lights (see pictura_lights) to the context: later
 * pictura_render_views calls draw them.  The context keeps the pointers, not
 * a copy: the arrays must stay valid while it renders, and their contents
 * may change between render calls (a signal changing state is a new cls
 * value, ordered on the render stream like any other input).  NULL, or
 * lights_per_world == 0, detaches.  EINVAL: num_worlds < 1, null arrays,
 * lights_per_world > 2^20, cos_max outside [0, 1]; a render call returns
 * EINVAL when num_worlds differs from its scene's.  ERANGE: more than
 * 2^31 - 1 lights.  No device work; synchronous. */
pictura_status pictura_set_lights(pictura_ctx ctx, const pictura_lights* lights);

/* One kinematic-bicycle step for every agent (the per-step agent motion of
 * the headline workload; the paper's simulation step is dt = 0.1 s, App. A.3,
 * Tab. hparams, and its agents follow a kinematic model whose exact form it
 * does not print, so the semi-implicit bicycle below is this library's
 * reading): v' = clamp(v + accel * dt, 0, vmax);
 * psi' = psi + v' / (0.6 length) * tan(steer) * dt wrapped into (-pi, pi];
 * x += v' cos(psi') dt; y += v' sin(psi') dt; cos_h/sin_h = cos/sin(psi').
 * steer[count] (radians) and accel[count] (m/s^2) are device arrays.
 * EINVAL: null pointers, count < 0, dt or vmax not finite.  Asynchronous. */
pictura_status pictura_agents_step(pictura_ctx ctx, const pictura_agent_state* state, const float* steer,
                                   const float* accel, float dt, float vmax, void* stream);

/* ---- introspection and test controls -------------------------------------- */

/* Reference for the achievable HBM write rate (the render's roofline is an
 * HBM write bound): writes `bytes` zero bytes to the device buffer dst with
 * 16-byte non-temporal stores, the store pattern of the render's write-out,
 * and nothing else.  dst must be 16-byte aligned and bytes a multiple of 16
 * (EINVAL otherwise); dst must hold at least `bytes` bytes.  Asynchronous on
 * `stream`: time it with events on that stream. */
pictura_status pictura_store_probe(pictura_ctx ctx, void* dst, uint64_t bytes, void* stream);

/* Grid geometry after pictura_bin_scene (host memory, synchronous: waits for
 * the binning to finish).  dims[w] = nx, ny; cell_base[w] = first cell of
 * world w (cell_base[num_worlds] = total cells); *total_prims = the number of
 * binned primitives.  A primitive is one input triangle, or a pair: input
 * triangles t and t + 1 of one world with the same class where t + 1 is
 * (a, c, d) for t = (a, b, c), bit for bit (a quad split along its diagonal),
 * paired greedily in input order.  The kernels cull and set up a pair once;
 * its two triangles are still drawn by the rules above, each with its own
 * depth plane.  Any pointer may be NULL. */
pictura_status pictura_bins_info(pictura_ctx ctx, int32_t* dims, int64_t* cell_base, int64_t* total_cells,
                                 int64_t* total_prims);

/* Copy the bins to host memory (synchronous).  cell_start[total_cells + 1]:
 * first re-laid-out primitive of each cell; cell_aabb[total_cells][6]: xmin
 * ymin zmin xmax ymax zmax of the cell's primitives (+inf/-inf when empty);
 * perm[total_prims]: for each re-laid-out primitive, the input index of its
 * first triangle, with bit 31 set for a pair. */
pictura_status pictura_bins_copy(pictura_ctx ctx, uint32_t* cell_start, float* cell_aabb, uint32_t* perm);

#define PICTURA_OPT_CULL   1 /* 1 (default): cell + triangle frustum culling; 0: every triangle of the world */
#define PICTURA_OPT_TILE   2 /* 0 (default): tiles of at most 64x64, split evenly over the view; n in 8..64: force n x n tiles (the last row and column ragged) */
#define PICTURA_OPT_STATS  3 /* 1: count the render kernel's work (cells, triangles, pixels); 0 (default): off */
/* Set a context option.  Images never depend on any option. */
pictura_status pictura_set_option(pictura_ctx ctx, int32_t option, int32_t value);

/* Copy the render kernel's accumulated work counters (PICTURA_OPT_STATS) to
 * host memory (synchronous): out[k], k < n, in this order: view tiles, cells
 * in the gathered rectangles, cells passing the rectangle prefilter, cells
 * passing the frustum test, triangles of those cells, boxes passing, box
 * triangles, first-pass survivors, exact batches, triangles clipped at near,
 * snapped triangles with pixels in the tile, of those rasterized by one lane,
 * pixels those lanes tested, triangles rasterized as records, of those on
 * the fp64 edge path, 8x8 blocks tested, blocks passing, first-pass
 * chunks of 64 candidates, then shader-clock cycles summed over waves spent
 * in:
 * prologue, cell and agent tests, first pass, exact pass (with records),
 * record raster (part of the exact pass), final barrier and write-out; then,
 * for the antialiased colour mode: surfaces whose fragments are evaluated
 * packed over the lanes, the window pixels and 64-pixel steps of those,
 * surfaces swept in 8x8 blocks, blocks swept, fragments written.
 * reset != 0 zeroes the counters. */
pictura_status pictura_stats_copy(pictura_ctx ctx, uint64_t* out, int32_t n, int32_t reset);

#define PICTURA_DEVERR_RING_WAIT 1u /* a raster record reserved in a view's record ring was never published */
/* Device-side errors the render kernels found (the kernels cannot return a
 * status): *out receives the OR of the PICTURA_DEVERR_* bits set by every
 * render call on this context since it was created or last reset; 0 means
 * none.  A set bit means an image may be incomplete (the kernel skipped the
 * work it could not do rather than hang).  Synchronous: waits for all work
 * on the context's device.  reset != 0 clears the word.  EINVAL: null out. */
pictura_status pictura_device_errors(pictura_ctx ctx, uint32_t* out, int32_t reset);

/* Device self-check of the reciprocal the kernels use in place of IEEE
 * division where |argument| lies in [2^-12, 2^20) (hardware reciprocal plus
 * one fused Newton step): *mismatches receives the number of fp32 values x
 * whose bit patterns lie in [lo_bits, lo_bits + count) for which it differs
 * from the correctly rounded 1.0f / x.  Synchronous.  EINVAL: null output or
 * a range reaching past the finite floats of lo_bits' sign. */
pictura_status pictura_selftest_rcp(pictura_ctx ctx, uint32_t lo_bits, uint32_t count, uint64_t* mismatches);

/* pictura_selftest_rcp without any device allocation, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, checks, result and
 * errors as pictura_selftest_rcp.  Its one piece of scratch, the 64-bit
 * mismatch counter, lives in a fixed 256-byte device array that the library
 * holds on every GPU it runs on until the process ends (its address is taken
 * by pictura_create); the counter does not grow with the range, so no range
 * the self-check accepts exceeds it.  The counter is cleared by a kernel at the
 * start of each call.  All contexts on one GPU share that array: calls that
 * overlap on the same GPU (from several host threads) race and may report
 * each other's counts.  ESTATE: the context's device has no scratch address.
 * Synchronous. */
pictura_status pictura_selftest_rcp_noalloc(pictura_ctx ctx, uint32_t lo_bits, uint32_t count, uint64_t* mismatches);

#ifdef __cplusplus
}
#endif

#endif /* PICTURA_H */
