/*
 * sqn.h -- C ABI of the MI355X (gfx950) cached SqueezeNeRF renderer.
 *
 * The library renders novel views from SqueezeNeRF caches (Wadhwani &
 * Kojima, "SqueezeNeRF: Further factorized FastNeRF for memory-efficient
 * inference", CVPR-W 2022).  For each pixel of each camera view it
 *   1. casts the pinhole ray through the pixel centre (Sec. 3.1),
 *   2. places N samples between the near and far planes (Sec. 3.1, 3.4),
 *   3. looks up sigma^j and (u^j, v^j, w^j) in the three factorized position
 *      sub-caches with nearest-neighbour lookup (Sec. 3.3, 3.4) and fuses
 *      them by Eq. 4 (sigma = product, k = sum over the planes) or, for
 *      caches made by sqn_create_linear_caches, by Eq. 5 (linear maps),
 *   4. looks up beta in the direction cache with bilinear interpolation
 *      (Sec. 3.4),
 *   5. forms colour c = sigmoid(beta^T (u, v, w)) (Eq. 2, then a sigmoid),
 *   6. composites colour and depth along the ray by Eq. 1, stopping once the
 *      transmittance T_i falls below eps.
 *
 * Conventions (not fixed by the paper; chosen here and used throughout):
 *   - pose: row-major 3x4 camera-to-world [R | c] in binary32; the camera
 *     looks down its -z axis, +x is right, +y is up;
 *   - pixel (u, v) is sampled at its centre (u + 1/2, v + 1/2); v = 0 is the
 *     top row; outputs are row-major [B][H][W];
 *   - the ray direction is d = R (a, b, -1) with a = (u + 1/2 - cx) / fx and
 *     b = -(v + 1/2 - cy) / fy, not normalised, so the sample parameter t is
 *     depth along the camera axis and near/far are planes;
 *   - uniform samples sit at t_i = near + i (far - near) / N; stratified
 *     samples at t_i = near + (i + xi_i) (far - near) / N with xi_i taken
 *     from SplitMix64 (counter = ray id * N + i, ray id = (b H + v) W + u);
 *   - delta_i = max(0, t_{i+1} - t_i) |d| with t_N = far;
 *   - plane j in (xy, yz, zx) is indexed [first axis][second axis]; grid
 *     nodes are vertex-aligned over the box (node 0 on bbox_min, node n_p-1
 *     on bbox_max); nearest node = floor(g + 1/2) clamped, g = (p - bmin)
 *     (n_p - 1) / (bmax - bmin); samples outside the box have sigma = 0;
 *   - sigma = max(0, (sigma^xy sigma^yz) sigma^zx) (Eq. 4; Eq. 5: see
 *     sqn_linear_decoder);
 *   - direction cache: theta = polar angle from world +z on n_theta nodes
 *     spanning [0, pi] (clamped), phi = atan2(d_y, d_x) on n_phi periodic
 *     nodes at -pi + b 2 pi / n_phi;
 *   - the optical depth before sample i is accumulated exactly in 64-bit
 *     fixed point (units of 2^-32, per-sample term truncated and capped at
 *     2^16); sample i is evaluated iff that sum is <= floor(-ln(eps) 2^32),
 *     i.e. T_i >= eps; eps = 0 disables termination;
 *   - no background colour; depth is sum_i w_i t_i (0 for empty rays).
 * Ray positions, sample positions, grid indices and termination decisions
 * are evaluated in IEEE binary32 with one rounding per operation and no
 * fused multiply-add, so they are reproducible bit for bit on any IEEE
 * implementation; colour, transmittance and the sums are binary32 with
 * binary64 accumulation.
 *
 * Threading and streams: every call is asynchronous on the given HIP stream
 * (NULL = the default stream) unless stated; a cache handle is read-only
 * while rendering, so renders on several streams may share one handle.
 * Device faults surface at the caller's next synchronisation.
 */
#ifndef SQN_H
#define SQN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    SQN_OK = 0,
    SQN_ERR_INVALID_ARG = 1,    /* argument out of range, bad pointer or size  */
    SQN_ERR_OUT_OF_MEMORY = 2,  /* device allocation failed                     */
    SQN_ERR_DEVICE = 3,         /* a HIP call or kernel launch failed           */
    SQN_ERR_UNSUPPORTED = 4     /* valid but not supported by this build        */
} sqn_status;

typedef enum { SQN_F32 = 0, SQN_F16 = 1 } sqn_dtype;

/* Opaque, library-owned device copy of the caches. */
typedef struct sqn_caches sqn_caches;

/* Cache description (Sec. 3.3).  The paper stores sigma^j in fp32 and
 * u^j, v^j, w^j and beta in fp16; each dtype is chosen independently. */
typedef struct {
    int32_t n_p;          /* position grid nodes per axis, 2..8192            */
    int32_t D;            /* radiance components per colour channel, 1..32    */
    int32_t n_theta;      /* direction grid, polar angle, >= 2                */
    int32_t n_phi;        /* direction grid, azimuth, >= 2                    */
    int32_t sigma_dtype;  /* sqn_dtype of the sigma^j planes                  */
    int32_t uvw_dtype;    /* sqn_dtype of the u^j, v^j, w^j planes            */
    int32_t beta_dtype;   /* sqn_dtype of the direction cache                 */
    int32_t stratified;   /* 0: uniform samples, 1: one seeded offset per bin */
    float bbox_min[3];    /* scene box spanned by the position grids          */
    float bbox_max[3];    /* (bbox_min < bbox_max on every axis, finite)      */
    float t_eps;          /* transmittance threshold in [0, 1]; 0 = no stop   */
    int32_t reserved;     /* must be 0                                        */
    uint64_t seed;        /* stratified-sampling seed                         */
} sqn_cache_desc;

/* Pinhole intrinsics in pixels, shared by every view of a call. */
typedef struct {
    float fx, fy, cx, cy;
    int32_t width, height;
} sqn_intrinsics;

/* Copy the caches into library-owned device memory on the current device.
 *   sigma_planes[j]: device pointer, [n_p][n_p] of sigma_dtype, planes in the
 *                    order xy, yz, zx (Sec. 3.2), indexed [first][second];
 *   uvw_planes[j]:   device pointer, [n_p][n_p][3D] of uvw_dtype, each texel
 *                    u[0..D) then v[0..D) then w[0..D) (Eq. 3 outputs);
 *   beta:            device pointer, [n_theta][n_phi][D] of beta_dtype;
 *   stream:          hipStream_t the copies are ordered on; the call waits
 *                    for them, so the caller may free its arrays on return.
 * Values must be finite.  On success *out owns the copy (free it with
 * sqn_destroy); on failure *out is NULL and nothing is leaked.
 * Errors: SQN_ERR_INVALID_ARG (NULL pointer, range, a pointer that is not
 * HIP device memory or whose allocation is smaller than the array),
 * SQN_ERR_UNSUPPORTED (a uvw plane or the direction cache of 2^32 bytes or
 * more: the kernels address them with 32-bit offsets),
 * SQN_ERR_OUT_OF_MEMORY, SQN_ERR_DEVICE. */
sqn_status sqn_create_caches(const sqn_cache_desc* desc,
                             const void* const sigma_planes[3],
                             const void* const uvw_planes[3],
                             const void* beta,
                             void* stream,
                             sqn_caches** out);

/* Parameters of the alternative decoder "SqueezeNeRF (alt)" (Sec. 3.2
 * Eq. 5), binary32, in host memory:
 *   sigma = max(0, W_sigma concat(sigma^xy, sigma^yz, sigma^zx) + b_sigma),
 *   k     = W_k concat(k^xy, k^yz, k^zx) + b_k   for k in (u, v, w),
 * with each sigma^j a d_sigma-vector (the paper uses 12) and each k^j a
 * D-vector.  The max(0, .) keeps Eq. 1's density non-negative (the paper
 * states no activation).  The binary32 density is evaluated as: for each
 * plane j, s^j = a chain of fused multiply-adds over its channels in order,
 * starting from zero (s = fma(W_sigma[j d_sigma + c], sigma^j[c], s)); then
 * ((s^xy + s^yz) + s^zx) + b_sigma, each sum rounded; a NaN counts as 0. */
typedef struct {
    int32_t d_sigma;        /* channels of each sigma^j, 1..64                 */
    float b_sigma;          /* density bias                                    */
    const float* w_sigma;   /* [3 d_sigma], columns in concat order xy, yz, zx */
    const float* w_uvw;     /* [3][D][3D]: W_u, W_v, W_w, row-major            */
    const float* b_uvw;     /* [3][D]: b_u, b_v, b_w                           */
} sqn_linear_decoder;

/* sqn_create_caches for the Eq. 5 decoder.
 *   decoder:         host pointer, read during the call only;
 *   sigma_planes[j]: device pointer, [n_p][n_p][d_sigma] of desc->sigma_dtype
 *                    (the paper stores every alt cache value in fp16);
 *   uvw_planes, beta, stream, out: as for sqn_create_caches.
 * The handle keeps, per plane texel, s^j in binary32 (the channels are
 * folded with W_sigma here) and the radiance weights; renders use four lanes
 * per ray.  Weights and biases must be finite.
 * Errors: as sqn_create_caches, plus SQN_ERR_INVALID_ARG for a NULL or
 * non-finite decoder parameter or d_sigma outside [1, 64]. */
sqn_status sqn_create_linear_caches(const sqn_cache_desc* desc,
                                    const sqn_linear_decoder* decoder,
                                    const void* const sigma_planes[3],
                                    const void* const uvw_planes[3],
                                    const void* beta,
                                    void* stream,
                                    sqn_caches** out);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, serving loops that swap scenes, harnesses that forbid hipMalloc):
 * sqn_create_caches into the device memory an existing handle already owns,
 * allocating nothing.  The handle (made by sqn_create_caches, Eq. 4) then
 * holds the caches desc describes; its lanes, leap and NDC settings stay.
 *   caches:      the handle; its device block must hold the new layout
 *                (sqn_cache_device_bytes of a handle created from desc);
 *   desc, sigma_planes, uvw_planes, beta: as for sqn_create_caches, with
 *                n_p <= 2048;
 *   stream:      hipStream_t the work is ordered on.
 * Unlike sqn_create_caches the call does not wait: the input arrays must
 * stay valid, and no render with the handle may run on another stream, until
 * the stream has finished the call's work; renders on `stream` after it see
 * the new caches.  The preparation uses a 20 MiB scratch array that each
 * device holds for the life of the process and that every call on that
 * device shares: calls on one device that overlap in time (two streams, two
 * threads) race on it and must be serialised by the caller.
 * Errors: SQN_ERR_INVALID_ARG (NULL, range, n_p > 2048, a layout larger than
 * the handle's block, input arrays that are not device allocations large
 * enough, wrong device), SQN_ERR_UNSUPPORTED (a handle made by
 * sqn_create_linear_caches, or a uvw plane or direction cache of 2^32 bytes
 * or more), SQN_ERR_DEVICE (a launch failed: the handle's contents are then
 * unspecified; destroy it or recreate it again). */
sqn_status sqn_recreate_caches(sqn_caches* caches, const sqn_cache_desc* desc,
                               const void* const sigma_planes[3],
                               const void* const uvw_planes[3],
                               const void* beta,
                               void* stream);

/* Render n_poses views (Sec. 3.4, Eq. 1).
 *   poses:      device pointer, [n_poses][3][4] binary32 camera-to-world;
 *   intrinsics: host pointer, read during the call only;
 *   near_plane < far_plane, both finite; 1 <= n_samples <= 32768;
 *   rgb_out:    device pointer, [n_poses][H][W][3] binary32, written;
 *   depth_out:  device pointer, [n_poses][H][W] binary32, written; may be NULL;
 *   stream:     hipStream_t the kernel is launched on.
 * n_poses == 0 is a no-op.  Allocates nothing; returns before the kernel
 * finishes.  The handle must belong to the current device.
 * Errors: SQN_ERR_INVALID_ARG (as above; output or pose buffers that are
 * not device allocations large enough; more than 2^31-1 rays),
 * SQN_ERR_DEVICE (launch failure). */
sqn_status sqn_render(const sqn_caches* caches,
                      const float* poses, int32_t n_poses,
                      const sqn_intrinsics* intrinsics,
                      float near_plane, float far_plane, int32_t n_samples,
                      float* rgb_out, float* depth_out,
                      void* stream);

/* sqn_render plus per-ray diagnostics for bit-exact checks:
 *   ray_stats: device pointer, [n_poses][H][W][4] uint32, written with
 *     { stop:    first sample index that is not evaluated (T_i < eps), or N;
 *       n_inbox: evaluated samples inside the box;
 *       n_occ:   evaluated samples inside the box with sigma > 0;
 *       hash:    32-bit FNV-1a over the little-endian words (i, ix, iy, iz)
 *                of the occupied samples in order of i }.
 * rgb_out may be NULL here.  Slower than sqn_render. */
sqn_status sqn_render_stats(const sqn_caches* caches,
                            const float* poses, int32_t n_poses,
                            const sqn_intrinsics* intrinsics,
                            float near_plane, float far_plane, int32_t n_samples,
                            float* rgb_out, float* depth_out,
                            uint32_t* ray_stats,
                            void* stream);

/* Launch shape of later renders with this handle: how many lanes of a
 * wavefront share one ray (1, 4 or 8; the L lanes take the L consecutive
 * samples of a chunk), or 0 (the default) to choose per call from the number
 * of rays (8 below 2^18 rays, 4 below 2^20, else 1).  Sample, index and
 * termination decisions are identical for every choice; colour and depth
 * agree up to the rounding of their sums.  Not thread-safe against
 * concurrent renders with the handle.
 * Errors: SQN_ERR_INVALID_ARG; SQN_ERR_UNSUPPORTED for 1 or 8 on a handle
 * made by sqn_create_linear_caches (always four lanes). */
sqn_status sqn_set_lanes_per_ray(sqn_caches* caches, int32_t lanes);

/* Hybrid launch of single views: the centred rectangle of blocks of 16 x 16
 * pixels spanning `fraction` of the image's blocks along each axis marches
 * with four lanes per ray (its workgroups are dispatched first), every other
 * block with one lane per ray.  The long chains of samples over a centred
 * object then end four times sooner while the rest of the image costs a
 * quarter of the instructions.  Applies to one view at a time on a handle
 * from sqn_create_caches with empty-space skipping and world rays; other
 * renders use the lanes-per-ray setting.  0 (the default) turns it off;
 * sqn_set_lanes_per_ray also turns it off.  Sample, index and termination
 * decisions are identical for every choice.  Not thread-safe against
 * concurrent renders with the handle.
 * Errors: SQN_ERR_INVALID_ARG for a fraction outside [0, 1] or a NULL
 * handle; SQN_ERR_UNSUPPORTED for a fraction > 0 on a handle made by
 * sqn_create_linear_caches. */
sqn_status sqn_set_centre_block(sqn_caches* caches, float fraction);

/* Measure the launch shapes on one batch and keep the fastest: renders the
 * batch (arguments as sqn_render) with 4, 1 and 8 lanes per ray and, for a
 * single view where sqn_set_centre_block applies, with hybrid launches of
 * centred fractions 0.15, 0.5 and 1 (four lanes only for a handle made by
 * sqn_create_linear_caches): each twice untimed, then in four rounds that
 * each render every candidate once untimed and 5 times between two HIP
 * events on `stream` (the rounds spread the drift of the GPU's clocks as
 * they settle over all candidates), then keeps the fastest (least total
 * time) as sqn_set_lanes_per_ray
 * and sqn_set_centre_block would, and writes the choice to lanes_out (the
 * lanes per ray, or -1 for a hybrid launch) and centre_out (the hybrid
 * fraction, 0 otherwise) where they are not NULL (for an empty batch the
 * settings stay and nothing is written).  No candidate changes a sample, index or
 * termination decision, only the time; which is fastest depends on the
 * image size, the number of views and the scene (the chains of samples),
 * which the default per-call choice sees only through the number of rays.
 * A single view deals its tiles in blocks of 2 x 2 from the centre of the
 * image outwards.  rgb_out and depth_out receive a render of
 * the batch.  Blocks until the timed renders finish; creates two HIP events
 * and allocates no device memory.  Not thread-safe against concurrent
 * renders with the handle.  Errors: those of sqn_render (the handle's
 * settings are then left as they were); SQN_ERR_DEVICE if the events
 * fail. */
sqn_status sqn_tune_lanes_per_ray(sqn_caches* caches, const float* poses, int32_t n_poses,
                                  const sqn_intrinsics* intrinsics, float near_plane, float far_plane,
                                  int32_t n_samples, float* rgb_out, float* depth_out, void* stream,
                                  int32_t* lanes_out, float* centre_out);

/* Leaps over empty space (1, the default) or a dense march (0).  sigma is
 * the product of the three planar sigma^j (Sec. 3.2 Eq. 4), so it vanishes
 * wherever one plane does; sqn_create_caches stores, next to each sigma^j,
 * the Chebyshev distance to the nearest texel with sigma^j != 0 (capped at
 * 255), and the march skips every sample whose texel in some plane stays
 * within that empty square.  For the Eq. 5 decoder a texel of plane j counts
 * as empty when its s^j plus the largest s^k the other two planes hold along
 * the row or column the texel shares with them, plus b_sigma, is <= 0 in the
 * same binary32 order, and a 3-D grid of cells (at most 128 per axis) marks a
 * cell empty when the three planes' largest s^j over its footprint, summed
 * with b_sigma in that order, is <= 0; a sample in an empty cell reads no
 * plane and leaps out of the empty cube around it.  Leaps land on the first
 * sample that may lie past the proven-empty run.  Only samples with
 * sigma = 0 are skipped, so results, sample counts and termination are those
 * of the dense march.
 * Errors: SQN_ERR_INVALID_ARG. */
sqn_status sqn_set_empty_space_skipping(sqn_caches* caches, int32_t enable);

/* ---- cache generation (Sec. 3.3; network shapes of Sec. 3.4) --------------
 *
 * The caches are the outputs of the trained networks on grids: each position
 * network F_pos^j on its plane's n_p x n_p vertex-aligned nodes over the
 * scene box (plane j = (first, second) axes of xy, yz, zx, indexed
 * [first][second]), the direction network F_dir on the n_theta x n_phi
 * direction nodes (theta_a = a pi / (n_theta - 1) from +z, phi_b =
 * -pi + b 2 pi / n_phi).  Inputs are NeRF's positional encoding, per
 * component c of the input: [c, then for k = 0..L-1: sin(2^k pi c),
 * cos(2^k pi c)], interleaved over the components per frequency, i.e.
 * [a, b, sin(pi a), sin(pi b), cos(pi a), cos(pi b), sin(2 pi a), ...].
 * Hidden layers apply ReLU, the last layer is linear.  F_pos^j emits
 * (sigma_0, w_sigma, w_u[D], u_0[D], w_v[D], v_0[D], w_w[D], w_0[D]) (the
 * order of Sec. 3.2) and the cache stores Eq. 3's sigma^j = sigma_0 w_sigma
 * and k^j = w_k * k_0; F_dir emits beta[D].
 * Arithmetic: binary16 weights and activations, binary32 accumulation,
 * biases, Eq. 3 products and outputs before their storage dtype. */

/* One network, host memory read during sqn_create_networks only. */
typedef struct {
    int32_t n_hidden;                 /* hidden layers, 1..16                         */
    int32_t width;                    /* units per hidden layer: 256 for F_pos^j, 128  */
                                      /* for F_dir (the sizes of Sec. 3.4)            */
    int32_t n_in;                     /* encoding size: 2 (1 + 2 pos_freq) or          */
                                      /* 3 (1 + 2 dir_freq), at most 64               */
    int32_t n_out;                    /* 2 + 6D for F_pos^j, D for F_dir               */
    const uint16_t* const* weights;   /* n_hidden + 1 binary16 matrices [out][in]      */
    const float* const* biases;       /* n_hidden + 1 binary32 vectors [out]           */
} sqn_mlp_desc;

/* Opaque, library-owned device copy of the four networks. */
typedef struct sqn_networks sqn_networks;

/* Upload the networks (pos[j] for planes xy, yz, zx, and dir) for outputs of
 * D components, with pos_freq / dir_freq encoding frequencies (NeRF: 10, 4).
 * Weights must be finite.  The call waits for its copies; *out is NULL on
 * failure.  Errors: SQN_ERR_INVALID_ARG (NULL, sizes, non-finite values),
 * SQN_ERR_UNSUPPORTED (other widths), SQN_ERR_OUT_OF_MEMORY,
 * SQN_ERR_DEVICE. */
sqn_status sqn_create_networks(const sqn_mlp_desc pos[3], const sqn_mlp_desc* dir,
                               int32_t D, int32_t pos_freq, int32_t dir_freq,
                               void* stream, sqn_networks** out);

/* Evaluate the networks on the grids desc describes (n_p, n_theta, n_phi,
 * D, bbox and the three dtypes; the sampling fields are ignored) and write
 * the caches in the layout sqn_create_caches reads:
 *   sigma_planes[j]: device, [n_p][n_p] of sigma_dtype;
 *   uvw_planes[j]:   device, [n_p][n_p][3D] of uvw_dtype;
 *   beta:            device, [n_theta][n_phi][D] of beta_dtype.
 * Asynchronous on `stream`; allocates nothing.  The handle keeps one
 * encoding table, so generations with one handle must not overlap.
 * Errors: SQN_ERR_INVALID_ARG (desc, D mismatch, output buffers that are
 * not device allocations large enough, wrong device), SQN_ERR_DEVICE. */
sqn_status sqn_generate_caches(sqn_networks* nets, const sqn_cache_desc* desc,
                               void* const sigma_planes[3], void* const uvw_planes[3],
                               void* beta, void* stream);

/* Bytes of device memory the networks handle owns. */
size_t sqn_networks_device_bytes(const sqn_networks* nets);

/* Free the networks; NULL is a no-op. */
void sqn_destroy_networks(sqn_networks* nets);

/* Ray space of later renders with this handle.  ndc_near = 0 (the default):
 * world rays as above.  ndc_near > 0: forward-facing captures (the LLFF
 * scenes the paper evaluates, Sec. 4), marched as in NeRF in the normalized
 * device coordinates of the pinhole camera looking down -z with near plane
 * ndc_near: a world point (x, y, z) maps to (-(fx/(W/2)) x/z,
 * -(fy/(H/2)) y/z, 1 + 2 ndc_near/z), so the frustum beyond the near plane
 * is [-1, 1]^3 (the caches' box).  Each ray is moved to its point on the
 * near plane, t_s = -(ndc_near + o_z)/d_z, and becomes o' + t' d'; near and
 * far of sqn_render are then t' bounds (0 and 1 span near plane to
 * infinity), delta_i uses |d'|, depth_out is sum w_i t'_i, and beta is
 * still looked up along the world direction.  Rays with d_z >= 0 have no
 * samples.  Binary32, one rounding per operation:
 *   o' = (-(sx (o_x/o_z)), -(sy (o_y/o_z)), 1 + (2n)/o_z),
 *   d' = (-(sx (d_x/d_z - o_x/o_z)), -(sy (d_y/d_z - o_y/o_z)), -((2n)/o_z)),
 *   sx = fx/(0.5 W), sy = fy/(0.5 H), o after the move.
 * Not thread-safe against concurrent renders with the handle.
 * Errors: SQN_ERR_INVALID_ARG (NULL, negative or non-finite). */
sqn_status sqn_set_ndc(sqn_caches* caches, float ndc_near);

/* Bytes of device memory the handle owns. */
size_t sqn_cache_device_bytes(const sqn_caches* caches);

/* Free the handle and its device memory; NULL is a no-op.  The caller must
 * ensure no render using the handle is still running. */
void sqn_destroy(sqn_caches* caches);

/* Static description of a status code. */
const char* sqn_status_string(sqn_status status);

/* Detail of the last failure on the calling thread ("" if none). */
const char* sqn_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* SQN_H */
