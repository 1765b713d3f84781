/*
 * CPU oracle for the cached SqueezeNeRF renderer -- TEST INFRASTRUCTURE.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * may load or call this library.  It is a plain, slow, obviously correct
 * restatement of what the renderer computes, and shares no code with the HIP
 * path (no common headers, helpers or tables).
 *
 * What it computes, per pixel ray (SqueezeNeRF Sec. 3.1 Eq. 1-2, Sec. 3.2
 * Eq. 4, Sec. 3.3, Sec. 3.4):
 *   - a pinhole ray from the camera centre through the pixel centre
 *     (Sec. 3.1); for forward-facing captures (the LLFF scenes of Sec. 4)
 *     optionally mapped to normalized device coordinates, the NeRF
 *     convention the paper inherits;
 *   - N samples between the near and far planes (Sec. 3.1), uniform or
 *     stratified with a seeded SplitMix64 offset per bin;
 *   - nearest-neighbour lookup of sigma^j and (u^j, v^j, w^j) in the three
 *     position sub-caches (Sec. 3.4), fused by Eq. 4: sigma = product of the
 *     sigma^j, k = sum of the k^j; or, for the alternative decoder
 *     ("SqueezeNeRF (alt)", Sec. 3.2 Eq. 5), sigma^j a D_sigma-vector and
 *     sigma = max(0, W_sigma concat(sigma^j) + b_sigma),
 *     k = W_k concat(k^j) + b_k for each k in (u, v, w);
 *   - bilinear lookup of beta in the direction cache at (theta, phi)
 *     (Sec. 3.4);
 *   - colour c = sigmoid(beta^T (u, v, w)) (Eq. 2 followed by a sigmoid);
 *   - Eq. 1 compositing with transmittance T_i = exp(-sum_{j<i} sigma_j
 *     delta_j), accumulated in 2^-32 fixed point, and early termination once
 *     T_i < eps.
 *
 * Precision: every step that decides an integer (ray, sample position, grid
 * index, termination) is evaluated in IEEE binary32 with one rounding per
 * operation and no fused multiply-add, except the Eq. 5 density, which is
 * defined as chains of correctly rounded binary32 fused multiply-adds (see
 * oracle.c); colour, transmittance, weights and the sums are evaluated in
 * binary64.
 */
#ifndef SQN_ORACLE_H
#define SQN_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    int32_t n_p;            /* position grid size per axis (>= 2)            */
    int32_t D;              /* radiance components (>= 1)                     */
    int32_t n_theta;        /* direction grid, polar angle (>= 2)             */
    int32_t n_phi;          /* direction grid, azimuth (>= 2)                 */
    int32_t sigma_f16;      /* 1: sigma planes are binary16, 0: binary32      */
    int32_t uvw_f16;        /* 1: uvw planes are binary16, 0: binary32        */
    int32_t beta_f16;       /* 1: direction cache is binary16, 0: binary32    */
    int32_t stratified;     /* 1: one seeded offset per bin, 0: uniform       */
    float bmin[3], bmax[3]; /* scene box the position grids span              */
    float t_eps;            /* transmittance threshold; 0 disables stopping   */
    int32_t pad0;
    uint64_t seed;          /* stratified-sampling seed                       */
    const void* sigma[3];   /* [n_p][n_p] each, planes xy, yz, zx             */
                            /* ([n_p][n_p][d_sigma] when d_sigma > 0)         */
    const void* uvw[3];     /* [n_p][n_p][3D] each: u[0..D) v[0..D) w[0..D)   */
    const void* beta;       /* [n_theta][n_phi][D]                            */
    /* Eq. 5 decoder (used when d_sigma > 0), binary32: */
    int32_t d_sigma;        /* 0: Eq. 4; > 0: channels of each sigma^j        */
    float b_sigma;          /* density bias                                   */
    const float* w_sigma;   /* [3 d_sigma], columns in concat order xy,yz,zx  */
    const float* w_uvw;     /* [3][D][3D]: W_u, W_v, W_w, row-major           */
    const float* b_uvw;     /* [3][D]: b_u, b_v, b_w                          */
} oracle_scene;

typedef struct {
    float fx, fy, cx, cy;   /* pinhole intrinsics, pixels                     */
    int32_t width, height;
    float ndc_near;         /* > 0: march in normalized device coordinates    */
                            /* of the forward-facing camera (see oracle.c)    */
    int32_t pad;
} oracle_camera;

typedef struct {
    double rgb[3];          /* composited colour                              */
    double depth;           /* sum of w_i t_i (camera-z depth)                */
    double acc;             /* sum of w_i                                     */
    int64_t tau_end;        /* fixed-point optical depth when the ray stopped */
    uint32_t stop;          /* first non-live sample index, or N              */
    uint32_t n_inbox;       /* live samples inside the box                    */
    uint32_t n_occ;         /* live samples inside the box with sigma > 0     */
    uint32_t hash;          /* FNV-1a over (i, ix, iy, iz) of occupied samples */
} oracle_ray;

/* Renders the rays listed in ray_ids (ray id = (b*H + v)*W + u), or every
 * ray of the n_poses views when ray_ids is NULL, into out[n_rays].
 * poses: [n_poses][3][4] camera-to-world.  Returns 0, or -1 on bad input. */
int oracle_render(const oracle_scene* sc, const float* poses, int32_t n_poses,
                  const oracle_camera* cam, float near_t, float far_t,
                  int32_t n_samples, const int64_t* ray_ids, int64_t n_rays,
                  oracle_ray* out, int32_t n_threads);

/* floor(-ln(eps) * 2^32), or INT64_MAX for eps <= 0. */
int64_t oracle_tau_eps_q(float eps);

/* Exact value of an IEEE binary16 bit pattern. */
double oracle_half_to_double(uint16_t bits);

/* The counter-th output (0-based) of SplitMix64 started at state `seed`. */
uint64_t oracle_splitmix64(uint64_t seed, uint64_t counter);

#ifdef __cplusplus
}
#endif
#endif
