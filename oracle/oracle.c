/*
 * CPU oracle for the cached SqueezeNeRF renderer -- TEST INFRASTRUCTURE.
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg use it.
 * See oracle.h for what is computed and in which precision.
 *
 * Build: gcc -O2 -std=c11 -ffp-contract=off -fPIC -shared -pthread (no
 * fast-math, no target-specific flags), so every binary32 operation below
 * rounds exactly once as written.
 */
#include "oracle.h"

#include <math.h>
#include <pthread.h>
#include <stdlib.h>
#include <string.h>

#ifndef M_PI
#define M_PI 3.14159265358979323846
#endif

/* ---- small definitions the renderer's inputs need ---------------------- */

/* IEEE 754 binary16: sign, 5-bit exponent (bias 15), 10-bit fraction. */
double oracle_half_to_double(uint16_t bits)
{
    int sign = (bits >> 15) & 1;
    int e = (bits >> 10) & 0x1f;
    int f = bits & 0x3ff;
    double v;
    if (e == 0)
        v = ldexp((double)f, -24);                 /* zero / subnormal */
    else if (e == 31)
        v = f ? NAN : INFINITY;
    else
        v = ldexp((double)(1024 + f), e - 25);     /* (1 + f/1024) 2^(e-15) */
    return sign ? -v : v;
}

/* SplitMix64 (Steele, Lea, Flood, OOPSLA 2014): the state advances by the
 * golden-ratio increment and each output is a 64-bit finaliser of the state.
 * The counter-th output of a generator started at `seed` is therefore the
 * finaliser of seed + (counter + 1) * increment. */
uint64_t oracle_splitmix64(uint64_t seed, uint64_t counter)
{
    uint64_t z = seed + (counter + 1) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* Transmittance threshold in 2^-32 fixed-point optical depth:
 * T >= eps  <=>  tau <= -ln(eps). */
int64_t oracle_tau_eps_q(float eps)
{
    if (!(eps > 0.0f))
        return INT64_MAX;
    double x = -log((double)eps) * 4294967296.0;
    if (x <= 0.0)
        return 0;
    return (int64_t)floor(x);
}

static float cache_value(const void* base, int is_f16, size_t idx)
{
    if (is_f16)
        return (float)oracle_half_to_double(((const uint16_t*)base)[idx]);
    return ((const float*)base)[idx];
}

static double cache_value64(const void* base, int is_f16, size_t idx)
{
    if (is_f16)
        return oracle_half_to_double(((const uint16_t*)base)[idx]);
    return (double)((const float*)base)[idx];
}

/* FNV-1a (32-bit) over the little-endian bytes of one 32-bit word. */
static uint32_t fnv1a_word(uint32_t h, uint32_t x)
{
    for (int k = 0; k < 4; ++k) {
        h ^= (x >> (8 * k)) & 0xffu;
        h *= 16777619u;
    }
    return h;
}

/* ---- Eq. 5, the alternative ("alt") decoder ----------------------------- */

/* Density: sigma = W_sigma concat(sigma^xy, sigma^yz, sigma^zx) + b_sigma,
 * then max(0, .) so that Eq. 1 sees a non-negative density.  The binary32
 * evaluation order is fixed here because sigma decides the optical depth and
 * hence termination (the paper gives none): for each plane the partial dot
 * product of its D_sigma channels with its block of W_sigma, as a chain of
 * correctly rounded fused multiply-adds starting from zero in channel order;
 * then the three partial sums added in plane order; then the bias.  A NaN
 * sum counts as zero density. */
static float alt_sigma(const oracle_scene* sc, const size_t texel[3])
{
    const int32_t ds = sc->d_sigma;
    float part[3];
    for (int j = 0; j < 3; ++j) {
        float s = 0.0f;
        for (int32_t c = 0; c < ds; ++c) {
            float f = cache_value(sc->sigma[j], sc->sigma_f16, texel[j] * (size_t)ds + c);
            s = fmaf(sc->w_sigma[j * ds + c], f, s);
        }
        part[j] = s;
    }
    float pre = part[0] + part[1];
    pre = pre + part[2];
    pre = pre + sc->b_sigma;
    return pre > 0.0f ? pre : 0.0f;
}

/* Colour logits (binary64): for each channel k in (u, v, w) the decoded
 * vector k = W_k concat(k^xy, k^yz, k^zx) + b_k (Eq. 5), then its inner
 * product with beta (Eq. 2). */
static void alt_logits(const oracle_scene* sc, const size_t rec[3], const double* beta,
                       double x[3])
{
    const int32_t D = sc->D;
    for (int c = 0; c < 3; ++c) {
        const float* W = sc->w_uvw + (size_t)c * D * 3 * D;
        double sum = 0.0;
        for (int32_t d = 0; d < D; ++d) {
            double k = (double)sc->b_uvw[c * D + d];
            for (int j = 0; j < 3; ++j)
                for (int32_t e = 0; e < D; ++e) {
                    double f = cache_value64(sc->uvw[j], sc->uvw_f16, rec[j] + (size_t)c * D + e);
                    k += (double)W[(size_t)d * 3 * D + (size_t)j * D + e] * f;
                }
            sum += beta[d] * k;
        }
        x[c] = sum;
    }
}

/* ---- normalized device coordinates ------------------------------------- */

/* Forward-facing captures (LLFF) are marched in the normalized device
 * coordinates of a pinhole camera looking down -z with near plane n: a world
 * point (x, y, z), z < 0, maps to
 *   x' = -(fx / (W/2)) x / z,  y' = -(fy / (H/2)) y / z,  z' = 1 + 2 n / z,
 * so the frustum from z = -n to infinity becomes [-1, 1]^3 and straight
 * lines stay straight.  The ray o + t d is first moved to its point on the
 * near plane (t_s = -(n + o_z) / d_z); in these coordinates it is then
 * o' + t' d' with t' in [0, 1) from the near plane to infinity:
 *   o' = (-(sx) o_x/o_z, -(sy) o_y/o_z, 1 + 2n/o_z),
 *   d' = (-(sx) (d_x/d_z - o_x/o_z), -(sy) (d_y/d_z - o_y/o_z), -2n/o_z),
 * sx = fx / (W/2), sy = fy / (H/2).  A ray with d_z >= 0 never reaches the
 * near plane and has no samples.  Binary32, one rounding per operation, in
 * the order written.  Returns 0 for a ray without samples. */
static int ndc_ray(const oracle_camera* cam, float o[3], float d[3])
{
    const float n = cam->ndc_near;
    if (!(d[2] < 0.0f))
        return 0;
    float ts = -(n + o[2]) / d[2];
    float os[3];
    for (int r = 0; r < 3; ++r) {
        float td = ts * d[r];
        os[r] = o[r] + td;
    }
    const float sx = cam->fx / (0.5f * (float)cam->width);
    const float sy = cam->fy / (0.5f * (float)cam->height);
    const float oxz = os[0] / os[2], oyz = os[1] / os[2];
    const float dxz = d[0] / d[2], dyz = d[1] / d[2];
    const float n2 = 2.0f * n;
    const float n2z = n2 / os[2];
    o[0] = -(sx * oxz);
    o[1] = -(sy * oyz);
    o[2] = 1.0f + n2z;
    d[0] = -(sx * (dxz - oxz));
    d[1] = -(sy * (dyz - oyz));
    d[2] = -n2z;
    return 1;
}

/* ---- one ray ------------------------------------------------------------ */

typedef struct {
    const oracle_scene* sc;
    const float* poses;
    const oracle_camera* cam;
    float near_t, far_t;
    int32_t N;
    int64_t tau_eps;
    float scale[3];       /* (n_p - 1) / (bmax - bmin) per axis, binary32 */
    float dt;             /* (far - near) / N, binary32 */
} job_t;

/* Sample position t_i along the ray, in the camera-z units of the near and
 * far planes: the left end of bin i, or a seeded point inside bin i. */
static float sample_t(const job_t* J, int64_t ray_id, int32_t i)
{
    float x = (float)i;
    if (J->sc->stratified) {
        uint64_t h = oracle_splitmix64(J->sc->seed, (uint64_t)ray_id * (uint64_t)J->N
                                                     + (uint64_t)i);
        float xi = (float)(h >> 40) * 0x1p-24f;      /* 24 random bits in [0,1) */
        x = x + xi;
    }
    return J->near_t + x * J->dt;
}

/* Nearest grid node along one axis: vertex-aligned nodes, ties round up. */
static int32_t nearest_node(float p, float lo, float scale, int32_t n_p)
{
    float g = (p - lo) * scale;
    int32_t i = (int32_t)floorf(g + 0.5f);
    return i < n_p - 1 ? i : n_p - 1;
}

/* Bilinear lookup of beta at direction d (Sec. 3.4).  theta is the polar
 * angle from +z on a clamped vertex-aligned grid of n_theta nodes over
 * [0, pi]; phi = atan2(d_y, d_x) on a periodic grid of n_phi nodes at
 * -pi + b * 2pi / n_phi. */
static void lookup_beta(const oracle_scene* sc, const float d[3], double* beta)
{
    double dx = d[0], dy = d[1], dz = d[2];
    double n = sqrt(dx * dx + dy * dy + dz * dz);
    double cz = dz / n;
    if (cz > 1.0) cz = 1.0;
    if (cz < -1.0) cz = -1.0;
    double theta = acos(cz);
    double phi = atan2(dy, dx);

    double gt = theta * (double)(sc->n_theta - 1) / M_PI;
    int32_t a0 = (int32_t)floor(gt);
    if (a0 > sc->n_theta - 2) a0 = sc->n_theta - 2;
    if (a0 < 0) a0 = 0;
    double ft = gt - (double)a0;
    if (ft < 0.0) ft = 0.0;
    if (ft > 1.0) ft = 1.0;

    double gp = (phi + M_PI) * (double)sc->n_phi / (2.0 * M_PI);
    double fb = floor(gp);
    double fp = gp - fb;
    int32_t b0 = (int32_t)fb;
    b0 = ((b0 % sc->n_phi) + sc->n_phi) % sc->n_phi;
    int32_t b1 = (b0 + 1) % sc->n_phi;

    const int32_t D = sc->D;
    for (int32_t k = 0; k < D; ++k) {
        double v00 = cache_value64(sc->beta, sc->beta_f16, ((size_t)a0 * sc->n_phi + b0) * D + k);
        double v01 = cache_value64(sc->beta, sc->beta_f16, ((size_t)a0 * sc->n_phi + b1) * D + k);
        double v10 = cache_value64(sc->beta, sc->beta_f16, ((size_t)(a0 + 1) * sc->n_phi + b0) * D + k);
        double v11 = cache_value64(sc->beta, sc->beta_f16, ((size_t)(a0 + 1) * sc->n_phi + b1) * D + k);
        beta[k] = (1.0 - ft) * ((1.0 - fp) * v00 + fp * v01)
                + ft * ((1.0 - fp) * v10 + fp * v11);
    }
}

static void render_ray(const job_t* J, int64_t ray_id, oracle_ray* out)
{
    const oracle_scene* sc = J->sc;
    const oracle_camera* cam = J->cam;
    const int32_t W = cam->width, H = cam->height, N = J->N, n_p = sc->n_p, D = sc->D;
    const int64_t pix = (int64_t)W * H;
    const int64_t b = ray_id / pix;
    const int32_t v = (int32_t)((ray_id % pix) / W);
    const int32_t u = (int32_t)(ray_id % W);
    const float* P = J->poses + 12 * b;

    memset(out, 0, sizeof(*out));

    /* Ray through the centre of pixel (u, v); v = 0 is the top row.  The
     * camera looks down -z, so the camera-space direction is (a, b, -1) and
     * t below is depth along the camera axis. */
    float a = (((float)u + 0.5f) - cam->cx) / cam->fx;
    float bb = -((((float)v + 0.5f) - cam->cy) / cam->fy);
    float o[3], d[3];
    for (int r = 0; r < 3; ++r) {
        float pa = P[4 * r + 0] * a;
        float pb = P[4 * r + 1] * bb;
        d[r] = (pa + pb) - P[4 * r + 2];
        o[r] = P[4 * r + 3];
    }
    /* Direction weights, once per ray, from the world direction. */
    double beta[64];
    lookup_beta(sc, d, beta);

    int no_samples = 0;
    if (cam->ndc_near > 0.0f && !ndc_ray(cam, o, d))
        no_samples = 1;
    float d00 = d[0] * d[0], d11 = d[1] * d[1], d22 = d[2] * d[2];
    float dnorm = sqrtf((d00 + d11) + d22);

    int64_t tau = 0;          /* sum_{j<i} sigma_j delta_j in units of 2^-32 */
    uint32_t hash = 2166136261u;
    uint32_t stop = (uint32_t)N, n_inbox = 0, n_occ = 0;
    double rgb[3] = {0.0, 0.0, 0.0}, depth = 0.0, acc = 0.0;

    for (int32_t i = 0; i < N; ++i) {
        /* Sample i is evaluated only while its transmittance T_i >= eps. */
        if (tau > J->tau_eps) {
            stop = (uint32_t)i;
            break;
        }
        float t = sample_t(J, ray_id, i);
        float t_next = (i + 1 < N) ? sample_t(J, ray_id, i + 1) : J->far_t;

        float p[3];
        int inside = !no_samples;
        for (int r = 0; r < 3; ++r) {
            float td = t * d[r];
            p[r] = o[r] + td;
            if (!(p[r] >= sc->bmin[r] && p[r] <= sc->bmax[r]))
                inside = 0;
        }

        float sigma = 0.0f;
        int32_t ix = 0, iy = 0, iz = 0;
        size_t texel[3] = {0, 0, 0};
        if (inside) {
            n_inbox++;
            ix = nearest_node(p[0], sc->bmin[0], J->scale[0], n_p);
            iy = nearest_node(p[1], sc->bmin[1], J->scale[1], n_p);
            iz = nearest_node(p[2], sc->bmin[2], J->scale[2], n_p);
            /* Plane (x,y) at [ix][iy], (y,z) at [iy][iz], (z,x) at [iz][ix]. */
            texel[0] = (size_t)ix * n_p + iy;
            texel[1] = (size_t)iy * n_p + iz;
            texel[2] = (size_t)iz * n_p + ix;
            if (sc->d_sigma > 0) {
                sigma = alt_sigma(sc, texel);
            } else {
                /* Eq. 4: sigma is the product of the three planar densities. */
                float sxy = cache_value(sc->sigma[0], sc->sigma_f16, texel[0]);
                float syz = cache_value(sc->sigma[1], sc->sigma_f16, texel[1]);
                float szx = cache_value(sc->sigma[2], sc->sigma_f16, texel[2]);
                float prod = sxy * syz;
                prod = prod * szx;
                sigma = fmaxf(0.0f, prod);
            }
        }

        /* delta_i: distance to the next sample (the far plane after the
         * last).  A sample without density adds nothing to the optical depth. */
        float gap = fmaxf(0.0f, t_next - t);
        float delta = gap * dnorm;
        float q = 0.0f;
        int64_t Q = 0;

        if (sigma > 0.0f) {
            q = sigma * delta;
            Q = (int64_t)(fminf(q, 65536.0f) * 4294967296.0f);
            n_occ++;
            hash = fnv1a_word(hash, (uint32_t)i);
            hash = fnv1a_word(hash, (uint32_t)ix);
            hash = fnv1a_word(hash, (uint32_t)iy);
            hash = fnv1a_word(hash, (uint32_t)iz);

            /* Eq. 4 (sum of the planar k^j) or Eq. 5, and Eq. 2 (inner
             * product with beta), then a sigmoid per channel. */
            size_t rec[3];
            for (int j = 0; j < 3; ++j)
                rec[j] = texel[j] * (size_t)(3 * D);
            double x[3] = {0.0, 0.0, 0.0};
            if (sc->d_sigma > 0) {
                alt_logits(sc, rec, beta, x);
            } else {
                for (int c = 0; c < 3; ++c)
                    for (int32_t k = 0; k < D; ++k) {
                        size_t off = (size_t)c * D + k;
                        double kxy = cache_value64(sc->uvw[0], sc->uvw_f16, rec[0] + off);
                        double kyz = cache_value64(sc->uvw[1], sc->uvw_f16, rec[1] + off);
                        double kzx = cache_value64(sc->uvw[2], sc->uvw_f16, rec[2] + off);
                        x[c] += beta[k] * ((kxy + kyz) + kzx);
                    }
            }
            double col[3];
            for (int c = 0; c < 3; ++c)
                col[c] = 1.0 / (1.0 + exp(-x[c]));

            /* Eq. 1: w_i = T_i (1 - exp(-sigma_i delta_i)). */
            double T = exp(-(double)tau * 0x1p-32);
            double alpha = -expm1(-(double)q);
            double w = T * alpha;
            for (int c = 0; c < 3; ++c)
                rgb[c] += w * col[c];
            depth += w * (double)t;
            acc += w;
        }
        tau += Q;
    }

    out->rgb[0] = rgb[0];
    out->rgb[1] = rgb[1];
    out->rgb[2] = rgb[2];
    out->depth = depth;
    out->acc = acc;
    out->tau_end = tau;
    out->stop = stop;
    out->n_inbox = n_inbox;
    out->n_occ = n_occ;
    out->hash = hash;
}

/* ---- threads over rays --------------------------------------------------- */

typedef struct {
    const job_t* J;
    const int64_t* ray_ids;
    int64_t n_rays;
    int32_t first, stride;   /* blocks first, first + stride, ... */
    oracle_ray* out;
} slice_t;

enum { BLOCK_RAYS = 64 };

/* Threads take interleaved blocks of rays so that cheap and expensive image
 * regions are spread over all of them. */
static void* run_slice(void* arg)
{
    slice_t* s = (slice_t*)arg;
    for (int64_t blk = s->first; blk * BLOCK_RAYS < s->n_rays; blk += s->stride) {
        int64_t end = (blk + 1) * BLOCK_RAYS;
        if (end > s->n_rays)
            end = s->n_rays;
        for (int64_t k = blk * BLOCK_RAYS; k < end; ++k) {
            int64_t id = s->ray_ids ? s->ray_ids[k] : k;
            render_ray(s->J, id, &s->out[k]);
        }
    }
    return NULL;
}

int oracle_render(const oracle_scene* sc, const float* poses, int32_t n_poses,
                  const oracle_camera* cam, float near_t, float far_t,
                  int32_t n_samples, const int64_t* ray_ids, int64_t n_rays,
                  oracle_ray* out, int32_t n_threads)
{
    if (!sc || !poses || !cam || !out || n_poses < 1 || n_samples < 1)
        return -1;
    if (sc->n_p < 2 || sc->D < 1 || sc->D > 64 || sc->n_theta < 2 || sc->n_phi < 2)
        return -1;
    if (sc->d_sigma < 0 || (sc->d_sigma > 0 && (!sc->w_sigma || !sc->w_uvw || !sc->b_uvw)))
        return -1;
    if (cam->width < 1 || cam->height < 1 || !(near_t < far_t))
        return -1;
    const int64_t total = (int64_t)n_poses * cam->width * cam->height;
    if (!ray_ids)
        n_rays = total;
    for (int64_t k = 0; ray_ids && k < n_rays; ++k)
        if (ray_ids[k] < 0 || ray_ids[k] >= total)
            return -1;

    job_t J;
    J.sc = sc;
    J.poses = poses;
    J.cam = cam;
    J.near_t = near_t;
    J.far_t = far_t;
    J.N = n_samples;
    J.tau_eps = oracle_tau_eps_q(sc->t_eps);
    for (int r = 0; r < 3; ++r)
        J.scale[r] = (float)(sc->n_p - 1) / (sc->bmax[r] - sc->bmin[r]);
    J.dt = (far_t - near_t) / (float)n_samples;

    if (n_threads < 1)
        n_threads = 1;
    if (n_threads > 256)
        n_threads = 256;
    if (n_rays < n_threads)
        n_threads = n_rays > 0 ? (int32_t)n_rays : 1;

    pthread_t th[256];
    int started[256];
    slice_t sl[256];
    for (int32_t k = 0; k < n_threads; ++k) {
        sl[k].J = &J;
        sl[k].ray_ids = ray_ids;
        sl[k].n_rays = n_rays;
        sl[k].first = k;
        sl[k].stride = n_threads;
        sl[k].out = out;
    }
    for (int32_t k = 1; k < n_threads; ++k)
        started[k] = pthread_create(&th[k], NULL, run_slice, &sl[k]) == 0;
    run_slice(&sl[0]);
    for (int32_t k = 1; k < n_threads; ++k) {
        if (started[k])
            pthread_join(th[k], NULL);
        else
            run_slice(&sl[k]);
    }
    return 0;
}
