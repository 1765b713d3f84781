// Render kernels of the cached SqueezeNeRF path for gfx950 (CDNA4).
//
// One lane renders one pixel ray; a wave64 covers an 8x8 pixel tile, a
// 256-thread workgroup a 16x16 tile.  Neighbouring rays of a tile sit a
// fraction of a texel apart at equal sample index (samples are equal-depth
// planes), so the nearest-node gathers of a wave hit a handful of texels and
// cache lines: the wave-wide gather is what coalesces, not the sample axis.
//
// Per ray: pinhole ray (Sec. 3.1), a conservative clip of the sample range
// to the scene box (samples outside it have sigma = 0 and contribute
// nothing), the bilinear direction lookup of beta (Sec. 3.4) once, then a
// march over the samples: nearest-node gather of the three sigma^j and
// their product (Eq. 4), the fixed-point optical depth and termination test
// (Eq. 1 with T_i >= eps), and only for live samples with sigma > 0 the
// three uvw records, their sum (Eq. 4), the inner product with beta (Eq. 2),
// a sigmoid and the Eq. 1 weights.
//
// This file must be compiled with -ffp-contract=off and correctly rounded
// binary32 division and square root: the ray, sample, index and termination
// arithmetic is specified as one rounding per written operation.  Fused
// multiply-adds are requested explicitly (fmaf) where only the value path
// uses them.
#include <math.h>

#include "sqn_internal.h"

namespace sqn {
namespace {

constexpr double kPi = 3.14159265358979323846;

__device__ __forceinline__ float widen(float x) { return x; }
__device__ __forceinline__ float widen(_Float16 x) { return static_cast<float>(x); }

template <typename T>
__device__ __forceinline__ float load_value(const void* base, uint32_t idx)
{
    return widen(static_cast<const T*>(base)[idx]);
}

// ---------------------------------------------------------------------------
// exact path (binary32, one rounding per operation)

// Nearest vertex-aligned node along one axis; ties round up.
__device__ __forceinline__ int32_t nearest_node(float p, float lo, float scale, int32_t n_p)
{
    float g = (p - lo) * scale;
    int32_t i = static_cast<int32_t>(floorf(g + 0.5f));
    return min(i, n_p - 1);
}

// trunc(min(q, 2^16) * 2^32) for q >= 0, without a float->int64 conversion:
// the integer part and the (exactly representable) fraction convert
// separately.
__device__ __forceinline__ int64_t fixed_q(float q)
{
    float qc = fminf(q, 65536.0f);
    float hi = floorf(qc);
    float frac = qc - hi;
    uint32_t lo = static_cast<uint32_t>(frac * 4294967296.0f);
    return static_cast<int64_t>((static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) | lo);
}

// SplitMix64 (Steele, Lea & Flood 2014): output number `counter` (0-based)
// of the generator whose state starts at `seed`.
__device__ __forceinline__ uint64_t splitmix64(uint64_t seed, uint64_t counter)
{
    uint64_t z = seed + (counter + 1ull) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// Sample position t_i (camera-axis depth): left end of bin i, or a seeded
// point inside it.
__device__ __forceinline__ float sample_t(const RenderParams& P, bool stratified,
                                          uint64_t ray_key, int32_t i)
{
    float x = static_cast<float>(i);
    if (stratified) {
        uint64_t h = splitmix64(P.seed, ray_key + static_cast<uint64_t>(i));
        float xi = static_cast<float>(static_cast<uint32_t>(h >> 40)) * 0x1p-24f;
        x = x + xi;
    }
    float xd = x * P.dt;
    return P.near_t + xd;
}

// Conservative sample-index range [i0, i1] of the scene box: every sample
// outside it fails the exact in-box test.  The face crossings are computed
// in binary64 and widened by far more than the binary32 evaluation of
// o + t d can misplace them, then widened by two more samples.
__device__ inline void clip_to_box(const RenderParams& P, const float o[3], const float d[3],
                                   int32_t& i0, int32_t& i1)
{
    double lo = -INFINITY, hi = INFINITY;
    for (int r = 0; r < 3; ++r) {
        if (d[r] == 0.0f) {
            // p_r = o_r exactly for every t
            if (!(o[r] >= P.bmin[r] && o[r] <= P.bmax[r])) {
                i0 = 1;
                i1 = 0;
                return;
            }
            continue;
        }
        const double dr = d[r], orr = o[r];
        const double ta = (static_cast<double>(P.bmin[r]) - orr) / dr;
        const double tb = (static_cast<double>(P.bmax[r]) - orr) / dr;
        const double tmin = fmin(ta, tb), tmax = fmax(ta, tb);
        const double bmag = fmax(fabs(static_cast<double>(P.bmin[r])),
                                 fabs(static_cast<double>(P.bmax[r])));
        const double m = 1e-5 * (fmax(fabs(tmin), fabs(tmax)) + (fabs(orr) + bmag) / fabs(dr));
        lo = fmax(lo, tmin - m);
        hi = fmin(hi, tmax + m);
    }
    if (!(lo <= hi)) {
        i0 = 1;
        i1 = 0;
        return;
    }
    const double n_last = static_cast<double>(P.n_samples - 1);
    const double dt = P.dt;
    double f0 = floor((lo - static_cast<double>(P.near_t)) / dt) - 2.0;
    double f1 = ceil((hi - static_cast<double>(P.near_t)) / dt) + 2.0;
    f0 = fmin(fmax(f0, 0.0), n_last + 1.0);
    f1 = fmin(fmax(f1, -1.0), n_last);
    i0 = static_cast<int32_t>(f0);
    i1 = static_cast<int32_t>(f1);
}

// ---------------------------------------------------------------------------
// value path

// Bilinear lookup of beta (Sec. 3.4), once per ray, in binary64: theta is
// the polar angle from +z on a clamped grid over [0, pi], phi = atan2 on a
// periodic grid starting at -pi.
template <int DC>
__device__ inline void lookup_beta(const RenderParams& P, const float d[3], float* beta)
{
    const double dx = d[0], dy = d[1], dz = d[2];
    const double theta = atan2(sqrt(dx * dx + dy * dy), dz);
    const double phi = atan2(dy, dx);

    const double gt = theta * static_cast<double>(P.n_theta - 1) / kPi;
    int32_t a0 = static_cast<int32_t>(floor(gt));
    a0 = max(0, min(a0, P.n_theta - 2));
    const double ft = fmin(fmax(gt - static_cast<double>(a0), 0.0), 1.0);

    const double gp = (phi + kPi) * static_cast<double>(P.n_phi) / (2.0 * kPi);
    const double fb = floor(gp);
    const double fp = gp - fb;
    int32_t b0 = static_cast<int32_t>(fb);
    b0 = ((b0 % P.n_phi) + P.n_phi) % P.n_phi;
    const int32_t b1 = (b0 + 1 == P.n_phi) ? 0 : b0 + 1;

    const int32_t D = DC > 0 ? DC : P.D;
    const uint32_t r0 = static_cast<uint32_t>(a0 * P.n_phi);
    const uint32_t r1 = static_cast<uint32_t>((a0 + 1) * P.n_phi);
    const uint32_t i00 = (r0 + b0) * D, i01 = (r0 + b1) * D;
    const uint32_t i10 = (r1 + b0) * D, i11 = (r1 + b1) * D;
    const double w00 = (1.0 - ft) * (1.0 - fp), w01 = (1.0 - ft) * fp;
    const double w10 = ft * (1.0 - fp), w11 = ft * fp;
#pragma unroll
    for (int32_t k = 0; k < (DC > 0 ? DC : 32); ++k) {
        if (DC == 0 && k >= D)
            break;
        double v00, v01, v10, v11;
        if (P.beta_f16) {
            v00 = load_value<_Float16>(P.beta, i00 + k);
            v01 = load_value<_Float16>(P.beta, i01 + k);
            v10 = load_value<_Float16>(P.beta, i10 + k);
            v11 = load_value<_Float16>(P.beta, i11 + k);
        } else {
            v00 = load_value<float>(P.beta, i00 + k);
            v01 = load_value<float>(P.beta, i01 + k);
            v10 = load_value<float>(P.beta, i10 + k);
            v11 = load_value<float>(P.beta, i11 + k);
        }
        beta[k] = static_cast<float>((w00 * v00 + w01 * v01) + (w10 * v10 + w11 * v11));
    }
}

__device__ __forceinline__ float sigmoid(float x)
{
    return __builtin_amdgcn_rcpf(1.0f + expf(-x));
}

// Colour of one occupied sample: the three uvw records summed over planes
// (Eq. 4), inner product with beta per channel (Eq. 2), sigmoid.
template <typename UT, int DC>
__device__ __forceinline__ void sample_colour(const RenderParams& P, uint32_t t0, uint32_t t1,
                                              uint32_t t2, const float* beta, float col[3])
{
    if constexpr (DC > 0 && (3 * DC * sizeof(UT)) % 16 == 0) {
        constexpr int NV = 3 * DC;
        constexpr int NB = NV * static_cast<int>(sizeof(UT));
        constexpr int NQ = NB / 16;
        const uint4* p0 = reinterpret_cast<const uint4*>(static_cast<const char*>(P.uvw[0]) + static_cast<size_t>(t0) * NB);
        const uint4* p1 = reinterpret_cast<const uint4*>(static_cast<const char*>(P.uvw[1]) + static_cast<size_t>(t1) * NB);
        const uint4* p2 = reinterpret_cast<const uint4*>(static_cast<const char*>(P.uvw[2]) + static_cast<size_t>(t2) * NB);
        uint4 q0[NQ], q1[NQ], q2[NQ];
#pragma unroll
        for (int k = 0; k < NQ; ++k) {
            q0[k] = p0[k];
            q1[k] = p1[k];
            q2[k] = p2[k];
        }
        UT v0[NV], v1[NV], v2[NV];
        __builtin_memcpy(v0, q0, NB);
        __builtin_memcpy(v1, q1, NB);
        __builtin_memcpy(v2, q2, NB);
#pragma unroll
        for (int c = 0; c < 3; ++c) {
            float x = 0.0f;
#pragma unroll
            for (int k = 0; k < DC; ++k) {
                const float U = (widen(v0[c * DC + k]) + widen(v1[c * DC + k])) + widen(v2[c * DC + k]);
                x = fmaf(beta[k], U, x);
            }
            col[c] = sigmoid(x);
        }
    } else {
        const int32_t D = P.D;
        const uint32_t nv = 3u * static_cast<uint32_t>(D);
        for (int c = 0; c < 3; ++c) {
            float x = 0.0f;
            for (int32_t k = 0; k < D; ++k) {
                const uint32_t off = static_cast<uint32_t>(c * D + k);
                const float U = (load_value<UT>(P.uvw[0], t0 * nv + off)
                                 + load_value<UT>(P.uvw[1], t1 * nv + off))
                                + load_value<UT>(P.uvw[2], t2 * nv + off);
                x = fmaf(beta[k], U, x);
            }
            col[c] = sigmoid(x);
        }
    }
}

__device__ __forceinline__ uint32_t fnv1a_word(uint32_t h, uint32_t x)
{
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        h ^= (x >> (8 * k)) & 0xffu;
        h *= 16777619u;
    }
    return h;
}

// Map the hardware workgroup id to a tile so that each XCD (workgroups are
// dealt round-robin over the 8 XCDs) receives one contiguous run of tiles
// and its L2 sees spatially coherent gathers.
__device__ __forceinline__ int32_t xcd_tile_order(int32_t bid, int32_t n)
{
    const int32_t xcd = bid & 7, local = bid >> 3;
    const int32_t per = n >> 3, rem = n & 7;
    return xcd * per + min(xcd, rem) + local;
}

template <typename ST, typename UT, int DC, bool STATS>
__global__ __launch_bounds__(kBlockThreads) void render_kernel(const RenderParams P)
{
    const int32_t g = xcd_tile_order(static_cast<int32_t>(blockIdx.x), P.n_groups);
    const int32_t tiles_per_view = P.tiles_x * P.tiles_y;
    const int32_t view = g / tiles_per_view;
    const int32_t tr = g - view * tiles_per_view;
    const int32_t ty = tr / P.tiles_x;
    const int32_t tx = tr - ty * P.tiles_x;
    const int32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int32_t u = tx * kTileW + (wave & 1) * 8 + (lane & 7);
    const int32_t v = ty * kTileH + (wave >> 1) * 8 + (lane >> 3);
    if (view >= P.n_views || u >= P.width || v >= P.height)
        return;

    const int64_t ray = (static_cast<int64_t>(view) * P.height + v) * P.width + u;
    const int32_t N = P.n_samples;
    const bool stratified = P.stratified != 0;
    const uint64_t ray_key = static_cast<uint64_t>(ray) * static_cast<uint64_t>(N);

    // --- ray through the pixel centre (camera looks down -z) ---
    const float* pose = P.poses + 12 * static_cast<int64_t>(view);
    float pm[12];
#pragma unroll
    for (int k = 0; k < 12; ++k)
        pm[k] = pose[k];
    const float a = ((static_cast<float>(u) + 0.5f) - P.cx) / P.fx;
    const float b = -(((static_cast<float>(v) + 0.5f) - P.cy) / P.fy);
    float o[3], d[3];
#pragma unroll
    for (int r = 0; r < 3; ++r) {
        const float pa = pm[4 * r + 0] * a;
        const float pb = pm[4 * r + 1] * b;
        d[r] = (pa + pb) - pm[4 * r + 2];
        o[r] = pm[4 * r + 3];
    }
    const float d00 = d[0] * d[0], d11 = d[1] * d[1], d22 = d[2] * d[2];
    const float dn = sqrtf((d00 + d11) + d22);

    int32_t i0, i1;
    clip_to_box(P, o, d, i0, i1);

    float beta[DC > 0 ? DC : 32];
    lookup_beta<DC>(P, d, beta);

    // --- march ---
    int64_t tau = 0;                 // optical depth before sample i, 2^-32 units
    double acc_r = 0.0, acc_g = 0.0, acc_b = 0.0, acc_t = 0.0;
    uint32_t n_inbox = 0, n_occ = 0, hash = 2166136261u;
    const int32_t n_p = P.n_p;

    int32_t i = i0;
    float t = (i0 <= i1) ? sample_t(P, stratified, ray_key, i0) : 0.0f;
    for (; i <= i1; ++i) {
        if (tau > P.tau_eps)
            break;
        const float tn = (i + 1 < N) ? sample_t(P, stratified, ray_key, i + 1) : P.far_t;
        float p[3];
        bool inside = true;
#pragma unroll
        for (int r = 0; r < 3; ++r) {
            const float td = t * d[r];
            p[r] = o[r] + td;
            inside = inside && (p[r] >= P.bmin[r]) && (p[r] <= P.bmax[r]);
        }
        if (inside) {
            const int32_t ix = nearest_node(p[0], P.bmin[0], P.scale[0], n_p);
            const int32_t iy = nearest_node(p[1], P.bmin[1], P.scale[1], n_p);
            const int32_t iz = nearest_node(p[2], P.bmin[2], P.scale[2], n_p);
            const uint32_t txy = static_cast<uint32_t>(ix * n_p + iy);
            const uint32_t tyz = static_cast<uint32_t>(iy * n_p + iz);
            const uint32_t tzx = static_cast<uint32_t>(iz * n_p + ix);
            const float sxy = load_value<ST>(P.sigma[0], txy);
            const float syz = load_value<ST>(P.sigma[1], tyz);
            const float szx = load_value<ST>(P.sigma[2], tzx);
            float prod = sxy * syz;
            prod = prod * szx;
            const float sigma = fmaxf(0.0f, prod);
            if constexpr (STATS)
                ++n_inbox;
            if (sigma > 0.0f) {
                const float gap = fmaxf(0.0f, tn - t);
                const float delta = gap * dn;
                const float q = sigma * delta;
                if constexpr (STATS) {
                    ++n_occ;
                    hash = fnv1a_word(hash, static_cast<uint32_t>(i));
                    hash = fnv1a_word(hash, static_cast<uint32_t>(ix));
                    hash = fnv1a_word(hash, static_cast<uint32_t>(iy));
                    hash = fnv1a_word(hash, static_cast<uint32_t>(iz));
                }
                float col[3];
                sample_colour<UT, DC>(P, txy, tyz, tzx, beta, col);
                const float T = expf(static_cast<float>(tau) * -0x1p-32f);
                const float alpha = -expm1f(-q);
                const double w = static_cast<double>(T * alpha);
                acc_r = fma(w, static_cast<double>(col[0]), acc_r);
                acc_g = fma(w, static_cast<double>(col[1]), acc_g);
                acc_b = fma(w, static_cast<double>(col[2]), acc_b);
                acc_t = fma(w, static_cast<double>(t), acc_t);
                tau += fixed_q(q);
            }
        }
        t = tn;
    }
    const uint32_t stop = (tau > P.tau_eps) ? static_cast<uint32_t>(i) : static_cast<uint32_t>(N);

    if (P.rgb) {
        P.rgb[3 * ray + 0] = static_cast<float>(acc_r);
        P.rgb[3 * ray + 1] = static_cast<float>(acc_g);
        P.rgb[3 * ray + 2] = static_cast<float>(acc_b);
    }
    if (P.depth)
        P.depth[ray] = static_cast<float>(acc_t);
    if constexpr (STATS) {
        uint4 s;
        s.x = stop;
        s.y = n_inbox;
        s.z = n_occ;
        s.w = hash;
        reinterpret_cast<uint4*>(P.stats)[ray] = s;
    }
}

template <typename ST, typename UT, int DC>
hipError_t launch_typed(const RenderParams& p, bool stats, hipStream_t stream)
{
    const dim3 grid(static_cast<uint32_t>(p.n_groups));
    const dim3 block(kBlockThreads);
    if (stats)
        render_kernel<ST, UT, DC, true><<<grid, block, 0, stream>>>(p);
    else
        render_kernel<ST, UT, DC, false><<<grid, block, 0, stream>>>(p);
    return hipGetLastError();
}

template <typename ST, typename UT>
hipError_t launch_d(const RenderParams& p, bool stats, hipStream_t stream)
{
    switch (p.D) {
    case 8:
        return launch_typed<ST, UT, 8>(p, stats, stream);
    case 16:
        return launch_typed<ST, UT, 16>(p, stats, stream);
    default:
        return launch_typed<ST, UT, 0>(p, stats, stream);
    }
}

}  // namespace

hipError_t launch_render(const RenderParams& p, int sigma_dtype, int uvw_dtype, bool stats,
                         hipStream_t stream)
{
    const bool s16 = sigma_dtype == SQN_F16, u16 = uvw_dtype == SQN_F16;
    if (s16 && u16)
        return launch_d<_Float16, _Float16>(p, stats, stream);
    if (s16)
        return launch_d<_Float16, float>(p, stats, stream);
    if (u16)
        return launch_d<float, _Float16>(p, stats, stream);
    return launch_d<float, float>(p, stats, stream);
}

}  // namespace sqn
