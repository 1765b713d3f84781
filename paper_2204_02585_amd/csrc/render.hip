// Render kernels of the cached SqueezeNeRF path for gfx950 (CDNA4).
//
// Work layout.  L consecutive lanes of a wave64 (L = 1, 4 or 8) share one
// pixel ray and walk its samples in chunks of L consecutive samples, one per
// lane; a wave holds 64/L rays laid out as a compact pixel tile.  Rays of a
// tile sit a fraction of a texel apart at equal sample index (samples lie on
// equal-depth planes), so the nearest-node gathers of one wave-wide load hit
// a few texels and cache lines.  L > 1 multiplies the number of waves of a
// frame (a single 800x800 view is only 10^4 waves at L = 1) at the price of a
// short cross-lane scan per chunk; the per-ray setup is then computed once
// per ray by the workgroup, not by each of its L lanes.
//
// Per ray: pinhole ray (Sec. 3.1); a conservative clip of the sample range to
// the scene box (samples outside it have sigma = 0 and add nothing); the
// bilinear direction lookup of beta (Sec. 3.4).  Per sample: nearest-node
// gathers of the three sigma^j and their product (Eq. 4), or of the three
// per-plane partial sums of Eq. 5 and their biased sum; the 2^-32
// fixed-point optical depth increment, scanned exactly across the L lanes;
// the termination test T_i >= eps (Eq. 1); and only for live samples with
// sigma > 0 the three uvw records, beta^T (sum of the planar uvw) (Eq. 4 and
// Eq. 2), a sigmoid and the Eq. 1 weight.
//
// Compile with -ffp-contract=off and correctly rounded binary32 division and
// square root: ray, sample, grid-index and termination arithmetic is
// specified as one rounding per written operation.  The value path requests
// fused multiply-adds explicitly.
#include <math.h>

#include "atan2_lookup.h"
#include "sqn_internal.h"

namespace sqn {
namespace {

constexpr double kPi = 3.14159265358979323846;
constexpr float kLog2e = 1.4426950408889634f;

__device__ __forceinline__ float widen(float x) { return x; }
__device__ __forceinline__ float widen(_Float16 x) { return static_cast<float>(x); }

// Element at byte offset `off` (32-bit) from a uniform base pointer.
template <typename T>
__device__ __forceinline__ T load_at(const void* base, uint32_t off)
{
    return *reinterpret_cast<const T*>(static_cast<const char*>(base) + off);
}

// ---------------------------------------------------------------------------
// lanes of one ray: L = 4 consecutive lanes of a quad, exchanged with DPP
// quad permutations, or L = 8 lanes of a half-row, whose two quads also
// exchange through the half-row mirror (lane i <-> 7 - i); the group is
// always entirely active or inactive

constexpr int qperm(int a, int b, int c, int d) { return a | (b << 2) | (c << 4) | (d << 6); }
constexpr int kHalfMirror = 0x141;   // DPP row_half_mirror

template <int CTRL>
__device__ __forceinline__ uint32_t dpp32(uint32_t x)
{
    return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(x), CTRL, 0xf, 0xf, true));
}

template <int CTRL>
__device__ __forceinline__ uint64_t dpp64(uint64_t x)
{
    const uint32_t lo = dpp32<CTRL>(static_cast<uint32_t>(x));
    const uint32_t hi = dpp32<CTRL>(static_cast<uint32_t>(x >> 32));
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

template <int CTRL>
__device__ __forceinline__ float dppf(float x)
{
    return __uint_as_float(dpp32<CTRL>(__float_as_uint(x)));
}

// value of lane s + 1 of the group (the last lane reads itself)
template <int L>
__device__ __forceinline__ float grp_next(float x)
{
    if constexpr (L == 4)
        return dppf<qperm(1, 2, 3, 3)>(x);
    else if constexpr (L == 8) {
        // lane 3 takes lane 4 from the other quad (7 - 3 = 4)
        const float a = dppf<qperm(1, 2, 3, 3)>(x);
        const float b = dppf<kHalfMirror>(x);
        return ((__lane_id() & 7) == 3) ? b : a;
    } else
        return x;
}

// value of lane 0 of the group
template <int L>
__device__ __forceinline__ float grp_first(float x)
{
    if constexpr (L == 4)
        return dppf<qperm(0, 0, 0, 0)>(x);
    else if constexpr (L == 8) {
        // the upper quad reads lane 0 where the mirror put it, in lane 7
        const float a = dppf<qperm(0, 0, 0, 0)>(x);
        const float b = dppf<qperm(3, 3, 3, 3)>(dppf<kHalfMirror>(x));
        return ((__lane_id() & 7) < 4) ? a : b;
    } else
        return x;
}

// Exclusive prefix sum of q over the group (lane order) and the group total.
template <int L>
__device__ __forceinline__ void grp_scan(uint64_t q, int s, uint64_t& excl, uint64_t& total)
{
    if constexpr (L == 1) {
        excl = 0;
        total = q;
    } else {
        const int sq = s & 3;
        uint64_t y = q;
        const uint64_t y1 = dpp64<qperm(0, 0, 1, 2)>(y);
        y += (sq >= 1) ? y1 : 0;
        const uint64_t y2 = dpp64<qperm(0, 0, 0, 1)>(y);
        y += (sq >= 2) ? y2 : 0;
        const uint64_t tq = dpp64<qperm(3, 3, 3, 3)>(y);
        if constexpr (L == 8) {
            // the other quad's total; the upper quad adds the lower one's
            const uint64_t other = dpp64<kHalfMirror>(tq);
            y += (s >= 4) ? other : 0;
            excl = y - q;
            total = tq + other;
        } else {
            excl = y - q;
            total = tq;
        }
    }
}

template <int L>
__device__ __forceinline__ float grp_sum(float x)
{
    if constexpr (L >= 2)
        x += dppf<qperm(1, 0, 3, 2)>(x);
    if constexpr (L >= 4)
        x += dppf<qperm(2, 3, 0, 1)>(x);
    if constexpr (L == 8)
        x += dppf<kHalfMirror>(x);
    return x;
}

template <int CTRL>
__device__ __forceinline__ double dppd(double x)
{
    return __longlong_as_double(static_cast<long long>(dpp64<CTRL>(static_cast<uint64_t>(__double_as_longlong(x)))));
}

template <int L>
__device__ __forceinline__ double grp_sum(double x)
{
    if constexpr (L >= 2)
        x += dppd<qperm(1, 0, 3, 2)>(x);
    if constexpr (L >= 4)
        x += dppd<qperm(2, 3, 0, 1)>(x);
    if constexpr (L == 8)
        x += dppd<kHalfMirror>(x);
    return x;
}

template <int L>
__device__ __forceinline__ int32_t grp_max(int32_t x)
{
    if constexpr (L >= 2)
        x = max(x, static_cast<int32_t>(dpp32<qperm(1, 0, 3, 2)>(static_cast<uint32_t>(x))));
    if constexpr (L >= 4)
        x = max(x, static_cast<int32_t>(dpp32<qperm(2, 3, 0, 1)>(static_cast<uint32_t>(x))));
    if constexpr (L == 8)
        x = max(x, static_cast<int32_t>(dpp32<kHalfMirror>(static_cast<uint32_t>(x))));
    return x;
}

template <int L>
__device__ __forceinline__ uint32_t grp_add(uint32_t x)
{
    if constexpr (L >= 2)
        x += dpp32<qperm(1, 0, 3, 2)>(x);
    if constexpr (L >= 4)
        x += dpp32<qperm(2, 3, 0, 1)>(x);
    if constexpr (L == 8)
        x += dpp32<kHalfMirror>(x);
    return x;
}

// ---------------------------------------------------------------------------
// exact path (binary32, one rounding per operation)

// (int)floor(x) in one instruction; exact for every x this code passes
// (finite, |x| < 2^31).
__device__ __forceinline__ int32_t floor_to_int(float x)
{
    int32_t r;
    asm("v_cvt_flr_i32_f32 %0, %1" : "=v"(r) : "v"(x));
    return r;
}

// Nearest vertex-aligned node along one axis; ties round up:
// floor(g + 1/2) with g = (p - lo) scale.  For a sample inside the box
// 1/2 <= g + 1/2 < n_p, so clamping g + 1/2 to [0, n_p - 1] before the floor
// gives min(floor(g + 1/2), n_p - 1) there and a valid index everywhere.
__device__ __forceinline__ uint32_t nearest_node(float p, float lo, float scale, float hi_node)
{
    const float g = (p - lo) * scale;
    const float h = g + 0.5f;
    return static_cast<uint32_t>(floor_to_int(__builtin_amdgcn_fmed3f(h, 0.0f, hi_node)));
}

// nearest_node for a sample inside the box, where 1/2 <= g + 1/2 <= n_p - 1/2
// (bmin <= p <= bmax, and binary32 subtraction and multiplication are
// monotone), so the clamp would change nothing.
__device__ __forceinline__ uint32_t nearest_node_inside(float p, float lo, float scale)
{
    const float g = (p - lo) * scale;
    const float h = g + 0.5f;
    return static_cast<uint32_t>(floor_to_int(h));
}

// trunc(min(q, 2^16) * 2^32) for q >= 0: the integer part and the (exactly
// representable) fraction convert separately.
__device__ __forceinline__ uint64_t fixed_q(float q)
{
    const float qc = fminf(q, 65536.0f);
    const float hi = floorf(qc);
    const float frac = qc - hi;
    const uint32_t lo = static_cast<uint32_t>(frac * 4294967296.0f);
    return (static_cast<uint64_t>(static_cast<uint32_t>(hi)) << 32) | lo;
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
        const uint64_t h = splitmix64(P.seed, ray_key + static_cast<uint64_t>(i));
        const float xi = static_cast<float>(static_cast<uint32_t>(h >> 40)) * 0x1p-24f;
        x = x + xi;
    }
    const float xd = x * P.dt;
    return P.near_t + xd;
}

// Normalized device coordinates of a camera looking down -z with near plane
// n (forward-facing captures): a world point (x, y, z) maps to
// (-(fx/(W/2)) x/z, -(fy/(H/2)) y/z, 1 + 2n/z), the frustum beyond the near
// plane to [-1, 1]^3.  The ray is moved to its point on the near plane,
// t_s = -(n + o_z)/d_z, and becomes o' + t' d' with t' in [0, 1) up to
// infinity.  Binary32, one rounding per operation, in this order.  A ray
// with d_z >= 0 never reaches the near plane: returns false (no samples).
__device__ __forceinline__ bool ndc_ray(const RenderParams& P, float o[3], float d[3])
{
    const float n = P.ndc_near;
    if (!(d[2] < 0.0f))
        return false;
    const float ts = -(n + o[2]) / d[2];
    float os[3];
#pragma unroll
    for (int r = 0; r < 3; ++r) {
        const float td = ts * d[r];
        os[r] = o[r] + td;
    }
    const float sx = P.fx / (0.5f * static_cast<float>(P.width));
    const float sy = P.fy / (0.5f * static_cast<float>(P.height));
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
    return true;
}

// Conservative sample-index range [i0, i1] of the scene box: every sample
// outside it fails the exact in-box test.  Face crossings are widened by
// 1e-5 relative (far beyond the few-ulp misplacement of the binary32
// position o + t d and of this estimate), then by two samples.  An axis with
// a (nearly) zero direction component constrains nothing here unless the
// component is exactly zero, where p = o holds exactly.
// [j0, j1] is the range of samples certainly inside: the crossings narrowed
// by the same margin and one more sample on each side, so every such sample
// passes the six exact box tests (its binary32 position is within a few ulp
// of the exact one, the margin is 160 times that) and needs no clamp of its
// node indices; empty when an axis has a tiny nonzero component.
__device__ __forceinline__ void clip_to_box(const RenderParams& P, const float o[3], const float d[3],
                                            int32_t& i0, int32_t& i1, int32_t& j0, int32_t& j1)
{
    float lo = -INFINITY, hi = INFINITY, lo_in = -INFINITY, hi_in = INFINITY;
    bool empty = false, no_inner = false;
#pragma unroll
    for (int r = 0; r < 3; ++r) {
        if (d[r] == 0.0f) {
            empty = empty || !(o[r] >= P.bmin[r] && o[r] <= P.bmax[r]);
        } else if (fabsf(d[r]) > 1e-20f) {
            const float inv = __builtin_amdgcn_rcpf(d[r]);
            const float ta = (P.bmin[r] - o[r]) * inv;
            const float tb = (P.bmax[r] - o[r]) * inv;
            const float tmin = fminf(ta, tb), tmax = fmaxf(ta, tb);
            const float bmag = fmaxf(fabsf(P.bmin[r]), fabsf(P.bmax[r]));
            const float m = 1e-5f * (fmaxf(fabsf(tmin), fabsf(tmax)) + (fabsf(o[r]) + bmag) * fabsf(inv));
            lo = fmaxf(lo, tmin - m);
            hi = fminf(hi, tmax + m);
            lo_in = fmaxf(lo_in, tmin + m);
            hi_in = fminf(hi_in, tmax - m);
        } else {
            no_inner = true;
        }
    }
    const float n_last = static_cast<float>(P.n_samples - 1);
    float f0 = floorf((lo - P.near_t) * P.inv_dt) - 2.0f;
    float f1 = ceilf((hi - P.near_t) * P.inv_dt) + 2.0f;
    f0 = fminf(fmaxf(f0, 0.0f), n_last + 1.0f);
    f1 = fminf(fmaxf(f1, -1.0f), n_last);
    if (empty || !(lo <= hi)) {
        f0 = 1.0f;
        f1 = 0.0f;
    }
    i0 = static_cast<int32_t>(f0);
    i1 = static_cast<int32_t>(f1);
    float g0 = ceilf((lo_in - P.near_t) * P.inv_dt) + 1.0f;
    float g1 = floorf((hi_in - P.near_t) * P.inv_dt) - 1.0f;
    // inside [i0, i1]; a NaN or an infinite bound gives the empty range
    g0 = fminf(fmaxf(g0, f0), n_last + 1.0f);
    g1 = fminf(fmaxf(g1, -1.0f), f1);
    if (empty || no_inner || !(lo_in <= hi_in) || !(g0 <= g1)) {
        g0 = 1.0f;
        g1 = 0.0f;
    }
    j0 = static_cast<int32_t>(g0);
    j1 = static_cast<int32_t>(g1);
}

// ---------------------------------------------------------------------------
// value path

// Bilinear lookup of beta (Sec. 3.4), once per ray by one lane.  The angles
// and grid coordinates are computed in binary64 (theta = polar angle from +z
// on a clamped grid over [0, pi]; phi = atan2 on a periodic grid from -pi).
// Component k goes to beta_lds[k * BS].
template <int DC, int BS>
__device__ __forceinline__ void lookup_beta(const RenderParams& P, const float d[3], float* beta_lds)
{
    const double dx = d[0], dy = d[1], dz = d[2];
    const double theta = atan2_lookup(sqrt(dx * dx + dy * dy), dz);
    const double phi = atan2_lookup(dy, dx);

    // grid coordinates: theta in [0, pi] and phi + pi in [0, 2 pi], scaled
    // by factors the host computes in binary64
    const double gt = theta * P.theta_scale;
    int32_t a0 = static_cast<int32_t>(floor(gt));
    a0 = max(0, min(a0, P.n_theta - 2));
    const double ft = fmin(fmax(gt - static_cast<double>(a0), 0.0), 1.0);

    const double gp = (phi + kPi) * P.phi_scale;
    const double fb = floor(gp);
    const double fp = gp - fb;
    // gp lies in [0, n_phi] (n_phi only at phi = pi), so one wrap suffices;
    // the clamps keep any input inside the table
    int32_t b0 = static_cast<int32_t>(fb);
    b0 = b0 >= P.n_phi ? b0 - P.n_phi : b0;
    b0 = min(max(b0, 0), P.n_phi - 1);
    const int32_t b1 = (b0 + 1 == P.n_phi) ? 0 : b0 + 1;

    const int32_t D = DC > 0 ? DC : P.D;
    const uint32_t row0 = static_cast<uint32_t>(a0 * P.n_phi);
    const uint32_t row1 = static_cast<uint32_t>((a0 + 1) * P.n_phi);
    // corners c = 0..3: (a0,b0) (a0,b1) (a0+1,b0) (a0+1,b1)
    const uint32_t texel[4] = {row0 + b0, row0 + b1, row1 + b0, row1 + b1};
    const float wgt[4] = {static_cast<float>((1.0 - ft) * (1.0 - fp)), static_cast<float>((1.0 - ft) * fp),
                          static_cast<float>(ft * (1.0 - fp)), static_cast<float>(ft * fp)};
    const uint32_t esz = P.beta_f16 ? 2u : 4u;
    auto component = [&](int k) {
        float acc = 0.0f;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const uint32_t off = (texel[c] * static_cast<uint32_t>(D) + k) * esz;
            const float v = P.beta_f16 ? widen(load_at<_Float16>(P.beta, off)) : load_at<float>(P.beta, off);
            acc = fmaf(wgt[c], v, acc);
        }
        return acc;
    };
    if constexpr (DC == 8) {
        // each corner record (D contiguous values) in 16-byte loads (at
        // D = 16 this measured slower than per-component loads)
        float acc[DC];
#pragma unroll
        for (int k = 0; k < DC; ++k)
            acc[k] = 0.0f;
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const float w = wgt[c];
            if (P.beta_f16) {
#pragma unroll
                for (int q = 0; q < DC / 8; ++q) {
                    const uint4 raw = load_at<uint4>(P.beta, texel[c] * (DC * 2u) + 16u * q);
                    _Float16 h[8];
                    __builtin_memcpy(h, &raw, 16);
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        acc[8 * q + e] = fmaf(w, widen(h[e]), acc[8 * q + e]);
                }
            } else {
#pragma unroll
                for (int q = 0; q < DC / 4; ++q) {
                    const float4 v = load_at<float4>(P.beta, texel[c] * (DC * 4u) + 16u * q);
                    acc[4 * q + 0] = fmaf(w, v.x, acc[4 * q + 0]);
                    acc[4 * q + 1] = fmaf(w, v.y, acc[4 * q + 1]);
                    acc[4 * q + 2] = fmaf(w, v.z, acc[4 * q + 2]);
                    acc[4 * q + 3] = fmaf(w, v.w, acc[4 * q + 3]);
                }
            }
        }
#pragma unroll
        for (int k = 0; k < DC; ++k)
            beta_lds[k * BS] = acc[k];
    } else if constexpr (DC > 0) {
#pragma unroll
        for (int k = 0; k < DC; ++k)
            beta_lds[k * BS] = component(k);
    } else {
        for (int k = 0; k < D; ++k)
            beta_lds[k * BS] = component(k);
    }
}

__device__ __forceinline__ float sigmoid(float x)
{
    return __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-x * kLog2e));
}

// Colour of one occupied sample: beta^T (k^xy + k^yz + k^zx) per channel
// (Eq. 4 and Eq. 2, summed plane by plane), then a sigmoid.
template <typename UT, int DC, int BS>
__device__ __forceinline__ void sample_colour(const RenderParams& P, uint32_t t0, uint32_t t1,
                                              uint32_t t2, const float* beta_lds, float col[3])
{
    // beta component k of this lane's ray lives at beta_lds[k * BS]
    auto beta = [&](int k) { return beta_lds[k * BS]; };
    if constexpr (DC > 0 && (3 * DC * sizeof(UT)) % 16 == 0) {
        constexpr int NV = 3 * DC;
        constexpr uint32_t NB = NV * static_cast<uint32_t>(sizeof(UT));
        constexpr int NQ = NB / 16;
        const uint32_t texel[3] = {t0, t1, t2};
        float x[3] = {0.0f, 0.0f, 0.0f};
        // one plane's record at a time keeps a single record in registers
#pragma unroll
        for (int j = 0; j < 3; ++j) {
            uint4 q[NQ];
#pragma unroll
            for (int k = 0; k < NQ; ++k)
                q[k] = load_at<uint4>(P.uvw[j], texel[j] * NB + 16u * k);
            UT rec[NV];
            __builtin_memcpy(rec, q, NB);
#pragma unroll
            for (int c = 0; c < 3; ++c)
#pragma unroll
                for (int k = 0; k < DC; ++k)
                    x[c] = fmaf(beta(k), widen(rec[c * DC + k]), x[c]);
        }
#pragma unroll
        for (int c = 0; c < 3; ++c)
            col[c] = sigmoid(x[c]);
    } else {
        const int32_t D = P.D;
        const uint32_t nv = 3u * static_cast<uint32_t>(D);
        const uint32_t esz = static_cast<uint32_t>(sizeof(UT));
        for (int c = 0; c < 3; ++c) {
            float x = 0.0f;
            for (int32_t k = 0; k < D; ++k) {
                const uint32_t off = static_cast<uint32_t>(c * D + k);
                const float bk = beta(k);
                x = fmaf(bk, widen(load_at<UT>(P.uvw[0], (t0 * nv + off) * esz)), x);
                x = fmaf(bk, widen(load_at<UT>(P.uvw[1], (t1 * nv + off) * esz)), x);
                x = fmaf(bk, widen(load_at<UT>(P.uvw[2], (t2 * nv + off) * esz)), x);
            }
            col[c] = sigmoid(x);
        }
    }
}

// Eq. 5 decoder, folded into Eq. 2 once per ray: with beta fixed along the
// ray, the logit of channel c is
//   beta^T (W_c concat_c + b_c) = sum_e (W_c^T beta)_e concat_c[e] + beta^T b_c,
// so each ray keeps the 9D values W_c^T beta and the three beta^T b_c (rows
// of lin_w: c*3D + e, then the biases) and every occupied sample costs one
// 3D-term inner product per channel, as with Eq. 4.  The L lanes of the ray
// compute every L-th row and store it in the ray's LDS row `lin`, where beta
// waits: in lin[0, D) for a compile-time D (read into registers before any
// row is written: LDS operations of one wavefront complete in order), else
// in lin[9D + 3, 10D + 3).
template <int DC, int L>
__device__ __forceinline__ void fold_decoder(const RenderParams& P, int s, float* lin)
{
    if constexpr (DC > 0) {
        constexpr int32_t rows = 9 * DC + 3;
        float b[DC];
#pragma unroll
        for (int k = 0; k < DC; ++k)
            b[k] = lin[k];
        __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
        for (int32_t o = s; o < rows; o += L) {
            const float4* w = reinterpret_cast<const float4*>(P.lin_w + o * DC);
            float acc = 0.0f;
#pragma unroll
            for (int k = 0; k < DC / 4; ++k) {
                const float4 w4 = w[k];
                acc = fmaf(b[4 * k + 0], w4.x, acc);
                acc = fmaf(b[4 * k + 1], w4.y, acc);
                acc = fmaf(b[4 * k + 2], w4.z, acc);
                acc = fmaf(b[4 * k + 3], w4.w, acc);
            }
            lin[o] = acc;
        }
    } else {
        const int32_t D = P.D;
        const int32_t rows = 9 * D + 3;
        for (int32_t o = s; o < rows; o += L) {
            const float* w = P.lin_w + o * D;
            float acc = 0.0f;
            for (int32_t k = 0; k < D; ++k)
                acc = fmaf(lin[rows + k], w[k], acc);
            lin[o] = acc;
        }
    }
    // the other lanes of the ray (same wavefront) read these rows; LDS
    // operations of one wavefront complete in order, so ordering the code
    // suffices
    __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
    __builtin_amdgcn_wave_barrier();
}

// Colour of one occupied sample under Eq. 5: per channel c,
// sigmoid(beta^T b_c + sum_j sum_e (W_c^T beta)[jD + e] k^j_c[e]).
template <typename UT, int DC>
__device__ __forceinline__ void sample_colour_lin(const RenderParams& P, uint32_t t0, uint32_t t1,
                                                  uint32_t t2, const float* lin, float col[3])
{
    const uint32_t texel[3] = {t0, t1, t2};
    if constexpr (DC > 0 && DC % 4 == 0 && (3 * DC * sizeof(UT)) % 16 == 0) {
        constexpr int NV = 3 * DC;
        constexpr uint32_t NB = NV * static_cast<uint32_t>(sizeof(UT));
        constexpr int NQ = NB / 16;
        float x[3] = {lin[9 * DC + 0], lin[9 * DC + 1], lin[9 * DC + 2]};
#pragma unroll
        for (int j = 0; j < 3; ++j) {
            uint4 q[NQ];
#pragma unroll
            for (int k = 0; k < NQ; ++k)
                q[k] = load_at<uint4>(P.uvw[j], texel[j] * NB + 16u * k);
            UT rec[NV];
            __builtin_memcpy(rec, q, NB);
#pragma unroll
            for (int c = 0; c < 3; ++c)
#pragma unroll
                for (int e = 0; e < DC; e += 4) {
                    const float4 w = *reinterpret_cast<const float4*>(lin + c * 3 * DC + j * DC + e);
                    x[c] = fmaf(w.x, widen(rec[c * DC + e + 0]), x[c]);
                    x[c] = fmaf(w.y, widen(rec[c * DC + e + 1]), x[c]);
                    x[c] = fmaf(w.z, widen(rec[c * DC + e + 2]), x[c]);
                    x[c] = fmaf(w.w, widen(rec[c * DC + e + 3]), x[c]);
                }
        }
#pragma unroll
        for (int c = 0; c < 3; ++c)
            col[c] = sigmoid(x[c]);
    } else {
        const int32_t D = P.D;
        const uint32_t nv = 3u * static_cast<uint32_t>(D);
        const uint32_t esz = static_cast<uint32_t>(sizeof(UT));
        for (int c = 0; c < 3; ++c) {
            float x = lin[9 * D + c];
            for (int j = 0; j < 3; ++j)
                for (int32_t e = 0; e < D; ++e) {
                    const uint32_t off = static_cast<uint32_t>(c * D + e);
                    x = fmaf(lin[c * 3 * D + j * D + e], widen(load_at<UT>(P.uvw[j], (texel[j] * nv + off) * esz)), x);
                }
            col[c] = sigmoid(x);
        }
    }
}

// exp(-tau 2^-32) for a 2^-32 fixed-point optical depth.
__device__ __forceinline__ float transmittance(uint64_t tau)
{
    const float hi = static_cast<float>(static_cast<uint32_t>(tau >> 32));
    const float lo = static_cast<float>(static_cast<uint32_t>(tau));
    const float x = fmaf(lo, 0x1p-32f, hi);
    return __builtin_amdgcn_exp2f(-x * kLog2e);
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

// Deferred colour.  An occupied live sample needs its three uvw records
// (nine 16-byte loads at D = 8, binary16) and 3 x 3D multiply-adds; issued
// where the sample is found, they run with only the wave's occupied lanes
// active, and a 16-byte gather costs the memory pipeline the same however few
// lanes take part.  Instead the sample's texels, its Eq. 1 weight
// w = T (1 - exp(-sigma delta)) and its ray go to a per-wave ring of kQueue
// entries in LDS, and whenever 64 are waiting the whole wave evaluates them,
// one per lane, adding w c into per-ray binary64 sums in LDS (the colour
// sums are independent of the order of the samples up to binary64
// rounding).  Depth, sum w t, needs no records and stays in registers.
constexpr uint32_t kQueue = 128;   // 63 waiting + 64 pushed at most

constexpr bool defers_colour(int DC, bool LIN) { return !LIN && (DC == 8 || DC == 16); }

struct ColourQueue {
    uint4* entries;        // [kQueue] wave-private ring: texel0 | slot << 26, texel1, texel2, w
    double* acc;           // [rays per wave][3] rgb sums of the wave's rays
    const float* beta;     // beta of ray slot 0 of the wave; slot r, component k at beta[r + k * BS]
};

// Evaluate the n oldest entries with every lane of the wave present here.
// With all 64 lanes present a quad takes an entry: lane c < 3 evaluates
// colour channel c, reading that channel's part of the entry's record in
// each plane (16 bytes at D = 8 binary16), so the three loads of a quad fall
// in the one or two 64-byte segments of a record instead of one segment per
// lane, which is what a gather costs the memory pipeline; the channel's
// logit sums plane by plane in the order sample_colour uses.  That takes
// four times the rounds, whose vector instructions the one-lane march at D
// = 8 (bound by vector-ALU issue with many views) cannot spare, so QUADS is
// set for rays of four or eight lanes and for D = 16, whose 96-byte records
// leave the vector ALUs idle waiting for HBM.  Otherwise, or in a wave at
// the image edge, one entry per lane.
template <typename UT, int DC, bool LIN, int BS, bool QUADS>  // Eq. 4 only (LIN false)
__device__ __forceinline__ void drain_colour(const RenderParams& P, const ColourQueue& cq, uint32_t& head,
                                             uint32_t n)
{
    const uint64_t ex = __builtin_amdgcn_read_exec();
    if (QUADS && ex == ~0ull) {
        constexpr uint32_t NB = 3u * DC * static_cast<uint32_t>(sizeof(UT));   // bytes of a record
        constexpr uint32_t CB = DC * static_cast<uint32_t>(sizeof(UT));        // bytes of a channel
        constexpr int NQ = CB / 16;
        static_assert(CB % 16 == 0, "channels of whole 16-byte pieces");
        const uint32_t lane = __lane_id();
        const uint32_t c = lane & 3u;
        for (uint32_t done = 0; done < n; done += 16) {
            const uint32_t k = done + (lane >> 2);
            if (k < n && c < 3u) {
                const uint4 e = cq.entries[(head + k) & (kQueue - 1)];
                const uint32_t slot = e.x >> 26;
                const uint32_t texel[3] = {e.x & ((1u << 26) - 1u), e.y, e.z};
                const float* beta = cq.beta + slot;
                float x = 0.0f;
#pragma unroll
                for (int j = 0; j < 3; ++j) {
                    uint4 q[NQ];
#pragma unroll
                    for (int r = 0; r < NQ; ++r)
                        q[r] = load_at<uint4>(P.uvw[j], texel[j] * NB + c * CB + 16u * r);
                    UT rec[DC];
                    __builtin_memcpy(rec, q, CB);
#pragma unroll
                    for (int r = 0; r < DC; ++r)
                        x = fmaf(beta[r * BS], widen(rec[r]), x);
                }
                const double w = static_cast<double>(__uint_as_float(e.w));
                atomicAdd(cq.acc + 3 * slot + c, w * static_cast<double>(sigmoid(x)));
            }
        }
    } else {
        const uint32_t workers = static_cast<uint32_t>(__builtin_popcountll(ex));
        const uint32_t rank = __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(ex >> 32),
                                                        __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(ex), 0u));
        for (uint32_t done = 0; done < n; done += workers) {
            const uint32_t k = done + rank;
            if (k < n) {
                const uint4 e = cq.entries[(head + k) & (kQueue - 1)];
                const uint32_t slot = e.x >> 26;
                const uint32_t t0 = e.x & ((1u << 26) - 1u);
                float col[3];
                sample_colour<UT, DC, BS>(P, t0, e.y, e.z, cq.beta + slot, col);
                const double w = static_cast<double>(__uint_as_float(e.w));
                double* a = cq.acc + 3 * slot;
                atomicAdd(a + 0, w * static_cast<double>(col[0]));
                atomicAdd(a + 1, w * static_cast<double>(col[1]));
                atomicAdd(a + 2, w * static_cast<double>(col[2]));
            }
        }
    }
    head = (head + n) & (kQueue - 1);
}

#ifndef SQN_XCD_BLOCK
#define SQN_XCD_BLOCK 4
#endif

// Packed position record of plane j at a texel: sigma^j and the Chebyshev
// distance (texels) to the nearest texel with sigma^j != 0 (0 = this one),
// see prepare.hip.  binary16 sigma: one word (sigma | dist << 16); binary32
// sigma: two words.
// Byte offset of record (a, b) in a packed plane of B-byte records, four
// rows interleaved: B ((a & ~3) n_p + 4 b + (a & 3)), so a 64-byte segment
// holds a 4 x 4 block of texels (4 x 2 with two-word records): the four
// samples of a ray that a quad gathers together, a texel or two apart,
// touch 2.3 segments per plane on an 800 x 800 view against 3.6 in
// row-major order (2.9 against 3.6 with two-word records), and a gather
// costs the memory pipeline by segments.  Written as row_part(a) + 4 B b
// with row_part(a) = B ((n_p - 1)(a & ~3) + a), each coordinate's part
// shared by its plane; bnm1 = B (n_p - 1).
template <uint32_t B>
__device__ __forceinline__ uint32_t row_part(uint32_t a, uint32_t bnm1)
{
    return __umul24(a & ~3u, bnm1) + a * B;
}
template <uint32_t B>
__device__ __forceinline__ uint32_t record_offset(uint32_t row_a, uint32_t b)
{
    return row_a + b * (4u * B);
}

template <typename ST>
struct SigmaRecord;

template <>
struct SigmaRecord<_Float16> {
    static constexpr uint32_t bytes = 4;
    static __device__ __forceinline__ void load(const void* plane, uint32_t off, float& sigma, uint32_t& dist)
    {
        const uint32_t w = load_at<uint32_t>(plane, off);
        sigma = static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(w & 0xffffu)));
        dist = w >> 16;
    }
};

template <>
struct SigmaRecord<float> {
    static constexpr uint32_t bytes = 8;
    static __device__ __forceinline__ void load(const void* plane, uint32_t off, float& sigma, uint32_t& dist)
    {
        const uint2 w = load_at<uint2>(plane, off);
        sigma = __uint_as_float(w.x);
        dist = w.y;
    }
};

// Sample index just past the exit parameter t_exit of a leap: every sample
// below it has t_k <= t_exit.  x = (t_exit - near) / dt is pulled in by
// 2^-19 (x + |near| / dt): y = t_exit k - c in one fused multiply-add, with
// k = (1 - 2^-19) / dt and c = near k + 2^-19 |near| / dt rounded from
// binary64 on the host.  The roundings of k, c and the fused multiply-add
// stay under 3 units of 2^-24 of |x| + |near| / dt, those of the binary32
// t_k = near + k dt under 8 more, and the pull-in is 32 units; a stratified
// sample k lies at or below t_{k+1} of the uniform grid, so it lands one
// index earlier.  Non-positive y gives an index <= 0 (the caller clamps),
// +inf stays +inf, NaN stays NaN.
__device__ __forceinline__ float leap_index(const RenderParams& P, float t_exit)
{
    const float y = fmaf(t_exit, P.leap_k, -P.leap_c);
    return floorf(y) + (P.stratified ? 0.0f : 1.0f);
}

// First sample index a leap may land on after sample i, whose nearest nodes
// are (c[0], c[1], c[2]) and whose plane `j` texel lies at Chebyshev
// distance D > 0 from every texel with sigma^j != 0.  Every sample whose
// plane-j texel stays within distance D - 1 is empty; along each of the
// plane's two axes the grid coordinate g = (p - bmin) scale moves affinely in
// t (g = g0 + t ds), and the node index stays inside the square while g is
// below c + D - 1/2 (or above c - D + 1/2 moving down).  The bound is pulled
// in by a margin of texels (the binary32 position and rounding error of g),
// so every sample up to the exit parameter is inside the square; `half` is
// 1/2 + that margin, formed once per ray.
// inv_ds[r] = 1 / ds[r], +inf for ds = 0, so that an axis the ray does not
// move along never ends the run (a non-positive distance to the bound there
// gives -inf or NaN, i.e. no leap or the other axis: never a longer one);
// its sign tells the direction.
__device__ __forceinline__ int32_t leap_target(const RenderParams& P, int j, uint32_t D, const uint32_t c[3],
                                               const float g0[3], const float inv_ds[3], float half, int32_t i)
{
    const float h = static_cast<float>(D) - half;
    float t[3];
#pragma unroll
    for (int r = 0; r < 3; ++r) {
        // c + h or c - h
        const float bound = static_cast<float>(c[r]) + copysignf(h, inv_ds[r]);
        t[r] = (bound - g0[r]) * inv_ds[r];
    }
    // plane 0 (xy) uses axes 0, 1; plane 1 (yz) 1, 2; plane 2 (zx) 2, 0
    const float t01 = fminf(t[0], t[1]), t12 = fminf(t[1], t[2]), t20 = fminf(t[2], t[0]);
    const float t_exit = j == 0 ? t01 : (j == 1 ? t12 : t20);
    const float f = leap_index(P, t_exit);
    // clamp to [i + 1, N]; a NaN f gives i + 1 (the median of three takes
    // the smallest when an operand is NaN)
    const float lo = static_cast<float>(i + 1), hi = static_cast<float>(P.n_samples);
    return static_cast<int32_t>(__builtin_amdgcn_fmed3f(f, lo, hi));
}

// First sample index a leap may land on after sample i, whose node indices
// lie in cell cc of the 3-D cell grid (cells of G x G x G nodes) at
// Chebyshev distance D > 0 (in cells) from every cell that may hold
// sigma > 0.  Every sample whose cell stays within distance D - 1 is empty:
// along each axis the node index stays inside cells cc - (D-1) .. cc + (D-1),
// i.e. g in [G (cc - D + 1) - 1/2, G (cc + D) - 1/2), while g = g0 + t ds
// moves affinely in t.  Margins and zero components as in leap_target.
__device__ __forceinline__ int32_t leap_cells(const RenderParams& P, uint32_t D, const uint32_t cc[3],
                                              const float g0[3], const float inv_ds[3], float margin, int32_t i)
{
    const float G = static_cast<float>(1 << P.cell_shift);
    const float Df = static_cast<float>(D);
    float t_exit = INFINITY;
#pragma unroll
    for (int r = 0; r < 3; ++r) {
        const float c = static_cast<float>(cc[r]);
        const float bound = inv_ds[r] > 0.0f ? G * (c + Df) - 0.5f - margin : G * (c - Df + 1.0f) - 0.5f + margin;
        t_exit = fminf(t_exit, (bound - g0[r]) * inv_ds[r]);
    }
    const float f = leap_index(P, t_exit);
    const float lo = static_cast<float>(i + 1), hi = static_cast<float>(P.n_samples);
    return static_cast<int32_t>(fminf(fmaxf(f, lo), hi));
}

// Map the hardware workgroup id to a tile.  Workgroups are dealt
// round-robin over the 8 XCDs.  SQN_XCD_BLOCK = 0: each XCD receives one
// contiguous run of tiles; K > 0: runs of K consecutive tiles are dealt to
// the XCDs in turn (K = 1 is the hardware order).
__device__ __forceinline__ int32_t xcd_tile_order(int32_t bid, int32_t n)
{
    const int32_t xcd = bid & 7, local = bid >> 3;
    if constexpr (SQN_XCD_BLOCK == 0) {
        const int32_t per = n >> 3, rem = n & 7;
        return xcd * per + min(xcd, rem) + local;
    } else {
        constexpr int32_t K = SQN_XCD_BLOCK;
        const int32_t n_full = (n / (8 * K)) * (8 * K);
        if (bid >= n_full)
            return bid;
        return (xcd + 8 * (local / K)) * K + (local % K);
    }
}

// Waves per SIMD the register allocation is asked to allow: a single
// 800x800 view is 10^4 waves at one lane per ray, so occupancy decides how
// much of the frame runs in a second round.  Larger records need more
// registers; the targets are the highest that compile without spilling.
constexpr int waves_per_simd(int record_bytes)
{
    return record_bytes == 0 ? 6 : (record_bytes <= 48 ? 8 : (record_bytes <= 96 ? 5 : 4));
}

// What the march needs of one ray besides beta: the ray (after the NDC map
// for forward-facing captures), |d|, the conservative sample range of the
// box and the affine grid coordinates of the leaps.
struct RayGeom {
    float o[3], d[3];
    float dn;
    float g0[3], inv_ds[3];   // grid coordinate g = g0 + t ds per axis, 1/ds
    float margin;             // texels a leap keeps from its square's edge
    int32_t i0, i1;           // samples that may lie in the box
    int32_t j0;               // samples certainly in the box: i - j0 <= jspan as unsigned
    uint32_t jspan;           // (j0 = INT_MIN, jspan = 0 when there are none)
};

// World ray through the pixel centre of (u, v) (camera looks down -z).
__device__ __forceinline__ void pixel_ray(const RenderParams& P, int32_t view, int32_t u, int32_t v,
                                          float o[3], float d[3])
{
    const float* pose = P.poses + 12 * static_cast<int64_t>(view);
    float pm[12];
#pragma unroll
    for (int k = 0; k < 12; ++k)
        pm[k] = pose[k];
    const float a = ((static_cast<float>(u) + 0.5f) - P.cx) / P.fx;
    const float b = -(((static_cast<float>(v) + 0.5f) - P.cy) / P.fy);
#pragma unroll
    for (int r = 0; r < 3; ++r) {
        const float pa = pm[4 * r + 0] * a;
        const float pb = pm[4 * r + 1] * b;
        d[r] = (pa + pb) - pm[4 * r + 2];
        o[r] = pm[4 * r + 3];
    }
}

// RayGeom from the world ray (o, d): NDC map, |d|, box clip, leap constants.
template <bool SKIP, bool NDC>
__device__ __forceinline__ void march_geometry(const RenderParams& P, const float o_w[3], const float d_w[3],
                                               RayGeom& g)
{
#pragma unroll
    for (int r = 0; r < 3; ++r) {
        g.o[r] = o_w[r];
        g.d[r] = d_w[r];
    }
    // forward-facing captures march in normalized device coordinates
    bool no_samples = false;
    if constexpr (NDC)
        no_samples = !ndc_ray(P, g.o, g.d);
    const float d00 = g.d[0] * g.d[0], d11 = g.d[1] * g.d[1], d22 = g.d[2] * g.d[2];
    g.dn = sqrtf((d00 + d11) + d22);
    int32_t j1;
    clip_to_box(P, g.o, g.d, g.i0, g.i1, g.j0, j1);
    if constexpr (NDC) {
        if (no_samples) {
            g.i0 = 1;
            g.i1 = 0;
            g.j0 = 1;
            j1 = 0;
        }
    }
    if (g.j0 <= j1) {
        g.jspan = static_cast<uint32_t>(j1 - g.j0);
    } else {
        g.j0 = INT32_MIN;
        g.jspan = 0;
    }
    g.margin = 0.0f;
    if constexpr (SKIP) {
#pragma unroll
        for (int r = 0; r < 3; ++r) {
            g.g0[r] = (g.o[r] - P.bmin[r]) * P.scale[r];
            const float ds = g.d[r] * P.scale[r];
            g.inv_ds[r] = ds == 0.0f ? INFINITY : __builtin_amdgcn_rcpf(ds);
        }
        // binary32 rounding of g along the exact path, of g + 1/2 at the node
        // boundary and of this affine estimate all stay below 2^-20 times
        // the magnitudes involved (about 16 units in the last place)
        float mag = static_cast<float>(P.n_p);
#pragma unroll
        for (int r = 0; r < 3; ++r)
            mag = fmaxf(mag, fabsf(g.g0[r]) + fabsf(g.d[r] * P.scale[r]) * fabsf(P.far_t)
                                 + P.scale[r] * (fabsf(P.bmin[r]) + fabsf(P.bmax[r])));
        g.margin = P.leap_margin + 0x1p-20f * mag;
    }
}

// One ray (or, with L lanes per ray, one L-lane group) at pixel (u, v) of
// view `view`; `lane` is the lane index in the wave.
// SKIP: leap over runs of samples that one plane's distance field proves
// empty (with L lanes per ray, the next chunk starts at the furthest end of
// the runs its lanes found).
// COOP: the workgroup computed the ray's geometry and beta once per ray
// (`pre`; beta at beta[k * BS]) instead of in each of its L lanes.
template <typename ST, typename UT, int DC, bool STATS, int L, bool SKIP, bool LIN, bool NDC, bool COOP = false,
          int BS = kBlockThreads>
__device__ __forceinline__ void render_ray(const RenderParams& P, int32_t view, int32_t u,
                                           int32_t v, int32_t lane, float* const beta, float* const lin,
                                           const ColourQueue& cq, int32_t slot, const RayGeom* pre = nullptr)
{
    static_assert(L == 1 || L == 4 || L == 8, "one, four or eight lanes per ray");
    const int32_t s = (L == 1) ? 0 : (lane & (L - 1));
    const int64_t ray = (static_cast<int64_t>(view) * P.height + v) * P.width + u;
    const int32_t N = P.n_samples;
    const bool stratified = P.stratified != 0;
    const uint64_t ray_key = static_cast<uint64_t>(ray) * static_cast<uint64_t>(N);

    RayGeom geo;
    if constexpr (COOP) {
        geo = *pre;
        // Eq. 5: beta waits in the ray's LDS row; the L lanes fold it
        if constexpr (LIN)
            fold_decoder<DC, L>(P, s, lin);
        if constexpr (!NDC) {
            // a world ray starts at the camera centre, the same for the whole
            // view: taken from the pose, it and its grid coordinates stay in
            // scalar registers (the same binary32 operations as the setup)
            const float* pose = P.poses + 12 * static_cast<int64_t>(view);
#pragma unroll
            for (int r = 0; r < 3; ++r) {
                geo.o[r] = pose[4 * r + 3];
                if constexpr (SKIP)
                    geo.g0[r] = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(
                                    int, (geo.o[r] - P.bmin[r]) * P.scale[r])));
            }
        }
    } else {
        float o_w[3], d_w[3];
        pixel_ray(P, view, u, v, o_w, d_w);
        // direction weights from the world direction
        if constexpr (LIN) {
            // beta goes to the ray's LDS row (the L lanes write equal values)
            lookup_beta<DC, 1>(P, d_w, DC > 0 ? lin : lin + 9 * P.D + 3);
            __builtin_amdgcn_fence(__ATOMIC_ACQ_REL, "wavefront");
            fold_decoder<DC, L>(P, s, lin);
        } else {
            lookup_beta<DC, BS>(P, d_w, beta);
        }
        march_geometry<SKIP, NDC>(P, o_w, d_w, geo);
    }
    const float* const o = geo.o;
    const float* const d = geo.d;
    const float dn = geo.dn;
    const int32_t i0 = geo.i0, i1 = geo.i1, j0 = geo.j0;
    const uint32_t jspan = geo.jspan;
    const float* const g0 = geo.g0;
    const float* const inv_ds = geo.inv_ds;
    const float leap_margin = geo.margin;
    const float leap_half = 0.5f + leap_margin;
    const int32_t n_p = P.n_p;
    const float hi_node = static_cast<float>(n_p - 1);
    // Eq. 4 at D = 8 and 16 defers colour to the wave's queue (measured:
    // 4-8% faster on every D = 8 workload; at D = 16, drained by quads, 7%
    // faster on the HBM-bound 1920x1080 view in its hybrid shape and 13%
    // with one lane); Eq. 5 keeps a row of folded weights per ray in LDS
    // and, like the other D, evaluates colour where the sample is found
    constexpr bool kDefer = defers_colour(DC, LIN);
    uint64_t tau = 0;              // optical depth before the chunk, 2^-32 units
    double acc_r = 0.0, acc_g = 0.0, acc_b = 0.0, acc_t = 0.0;
    int32_t last_live = -1;
    uint32_t n_inbox = 0, n_occ = 0, hash = 2166136261u;
    // the ray's colour sums, written by whichever lanes evaluate its samples
    if (kDefer && s == 0) {
        cq.acc[3 * slot + 0] = 0.0;
        cq.acc[3 * slot + 1] = 0.0;
        cq.acc[3 * slot + 2] = 0.0;
    }
    uint32_t q_head = 0, q_count = 0;   // the wave's queue, wave-uniform

    int32_t base = i0;
    // t of this lane's sample in the current chunk
    float t = (base <= i1) ? sample_t(P, stratified, ray_key, base + s) : 0.0f;
    // with deferred colour every lane present stays in the loop until the
    // wave is done, so that the whole wave evaluates the queued colours;
    // otherwise a lane leaves as soon as its ray is done
    for (;;) {
        const bool active = base <= i1 && tau <= static_cast<uint64_t>(P.tau_eps);
        if constexpr (kDefer) {
            if (__builtin_amdgcn_ballot_w64(active) == 0)
                break;
        } else if (!active) {
            break;
        }
        bool pushed = false;
        if (active) {
        const int32_t i = base + s;
        const bool in_range = i <= i1;
        const float t_next_chunk = sample_t(P, stratified, ray_key, base + L + s);

        float p[3];
#pragma unroll
        for (int r = 0; r < 3; ++r) {
            const float td = t * d[r];
            p[r] = o[r] + td;
        }
        bool inside;
        uint32_t ix, iy, iz;
        // when every lane's sample is certainly in the box the six exact
        // tests would all pass and the node indices need no clamp (a
        // wave-uniform branch)
        // 0 <= i - j0 <= jspan, one unsigned compare (i >= 0 > INT_MIN)
        const bool deep = static_cast<uint32_t>(i) - static_cast<uint32_t>(j0) <= jspan;
        if (__builtin_amdgcn_ballot_w64(deep) == __builtin_amdgcn_read_exec()) {
            inside = true;
            ix = nearest_node_inside(p[0], P.bmin[0], P.scale[0]);
            iy = nearest_node_inside(p[1], P.bmin[1], P.scale[1]);
            iz = nearest_node_inside(p[2], P.bmin[2], P.scale[2]);
        } else {
            inside = in_range & (p[0] >= P.bmin[0]) & (p[0] <= P.bmax[0]) & (p[1] >= P.bmin[1])
                     & (p[1] <= P.bmax[1]) & (p[2] >= P.bmin[2]) & (p[2] <= P.bmax[2]);
            // node indices are clamped to the grid for any position; they
            // are used only for samples inside the box
            ix = nearest_node(p[0], P.bmin[0], P.scale[0], hi_node);
            iy = nearest_node(p[1], P.bmin[1], P.scale[1], hi_node);
            iz = nearest_node(p[2], P.bmin[2], P.scale[2], hi_node);
        }
        float sigma = 0.0f;
        int32_t leap = 0;
        if (inside) {
            // Eq. 5: a sample in an empty cell of the 3-D cell grid has
            // sigma = 0 without reading the planes
            bool dead = false;
            if constexpr (LIN && SKIP) {
                const uint32_t cc[3] = {ix >> P.cell_shift, iy >> P.cell_shift, iz >> P.cell_shift};
                const uint32_t cd = P.cell_dist[(cc[0] * P.cell_m + cc[1]) * P.cell_m + cc[2]];
                if (cd != 0) {
                    dead = true;
                    leap = leap_cells(P, cd, cc, g0, inv_ds, leap_margin, i);
                }
            }
            if (!dead) {
                float sxy, syz, szx;
                uint32_t dxy, dyz, dzx;
                constexpr uint32_t RB = SigmaRecord<ST>::bytes;
                const uint32_t bnm1 = RB * static_cast<uint32_t>(n_p - 1);
                SigmaRecord<ST>::load(P.sigma[0], record_offset<RB>(row_part<RB>(ix, bnm1), iy), sxy, dxy);
                SigmaRecord<ST>::load(P.sigma[1], record_offset<RB>(row_part<RB>(iy, bnm1), iz), syz, dyz);
                SigmaRecord<ST>::load(P.sigma[2], record_offset<RB>(row_part<RB>(iz, bnm1), ix), szx, dzx);
                if constexpr (LIN) {
                    // Eq. 5 on the folded per-plane partial sums
                    float pre = sxy + syz;
                    pre = pre + szx;
                    pre = pre + P.b_sigma;
                    sigma = pre > 0.0f ? pre : 0.0f;
                } else {
                    // Eq. 4
                    float prod = sxy * syz;
                    prod = prod * szx;
                    sigma = fmaxf(0.0f, prod);
                }
                if constexpr (SKIP) {
                    const uint32_t dmax = max(dxy, max(dyz, dzx));
                    if (dmax != 0) {
                        const int j = (dxy == dmax) ? 0 : ((dyz == dmax) ? 1 : 2);
                        const uint32_t c[3] = {ix, iy, iz};
                        leap = leap_target(P, j, dmax, c, g0, inv_ds, leap_half, i);
                    }
                }
            }
        }
        // in-box samples among first .. last-1 (diagnostics of a leap)
        auto count_inbox = [&](int32_t first, int32_t last) {
            uint32_t n = 0;
            for (int32_t k = first; k < last; ++k) {
                const float tk = sample_t(P, stratified, ray_key, k);
                bool in_k = true;
#pragma unroll
                for (int r = 0; r < 3; ++r) {
                    const float pk = o[r] + tk * d[r];
                    in_k = in_k & (pk >= P.bmin[r]) & (pk <= P.bmax[r]);
                }
                n += in_k ? 1u : 0u;
            }
            return n;
        };
        bool leapt = false;
        if constexpr (SKIP && L == 1) {
            if (leap != 0) {
                // samples i .. leap-1 are empty: sample i has sigma^j = 0 in
                // the plane with distance dmax, the rest stay within its
                // empty square
                if constexpr (STATS)
                    n_inbox += count_inbox(i, leap);
                base = leap;
                t = sample_t(P, stratified, ray_key, base);
                leapt = true;
            }
        }
        if (!leapt) {
        float q = 0.0f;
        uint64_t excl = 0, total = 0;
        // a chunk in which no lane of the wave is occupied adds nothing to
        // the optical depth: the exchange of t and the scan are skipped (a
        // wave-uniform branch, so every group is whole inside it)
        if (L == 1 || __builtin_amdgcn_ballot_w64(sigma > 0.0f) != 0) {
            // t_{i+1}: the next lane's t, or for the group's last lane the
            // first sample of the next chunk
            const float t_first_next = grp_first<L>(t_next_chunk);
            const float t_lane_next = grp_next<L>(t);
            float tn = (s == L - 1) ? t_first_next : t_lane_next;
            if (i + 1 >= N)
                tn = P.far_t;
            uint64_t Q = 0;
            if (sigma > 0.0f) {
                const float gap = fmaxf(0.0f, tn - t);
                const float delta = gap * dn;
                q = sigma * delta;
                Q = fixed_q(q);
            }
            grp_scan<L>(Q, s, excl, total);
        }
        const uint64_t tau_i = tau + excl;
        // with one lane per ray the loop condition already guarantees
        // tau_i = tau <= tau_eps and i <= i1
        const bool live = (L == 1) || (in_range & (tau_i <= static_cast<uint64_t>(P.tau_eps)));
        const bool occ = live & (sigma > 0.0f);
        // queue positions of this step's occupied samples, in lane order
        const uint64_t occ_mask = kDefer ? __builtin_amdgcn_ballot_w64(occ) : 0;
        if (occ && !kDefer) {
            float col[3];
            if constexpr (LIN)
                sample_colour_lin<UT, DC>(P, __umul24(ix, n_p) + iy, __umul24(iy, n_p) + iz,
                                          __umul24(iz, n_p) + ix, lin, col);
            else
                sample_colour<UT, DC, BS>(P, __umul24(ix, n_p) + iy, __umul24(iy, n_p) + iz,
                                          __umul24(iz, n_p) + ix, beta, col);
            const float T = transmittance(tau_i);
            const float alpha = -expm1f(-q);
            const double w = static_cast<double>(T * alpha);
            acc_r = fma(w, static_cast<double>(col[0]), acc_r);
            acc_g = fma(w, static_cast<double>(col[1]), acc_g);
            acc_b = fma(w, static_cast<double>(col[2]), acc_b);
            acc_t = fma(w, static_cast<double>(t), acc_t);
        }
        if (occ && kDefer) {
            const float T = transmittance(tau_i);
            const float alpha = -expm1f(-q);
            const float w = T * alpha;
            acc_t = fma(static_cast<double>(w), static_cast<double>(t), acc_t);
            const uint32_t rank = __builtin_amdgcn_mbcnt_hi(static_cast<uint32_t>(occ_mask >> 32),
                                                            __builtin_amdgcn_mbcnt_lo(static_cast<uint32_t>(occ_mask), 0u));
            cq.entries[(q_head + q_count + rank) & (kQueue - 1)] =
                make_uint4((__umul24(ix, n_p) + iy) | (static_cast<uint32_t>(slot) << 26), __umul24(iy, n_p) + iz,
                           __umul24(iz, n_p) + ix, __float_as_uint(w));
            pushed = true;
        }
        if (L > 1 && live)
            last_live = i;
        if constexpr (STATS) {
            n_inbox += (live & inside) ? 1u : 0u;
            n_occ += occ ? 1u : 0u;
            // FNV-1a over the occupied samples of the group in sample order
#pragma unroll
            for (int k = 0; k < L; ++k) {
                const int src = (lane & ~(L - 1)) + k;
                const bool o_k = __shfl(occ ? 1 : 0, src) != 0;
                const uint32_t i_k = static_cast<uint32_t>(__shfl(i, src));
                const uint32_t x_k = static_cast<uint32_t>(__shfl(static_cast<int>(ix), src));
                const uint32_t y_k = static_cast<uint32_t>(__shfl(static_cast<int>(iy), src));
                const uint32_t z_k = static_cast<uint32_t>(__shfl(static_cast<int>(iz), src));
                if (o_k) {
                    hash = fnv1a_word(hash, i_k);
                    hash = fnv1a_word(hash, x_k);
                    hash = fnv1a_word(hash, y_k);
                    hash = fnv1a_word(hash, z_k);
                }
            }
        }
        tau += total;
        int32_t next = base + L;
        if constexpr (SKIP && L > 1) {
            // every lane's empty run [i, leap) is a valid leap: the next chunk
            // starts at the furthest one that ends past this chunk
            const int32_t last_leap = grp_max<L>(leap);
            if (last_leap > next && tau <= static_cast<uint64_t>(P.tau_eps)) {
                if constexpr (STATS) {
                    if (s == 0)
                        n_inbox += count_inbox(next, last_leap);
                }
                next = last_leap;
            }
        }
        t = (next == base + L) ? t_next_chunk : sample_t(P, stratified, ray_key, next + s);
        base = next;
        }   // !leapt
        }   // active
        if constexpr (kDefer) {
            // whole wave: count the pushes; evaluate 64 once they are waiting
            q_count += static_cast<uint32_t>(__builtin_popcountll(__builtin_amdgcn_ballot_w64(pushed)));
            if (q_count >= 64) {
                drain_colour<UT, DC, LIN, BS, (L > 1 || DC == 16)>(P, cq, q_head, 64);
                q_count -= 64;
            }
        }
    }
    if constexpr (kDefer)
        drain_colour<UT, DC, LIN, BS, (L > 1 || DC == 16)>(P, cq, q_head, q_count);

    // combine the lanes of the ray
    if constexpr (!kDefer) {
        acc_r = grp_sum<L>(acc_r);
        acc_g = grp_sum<L>(acc_g);
        acc_b = grp_sum<L>(acc_b);
    }
    acc_t = grp_sum<L>(acc_t);
    // the first non-live sample: with one lane per ray the loop leaves as
    // soon as the optical depth crosses, at the index after the last sample
    const bool terminated = tau > static_cast<uint64_t>(P.tau_eps);
    const int32_t stop = !terminated ? N : (L == 1 ? base : grp_max<L>(last_live) + 1);
    if constexpr (STATS) {
        n_inbox = grp_add<L>(n_inbox);
        n_occ = grp_add<L>(n_occ);
    }
    if (s != 0)
        return;
    // outputs are written once and never read here: streaming stores keep
    // the partially written lines of a pixel tile from being allocated in
    // L2 and written back piecemeal while the gathers churn it
    if (P.rgb) {
        if constexpr (kDefer) {
            acc_r = cq.acc[3 * slot + 0];
            acc_g = cq.acc[3 * slot + 1];
            acc_b = cq.acc[3 * slot + 2];
        }
        __builtin_nontemporal_store(static_cast<float>(acc_r), P.rgb + 3 * ray + 0);
        __builtin_nontemporal_store(static_cast<float>(acc_g), P.rgb + 3 * ray + 1);
        __builtin_nontemporal_store(static_cast<float>(acc_b), P.rgb + 3 * ray + 2);
    }
    if (P.depth)
        __builtin_nontemporal_store(static_cast<float>(acc_t), P.depth + ray);
    if constexpr (STATS) {
        uint4 st;
        st.x = static_cast<uint32_t>(stop);
        st.y = n_inbox;
        st.z = n_occ;
        st.w = hash;
        reinterpret_cast<uint4*>(P.stats)[ray] = st;
    }
}

// Launch shapes: L = 1, 4 or 8 lanes per ray over workgroup tiles of
// kTileW(L) x kTileH(L) pixels, with or without leaps over empty space.
// LDS floats of the folded Eq. 5 weights per workgroup (64 rays); a run-time
// D also keeps beta after the rows.
template <int DC, bool LIN>
constexpr int lin_smem_floats()
{
    return LIN ? (DC > 0 ? lin_stride(DC) : lin_stride_generic(32)) * (kBlockThreads / 4) : 4;
}

// LDS floats of beta per workgroup: one copy per lane with one lane per
// ray, one per ray (64) with four; Eq. 5 keeps it in the folded rows.
template <int DC, bool LIN, int L = 1>
constexpr int beta_smem_floats()
{
    return LIN ? 4 : (DC > 0 ? DC : 32) * (L == 4 ? 64 : kBlockThreads);
}

// Waves per SIMD: the register target, capped by how many 4-wave workgroups
// the 160 KiB of LDS of a compute unit holds.
template <typename UT, int DC, bool LIN, bool NDC = false, int L = 1>
constexpr int occupancy()
{
    // the Eq. 5 path holds more per-ray state (LDS row pointers, folded
    // biases); six waves leave it room without spilling.  The NDC map keeps
    // a few more values across the march (at eight waves the forward-facing
    // kernel spilled three registers and ran 7% slower), and the four-lane
    // kernels that read their ray setup from LDS (four or eight lanes)
    // measured 3-4% faster at seven waves than at eight: one wave less for
    // both.
    constexpr int rec0 = waves_per_simd(3 * DC * static_cast<int>(sizeof(UT)));
    constexpr int rec = (NDC || (L >= 4 && !LIN)) && rec0 > 4 ? rec0 - 1 : rec0;
    constexpr int regs = LIN && rec > 6 ? 6 : rec;
    constexpr int lds = 4 * (lin_smem_floats<DC, LIN>() + beta_smem_floats<DC, LIN>())
                        + (defers_colour(DC, LIN) ? 4 * static_cast<int>(kQueue) * 16 + 4 * (64 / L) * 3 * 8 : 0);
    constexpr int by_lds = 163840 / lds;
    return regs < by_lds ? regs : (by_lds < 1 ? 1 : by_lds);
}

// One workgroup's rays at tile (tx, ty) of view `view`, with the LDS arrays
// of the launch shape: beta, the Eq. 5 rows, the colour queue and sums, and
// (four or eight lanes) the rays' march geometry.
template <typename ST, typename UT, int DC, bool STATS, int L, bool SKIP, bool LIN, bool NDC>
__device__ __forceinline__ void workgroup_rays(const RenderParams& P, int32_t view, int32_t tx, int32_t ty,
                                               float* beta_smem, float* lin_smem, uint4* queue_smem,
                                               double* qacc_smem, RayGeom* geom)
{
    const int32_t lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    constexpr int32_t WW = kWaveW(L), WH = kWaveH(L);
    const int32_t slot = lane / L;
    const int32_t u = tx * kTileW(L) + (wave & 1) * WW + (slot % WW);
    const int32_t v = ty * kTileH(L) + (wave >> 1) * WH + (slot / WW);
    if constexpr (L >= 4) {
        // Four or eight lanes per ray: the first wave computes beta and the
        // second the march geometry of the workgroup's 256 / L rays, one lane
        // per ray, and the four waves march from them; the ray setup then
        // costs one wave's instructions per workgroup instead of L (the
        // march is bound by vector-ALU issue).  Eq. 5 (four lanes) keeps
        // beta in the ray's row of folded weights, which its lanes fold.
        constexpr int32_t stride = LIN && DC > 0 ? lin_stride(DC) : 0;
        auto lin_row = [&](int32_t r) { return lin_smem + r * (DC > 0 ? stride : P.lin_stride); };
        constexpr int32_t RPW = 64 / L;   // rays per wave
        if (wave < 2 && lane < 4 * RPW) {
            const int32_t w = lane / RPW, sl = lane % RPW;
            const int32_t ur = tx * kTileW(L) + (w & 1) * WW + (sl % WW);
            const int32_t vr = ty * kTileH(L) + (w >> 1) * WH + (sl / WW);
            if (view < P.n_views && ur < P.width && vr < P.height) {
                float o_w[3], d_w[3];
                pixel_ray(P, view, ur, vr, o_w, d_w);
                // wave 0: beta, wave 1: the march geometry
                if (wave == 0) {
                    if constexpr (LIN)
                        lookup_beta<DC, 1>(P, d_w, DC > 0 ? lin_row(lane) : lin_row(lane) + 9 * P.D + 3);
                    else
                        lookup_beta<DC, 64>(P, d_w, beta_smem + lane);
                } else {
                    march_geometry<SKIP, NDC>(P, o_w, d_w, geom[lane]);
                }
            }
        }
        __syncthreads();
        const int32_t r = wave * RPW + slot;
        ColourQueue cq;
        cq.entries = queue_smem + wave * kQueue;
        cq.acc = qacc_smem + wave * RPW * 3;
        cq.beta = beta_smem + wave * RPW;
        if (view < P.n_views && u < P.width && v < P.height)
            render_ray<ST, UT, DC, STATS, L, SKIP, LIN, NDC, true, 64>(P, view, u, v, lane, beta_smem + r,
                                                                      LIN ? lin_row(r) : nullptr, cq, slot, &geom[r]);
    } else {
        // all lanes of a ray agree on this, so a lane group is never split
        static_assert(!LIN, "the Eq. 5 decoder runs with four lanes per ray");
        if (view < P.n_views && u < P.width && v < P.height) {
            ColourQueue cq;
            cq.entries = queue_smem + wave * kQueue;
            cq.acc = qacc_smem + wave * 64 * 3;
            cq.beta = beta_smem + wave * 64;
            render_ray<ST, UT, DC, STATS, L, SKIP, LIN, NDC>(P, view, u, v, lane, beta_smem + threadIdx.x, nullptr,
                                                        cq, slot);
        }
    }
}

// k -> n/2, n/2 - 1, n/2 + 1, ...: a bijection of [0, n) that starts at the
// middle
__device__ __forceinline__ int32_t centre_first(int32_t k, int32_t n)
{
    return (k & 1) == 0 ? n / 2 + k / 2 : n / 2 - 1 - k / 2;
}

template <typename ST, typename UT, int DC, bool STATS, int L, bool SKIP, bool LIN, bool NDC>
__global__ __launch_bounds__(kBlockThreads, (occupancy<UT, DC, LIN, NDC, L>())) void render_kernel(const RenderParams P)
{
    // beta of every lane's ray, component-major so that a wave-wide read of
    // one component touches consecutive LDS words; each lane reads only what
    // it wrote, so no barrier is needed
    __shared__ float beta_smem[beta_smem_floats<DC, LIN, L>()];
    // Eq. 5: one row of folded weights per ray, written and read only by
    // the ray's own lanes
    __shared__ __align__(16) float lin_smem[lin_smem_floats<DC, LIN>()];
    // deferred colour: a ring of queued samples and the rays' rgb sums per wave
    constexpr bool kDefer = defers_colour(DC, LIN);
    __shared__ uint4 queue_smem[kDefer ? 4 * kQueue : 1];
    __shared__ double qacc_smem[kDefer ? 4 * (64 / L) * 3 : 1];
    __shared__ RayGeom geom_smem[L >= 4 ? 64 : 1];
    int32_t view, tx, ty;
    if (P.block_order) {
        // one view: blocks of 2 x 2 tiles from the centre outwards (the
        // waves over a centred object carry the longest chains of samples
        // and set the view's time, so they start first and the light edge
        // tiles fill the end of the launch), the four workgroups of a block
        // the ones 8 apart in dispatch order (one XCD, whose L2 then holds
        // their shared texels); the grid covers whole blocks, and tiles past
        // the image edge render nothing
        const int32_t bx = (P.tiles_x + 1) >> 1, by = (P.tiles_y + 1) >> 1;
        const int32_t bid = static_cast<int32_t>(blockIdx.x);
        int32_t blk = bid >> 2, sub = bid & 3;
        if (bid < (P.n_groups & ~31)) {
            const int32_t li = bid >> 3;
            blk = 8 * (li >> 2) + (bid & 7);
            sub = li & 3;
        }
        view = 0;
        tx = 2 * centre_first(blk % bx, bx) + (sub & 1);
        ty = 2 * centre_first(blk / bx, by) + (sub >> 1);
    } else {
        const int32_t tile = xcd_tile_order(static_cast<int32_t>(blockIdx.x), P.n_groups);
        const int32_t tiles_per_view = P.tiles_x * P.tiles_y;
        view = tile / tiles_per_view;
        const int32_t tr = tile - view * tiles_per_view;
        ty = tr / P.tiles_x;
        tx = tr - ty * P.tiles_x;
    }
    workgroup_rays<ST, UT, DC, STATS, L, SKIP, LIN, NDC>(P, view, tx, ty, beta_smem, lin_smem, queue_smem, qacc_smem,
                                                         geom_smem);
}

// LDS bytes of one workgroup of a hybrid launch with L lanes per ray: the
// colour queue, the rays' rgb sums, (four lanes) the march geometry, beta;
// both shapes carve them from one buffer, 16-byte aligned.
template <typename UT, int DC, int L>
constexpr int hybrid_lds_bytes()
{
    constexpr bool defer = defers_colour(DC, false);
    return (defer ? 4 * static_cast<int>(kQueue) * 16 : 16) + (defer ? 4 * (64 / L) * 3 * 8 : 16)
           + (L >= 4 ? 64 * static_cast<int>(sizeof(RayGeom)) : 0) + 4 * beta_smem_floats<DC, false, L>();
}

template <typename UT, int DC>
constexpr int hybrid_occupancy()
{
    constexpr int a = occupancy<UT, DC, false, false, 1>(), b = occupancy<UT, DC, false, false, 4>();
    constexpr int bytes = hybrid_lds_bytes<UT, DC, 1>() > hybrid_lds_bytes<UT, DC, 4>()
                              ? hybrid_lds_bytes<UT, DC, 1>()
                              : hybrid_lds_bytes<UT, DC, 4>();
    constexpr int by_lds = 163840 / bytes;
    constexpr int m = a < b ? a : b;
    return m < by_lds ? m : by_lds;
}

// One view, leaps, world rays, Eq. 4.  The image is cut into blocks of 16 x
// 16 pixels (one workgroup of one lane per ray, four of four lanes); the
// first n_heavy workgroups march a centred rectangle of hy_w x hy_h blocks
// with four lanes per ray (the long chains of samples over a centred object
// become four times shorter), the others march every other block with one
// lane per ray (a quarter of the instructions).  Workgroups are either kind
// as a whole, so the barrier of the four-lane setup is taken by all or none
// of a workgroup's waves.
template <typename ST, typename UT, int DC, bool STATS>
__global__ __launch_bounds__(kBlockThreads, (hybrid_occupancy<UT, DC>())) void render_kernel_hybrid(
    const RenderParams P)
{
    constexpr bool kDefer = defers_colour(DC, false);
    constexpr int kQ = kDefer ? 4 * static_cast<int>(kQueue) * 16 : 16;
    constexpr int kBytes = hybrid_lds_bytes<UT, DC, 1>() > hybrid_lds_bytes<UT, DC, 4>()
                               ? hybrid_lds_bytes<UT, DC, 1>()
                               : hybrid_lds_bytes<UT, DC, 4>();
    __shared__ __align__(16) unsigned char lds[kBytes];
    uint4* queue = reinterpret_cast<uint4*>(lds);
    const int32_t bid = static_cast<int32_t>(blockIdx.x);
    if (bid < P.n_heavy) {
        // four workgroups (8 x 8 pixels each) per block; blocks from the
        // middle of the rectangle outwards
        constexpr int kAcc = kDefer ? 4 * 16 * 3 * 8 : 16;
        double* acc = reinterpret_cast<double*>(lds + kQ);
        RayGeom* geom = reinterpret_cast<RayGeom*>(lds + kQ + kAcc);
        float* beta = reinterpret_cast<float*>(lds + kQ + kAcc + 64 * sizeof(RayGeom));
        // consecutive workgroups go to the 8 XCDs in turn: the four of a
        // block are the ones 8 apart, so they share one XCD's L2 (a full
        // group of 8 blocks at a time; the last partial group in order)
        int32_t blk = bid >> 2, sub = bid & 3;
        if (bid < (P.n_heavy & ~31)) {
            const int32_t xcd = bid & 7, li = bid >> 3;
            blk = 8 * (li >> 2) + xcd;
            sub = li & 3;
        }
        const int32_t by = P.hy_y0 + centre_first(blk / P.hy_w, P.hy_h);
        const int32_t bx = P.hy_x0 + centre_first(blk % P.hy_w, P.hy_w);
        workgroup_rays<ST, UT, DC, STATS, 4, true, false, false>(P, 0, 2 * bx + (sub & 1), 2 * by + (sub >> 1), beta,
                                                                 nullptr, queue, acc, geom);
    } else {
        // the blocks outside the rectangle, row by row: the rows above it,
        // the rows beside it (left part, then right part), the rows below
        constexpr int kAcc = kDefer ? 4 * 64 * 3 * 8 : 16;
        double* acc = reinterpret_cast<double*>(lds + kQ);
        float* beta = reinterpret_cast<float*>(lds + kQ + kAcc);
        int32_t l = bid - P.n_heavy, bx, by;
        const int32_t above = P.hy_y0 * P.hy_bx, side = P.hy_bx - P.hy_w;
        if (l < above) {
            by = l / P.hy_bx;
            bx = l - by * P.hy_bx;
        } else if ((l -= above) < P.hy_h * side) {
            const int32_t r = l / side, k = l - r * side;
            by = P.hy_y0 + r;
            bx = k < P.hy_x0 ? k : k + P.hy_w;
        } else {
            l -= P.hy_h * side;
            const int32_t r = l / P.hy_bx;
            by = P.hy_y0 + P.hy_h + r;
            bx = l - r * P.hy_bx;
        }
        workgroup_rays<ST, UT, DC, STATS, 1, true, false, false>(P, 0, bx, by, beta, nullptr, queue, acc, nullptr);
    }
}

template <typename ST, typename UT, int DC>
hipError_t launch_hybrid(const RenderParams& p, bool stats, hipStream_t stream)
{
    const dim3 grid(static_cast<uint32_t>(p.n_groups));
    const dim3 block(kBlockThreads);
    if (stats)
        render_kernel_hybrid<ST, UT, DC, true><<<grid, block, 0, stream>>>(p);
    else
        render_kernel_hybrid<ST, UT, DC, false><<<grid, block, 0, stream>>>(p);
    return hipGetLastError();
}

template <typename ST, typename UT, int DC, int L, bool SKIP, bool LIN, bool NDC>
hipError_t launch_ray_space(const RenderParams& p, bool stats, hipStream_t stream)
{
    const dim3 grid(static_cast<uint32_t>(p.n_groups));
    const dim3 block(kBlockThreads);
    if (stats)
        render_kernel<ST, UT, DC, true, L, SKIP, LIN, NDC><<<grid, block, 0, stream>>>(p);
    else
        render_kernel<ST, UT, DC, false, L, SKIP, LIN, NDC><<<grid, block, 0, stream>>>(p);
    return hipGetLastError();
}

// world rays, or forward-facing rays in normalized device coordinates
template <typename ST, typename UT, int DC, int L, bool SKIP, bool LIN>
hipError_t launch_shape(const RenderParams& p, bool stats, hipStream_t stream)
{
    return p.ndc_near > 0.0f ? launch_ray_space<ST, UT, DC, L, SKIP, LIN, true>(p, stats, stream)
                             : launch_ray_space<ST, UT, DC, L, SKIP, LIN, false>(p, stats, stream);
}

template <typename ST, typename UT, int DC>
hipError_t launch_typed(const RenderParams& p, bool stats, hipStream_t stream)
{
    if (p.hybrid)
        return launch_hybrid<ST, UT, DC>(p, stats, stream);
    if (p.lanes == 1)
        return p.skip ? launch_shape<ST, UT, DC, 1, true, false>(p, stats, stream)
                      : launch_shape<ST, UT, DC, 1, false, false>(p, stats, stream);
    if (p.lanes == 8)
        return p.skip ? launch_shape<ST, UT, DC, 8, true, false>(p, stats, stream)
                      : launch_shape<ST, UT, DC, 8, false, false>(p, stats, stream);
    return p.skip ? launch_shape<ST, UT, DC, 4, true, false>(p, stats, stream)
                  : launch_shape<ST, UT, DC, 4, false, false>(p, stats, stream);
}

// Eq. 5: binary32 partial-sum records, four lanes per ray.
template <typename UT, int DC>
hipError_t launch_linear(const RenderParams& p, bool stats, hipStream_t stream)
{
    return p.skip ? launch_shape<float, UT, DC, 4, true, true>(p, stats, stream)
                  : launch_shape<float, UT, DC, 4, false, true>(p, stats, stream);
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

template <typename UT>
hipError_t launch_linear_d(const RenderParams& p, bool stats, hipStream_t stream)
{
    switch (p.D) {
    case 8:
        return launch_linear<UT, 8>(p, stats, stream);
    case 16:
        return launch_linear<UT, 16>(p, stats, stream);
    default:
        return launch_linear<UT, 0>(p, stats, stream);
    }
}

}  // namespace

hipError_t launch_render(const RenderParams& p, int sigma_dtype, int uvw_dtype, bool stats,
                         hipStream_t stream)
{
    const bool s16 = sigma_dtype == SQN_F16, u16 = uvw_dtype == SQN_F16;
    if (p.linear)
        return u16 ? launch_linear_d<_Float16>(p, stats, stream) : launch_linear_d<float>(p, stats, stream);
    if (s16 && u16)
        return launch_d<_Float16, _Float16>(p, stats, stream);
    if (s16)
        return launch_d<_Float16, float>(p, stats, stream);
    if (u16)
        return launch_d<float, _Float16>(p, stats, stream);
    return launch_d<float, float>(p, stats, stream);
}

}  // namespace sqn
