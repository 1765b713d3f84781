// Create-time preparation of the position planes: for each plane j a mask of
// the texels whose samples may have sigma > 0, the Chebyshev (L-infinity)
// distance in texels from every texel to the nearest such texel (capped at
// kDistCap), and a record that packs the distance next to the value the
// render kernel reads.
//
// Eq. 4: sigma = sigma^xy sigma^yz sigma^zx vanishes wherever one factor
// does, so a texel is live unless its sigma^j compares equal to zero (NaN
// counts as live).
//
// Eq. 5 (linear decoder): sigma = max(0, W_sigma concat(sigma^j) + b_sigma)
// is evaluated as ((s^xy + s^yz) + s^zx) + b_sigma from per-plane partial
// sums s^j (a chain of fused multiply-adds over the channels of plane j).
// The partial sums are folded here, once, into the records.  A texel of plane
// j is dead when the same expression with the other two partial sums replaced
// by their maxima over the samples that can share this texel (a row or column
// of the other planes) is <= 0: binary32 addition is monotone, so every such
// sample then has a sum <= 0 or NaN, i.e. sigma = 0.
//
// A sample whose plane-j texel has distance D > 0 is empty, and so is every
// sample whose plane-j texel stays within Chebyshev distance D - 1 of it: the
// render kernel leaps over such runs.  L-infinity distance is separable: with
// f(a, b) the distance along row a from column b to the nearest live texel of
// that row, dist(a, b) = min over a' of max(|a - a'|, f(a', b)).
#include <math.h>

#include "sqn_internal.h"

namespace sqn {
namespace {

__device__ __forceinline__ float widen(float x) { return x; }
__device__ __forceinline__ float widen(_Float16 x) { return static_cast<float>(x); }

// Eq. 4 planes: live unless sigma^j == 0.
template <typename ST>
__global__ void nonzero_mask(const ST* __restrict__ plane, uint8_t* __restrict__ live, uint32_t n)
{
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n)
        live[i] = (static_cast<float>(plane[i]) == 0.0f) ? 0 : 1;
}

// One thread per row: forward and backward sweeps give the distance along
// the row to the nearest live texel, capped at cap + 1.
__global__ void row_distance(const uint8_t* __restrict__ live, uint16_t* __restrict__ f, int32_t n_p,
                             int32_t cap)
{
    const int32_t a = blockIdx.x * blockDim.x + threadIdx.x;
    if (a >= n_p)
        return;
    const uint32_t row = static_cast<uint32_t>(a) * static_cast<uint32_t>(n_p);
    const int32_t far = cap + 1;
    int32_t last = -(1 << 30);
    for (int32_t b = 0; b < n_p; ++b) {
        if (live[row + b])
            last = b;
        f[row + b] = static_cast<uint16_t>(min(far, b - last));
    }
    last = 1 << 30;
    for (int32_t b = n_p - 1; b >= 0; --b) {
        if (live[row + b])
            last = b;
        const int32_t fb = min(far, last - b);
        if (fb < f[row + b])
            f[row + b] = static_cast<uint16_t>(fb);
    }
}

// One thread per texel: the column pass, capped at cap.
__global__ void column_distance(const uint16_t* __restrict__ f, uint16_t* __restrict__ dist,
                                int32_t n_p, int32_t cap)
{
    const int32_t b = blockIdx.x * blockDim.x + threadIdx.x;
    const int32_t a = blockIdx.y;
    if (b >= n_p || a >= n_p)
        return;
    int32_t best = f[static_cast<uint32_t>(a) * n_p + b];
    for (int32_t k = 1; k < best && k <= cap; ++k) {
        if (a - k >= 0)
            best = min(best, max(k, static_cast<int32_t>(f[static_cast<uint32_t>(a - k) * n_p + b])));
        if (a + k < n_p)
            best = min(best, max(k, static_cast<int32_t>(f[static_cast<uint32_t>(a + k) * n_p + b])));
    }
    dist[static_cast<uint32_t>(a) * n_p + b] = static_cast<uint16_t>(min(best, cap));
}

// Packed record: binary16 sigma -> one 32-bit word (sigma bits | dist << 16);
// binary32 sigma -> two words (sigma bits, dist).  Record (a, b) of a plane
// lands at (a & ~3) n_p + 4 b + (a & 3): four rows interleaved, so that a
// 64-byte segment holds a 4 x 4 block of texels (4 x 2 with two-word
// records), which a quad's four samples along a ray share far more often
// than a run of one row (sigma_texel in render.hip); rows are padded to a
// multiple of four.  The linear decoder's planes are built row-major (their
// passes read rows and columns) and interleaved at the end
// (interleave_linear_planes).
__device__ __forceinline__ uint32_t interleaved(uint32_t i, uint32_t n_p)
{
    const uint32_t a = i / n_p, b = i - a * n_p;
    return (a & ~3u) * n_p + 4u * b + (a & 3u);
}

__global__ void pack_f16(const uint16_t* __restrict__ sigma, const uint16_t* __restrict__ dist,
                         uint32_t* __restrict__ out, uint32_t n, uint32_t n_p)
{
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n)
        out[interleaved(i, n_p)] = static_cast<uint32_t>(sigma[i]) | (static_cast<uint32_t>(dist[i]) << 16);
}

__global__ void scatter_interleaved(const uint2* __restrict__ rows, uint2* __restrict__ out, uint32_t n,
                                    uint32_t n_p)
{
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n)
        out[interleaved(i, n_p)] = rows[i];
}

__global__ void pack_f32(const uint32_t* __restrict__ sigma, const uint16_t* __restrict__ dist,
                         uint2* __restrict__ out, uint32_t n, uint32_t n_p)
{
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n)
        out[interleaved(i, n_p)] = make_uint2(sigma[i], static_cast<uint32_t>(dist[i]));
}

// Distance and packing of one plane whose live mask is in work.live.
hipError_t distance_transform(int32_t n_p, const PrepareWork& work, hipStream_t stream)
{
    const int32_t cap = kDistCap;
    row_distance<<<dim3((n_p + 63) / 64), 64, 0, stream>>>(work.live, work.f, n_p, cap);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    column_distance<<<dim3((n_p + 255) / 256, n_p), 256, 0, stream>>>(work.f, work.dist, n_p, cap);
    return hipGetLastError();
}

// ---- linear decoder -------------------------------------------------------

// s^j at every texel: fma chain over the d_sigma channels from zero, in
// channel order (the evaluation order of the density, see the file head).
template <typename ST>
__global__ void fold_partials(const ST* __restrict__ sigma, const float* __restrict__ w, int32_t ds,
                              uint2* __restrict__ packed, uint32_t n)
{
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n)
        return;
    const ST* v = sigma + static_cast<size_t>(i) * static_cast<size_t>(ds);
    float s = 0.0f;
    for (int32_t c = 0; c < ds; ++c)
        s = __builtin_fmaf(w[c], widen(v[c]), s);
    packed[i] = make_uint2(__float_as_uint(s), 0u);
}

// max over b of s[a][b] for each row a (one workgroup per row).  fmaxf skips
// NaN, whose samples have zero density anyway; an all-NaN row gives -inf.
__global__ void row_max(const uint2* __restrict__ packed, float* __restrict__ out, int32_t n_p)
{
    __shared__ float part[256];
    const int32_t a = blockIdx.x;
    const uint32_t row = static_cast<uint32_t>(a) * static_cast<uint32_t>(n_p);
    float m = -INFINITY;
    for (int32_t b = threadIdx.x; b < n_p; b += blockDim.x)
        m = fmaxf(m, __uint_as_float(packed[row + b].x));
    part[threadIdx.x] = m;
    __syncthreads();
    for (int32_t k = blockDim.x / 2; k > 0; k >>= 1) {
        if (static_cast<int32_t>(threadIdx.x) < k)
            part[threadIdx.x] = fmaxf(part[threadIdx.x], part[threadIdx.x + k]);
        __syncthreads();
    }
    if (threadIdx.x == 0)
        out[a] = part[0];
}

// max over a of s[a][b] for each column b (one thread per column).
__global__ void col_max(const uint2* __restrict__ packed, float* __restrict__ out, int32_t n_p)
{
    const int32_t b = blockIdx.x * blockDim.x + threadIdx.x;
    if (b >= n_p)
        return;
    float m = -INFINITY;
    for (int32_t a = 0; a < n_p; ++a)
        m = fmaxf(m, __uint_as_float(packed[static_cast<uint32_t>(a) * n_p + b].x));
    out[b] = m;
}

// Live mask of plane j.  maxima[2k] / maxima[2k + 1] are the row / column
// maxima of plane k (planes xy = [x][y], yz = [y][z], zx = [z][x]); the
// texel (a, b) of plane j shares samples with
//   xy (x=a, y=b): s^yz over row y, s^zx over column x
//   yz (y=a, z=b): s^xy over column y, s^zx over row z
//   zx (z=a, x=b): s^xy over row x, s^yz over column z
// and the bound keeps the evaluation order ((s^xy + s^yz) + s^zx) + b.
__global__ void linear_live(const uint2* __restrict__ packed, const float* __restrict__ maxima, int32_t j,
                            int32_t n_p, float b_sigma, uint8_t* __restrict__ live)
{
    const int32_t b = blockIdx.x * blockDim.x + threadIdx.x;
    const int32_t a = blockIdx.y;
    if (b >= n_p)
        return;
    const uint32_t i = static_cast<uint32_t>(a) * static_cast<uint32_t>(n_p) + b;
    const float s = __uint_as_float(packed[i].x);
    const float* m = maxima;
    float s_xy, s_yz, s_zx;
    if (j == 0) {
        s_xy = s;
        s_yz = m[2 * n_p + b];
        s_zx = m[5 * n_p + a];
    } else if (j == 1) {
        s_xy = m[1 * n_p + a];
        s_yz = s;
        s_zx = m[4 * n_p + b];
    } else {
        s_xy = m[0 * n_p + b];
        s_yz = m[3 * n_p + a];
        s_zx = s;
    }
    float bound = s_xy + s_yz;
    bound = bound + s_zx;
    bound = bound + b_sigma;
    live[i] = (bound <= 0.0f) ? 0 : 1;
}

__global__ void set_distance(const uint16_t* __restrict__ dist, uint2* __restrict__ packed, uint32_t n)
{
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n)
        packed[i].y = static_cast<uint32_t>(dist[i]);
}

// ---- cell grid of the linear decoder ---------------------------------------

// max of s^j over the g x g texels of each cell of plane j (cells [m][m]).
__global__ void cell_max(const uint2* __restrict__ packed, int32_t n_p, int32_t shift, int32_t m,
                         float* __restrict__ out)
{
    const int32_t cb = blockIdx.x * blockDim.x + threadIdx.x;
    const int32_t ca = blockIdx.y;
    if (cb >= m)
        return;
    const int32_t g = 1 << shift;
    const int32_t a1 = min(n_p, (ca + 1) * g), b1 = min(n_p, (cb + 1) * g);
    float mx = -INFINITY;
    for (int32_t a = ca * g; a < a1; ++a)
        for (int32_t b = cb * g; b < b1; ++b)
            mx = fmaxf(mx, __uint_as_float(packed[static_cast<uint32_t>(a) * n_p + b].x));
    out[ca * m + cb] = mx;
}

// live[(cx m + cy) m + cz]: the bound ((M_xy + M_yz) + M_zx) + b is not <= 0.
__global__ void cell_live(const float* __restrict__ cmax, int32_t m, float b_sigma, uint8_t* __restrict__ live)
{
    const int32_t cz = blockIdx.x * blockDim.x + threadIdx.x;
    const int32_t cy = blockIdx.y, cx = blockIdx.z;
    if (cz >= m)
        return;
    const float* mxy = cmax;
    const float* myz = cmax + m * m;
    const float* mzx = cmax + 2 * m * m;
    float bound = mxy[cx * m + cy] + myz[cy * m + cz];
    bound = bound + mzx[cz * m + cx];
    bound = bound + b_sigma;
    live[(static_cast<uint32_t>(cx) * m + cy) * m + cz] = (bound <= 0.0f) ? 0 : 1;
}

// Distance along z (innermost) to the nearest live cell, capped at cap + 1.
__global__ void cell_dist_z(const uint8_t* __restrict__ live, uint16_t* __restrict__ f, int32_t m, int32_t cap)
{
    const int32_t row = blockIdx.x * blockDim.x + threadIdx.x;
    if (row >= m * m)
        return;
    const uint32_t base = static_cast<uint32_t>(row) * m;
    const int32_t far = cap + 1;
    int32_t last = -(1 << 30);
    for (int32_t z = 0; z < m; ++z) {
        if (live[base + z])
            last = z;
        f[base + z] = static_cast<uint16_t>(min(far, z - last));
    }
    last = 1 << 30;
    for (int32_t z = m - 1; z >= 0; --z) {
        if (live[base + z])
            last = z;
        const int32_t fz = min(far, last - z);
        if (fz < f[base + z])
            f[base + z] = static_cast<uint16_t>(fz);
    }
}

// One separable Chebyshev pass along axis y (stride m) or x (stride m^2):
// out = min over k of max(|k|, in at offset k), capped at cap + 1.
__global__ void cell_dist_pass(const uint16_t* __restrict__ in, uint16_t* __restrict__ out, int32_t m,
                               int32_t along_x, int32_t cap)
{
    const int32_t cz = blockIdx.x * blockDim.x + threadIdx.x;
    const int32_t cy = blockIdx.y, cx = blockIdx.z;
    if (cz >= m)
        return;
    const int32_t pos = along_x ? cx : cy;
    const int32_t stride = along_x ? m * m : m;
    const uint32_t idx = (static_cast<uint32_t>(cx) * m + cy) * m + cz;
    int32_t best = in[idx];
    for (int32_t k = 1; k < best && k <= cap; ++k) {
        if (pos - k >= 0)
            best = min(best, max(k, static_cast<int32_t>(in[idx - k * stride])));
        if (pos + k < m)
            best = min(best, max(k, static_cast<int32_t>(in[idx + k * stride])));
    }
    out[idx] = static_cast<uint16_t>(min(best, cap + 1));
}

__global__ void cell_store(const uint16_t* __restrict__ f, uint8_t* __restrict__ dist, uint32_t n, int32_t cap)
{
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n)
        dist[i] = static_cast<uint8_t>(min(static_cast<int32_t>(f[i]), cap));
}

}  // namespace

hipError_t prepare_linear_cells(const void* const packed[3], int32_t n_p, float b_sigma, int32_t shift,
                                int32_t m, uint8_t* cell_dist, const PrepareWork& work, hipStream_t stream)
{
    hipError_t e = hipSuccess;
    for (int j = 0; j < 3; ++j) {
        cell_max<<<dim3((m + 63) / 64, m), 64, 0, stream>>>(static_cast<const uint2*>(packed[j]), n_p, shift, m,
                                                            work.cell_max + j * m * m);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
    }
    const dim3 cells((m + 63) / 64, m, m);
    cell_live<<<cells, 64, 0, stream>>>(work.cell_max, m, b_sigma, work.cell_live);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    const int32_t cap = 255;
    cell_dist_z<<<dim3((m * m + 63) / 64), 64, 0, stream>>>(work.cell_live, work.cell_f, m, cap);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    cell_dist_pass<<<cells, 64, 0, stream>>>(work.cell_f, work.cell_f2, m, 0, cap);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    cell_dist_pass<<<cells, 64, 0, stream>>>(work.cell_f2, work.cell_f, m, 1, cap);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    const uint32_t n = static_cast<uint32_t>(m) * m * m;
    cell_store<<<dim3((n + 255) / 256), 256, 0, stream>>>(work.cell_f, cell_dist, n, cap);
    return hipGetLastError();
}

hipError_t prepare_sigma_plane(const void* sigma, int sigma_dtype, int32_t n_p, void* packed,
                               const PrepareWork& work, hipStream_t stream)
{
    const uint32_t n = static_cast<uint32_t>(n_p) * static_cast<uint32_t>(n_p);
    const dim3 grid((n + 255) / 256);
    if (sigma_dtype == SQN_F16)
        nonzero_mask<_Float16><<<grid, 256, 0, stream>>>(static_cast<const _Float16*>(sigma), work.live, n);
    else
        nonzero_mask<float><<<grid, 256, 0, stream>>>(static_cast<const float*>(sigma), work.live, n);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    if ((e = distance_transform(n_p, work, stream)) != hipSuccess)
        return e;
    if (sigma_dtype == SQN_F16)
        pack_f16<<<grid, 256, 0, stream>>>(static_cast<const uint16_t*>(sigma), work.dist,
                                           static_cast<uint32_t*>(packed), n, static_cast<uint32_t>(n_p));
    else
        pack_f32<<<grid, 256, 0, stream>>>(static_cast<const uint32_t*>(sigma), work.dist,
                                           static_cast<uint2*>(packed), n, static_cast<uint32_t>(n_p));
    return hipGetLastError();
}

hipError_t prepare_linear_planes(const void* const sigma[3], int sigma_dtype, int32_t n_p,
                                 int32_t d_sigma, float b_sigma, void* const packed[3],
                                 const PrepareWork& work, hipStream_t stream)
{
    const uint32_t n = static_cast<uint32_t>(n_p) * static_cast<uint32_t>(n_p);
    const dim3 grid((n + 255) / 256);
    hipError_t e = hipSuccess;
    for (int j = 0; j < 3; ++j) {
        uint2* rec = static_cast<uint2*>(packed[j]);
        const float* w = work.w_sigma + j * d_sigma;
        if (sigma_dtype == SQN_F16)
            fold_partials<_Float16><<<grid, 256, 0, stream>>>(static_cast<const _Float16*>(sigma[j]), w,
                                                              d_sigma, rec, n);
        else
            fold_partials<float><<<grid, 256, 0, stream>>>(static_cast<const float*>(sigma[j]), w, d_sigma,
                                                           rec, n);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
        row_max<<<dim3(n_p), 256, 0, stream>>>(rec, work.maxima + (2 * j) * n_p, n_p);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
        col_max<<<dim3((n_p + 255) / 256), 256, 0, stream>>>(rec, work.maxima + (2 * j + 1) * n_p, n_p);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
    }
    for (int j = 0; j < 3; ++j) {
        uint2* rec = static_cast<uint2*>(packed[j]);
        linear_live<<<dim3((n_p + 255) / 256, n_p), 256, 0, stream>>>(rec, work.maxima, j, n_p, b_sigma,
                                                                      work.live);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
        if ((e = distance_transform(n_p, work, stream)) != hipSuccess)
            return e;
        set_distance<<<grid, 256, 0, stream>>>(work.dist, rec, n);
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
    }
    return hipSuccess;
}

hipError_t interleave_linear_planes(void* const packed[3], int32_t n_p, const PrepareWork& work,
                                    hipStream_t stream)
{
    const uint32_t n = static_cast<uint32_t>(n_p) * static_cast<uint32_t>(n_p);
    const dim3 grid((n + 255) / 256);
    for (int j = 0; j < 3; ++j) {
        hipError_t e = hipMemcpyAsync(work.rows, packed[j], static_cast<size_t>(n) * sizeof(uint2),
                                      hipMemcpyDeviceToDevice, stream);
        if (e != hipSuccess)
            return e;
        scatter_interleaved<<<grid, 256, 0, stream>>>(work.rows, static_cast<uint2*>(packed[j]), n,
                                                      static_cast<uint32_t>(n_p));
        if ((e = hipGetLastError()) != hipSuccess)
            return e;
    }
    return hipSuccess;
}

}  // namespace sqn
