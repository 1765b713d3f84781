// Create-time preparation of the position planes: for each plane j the
// Chebyshev (L-infinity) distance, in texels, from every texel to the
// nearest texel with sigma^j != 0, capped at kDistCap, packed next to sigma^j.
//
// sigma = sigma^xy sigma^yz sigma^zx (Eq. 4) vanishes wherever one factor
// does, so a sample whose plane-j texel has distance D > 0 is empty, and so
// is every sample whose plane-j texel stays within Chebyshev distance D - 1
// of it: the render kernel leaps over such runs.  A texel counts as
// occupied unless its stored value compares equal to zero (NaN counts as
// occupied), so distances never overstate the empty space.
//
// L-infinity distance is separable: with f(a, b) the distance along row a
// from column b to the nearest occupied texel of that row,
//   dist(a, b) = min over a' of max(|a - a'|, f(a', b)).
#include "sqn_internal.h"

namespace sqn {
namespace {

template <typename ST>
__device__ __forceinline__ bool occupied(const ST* plane, uint32_t idx)
{
    return !(static_cast<float>(plane[idx]) == 0.0f);
}

// One thread per row: forward and backward sweeps give the distance along
// the row to the nearest occupied texel, capped at cap + 1.
template <typename ST>
__global__ void row_distance(const ST* __restrict__ plane, uint16_t* __restrict__ f, int32_t n_p,
                             int32_t cap)
{
    const int32_t a = blockIdx.x * blockDim.x + threadIdx.x;
    if (a >= n_p)
        return;
    const uint32_t row = static_cast<uint32_t>(a) * static_cast<uint32_t>(n_p);
    const int32_t far = cap + 1;
    int32_t last = -(1 << 30);
    for (int32_t b = 0; b < n_p; ++b) {
        if (occupied(plane, row + b))
            last = b;
        f[row + b] = static_cast<uint16_t>(min(far, b - last));
    }
    last = 1 << 30;
    for (int32_t b = n_p - 1; b >= 0; --b) {
        if (occupied(plane, row + b))
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
// binary32 sigma -> two words (sigma bits, dist).
__global__ void pack_f16(const uint16_t* __restrict__ sigma, const uint16_t* __restrict__ dist,
                         uint32_t* __restrict__ out, uint32_t n)
{
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n)
        out[i] = static_cast<uint32_t>(sigma[i]) | (static_cast<uint32_t>(dist[i]) << 16);
}

__global__ void pack_f32(const uint32_t* __restrict__ sigma, const uint16_t* __restrict__ dist,
                         uint2* __restrict__ out, uint32_t n)
{
    const uint32_t i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n)
        out[i] = make_uint2(sigma[i], static_cast<uint32_t>(dist[i]));
}

}  // namespace

hipError_t prepare_sigma_plane(const void* sigma, int sigma_dtype, int32_t n_p, void* packed,
                               uint16_t* work_f, uint16_t* work_dist, hipStream_t stream)
{
    const uint32_t n = static_cast<uint32_t>(n_p) * static_cast<uint32_t>(n_p);
    const int32_t cap = kDistCap;
    const dim3 rows((n_p + 63) / 64);
    if (sigma_dtype == SQN_F16)
        row_distance<_Float16><<<rows, 64, 0, stream>>>(static_cast<const _Float16*>(sigma), work_f, n_p, cap);
    else
        row_distance<float><<<rows, 64, 0, stream>>>(static_cast<const float*>(sigma), work_f, n_p, cap);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess)
        return e;
    column_distance<<<dim3((n_p + 255) / 256, n_p), 256, 0, stream>>>(work_f, work_dist, n_p, cap);
    if ((e = hipGetLastError()) != hipSuccess)
        return e;
    const dim3 grid((n + 255) / 256);
    if (sigma_dtype == SQN_F16)
        pack_f16<<<grid, 256, 0, stream>>>(static_cast<const uint16_t*>(sigma), work_dist,
                                           static_cast<uint32_t*>(packed), n);
    else
        pack_f32<<<grid, 256, 0, stream>>>(static_cast<const uint32_t*>(sigma), work_dist,
                                           static_cast<uint2*>(packed), n);
    return hipGetLastError();
}

}  // namespace sqn
