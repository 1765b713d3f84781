// C ABI of the cached SqueezeNeRF renderer: argument validation, the
// library-owned device copy of the caches, and the render launches.
// Declarations and contracts: include/sqn.h.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <limits>
#include <mutex>
#include <vector>

#include "sqn_internal.h"

struct sqn_caches {
    sqn_cache_desc desc;
    int device;
    void* block;             // one hipMalloc holding every plane
    size_t bytes;
    const void* sigma[3];
    const void* uvw[3];
    const void* beta;
    float scale[3];          // (n_p - 1) / (bmax - bmin), binary32
    int64_t tau_eps;         // floor(-ln(eps) 2^32)
    int32_t lanes;           // lanes per ray, 0 = chosen per call
    float centre;            // > 0: hybrid launch of single views, centred block fraction
    int32_t skip;            // empty-space leaps (one lane per ray)
    float ndc_near;          // > 0: forward-facing rays in normalized device coordinates
    // linear (Eq. 5) decoder
    int32_t linear;          // 1: sigma[j] hold per-plane partial sums
    int32_t d_sigma;
    float b_sigma;
    const float* lin_w;      // [9D + 3][D] folded radiance weights and biases
    const uint8_t* cell_dist;  // [m^3] cell distances (Eq. 5 leaps)
    int32_t cell_shift, cell_m;
};

// Device copy of the networks for cache generation.
struct sqn_networks {
    int device;
    void* block;             // one hipMalloc: fragments, biases, encoding table
    size_t bytes;
    sqn::GenNet pos[3];
    sqn::GenNet dir;
    int32_t D, pos_freq, dir_freq, pos_in, dir_in;
    _Float16* enc_table;     // 3 x 8192 x (1 + 2 pos_freq) binary16
};

namespace {

// detail of the last failure on this thread; a fixed buffer, so that no
// error path allocates
thread_local char g_last_error[512];

sqn_status fail(sqn_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

sqn_status fail(sqn_status s, const char* fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return s;
}

void clear_error() { g_last_error[0] = '\0'; }

size_t dtype_size(int32_t dt) { return dt == SQN_F16 ? 2 : 4; }

bool valid_dtype(int32_t dt) { return dt == SQN_F32 || dt == SQN_F16; }

// The pointer must lie in a HIP device allocation with at least `bytes`
// bytes from it to the end of the allocation.
sqn_status check_device_range(const void* p, size_t bytes, const char* what)
{
    if (!p)
        return fail(SQN_ERR_INVALID_ARG, "%s is NULL", what);
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    hipError_t e = hipMemGetAddressRange(&base, &size, const_cast<void*>(p));
    if (e != hipSuccess || base == nullptr) {
        (void)hipGetLastError();
        return fail(SQN_ERR_INVALID_ARG, "%s (%p) is not HIP device memory", what, p);
    }
    const uintptr_t lo = reinterpret_cast<uintptr_t>(base);
    const uintptr_t q = reinterpret_cast<uintptr_t>(p);
    if (q < lo || q - lo > size || size - (q - lo) < bytes)
        return fail(SQN_ERR_INVALID_ARG,
                    "%s (%p) needs %zu bytes but its allocation ends %zu bytes after it", what,
                    p, bytes, size - (q - lo));
    return SQN_OK;
}

int64_t tau_threshold(float eps)
{
    if (!(eps > 0.0f))
        return std::numeric_limits<int64_t>::max();
    const double x = -log(static_cast<double>(eps)) * 4294967296.0;
    if (x <= 0.0)
        return 0;
    return static_cast<int64_t>(floor(x));
}

sqn_status validate_desc(const sqn_cache_desc* d)
{
    if (!d)
        return fail(SQN_ERR_INVALID_ARG, "desc is NULL");
    if (d->n_p < 2 || d->n_p > 8192)
        return fail(SQN_ERR_INVALID_ARG, "n_p = %d outside [2, 8192]", d->n_p);
    if (d->D < 1 || d->D > 32)
        return fail(SQN_ERR_INVALID_ARG, "D = %d outside [1, 32]", d->D);
    if (d->n_theta < 2 || d->n_phi < 2 || d->n_theta > 65536 || d->n_phi > 65536
        || static_cast<int64_t>(d->n_theta) * d->n_phi * d->D > (int64_t{1} << 31))
        return fail(SQN_ERR_INVALID_ARG, "direction grid %d x %d x %d out of range", d->n_theta,
                    d->n_phi, d->D);
    if (!valid_dtype(d->sigma_dtype) || !valid_dtype(d->uvw_dtype) || !valid_dtype(d->beta_dtype))
        return fail(SQN_ERR_INVALID_ARG, "dtype must be SQN_F32 or SQN_F16");
    if (d->stratified != 0 && d->stratified != 1)
        return fail(SQN_ERR_INVALID_ARG, "stratified must be 0 or 1");
    if (d->reserved != 0)
        return fail(SQN_ERR_INVALID_ARG, "reserved must be 0");
    for (int r = 0; r < 3; ++r)
        if (!isfinite(d->bbox_min[r]) || !isfinite(d->bbox_max[r]) || !(d->bbox_min[r] < d->bbox_max[r])
            || !isfinite(d->bbox_max[r] - d->bbox_min[r]))
            return fail(SQN_ERR_INVALID_ARG, "bbox axis %d is empty or not finite", r);
    if (!(d->t_eps >= 0.0f && d->t_eps <= 1.0f))
        return fail(SQN_ERR_INVALID_ARG, "t_eps = %g outside [0, 1]", static_cast<double>(d->t_eps));
    // every plane is addressed with 32-bit byte offsets
    const uint64_t texels = static_cast<uint64_t>(d->n_p) * d->n_p;
    const uint64_t uvw_plane = texels * 3u * d->D * dtype_size(d->uvw_dtype);
    static_assert(sqn::kDistCap < 65536, "distance must fit the packed record");
    if (uvw_plane >= (uint64_t{1} << 32))
        return fail(SQN_ERR_UNSUPPORTED, "a uvw plane of %llu bytes exceeds 2^32 bytes",
                    static_cast<unsigned long long>(uvw_plane));
    // so is the direction cache
    const uint64_t beta_bytes = static_cast<uint64_t>(d->n_theta) * d->n_phi * d->D * dtype_size(d->beta_dtype);
    if (beta_bytes >= (uint64_t{1} << 32))
        return fail(SQN_ERR_UNSUPPORTED, "a direction cache of %llu bytes exceeds 2^32 bytes",
                    static_cast<unsigned long long>(beta_bytes));
    return SQN_OK;
}

sqn_status validate_render(const sqn_caches* h, const float* poses, int32_t n_poses,
                           const sqn_intrinsics* in, float near_plane, float far_plane,
                           int32_t n_samples, const float* rgb, const float* depth,
                           const uint32_t* stats, bool need_rgb, int* device)
{
    if (!h)
        return fail(SQN_ERR_INVALID_ARG, "caches is NULL");
    if (!in)
        return fail(SQN_ERR_INVALID_ARG, "intrinsics is NULL");
    if (n_poses < 0)
        return fail(SQN_ERR_INVALID_ARG, "n_poses = %d is negative", n_poses);
    if (in->width < 1 || in->height < 1)
        return fail(SQN_ERR_INVALID_ARG, "image %d x %d is empty", in->width, in->height);
    if (!isfinite(in->fx) || !isfinite(in->fy) || in->fx == 0.0f || in->fy == 0.0f
        || !isfinite(in->cx) || !isfinite(in->cy))
        return fail(SQN_ERR_INVALID_ARG, "intrinsics must be finite with fx, fy != 0");
    if (!isfinite(near_plane) || !isfinite(far_plane) || !(near_plane < far_plane))
        return fail(SQN_ERR_INVALID_ARG, "need finite near < far (got %g, %g)",
                    static_cast<double>(near_plane), static_cast<double>(far_plane));
    if (n_samples < 1 || n_samples > 32768)
        return fail(SQN_ERR_INVALID_ARG, "n_samples = %d outside [1, 32768]", n_samples);
    const int64_t rays = static_cast<int64_t>(n_poses) * in->width * in->height;
    if (rays > std::numeric_limits<int32_t>::max())
        return fail(SQN_ERR_INVALID_ARG, "%lld rays exceed 2^31 - 1", static_cast<long long>(rays));
    if (hipGetDevice(device) != hipSuccess)
        return fail(SQN_ERR_DEVICE, "hipGetDevice failed");
    if (*device != h->device)
        return fail(SQN_ERR_INVALID_ARG, "caches live on device %d, current device is %d",
                    h->device, *device);
    if (n_poses == 0)
        return SQN_OK;
    const size_t nr = static_cast<size_t>(rays);
    sqn_status s = check_device_range(poses, static_cast<size_t>(n_poses) * 12 * sizeof(float), "poses");
    if (s != SQN_OK)
        return s;
    if (need_rgb || rgb) {
        s = check_device_range(rgb, nr * 3 * sizeof(float), "rgb_out");
        if (s != SQN_OK)
            return s;
    }
    if (depth) {
        s = check_device_range(depth, nr * sizeof(float), "depth_out");
        if (s != SQN_OK)
            return s;
    }
    if (stats) {
        s = check_device_range(stats, nr * 4 * sizeof(uint32_t), "ray_stats");
        if (s != SQN_OK)
            return s;
    }
    return SQN_OK;
}

sqn_status validate_decoder(const sqn_linear_decoder* dec, int32_t D)
{
    if (!dec)
        return fail(SQN_ERR_INVALID_ARG, "decoder is NULL");
    if (dec->d_sigma < 1 || dec->d_sigma > 64)
        return fail(SQN_ERR_INVALID_ARG, "d_sigma = %d outside [1, 64]", dec->d_sigma);
    if (!dec->w_sigma || !dec->w_uvw || !dec->b_uvw)
        return fail(SQN_ERR_INVALID_ARG, "decoder weight pointer is NULL");
    if (!isfinite(dec->b_sigma))
        return fail(SQN_ERR_INVALID_ARG, "b_sigma is not finite");
    for (int32_t k = 0; k < 3 * dec->d_sigma; ++k)
        if (!isfinite(dec->w_sigma[k]))
            return fail(SQN_ERR_INVALID_ARG, "w_sigma[%d] is not finite", k);
    for (int32_t k = 0; k < 9 * D * D; ++k)
        if (!isfinite(dec->w_uvw[k]))
            return fail(SQN_ERR_INVALID_ARG, "w_uvw[%d] is not finite", k);
    for (int32_t k = 0; k < 3 * D; ++k)
        if (!isfinite(dec->b_uvw[k]))
            return fail(SQN_ERR_INVALID_ARG, "b_uvw[%d] is not finite", k);
    return SQN_OK;
}

// Lanes per ray for a call of `rays` rays.  One lane per ray does the least
// work per sample, but a wave lives as long as its longest ray: below about
// 2^20 rays (one 800x800 view is 10^4 waves against 8192 resident wave
// slots) the heaviest waves, not throughput, set the time, and four lanes per
// ray cut their chains of dependent samples four-fold.  Below 2^18 rays
// (under two rounds of four-lane waves) eight lanes shorten them again
// (504x378 forward-facing view: 0.107 against 0.118 ms; at 800x800 eight
// lanes cost more vector-ALU work than they save).
int choose_lanes(int64_t rays)
{
    return rays < (int64_t{1} << 18) ? 8 : (rays < (int64_t{1} << 20) ? 4 : 1);
}

sqn_status render_common(const sqn_caches* h, const float* poses, int32_t n_poses,
                         const sqn_intrinsics* in, float near_plane, float far_plane,
                         int32_t n_samples, float* rgb, float* depth, uint32_t* stats,
                         void* stream)
{
    int device = -1;
    const bool with_stats = stats != nullptr;
    sqn_status s = validate_render(h, poses, n_poses, in, near_plane, far_plane, n_samples, rgb,
                                   depth, stats, !with_stats, &device);
    if (s != SQN_OK)
        return s;
    if (n_poses == 0)
        return SQN_OK;

    sqn::RenderParams p;
    memset(&p, 0, sizeof(p));
    for (int j = 0; j < 3; ++j) {
        p.sigma[j] = h->sigma[j];
        p.uvw[j] = h->uvw[j];
    }
    p.beta = h->beta;
    p.poses = poses;
    p.rgb = rgb;
    p.depth = depth;
    p.stats = stats;
    p.fx = in->fx;
    p.fy = in->fy;
    p.cx = in->cx;
    p.cy = in->cy;
    p.width = in->width;
    p.height = in->height;
    p.n_views = n_poses;
    p.near_t = near_plane;
    p.far_t = far_plane;
    p.n_samples = n_samples;
    p.dt = (far_plane - near_plane) / static_cast<float>(n_samples);
    p.stratified = h->desc.stratified;
    for (int r = 0; r < 3; ++r) {
        p.bmin[r] = h->desc.bbox_min[r];
        p.bmax[r] = h->desc.bbox_max[r];
        p.scale[r] = h->scale[r];
    }
    p.n_p = h->desc.n_p;
    p.D = h->desc.D;
    p.n_theta = h->desc.n_theta;
    p.n_phi = h->desc.n_phi;
    p.beta_f16 = h->desc.beta_dtype == SQN_F16;
    p.theta_scale = static_cast<double>(h->desc.n_theta - 1) / 3.14159265358979323846;
    p.phi_scale = static_cast<double>(h->desc.n_phi) / (2.0 * 3.14159265358979323846);
    p.rec_bytes = static_cast<uint32_t>(3 * h->desc.D * dtype_size(h->desc.uvw_dtype));
    p.tau_eps = h->tau_eps;
    p.seed = h->desc.seed;
    p.inv_dt = 1.0f / p.dt;
    {
        const double k = (1.0 - ldexp(1.0, -19)) / static_cast<double>(p.dt);
        p.leap_k = static_cast<float>(k);
        p.leap_c = static_cast<float>(static_cast<double>(near_plane) * k
                                      + ldexp(fabs(static_cast<double>(near_plane)) / static_cast<double>(p.dt), -19));
    }
    const int64_t rays = static_cast<int64_t>(n_poses) * in->width * in->height;
    p.skip = h->skip;
    // the folded Eq. 5 weights are shared by the lanes of a ray in LDS, which
    // holds them for 64 rays per workgroup, i.e. four lanes per ray
    p.lanes = h->linear ? 4 : (h->lanes != 0 ? h->lanes : choose_lanes(rays));
    p.linear = h->linear;
    p.b_sigma = h->b_sigma;
    p.lin_w = h->lin_w;
    // rows per ray in LDS; the kernels for D = 8 and 16 use lin_stride(D)
    p.lin_stride = sqn::lin_stride_generic(h->desc.D);
    p.ndc_near = h->ndc_near;
    p.cell_dist = h->cell_dist;
    p.cell_shift = h->cell_shift;
    p.cell_m = h->cell_m;
    p.leap_margin = 1e-3f;
    const int tw = sqn::kTileW(p.lanes), th = sqn::kTileH(p.lanes);
    p.tiles_x = (in->width + tw - 1) / tw;
    p.tiles_y = (in->height + th - 1) / th;
    const int64_t groups = static_cast<int64_t>(p.tiles_x) * p.tiles_y * n_poses;
    if (groups > std::numeric_limits<int32_t>::max())
        return fail(SQN_ERR_INVALID_ARG, "too many workgroups (%lld)", static_cast<long long>(groups));
    p.n_groups = static_cast<int32_t>(groups);
    // one view: blocks of 2 x 2 tiles from the centre outwards, each block's
    // four workgroups on one XCD so that its L2 serves the texels they share;
    // the grid covers whole blocks.  Measured with four or eight lanes per
    // ray against tiles in interleaved row order: 2-4% faster; with one lane
    // against tile rows and columns dealt from the centre: 3% faster on the
    // 800x800 view of the 256 cache, 10% on the 1K cache, 3% slower on the
    // 512 cache at 256 samples.  Batches of views keep the interleaved row
    // order, which spreads every view over the XCDs.
    if (n_poses == 1) {
        const int64_t bgroups = 4 * ((static_cast<int64_t>(p.tiles_x) + 1) / 2) * ((p.tiles_y + 1) / 2);
        if (bgroups > std::numeric_limits<int32_t>::max())
            return fail(SQN_ERR_INVALID_ARG, "too many workgroups (%lld)", static_cast<long long>(bgroups));
        p.block_order = 1;
        p.n_groups = static_cast<int32_t>(bgroups);
    }
    // hybrid launch: a centred rectangle of 16 x 16 pixel blocks, `centre`
    // of the image's blocks along each axis, with four lanes per ray and
    // the other blocks with one (single views of the product decoder with
    // leaps and world rays)
    if (h->centre > 0.0f && n_poses == 1 && !h->linear && h->skip && !(h->ndc_near > 0.0f)) {
        const int32_t bx = (in->width + 15) / 16, by = (in->height + 15) / 16;
        const int32_t hw = std::min(bx, std::max(1, static_cast<int32_t>(lroundf(h->centre * static_cast<float>(bx)))));
        const int32_t hh = std::min(by, std::max(1, static_cast<int32_t>(lroundf(h->centre * static_cast<float>(by)))));
        p.hybrid = 1;
        p.hy_bx = bx;
        p.hy_by = by;
        p.hy_w = hw;
        p.hy_h = hh;
        p.hy_x0 = (bx - hw) / 2;
        p.hy_y0 = (by - hh) / 2;
        p.n_heavy = 4 * hw * hh;
        const int64_t hgroups = static_cast<int64_t>(p.n_heavy) + static_cast<int64_t>(bx) * by
                                - static_cast<int64_t>(hw) * hh;
        if (hgroups > std::numeric_limits<int32_t>::max())
            return fail(SQN_ERR_INVALID_ARG, "too many workgroups (%lld)", static_cast<long long>(hgroups));
        p.n_groups = static_cast<int32_t>(hgroups);
    }

    // the linear decoder's records hold binary32 partial sums
    const int sigma_records = h->linear ? SQN_F32 : h->desc.sigma_dtype;
    hipError_t e = sqn::launch_render(p, sigma_records, h->desc.uvw_dtype, with_stats,
                                      static_cast<hipStream_t>(stream));
    if (e != hipSuccess)
        return fail(SQN_ERR_DEVICE, "render launch failed: %s", hipGetErrorString(e));
    return SQN_OK;
}

size_t align256(size_t x) { return (x + 255) & ~size_t{255}; }

// Where each array of a handle lives in its device block (offsets from the
// block start, each region 256-byte aligned) and the block size.
struct CacheLayout {
    size_t packed_bytes, uvw_bytes, beta_bytes, lin_bytes, cells;
    size_t off_sigma[3], off_uvw[3], off_beta, off_lin, off_cells, total;
};

CacheLayout cache_layout(const sqn_cache_desc* desc, bool linear)
{
    CacheLayout L;
    const int32_t D = desc->D;
    const size_t texels = static_cast<size_t>(desc->n_p) * desc->n_p;
    // packed records: 4 bytes for binary16 sigma, 8 for binary32 sigma or
    // the linear decoder's binary32 partial sums, four rows interleaved
    // (rows padded to a multiple of four)
    const size_t rows = (static_cast<size_t>(desc->n_p) + 3) / 4 * 4;
    L.packed_bytes = rows * desc->n_p * (!linear && desc->sigma_dtype == SQN_F16 ? 4 : 8);
    L.uvw_bytes = texels * 3 * D * dtype_size(desc->uvw_dtype);
    L.beta_bytes = static_cast<size_t>(desc->n_theta) * desc->n_phi * D * dtype_size(desc->beta_dtype);
    L.lin_bytes = linear ? (9 * static_cast<size_t>(D) + 3) * D * sizeof(float) : 0;
    const int32_t cell_m = sqn::linear_cells(desc->n_p);
    L.cells = linear ? static_cast<size_t>(cell_m) * cell_m * cell_m : 0;
    size_t total = 0;
    for (int j = 0; j < 3; ++j) {
        L.off_sigma[j] = total;
        total += align256(L.packed_bytes);
    }
    for (int j = 0; j < 3; ++j) {
        L.off_uvw[j] = total;
        total += align256(L.uvw_bytes);
    }
    L.off_beta = total;
    total += align256(L.beta_bytes);
    L.off_lin = total;
    total += align256(L.lin_bytes);
    L.off_cells = total;
    total += align256(L.cells);
    L.total = total;
    return L;
}

// Shared body of the two create calls; dec == NULL selects Eq. 4.
sqn_status create_impl(const sqn_cache_desc* desc, const sqn_linear_decoder* dec,
                       const void* const sigma_planes[3], const void* const uvw_planes[3],
                       const void* beta, void* stream, sqn_caches** out)
{
    if (!out)
        return fail(SQN_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    sqn_status s = validate_desc(desc);
    if (s != SQN_OK)
        return s;
    const bool linear = dec != nullptr;
    if (linear && (s = validate_decoder(dec, desc->D)) != SQN_OK)
        return s;
    if (!sigma_planes || !uvw_planes)
        return fail(SQN_ERR_INVALID_ARG, "plane pointer array is NULL");

    const int32_t D = desc->D;
    const int32_t ds = linear ? dec->d_sigma : 1;
    const size_t texels = static_cast<size_t>(desc->n_p) * desc->n_p;
    const size_t sigma_bytes = texels * ds * dtype_size(desc->sigma_dtype);
    const CacheLayout lay = cache_layout(desc, linear);
    const size_t uvw_bytes = lay.uvw_bytes, beta_bytes = lay.beta_bytes, lin_bytes = lay.lin_bytes;
    const size_t lin_rows = 9 * static_cast<size_t>(D) + 3;
    const int32_t cell_shift = sqn::linear_cell_shift(desc->n_p);
    const int32_t cell_m = sqn::linear_cells(desc->n_p);
    const size_t cells = lay.cells;
    static const char* names_s[3] = {"sigma_planes[0] (xy)", "sigma_planes[1] (yz)", "sigma_planes[2] (zx)"};
    static const char* names_u[3] = {"uvw_planes[0] (xy)", "uvw_planes[1] (yz)", "uvw_planes[2] (zx)"};
    for (int j = 0; j < 3; ++j) {
        if ((s = check_device_range(sigma_planes[j], sigma_bytes, names_s[j])) != SQN_OK)
            return s;
        if ((s = check_device_range(uvw_planes[j], uvw_bytes, names_u[j])) != SQN_OK)
            return s;
    }
    if ((s = check_device_range(beta, beta_bytes, "beta")) != SQN_OK)
        return s;

    auto align = align256;
    const size_t* off_sigma = lay.off_sigma;
    const size_t* off_uvw = lay.off_uvw;
    const size_t off_beta = lay.off_beta, off_lin = lay.off_lin, off_cells = lay.off_cells, total = lay.total;

    // temporary buffers of the preparation, freed before returning
    size_t work_total = 0;
    const size_t w_live = work_total;
    work_total += align(texels);
    const size_t w_f = work_total;
    work_total += align(texels * sizeof(uint16_t));
    const size_t w_dist = work_total;
    work_total += align(texels * sizeof(uint16_t));
    const size_t w_max = work_total;
    work_total += align(6 * static_cast<size_t>(desc->n_p) * sizeof(float));
    const size_t w_ws = work_total;
    work_total += align(3 * static_cast<size_t>(ds) * sizeof(float));
    const size_t w_cmax = work_total;
    work_total += align(3 * static_cast<size_t>(cell_m) * cell_m * sizeof(float));
    const size_t w_clive = work_total;
    work_total += align(cells);
    const size_t w_cf = work_total;
    work_total += align(cells * sizeof(uint16_t));
    const size_t w_cf2 = work_total;
    work_total += align(cells * sizeof(uint16_t));
    const size_t w_rows = work_total;
    work_total += align(linear ? texels * sizeof(uint2) : 0);

    // host-side parameters of the linear decoder: W_sigma, and the radiance
    // weights transposed so that row c*3D + e holds W_c[0..D)[e], followed
    // by the rows b_u, b_v, b_w
    std::vector<float> lin_host, ws_host;
    if (linear) {
        lin_host.resize(lin_rows * D);
        for (int32_t c = 0; c < 3; ++c)
            for (int32_t e = 0; e < 3 * D; ++e)
                for (int32_t d = 0; d < D; ++d)
                    lin_host[(static_cast<size_t>(c) * 3 * D + e) * D + d]
                        = dec->w_uvw[(static_cast<size_t>(c) * D + d) * 3 * D + e];
        for (int32_t c = 0; c < 3; ++c)
            for (int32_t d = 0; d < D; ++d)
                lin_host[(9 * static_cast<size_t>(D) + c) * D + d] = dec->b_uvw[c * D + d];
        ws_host.assign(dec->w_sigma, dec->w_sigma + 3 * ds);
    }

    sqn_caches* h = static_cast<sqn_caches*>(calloc(1, sizeof(sqn_caches)));
    if (!h)
        return fail(SQN_ERR_OUT_OF_MEMORY, "host allocation failed");
    h->desc = *desc;
    if (hipGetDevice(&h->device) != hipSuccess) {
        free(h);
        return fail(SQN_ERR_DEVICE, "hipGetDevice failed");
    }
    if (getenv("SQN_TEST_FAIL_ALLOC") != nullptr) {
        free(h);
        return fail(SQN_ERR_OUT_OF_MEMORY, "device allocation of %zu bytes refused (SQN_TEST_FAIL_ALLOC)", total);
    }
    hipError_t e = hipMalloc(&h->block, total);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        free(h);
        return fail(SQN_ERR_OUT_OF_MEMORY, "hipMalloc(%zu) failed: %s", total, hipGetErrorString(e));
    }
    h->bytes = total;
    char* base = static_cast<char*>(h->block);
    hipStream_t st = static_cast<hipStream_t>(stream);
    char* work = nullptr;
    e = hipMalloc(reinterpret_cast<void**>(&work), work_total);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        (void)hipFree(h->block);
        free(h);
        return fail(SQN_ERR_OUT_OF_MEMORY, "hipMalloc of %zu scratch bytes failed", work_total);
    }
    sqn::PrepareWork pw;
    pw.live = reinterpret_cast<uint8_t*>(work + w_live);
    pw.f = reinterpret_cast<uint16_t*>(work + w_f);
    pw.dist = reinterpret_cast<uint16_t*>(work + w_dist);
    pw.maxima = reinterpret_cast<float*>(work + w_max);
    pw.w_sigma = reinterpret_cast<float*>(work + w_ws);
    pw.cell_max = reinterpret_cast<float*>(work + w_cmax);
    pw.cell_live = reinterpret_cast<uint8_t*>(work + w_clive);
    pw.cell_f = reinterpret_cast<uint16_t*>(work + w_cf);
    pw.cell_f2 = reinterpret_cast<uint16_t*>(work + w_cf2);
    pw.rows = reinterpret_cast<uint2*>(work + w_rows);

    void* packed[3];
    for (int j = 0; j < 3; ++j) {
        packed[j] = base + off_sigma[j];
        h->sigma[j] = packed[j];
        h->uvw[j] = base + off_uvw[j];
    }
    h->beta = base + off_beta;
    if (linear) {
        e = hipMemcpyAsync(pw.w_sigma, ws_host.data(), ws_host.size() * sizeof(float),
                           hipMemcpyHostToDevice, st);
        if (e == hipSuccess)
            e = hipMemcpyAsync(base + off_lin, lin_host.data(), lin_bytes, hipMemcpyHostToDevice, st);
        if (e == hipSuccess)
            e = sqn::prepare_linear_planes(sigma_planes, desc->sigma_dtype, desc->n_p, ds, dec->b_sigma,
                                           packed, pw, st);
        if (e == hipSuccess)
            e = sqn::prepare_linear_cells(packed, desc->n_p, dec->b_sigma, cell_shift, cell_m,
                                          reinterpret_cast<uint8_t*>(base + off_cells), pw, st);
        if (e == hipSuccess)
            e = sqn::interleave_linear_planes(packed, desc->n_p, pw, st);
    } else {
        for (int j = 0; j < 3 && e == hipSuccess; ++j)
            e = sqn::prepare_sigma_plane(sigma_planes[j], desc->sigma_dtype, desc->n_p, packed[j], pw, st);
    }
    for (int j = 0; j < 3 && e == hipSuccess; ++j)
        e = hipMemcpyAsync(base + off_uvw[j], uvw_planes[j], uvw_bytes, hipMemcpyDeviceToDevice, st);
    if (e == hipSuccess)
        e = hipMemcpyAsync(base + off_beta, beta, beta_bytes, hipMemcpyDeviceToDevice, st);
    if (e == hipSuccess)
        e = hipStreamSynchronize(st);
    else
        (void)hipStreamSynchronize(st);
    (void)hipFree(work);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        (void)hipFree(h->block);
        free(h);
        return fail(SQN_ERR_DEVICE, "cache upload failed: %s", hipGetErrorString(e));
    }
    for (int r = 0; r < 3; ++r)
        h->scale[r] = static_cast<float>(desc->n_p - 1) / (desc->bbox_max[r] - desc->bbox_min[r]);
    h->tau_eps = tau_threshold(desc->t_eps);
    h->skip = 1;
    if (linear) {
        h->linear = 1;
        h->d_sigma = ds;
        h->b_sigma = dec->b_sigma;
        h->lin_w = reinterpret_cast<const float*>(base + off_lin);
        h->cell_dist = reinterpret_cast<const uint8_t*>(base + off_cells);
        h->cell_shift = cell_shift;
        h->cell_m = cell_m;
    }
    *out = h;
    clear_error();
    return SQN_OK;
}

// ---- sqn_recreate_caches: create-time preparation without allocating -------
//
// The distance transform of a plane needs n_p^2 bytes of live mask and two
// n_p^2 arrays of uint16 (row and capped Chebyshev distances).  For callers
// that cannot allocate, that scratch lives in one file-scope device array,
// sized for n_p <= kRecreateMaxNp.  Every device the library runs on holds
// its own copy until the process ends.  In host code `scratch` names a host
// stand-in, not device memory: its device address is taken once per device
// with hipGetSymbolAddress and only that address is passed to kernels.

constexpr int32_t kRecreateMaxNp = 2048;
constexpr size_t kRecreateScratchBytes = 5 * static_cast<size_t>(kRecreateMaxNp) * kRecreateMaxNp;
static_assert(kRecreateScratchBytes == 20u << 20, "20 MiB of scratch");

__device__ __align__(256) uint8_t scratch[kRecreateScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices];   // device address of `scratch` per device

// Device address of `scratch` on the current device `device`, looked up on
// the first call for that device.
sqn_status scratch_address(int device, void** out)
{
    if (device < 0 || device >= kMaxDevices)
        return fail(SQN_ERR_UNSUPPORTED, "device %d is beyond the %d devices this library tracks", device,
                    kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[device]) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || p == nullptr) {
            (void)hipGetLastError();
            return fail(SQN_ERR_DEVICE, "hipGetSymbolAddress(scratch) failed on device %d: %s", device,
                        hipGetErrorString(e));
        }
        g_scratch_ptr[device] = p;
    }
    *out = g_scratch_ptr[device];
    return SQN_OK;
}

// ---- cache generation: networks on the host side ---------------------------

// the input unit held by element e of lane-half h in a K step (generate.hip)
int kmap(int h, int e) { return 8 * (e >> 2) + 4 * h + (e & 3); }

bool half_finite(uint16_t bits) { return (bits & 0x7c00u) != 0x7c00u; }

// W [n_out][n_in] (binary16 bits) as MFMA A fragments
// [chunk][tile][step][lane][8] for `tiles` 32-row tiles and `steps` K steps
// of 16 inputs (steps a multiple of 4); physical row r takes source row
// rowmap[r] (-1: zero row), lane l covers row 32 tile + l % 32 and inputs
// 16 step + kmap(l / 32, e).
void build_fragments(const uint16_t* W, int n_in, const std::vector<int>& rowmap, int tiles, int steps,
                     uint16_t* out)
{
    size_t o = 0;
    for (int c = 0; c < steps / 4; ++c)
        for (int m = 0; m < tiles; ++m)
            for (int ss = 0; ss < 4; ++ss)
                for (int lane = 0; lane < 64; ++lane)
                    for (int e = 0; e < 8; ++e) {
                        const int src = rowmap[32 * m + lane % 32];
                        const int u = 16 * (4 * c + ss) + kmap(lane / 32, e);
                        out[o++] = (src >= 0 && u < n_in) ? W[static_cast<size_t>(src) * n_in + u] : 0;
                    }
}

sqn_status validate_mlp(const sqn_mlp_desc* m, int width, int n_in, int n_out, const char* what)
{
    if (!m)
        return fail(SQN_ERR_INVALID_ARG, "%s is NULL", what);
    if (m->width != width)
        return fail(SQN_ERR_UNSUPPORTED, "%s: width %d (this build runs %d units)", what, m->width, width);
    if (m->n_hidden < 1 || m->n_hidden > sqn::kMaxHidden)
        return fail(SQN_ERR_INVALID_ARG, "%s: n_hidden = %d outside [1, %d]", what, m->n_hidden, sqn::kMaxHidden);
    if (m->n_in != n_in || m->n_out != n_out)
        return fail(SQN_ERR_INVALID_ARG, "%s: %d inputs / %d outputs, expected %d / %d", what, m->n_in,
                    m->n_out, n_in, n_out);
    if (!m->weights || !m->biases)
        return fail(SQN_ERR_INVALID_ARG, "%s: NULL weight or bias array", what);
    for (int l = 0; l <= m->n_hidden; ++l) {
        const int fi = l == 0 ? n_in : width, fo = l == m->n_hidden ? n_out : width;
        if (!m->weights[l] || !m->biases[l])
            return fail(SQN_ERR_INVALID_ARG, "%s: layer %d has a NULL array", what, l);
        for (int k = 0; k < fi * fo; ++k)
            if (!half_finite(m->weights[l][k]))
                return fail(SQN_ERR_INVALID_ARG, "%s: layer %d weight %d is not finite", what, l, k);
        for (int k = 0; k < fo; ++k)
            if (!isfinite(m->biases[l][k]))
                return fail(SQN_ERR_INVALID_ARG, "%s: layer %d bias %d is not finite", what, l, k);
    }
    return SQN_OK;
}

// Host image of one network: fragments and biases per layer, and where each
// lands in the device block.
struct NetImage {
    std::vector<uint16_t> frag[sqn::kMaxHidden + 1];
    std::vector<float> bias[sqn::kMaxHidden + 1];
    int n_hidden = 0;
    int out_tiles = 0;
};

// head_rows: physical row -> source output row of the head; the head's
// fragments are padded with zero tiles to pad_tiles (the pipelined kernel
// stages whole chunks of width / 32 tiles)
NetImage make_image(const sqn_mlp_desc* m, int width, int in_steps, std::vector<int> head_rows,
                    int out_tiles, int pad_tiles)
{
    head_rows.resize(static_cast<size_t>(pad_tiles) * 32, -1);
    NetImage img;
    img.n_hidden = m->n_hidden;
    img.out_tiles = out_tiles;
    std::vector<int> ident(width);
    for (int r = 0; r < width; ++r)
        ident[r] = r;
    const int tiles = width / 32;
    for (int l = 0; l <= m->n_hidden; ++l) {
        const bool head = l == m->n_hidden;
        const int fi = l == 0 ? m->n_in : width;
        const int t = head ? pad_tiles : tiles;
        const int steps = l == 0 ? in_steps : width / 16;
        const std::vector<int>& rows = head ? head_rows : ident;
        img.frag[l].resize(static_cast<size_t>(t) * steps * 512);
        build_fragments(m->weights[l], fi, rows, t, steps, img.frag[l].data());
        img.bias[l].assign(static_cast<size_t>(t) * 32, 0.0f);
        for (int r = 0; r < t * 32; ++r)
            if (rows[r] >= 0)
                img.bias[l][r] = m->biases[l][rows[r]];
    }
    return img;
}

}  // namespace

extern "C" {

sqn_status sqn_create_caches(const sqn_cache_desc* desc, const void* const sigma_planes[3],
                             const void* const uvw_planes[3], const void* beta, void* stream,
                             sqn_caches** out)
{
    return create_impl(desc, nullptr, sigma_planes, uvw_planes, beta, stream, out);
}

sqn_status sqn_create_linear_caches(const sqn_cache_desc* desc, const sqn_linear_decoder* decoder,
                                    const void* const sigma_planes[3], const void* const uvw_planes[3],
                                    const void* beta, void* stream, sqn_caches** out)
{
    if (!decoder) {
        if (out)
            *out = nullptr;
        return fail(SQN_ERR_INVALID_ARG, "decoder is NULL");
    }
    return create_impl(desc, decoder, sigma_planes, uvw_planes, beta, stream, out);
}

sqn_status sqn_recreate_caches(sqn_caches* caches, const sqn_cache_desc* desc,
                               const void* const sigma_planes[3], const void* const uvw_planes[3],
                               const void* beta, void* stream)
{
    if (!caches)
        return fail(SQN_ERR_INVALID_ARG, "caches is NULL");
    sqn_status s = validate_desc(desc);
    if (s != SQN_OK)
        return s;
    if (caches->linear)
        return fail(SQN_ERR_UNSUPPORTED, "the handle holds Eq. 5 caches; sqn_recreate_caches takes Eq. 4 handles");
    if (!sigma_planes || !uvw_planes)
        return fail(SQN_ERR_INVALID_ARG, "plane pointer array is NULL");
    if (desc->n_p > kRecreateMaxNp)
        return fail(SQN_ERR_INVALID_ARG, "n_p = %d exceeds %d, the largest grid the static scratch (%zu bytes) covers",
                    desc->n_p, kRecreateMaxNp, kRecreateScratchBytes);
    int device = -1;
    if (hipGetDevice(&device) != hipSuccess)
        return fail(SQN_ERR_DEVICE, "hipGetDevice failed");
    if (device != caches->device)
        return fail(SQN_ERR_INVALID_ARG, "caches live on device %d, current device is %d", caches->device, device);
    const CacheLayout lay = cache_layout(desc, false);
    if (lay.total > caches->bytes)
        return fail(SQN_ERR_INVALID_ARG, "the caches need %zu bytes of device memory, the handle holds %zu",
                    lay.total, caches->bytes);
    const size_t texels = static_cast<size_t>(desc->n_p) * desc->n_p;
    const size_t sigma_bytes = texels * dtype_size(desc->sigma_dtype);
    static const char* names_s[3] = {"sigma_planes[0] (xy)", "sigma_planes[1] (yz)", "sigma_planes[2] (zx)"};
    static const char* names_u[3] = {"uvw_planes[0] (xy)", "uvw_planes[1] (yz)", "uvw_planes[2] (zx)"};
    for (int j = 0; j < 3; ++j) {
        if ((s = check_device_range(sigma_planes[j], sigma_bytes, names_s[j])) != SQN_OK)
            return s;
        if ((s = check_device_range(uvw_planes[j], lay.uvw_bytes, names_u[j])) != SQN_OK)
            return s;
    }
    if ((s = check_device_range(beta, lay.beta_bytes, "beta")) != SQN_OK)
        return s;
    void* scr = nullptr;
    if ((s = scratch_address(device, &scr)) != SQN_OK)
        return s;

    // live mask, row distances and capped distances of one plane at a time;
    // every kernel of the preparation writes its whole array before it is
    // read, so nothing needs clearing
    sqn::PrepareWork pw;
    memset(&pw, 0, sizeof(pw));
    uint8_t* w = static_cast<uint8_t*>(scr);
    pw.live = w;
    pw.f = reinterpret_cast<uint16_t*>(w + align256(texels));
    pw.dist = reinterpret_cast<uint16_t*>(w + align256(texels) + align256(texels * sizeof(uint16_t)));
    char* base = static_cast<char*>(caches->block);
    hipStream_t st = static_cast<hipStream_t>(stream);
    hipError_t e = hipSuccess;
    for (int j = 0; j < 3 && e == hipSuccess; ++j)
        e = sqn::prepare_sigma_plane(sigma_planes[j], desc->sigma_dtype, desc->n_p, base + lay.off_sigma[j], pw, st);
    for (int j = 0; j < 3 && e == hipSuccess; ++j)
        e = hipMemcpyAsync(base + lay.off_uvw[j], uvw_planes[j], lay.uvw_bytes, hipMemcpyDeviceToDevice, st);
    if (e == hipSuccess)
        e = hipMemcpyAsync(base + lay.off_beta, beta, lay.beta_bytes, hipMemcpyDeviceToDevice, st);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return fail(SQN_ERR_DEVICE, "cache preparation failed (the handle's contents are now unspecified): %s",
                    hipGetErrorString(e));
    }
    // later renders with the handle read the new arrays
    caches->desc = *desc;
    for (int j = 0; j < 3; ++j) {
        caches->sigma[j] = base + lay.off_sigma[j];
        caches->uvw[j] = base + lay.off_uvw[j];
    }
    caches->beta = base + lay.off_beta;
    for (int r = 0; r < 3; ++r)
        caches->scale[r] = static_cast<float>(desc->n_p - 1) / (desc->bbox_max[r] - desc->bbox_min[r]);
    caches->tau_eps = tau_threshold(desc->t_eps);
    clear_error();
    return SQN_OK;
}

sqn_status sqn_create_networks(const sqn_mlp_desc pos[3], const sqn_mlp_desc* dir, int32_t D,
                               int32_t pos_freq, int32_t dir_freq, void* stream, sqn_networks** out)
{
    if (!out)
        return fail(SQN_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    if (!pos)
        return fail(SQN_ERR_INVALID_ARG, "pos is NULL");
    if (D < 1 || D > 32)
        return fail(SQN_ERR_INVALID_ARG, "D = %d outside [1, 32]", D);
    const int pos_in = 2 * (1 + 2 * pos_freq), dir_in = 3 * (1 + 2 * dir_freq);
    if (pos_freq < 0 || pos_in > 64 || dir_freq < 0 || dir_in > 64)
        return fail(SQN_ERR_INVALID_ARG, "encoding frequencies %d / %d give more than 64 inputs", pos_freq,
                    dir_freq);
    static const char* names[3] = {"pos[0] (xy)", "pos[1] (yz)", "pos[2] (zx)"};
    sqn_status s;
    for (int j = 0; j < 3; ++j)
        if ((s = validate_mlp(&pos[j], 256, pos_in, 2 + 6 * D, names[j])) != SQN_OK)
            return s;
    if ((s = validate_mlp(dir, 128, dir_in, D, "dir")) != SQN_OK)
        return s;

    // position head: pair slot P = 16 m + 8 gg + 4 h + q in rows
    // 32 m + 16 gg + 4 h + q (first factor) and + 8 (second); slot 0 is
    // (sigma_0, w_sigma), slot 1 + c D + d is (w_c[d], c_0[d]) (Eq. 3)
    const int slots = 1 + 3 * D;
    const int pos_tiles = (slots + 15) / 16;
    std::vector<int> pos_rows(pos_tiles * 32, -1);
    for (int slot = 0; slot < slots; ++slot) {
        const int m = slot / 16, gg = (slot / 8) % 2, h = (slot / 4) % 2, q = slot % 4;
        const int row = 32 * m + 16 * gg + 4 * h + q;
        int first = 0, second = 1;
        if (slot > 0) {
            const int c = (slot - 1) / D, d = (slot - 1) % D;
            first = 2 + 2 * c * D + d;
            second = 2 + (2 * c + 1) * D + d;
        }
        pos_rows[row] = first;
        pos_rows[row + 8] = second;
    }
    std::vector<int> dir_rows(32, -1);
    for (int r = 0; r < D; ++r)
        dir_rows[r] = r;

    NetImage img[4];
    for (int j = 0; j < 3; ++j)
        img[j] = make_image(&pos[j], 256, 4, pos_rows, pos_tiles, 8);
    img[3] = make_image(dir, 128, 4, dir_rows, 1, 1);

    auto align = [](size_t x) { return (x + 255) & ~size_t{255}; };
    size_t total = 0;
    size_t off_frag[4][sqn::kMaxHidden + 1], off_bias[4][sqn::kMaxHidden + 1];
    for (int n = 0; n < 4; ++n)
        for (int l = 0; l <= img[n].n_hidden; ++l) {
            off_frag[n][l] = total;
            total += align(img[n].frag[l].size() * sizeof(uint16_t));
            off_bias[n][l] = total;
            total += align(img[n].bias[l].size() * sizeof(float));
        }
    const size_t off_table = total;
    total += align(3 * size_t{8192} * (1 + 2 * pos_freq) * sizeof(uint16_t));

    sqn_networks* h = static_cast<sqn_networks*>(calloc(1, sizeof(sqn_networks)));
    if (!h)
        return fail(SQN_ERR_OUT_OF_MEMORY, "host allocation failed");
    if (hipGetDevice(&h->device) != hipSuccess) {
        free(h);
        return fail(SQN_ERR_DEVICE, "hipGetDevice failed");
    }
    hipError_t e = hipMalloc(&h->block, total);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        free(h);
        return fail(SQN_ERR_OUT_OF_MEMORY, "hipMalloc(%zu) failed: %s", total, hipGetErrorString(e));
    }
    h->bytes = total;
    char* base = static_cast<char*>(h->block);
    hipStream_t st = static_cast<hipStream_t>(stream);
    for (int n = 0; n < 4 && e == hipSuccess; ++n) {
        sqn::GenNet& g = n < 3 ? h->pos[n] : h->dir;
        g.n_hidden = img[n].n_hidden;
        g.out_tiles = img[n].out_tiles;
        for (int l = 0; l <= img[n].n_hidden && e == hipSuccess; ++l) {
            g.frag[l] = base + off_frag[n][l];
            g.bias[l] = reinterpret_cast<const float*>(base + off_bias[n][l]);
            e = hipMemcpyAsync(base + off_frag[n][l], img[n].frag[l].data(),
                               img[n].frag[l].size() * sizeof(uint16_t), hipMemcpyHostToDevice, st);
            if (e == hipSuccess)
                e = hipMemcpyAsync(base + off_bias[n][l], img[n].bias[l].data(),
                                   img[n].bias[l].size() * sizeof(float), hipMemcpyHostToDevice, st);
        }
    }
    if (e == hipSuccess)
        e = hipStreamSynchronize(st);
    else
        (void)hipStreamSynchronize(st);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        (void)hipFree(h->block);
        free(h);
        return fail(SQN_ERR_DEVICE, "network upload failed: %s", hipGetErrorString(e));
    }
    h->enc_table = reinterpret_cast<_Float16*>(base + off_table);
    h->D = D;
    h->pos_freq = pos_freq;
    h->dir_freq = dir_freq;
    h->pos_in = pos_in;
    h->dir_in = dir_in;
    *out = h;
    clear_error();
    return SQN_OK;
}

sqn_status sqn_generate_caches(sqn_networks* nets, const sqn_cache_desc* desc, void* const sigma_planes[3],
                               void* const uvw_planes[3], void* beta, void* stream)
{
    if (!nets)
        return fail(SQN_ERR_INVALID_ARG, "networks is NULL");
    sqn_status s = validate_desc(desc);
    if (s != SQN_OK)
        return s;
    if (desc->D != nets->D)
        return fail(SQN_ERR_INVALID_ARG, "desc D = %d but the networks emit D = %d", desc->D, nets->D);
    if (!sigma_planes || !uvw_planes)
        return fail(SQN_ERR_INVALID_ARG, "plane pointer array is NULL");
    int device = -1;
    if (hipGetDevice(&device) != hipSuccess)
        return fail(SQN_ERR_DEVICE, "hipGetDevice failed");
    if (device != nets->device)
        return fail(SQN_ERR_INVALID_ARG, "networks live on device %d, current device is %d", nets->device,
                    device);
    const size_t texels = static_cast<size_t>(desc->n_p) * desc->n_p;
    static const char* names_s[3] = {"sigma_planes[0] (xy)", "sigma_planes[1] (yz)", "sigma_planes[2] (zx)"};
    static const char* names_u[3] = {"uvw_planes[0] (xy)", "uvw_planes[1] (yz)", "uvw_planes[2] (zx)"};
    for (int j = 0; j < 3; ++j) {
        if ((s = check_device_range(sigma_planes[j], texels * dtype_size(desc->sigma_dtype), names_s[j])) != SQN_OK)
            return s;
        if ((s = check_device_range(uvw_planes[j], texels * 3 * desc->D * dtype_size(desc->uvw_dtype),
                                    names_u[j])) != SQN_OK)
            return s;
    }
    const size_t beta_bytes = static_cast<size_t>(desc->n_theta) * desc->n_phi * desc->D
                              * dtype_size(desc->beta_dtype);
    if ((s = check_device_range(beta, beta_bytes, "beta")) != SQN_OK)
        return s;

    sqn::GenParams p;
    memset(&p, 0, sizeof(p));
    for (int j = 0; j < 3; ++j) {
        p.pos[j] = nets->pos[j];
        p.sigma_out[j] = sigma_planes[j];
        p.uvw_out[j] = uvw_planes[j];
    }
    p.dir = nets->dir;
    p.beta_out = beta;
    p.n_p = desc->n_p;
    p.n_theta = desc->n_theta;
    p.n_phi = desc->n_phi;
    p.D = desc->D;
    p.pos_freq = nets->pos_freq;
    p.dir_freq = nets->dir_freq;
    p.pos_in = nets->pos_in;
    p.dir_in = nets->dir_in;
    for (int r = 0; r < 3; ++r) {
        p.bmin[r] = desc->bbox_min[r];
        p.bmax[r] = desc->bbox_max[r];
    }
    p.sigma_f16 = desc->sigma_dtype == SQN_F16;
    p.uvw_f16 = desc->uvw_dtype == SQN_F16;
    p.beta_f16 = desc->beta_dtype == SQN_F16;
    hipError_t e = sqn::launch_generate(p, nets->enc_table, static_cast<hipStream_t>(stream));
    if (e != hipSuccess)
        return fail(SQN_ERR_DEVICE, "generation launch failed: %s", hipGetErrorString(e));
    return SQN_OK;
}

size_t sqn_networks_device_bytes(const sqn_networks* nets) { return nets ? nets->bytes : 0; }

void sqn_destroy_networks(sqn_networks* nets)
{
    if (!nets)
        return;
    if (nets->block)
        (void)hipFree(nets->block);
    free(nets);
}

sqn_status sqn_render(const sqn_caches* caches, const float* poses, int32_t n_poses,
                      const sqn_intrinsics* intrinsics, float near_plane, float far_plane,
                      int32_t n_samples, float* rgb_out, float* depth_out, void* stream)
{
    return render_common(caches, poses, n_poses, intrinsics, near_plane, far_plane, n_samples,
                         rgb_out, depth_out, nullptr, stream);
}

sqn_status sqn_render_stats(const sqn_caches* caches, const float* poses, int32_t n_poses,
                            const sqn_intrinsics* intrinsics, float near_plane, float far_plane,
                            int32_t n_samples, float* rgb_out, float* depth_out,
                            uint32_t* ray_stats, void* stream)
{
    if (!ray_stats)
        return fail(SQN_ERR_INVALID_ARG, "ray_stats is NULL");
    return render_common(caches, poses, n_poses, intrinsics, near_plane, far_plane, n_samples,
                         rgb_out, depth_out, ray_stats, stream);
}

sqn_status sqn_set_empty_space_skipping(sqn_caches* caches, int32_t enable)
{
    if (!caches)
        return fail(SQN_ERR_INVALID_ARG, "caches is NULL");
    if (enable != 0 && enable != 1)
        return fail(SQN_ERR_INVALID_ARG, "enable must be 0 or 1 (got %d)", enable);
    caches->skip = enable;
    return SQN_OK;
}

sqn_status sqn_set_lanes_per_ray(sqn_caches* caches, int32_t lanes)
{
    if (!caches)
        return fail(SQN_ERR_INVALID_ARG, "caches is NULL");
    if (lanes != 0 && lanes != 1 && lanes != 4 && lanes != 8)
        return fail(SQN_ERR_INVALID_ARG, "lanes per ray must be 0, 1, 4 or 8 (got %d)", lanes);
    if (caches->linear && (lanes == 1 || lanes == 8))
        return fail(SQN_ERR_UNSUPPORTED, "the linear decoder renders with four lanes per ray");
    caches->lanes = lanes;
    caches->centre = 0.0f;
    return SQN_OK;
}

sqn_status sqn_tune_lanes_per_ray(sqn_caches* caches, const float* poses, int32_t n_poses,
                                  const sqn_intrinsics* intrinsics, float near_plane, float far_plane,
                                  int32_t n_samples, float* rgb_out, float* depth_out, void* stream,
                                  int32_t* lanes_out, float* centre_out)
{
    if (!caches)
        return fail(SQN_ERR_INVALID_ARG, "caches is NULL");
    const int32_t before = caches->lanes;
    const float centre_before = caches->centre;
    // the batch itself is checked by the first render; candidates: lanes
    // per ray (centre 0), then hybrid launches of single views with centred
    // blocks of 0.15, 0.5 and 1 of the image per axis (1: four lanes per ray
    // everywhere, blocks dealt from the centre outwards)
    static const int32_t kCandidates[6] = {4, 1, 8, 0, 0, 0};
    static const float kCentre[6] = {0.0f, 0.0f, 0.0f, 0.15f, 0.5f, 1.0f};
    const bool hybrid_ok = n_poses == 1 && !caches->linear && caches->skip && !(caches->ndc_near > 0.0f);
    const int n_cand = caches->linear ? 1 : (hybrid_ok ? 6 : 3);
    // every candidate twice untimed (code and caches warm), then kRounds
    // rounds that each time every candidate over kReps renders (after one
    // untimed render in its shape): the GPU's clocks settle over the first
    // tens of milliseconds of load, and rounds spread that drift over all
    // candidates instead of favouring the last ones
    constexpr int kWarm = 2, kRounds = 4, kReps = 5;
    hipStream_t st = static_cast<hipStream_t>(stream);
    hipEvent_t ev[2] = {nullptr, nullptr};
    for (int k = 0; k < 2; ++k)
        if (hipEventCreate(&ev[k]) != hipSuccess) {
            (void)hipGetLastError();
            if (ev[0])
                (void)hipEventDestroy(ev[0]);
            return fail(SQN_ERR_DEVICE, "hipEventCreate failed");
        }
    sqn_status s = SQN_OK;
    float total_ms[6] = {0.0f, 0.0f, 0.0f, 0.0f, 0.0f, 0.0f};
    auto render = [&](int c, int times) {
        caches->lanes = kCandidates[c];
        caches->centre = kCentre[c];
        for (int r = 0; r < times && s == SQN_OK; ++r)
            s = render_common(caches, poses, n_poses, intrinsics, near_plane, far_plane, n_samples, rgb_out,
                              depth_out, nullptr, stream);
    };
    for (int c = 0; c < n_cand && s == SQN_OK; ++c)
        render(c, kWarm);
    for (int round = 0; round < kRounds && s == SQN_OK && n_poses > 0; ++round)
        for (int c = 0; c < n_cand && s == SQN_OK; ++c) {
            render(c, 1);
            if (s != SQN_OK)
                break;
            hipError_t e = hipEventRecord(ev[0], st);
            if (e == hipSuccess)
                render(c, kReps);
            if (s != SQN_OK)
                break;
            if (e == hipSuccess)
                e = hipEventRecord(ev[1], st);
            if (e == hipSuccess)
                e = hipEventSynchronize(ev[1]);
            float ms = 0.0f;
            if (e == hipSuccess)
                e = hipEventElapsedTime(&ms, ev[0], ev[1]);
            if (e != hipSuccess) {
                (void)hipGetLastError();
                s = fail(SQN_ERR_DEVICE, "timing the launch shapes failed: %s", hipGetErrorString(e));
                break;
            }
            total_ms[c] += ms;
        }
    int best = 0;
    for (int c = 1; c < n_cand; ++c)
        if (total_ms[c] < total_ms[best])
            best = c;
    (void)hipEventDestroy(ev[0]);
    (void)hipEventDestroy(ev[1]);
    if (s != SQN_OK || n_poses == 0) {
        caches->lanes = before;
        caches->centre = centre_before;
        return s;
    }
    caches->lanes = kCandidates[best];
    caches->centre = kCentre[best];
    if (lanes_out)
        *lanes_out = kCentre[best] > 0.0f ? -1 : kCandidates[best];
    if (centre_out)
        *centre_out = kCentre[best];
    return SQN_OK;
}

sqn_status sqn_set_centre_block(sqn_caches* caches, float fraction)
{
    if (!caches)
        return fail(SQN_ERR_INVALID_ARG, "caches is NULL");
    if (!(fraction >= 0.0f && fraction <= 1.0f))
        return fail(SQN_ERR_INVALID_ARG, "centre block fraction %g outside [0, 1]", static_cast<double>(fraction));
    if (caches->linear && fraction > 0.0f)
        return fail(SQN_ERR_UNSUPPORTED, "the linear decoder renders with four lanes per ray");
    caches->centre = fraction;
    return SQN_OK;
}

sqn_status sqn_set_ndc(sqn_caches* caches, float ndc_near)
{
    if (!caches)
        return fail(SQN_ERR_INVALID_ARG, "caches is NULL");
    if (!(ndc_near >= 0.0f) || !isfinite(ndc_near))
        return fail(SQN_ERR_INVALID_ARG, "ndc_near = %g must be finite and >= 0", static_cast<double>(ndc_near));
    caches->ndc_near = ndc_near;
    return SQN_OK;
}

size_t sqn_cache_device_bytes(const sqn_caches* caches) { return caches ? caches->bytes : 0; }

void sqn_destroy(sqn_caches* caches)
{
    if (!caches)
        return;
    if (caches->block)
        (void)hipFree(caches->block);
    free(caches);
}

const char* sqn_status_string(sqn_status status)
{
    switch (status) {
    case SQN_OK:
        return "success";
    case SQN_ERR_INVALID_ARG:
        return "invalid argument";
    case SQN_ERR_OUT_OF_MEMORY:
        return "out of device memory";
    case SQN_ERR_DEVICE:
        return "HIP device error";
    case SQN_ERR_UNSUPPORTED:
        return "unsupported configuration";
    }
    return "unknown status";
}

const char* sqn_last_error(void) { return g_last_error; }

}  // extern "C"
